// Matrix-core scoring pass of two-hidden-layer policies (dc_mlp.hip).
#pragma once
#include "dc_kernels.hpp"

namespace dc {

// Scores and ranking keys of every row of every unit (keys[u * kstride + r]).
int launch_score_mlp2(const EvictArgs& a, uint64_t* keys, int kstride, void* stream);

}  // namespace dc
