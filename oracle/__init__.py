"""CPU oracle for the DistillCache budgeted decode step — TEST INFRASTRUCTURE ONLY.

Plain, slow, binary64 numpy code written from the paper's definitions, one
function per step of the decode step.  It exists to check the HIP path and is
imported only by the tests, by ``__graft_entry__.smoke()`` and by the
``cpu_baseline`` leg of ``bench.py``.  The product library never imports, links
or executes anything here, and nothing here imports the product library.

Every value is computed in binary64 from the exact stored input values
(bfloat16/binary32 upcast).  Modules:

* ``attention``  – decode attention and per-query entropy (Sec. 3.1.1 state
  features; the reward motivation of Sec. 3.1.4 writes o_t = sum_i a_{t,i} v_i).
* ``features``   – the per-token state x_i = [alpha_i, ||v_i||_2, H_i, pos_i]
  (Sec. 3.1.1, with sigma_i left out) and the windowed entropy H_i.
* ``policy``     – the scoring MLP s_i = f_phi(x_i) (Sec. 3.1.2, App. D).
* ``select``     – deterministic argtop_B (Sec. 3.3, Algorithm 1).
* ``compact``    – storage order of the pruned cache (hole filling; the
  paper fixes none).
* ``kl``         – the per-step reward R_t = -KL(P_t || P^_t) (Sec. 3.1.4).
* ``sampling``   – training-mode selection: Gumbel-perturbed top-B, the exact
  log-partition log Z(s, B, tau) and log pi(a | s) (Sec. 3.1.2, App. C).
* ``reinforce``  – rollout reward math of the REINFORCE update: discounted
  returns, RLOO and EMA baselines, entropy surrogate, loss (Sec. 3.2).
* ``unit``       – one unit's cache and feature state stepped through
  append -> attention -> features -> score -> select -> prune (Algorithm 1,
  Sec. 3.1.3 for the student/teacher caches).

Parity status of each function is stated in its module docstring; every one is
pinned by the ``-m "not gpu"`` tests (closed forms, invariants, brute force,
library cross-checks) listed in tests/test_oracle_*.py.
"""
