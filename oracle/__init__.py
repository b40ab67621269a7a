"""CPU oracle for the hashed shared-memory embedding layer (ROBE-Z style PSS).

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this package: only the test-suite, the graft smoke check and the
``cpu_baseline`` leg of the benchmark use it.  It shares no code with the HIP
library; the only thing both sides consume is the seeded input generator in
``synth/``, which holds none of the method's arithmetic.

Contents
  pss_oracle  plain NumPy/float64 definition of the forward, the dense
              gradient (Alg. 1 dense branch), the sparse gradient (Alg. 1
              sparse branch) and the SGD / Adagrad updates.
  brute       pure-Python loop version on tiny inputs, including the explicit
              0/1 sketch matrix S of Thm. 2 (M = S E, lookup = (S e_i)^T M).
"""
from . import pss_oracle, brute  # noqa: F401
