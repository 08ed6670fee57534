"""Plain fp64 CPU oracle for Tactic's decode-time sparse attention.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package.  It shares no code with the HIP
library (no kernels, headers, helpers or tables) and never imports it; the
only thing both sides consume is the seeded input generator in ``synth``.

Modules
-------
numerics   bf16 round-to-nearest-even of fp64 values (storage precision).
attention  dense and subset attention (Eq. 2, Eq. 3), attention distance
           (Eq. 4), cumulative attention score (Eq. 5), the error bound
           (Eq. 6 / Appendix A) and the optimal selection of Sec. 3.4.
tactic     the decode path of Sec. 4.3-4.6 and Algorithm 1: cluster ranking,
           unpacking, distribution fit, cutoff, GQA union, attention.
kmeans     the prefill clustering of Sec. 4.2 and the cluster-contiguous
           layout (offsets + permutation) it defines.

Everything is computed in float64 on NumPy arrays; bf16 inputs are upcast
exactly.  Each function cites the passage of the paper it follows.
"""
from . import numerics, attention, tactic, kmeans  # noqa: F401
