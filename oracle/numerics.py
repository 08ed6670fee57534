"""Storage-precision helper for the oracle (test infrastructure only).

The key cache, the queries and the cluster centroids are stored as bf16
(8 significant bits, round to nearest even).  The oracle computes in fp64 and
rounds only where a value is stored in bf16 (the K-means centroids).
"""
import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round fp64 values to the nearest bf16 value, ties to even.

    A finite x is m * 2**e with 0.5 <= |m| < 1 (frexp); bf16 keeps 8
    significant bits, so m * 2**8 is rounded to an integer with ties to even
    (np.rint) and scaled back.  bf16 subnormals (|x| < 2**-126) and overflow
    are outside the range of any value this code stores and are not treated
    specially.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)
