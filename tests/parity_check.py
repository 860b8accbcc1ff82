"""Element-wise acceptance bound for fp32 outputs of the bf16 products.

Every product of two bf16 values is exact in fp32, so the only error in an
fp32 output is the rounding of its sums.  For a sum of K terms taken in any
order with fp32 additions, the classic bound (Higham, "Accuracy and Stability
of Numerical Algorithms", 2nd ed., Section 3.1, the gamma_n bound of a
recursive summation) is

    |fl(sum) - sum| <= gamma_{K-1} * sum_k |term_k|,  gamma_n = n u / (1 - n u),

with u = 2^-24.  The check below allows twice that (K + extra rounding steps:
the NVFP4 epilogue multiply, the code multiply and block sum of dS) and
applies it to every output element, beside the normwise gate.  An element
computed from the wrong operands (a stage read before it landed, a tile
written to the wrong place) misses it by orders of magnitude, whereas the
normwise error over a large output would hide a single such element.
"""

import numpy as np

U = 2.0 ** -24


def gamma(n):
    return n * U / (1.0 - n * U)


def elementwise_bound(absref, depth):
    """Allowed |got - ref| for outputs whose terms have absolute sum absref,
    accumulated over `depth` roundings."""
    return 2.0 * gamma(depth) * np.asarray(absref, np.float64) + 1e-38


def check_elements(got, ref, absref, depth):
    """Indices of the elements of got (fp32 results) outside the bound."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    bad = ~(np.abs(got - ref) <= elementwise_bound(absref, depth))   # NaN counts as bad
    return np.argwhere(bad)


def assert_elements(got, ref, absref, depth, what=""):
    bad = check_elements(got, ref, absref, depth)
    if bad.size:
        i = tuple(bad[0])
        raise AssertionError(f"{what}: {len(bad)} elements outside the per-element bound, first at {i}: "
                             f"got {np.asarray(got)[i]!r} ref {np.asarray(ref)[i]!r} "
                             f"allowed {elementwise_bound(np.asarray(absref)[i], depth)!r}")
