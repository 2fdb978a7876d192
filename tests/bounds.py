"""Per-element error terms that the GPU path's 16-bit handoffs add to the
strict fp64 reference, derived from the reference's own quantities.

The reference (the oracle) computes every step in fp64 from the bf16 inputs
and never rounds in between.  The GPU path stores some intermediates in
bfloat16 (Sec. 5 trains in 16-bit precision): H between fc1 and fc2, fc1's
upstream gradient dh_pre between fc2's input-gradient reduction and fc1's
backward, and, in the 16-bit-partials variant, each member's Partial(SUM)
block.  Rounding a value v to bfloat16 (8 significant bits, nearest even)
moves it by at most half the spacing ulp(v) of bfloat16 numbers at |v|.

* A single rounding that reaches an output directly adds at most
  ulp(v)/2 there (times |f'(v)| when an epilogue f follows).
* A rounded tensor V that feeds a product, Y = V W (or X^T V, or column
  sums of V), adds sum_k delta_k W_kn to each output, a sum of many
  independent rounding errors.  Each delta_k is modelled as uniform on
  [-ulp(V_k)/2, ulp(V_k)/2] (variance ulp^2 / 12), so the added error has
  standard deviation sqrt(sum_k ulp(V_k)^2 / 12 * W_kn^2); the bound is
  SIGMAS of those.  For sums of at most 12 terms six standard deviations
  also bound the worst case (6 sqrt(N/12) >= N/2).

These terms are added to the stated elementwise tolerance
1e-2 (|ref| + 1); nothing here reads a GPU value.
"""
import numpy as np

SIGMAS = 6.0


def ulp_bf16(x) -> np.ndarray:
    """Spacing of bfloat16 numbers at |x|: 2^(e-7) for |x| in [2^e, 2^(e+1));
    the subnormal spacing 2^-133 below 2^-126."""
    a = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return np.exp2(e - 7.0)


def rounding_var(v) -> np.ndarray:
    """Variance of one bfloat16 rounding of v (uniform error model)."""
    return ulp_bf16(v) ** 2 / 12.0


def single(v, scale=None) -> np.ndarray:
    """Bound of one rounding of v reaching the output, times |scale|."""
    b = 0.5 * ulp_bf16(v)
    return b if scale is None else b * np.abs(np.asarray(scale, dtype=np.float64))


def left(var, w) -> np.ndarray:
    """Y = V W with V carrying independent errors of variance `var` (an
    array shaped like V): SIGMAS standard deviations of each output."""
    w = np.asarray(w, dtype=np.float64)
    return SIGMAS * np.sqrt(np.asarray(var, dtype=np.float64) @ (w * w))


def right(x, var) -> np.ndarray:
    """Y = X^T V (a weight gradient) with V carrying errors of variance var."""
    x = np.asarray(x, dtype=np.float64)
    return SIGMAS * np.sqrt((x * x).T @ np.asarray(var, dtype=np.float64))


def colsum(var) -> np.ndarray:
    """Column sums of V with V carrying errors of variance var."""
    return SIGMAS * np.sqrt(np.asarray(var, dtype=np.float64).sum(axis=0))
