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

import oracle as O

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


def delta_bounds(q, k, v, do):
    """Error terms for dQ and dK of one (sequence, head) from delta_t = dO_t . O_t
    taken over the stored bf16 output (the kernels never see the exact O).
    The stored O carries two roundings of relative size 2^-9 (the bf16
    probabilities that enter P V, and the output's own rounding), so
    |dO_t[e]| (|O_t[e]| + (P |V|)_t[e]) scales the error of each term; taken
    as independent uniform roundings, delta_t's error has RMS
        r_t = 2^-9 / sqrt(3) * sqrt(sum_e dO_t[e]^2 (O_t[e]^2 + (P|V|)_t[e]^2)).
    It enters dS[t, u] = P[t, u] (dP[t, u] - delta_t), hence
        dK_u[e] error RMS = sqrt(sum_t P[t,u]^2 r_t^2 q_t[e]^2) / sqrt(d),
        dQ_t[e] error RMS = r_t sqrt(sum_u P[t,u]^2 k_u[e]^2) / sqrt(d);
    the bounds are six times these RMS values.  P, O come from the oracle."""
    q, k, v, do = (np.asarray(O._f64(a)) for a in (q, k, v, do))
    S, d = q.shape
    o, lse = O.attention_fwd(q, k, v)
    s = q @ k.T / np.sqrt(d)
    s[np.triu(np.ones((S, S), dtype=bool), 1)] = -np.inf
    P = np.exp(s - lse[:, None])
    r = 2.0 ** -9 / np.sqrt(3) * np.sqrt((do * do * (o * o + (P @ np.abs(v)) ** 2)).sum(1))
    bk = 6 / np.sqrt(d) * np.sqrt((P * P).T @ ((r * r)[:, None] * q * q))
    bq = 6 / np.sqrt(d) * r[:, None] * np.sqrt((P * P) @ (k * k))
    return bq, bk


def attention_dout_sensitivity(q, k, v, var_do):
    """Variances that a bf16 handoff of the output gradient dO (independent
    errors of variance var_do [S, d]) adds to the causal attention backward
    of one (sequence, head), from the oracle's q, k, v.  For fixed P the
    backward is linear in dO:
        dV_u = sum_t P[t,u] dO_t,
        dS[t,u] = P[t,u] (dO_t . (V_u - O_t))        (dP - delta, delta = dO_t . O_t),
        dQ_t = sum_u dS[t,u] K_u / sqrt(d),  dK_u = sum_t dS[t,u] Q_t / sqrt(d).
    Returns the per-element variances of dQ, dK, dV ([S, d] each) and the
    variances of their column sums over the tokens ([d] each), taken from the
    same linear maps (the column sums are not sums of the per-element
    variances: sum_u dV_u = sum_t dO_t, sum_u dK_u = 0 whatever dO is)."""
    q, k, v = (np.asarray(O._f64(a)) for a in (q, k, v))
    var = np.asarray(var_do, dtype=np.float64)
    S, d = q.shape
    o, lse = O.attention_fwd(q, k, v)
    s = q @ k.T / np.sqrt(d)
    s[np.triu(np.ones((S, S), dtype=bool), 1)] = -np.inf
    P = np.exp(s - lse[:, None])
    P2 = P * P
    var_dv = P2.T @ var
    # dQ_t[f] = sum_e dO_t[e] C[t, e, f],
    # C[t, e, f] = (sum_u P[t,u] V[u,e] K[u,f] - O[t,e] (P K)[t,f]) / sqrt(d)
    vk = (v[:, :, None] * k[:, None, :]).reshape(S, d * d)
    C = ((P @ vk).reshape(S, d, d) - o[:, :, None] * (P @ k)[:, None, :]) / np.sqrt(d)
    var_dq = np.einsum("tef,te->tf", C * C, var)
    # dK_u[f] = sum_t P[t,u] (dO_t . (V_u - O_t)) Q_t[f] / sqrt(d)
    w2 = var @ (v * v).T - 2.0 * (o * var) @ v.T + (o * o * var).sum(1)[:, None]
    var_dk = (P2 * w2).T @ (q * q) / d
    return dict(dq=var_dq, dk=var_dk, dv=var_dv, sum_dq=var_dq.sum(0),
                sum_dk=np.zeros(d), sum_dv=var.sum(0))


def attention_qkv_sensitivity(q, k, v, var_q, var_k, var_v):
    """Variance that independent errors in q, k, v (variances var_* [S, d],
    e.g. their bf16 handoff) add to each output O_t[e] of the causal
    attention of one (sequence, head), to first order:
        dO_t = sum_u P[t,u] dV_u + sum_u P[t,u] (V_u - O_t) ds_tu,
        ds_tu = (dQ_t . K_u + Q_t . dK_u) / sqrt(d).
    dQ_t is shared by every u of row t; dK_u and dV_u are independent."""
    q, k, v = (np.asarray(O._f64(a)) for a in (q, k, v))
    vq, vk_, vv = (np.asarray(a, dtype=np.float64) for a in (var_q, var_k, var_v))
    S, d = q.shape
    o, lse = O.attention_fwd(q, k, v)
    s = q @ k.T / np.sqrt(d)
    s[np.triu(np.ones((S, S), dtype=bool), 1)] = -np.inf
    P = np.exp(s - lse[:, None])
    P2 = P * P
    out = P2 @ vv
    # the row's dQ: C[t, e, f] = sum_u P[t,u] (V[u,e] - O[t,e]) K[u,f] / sqrt(d)
    vkp = (v[:, :, None] * k[:, None, :]).reshape(S, d * d)
    C = ((P @ vkp).reshape(S, d, d) - o[:, :, None] * (P @ k)[:, None, :]) / np.sqrt(d)
    out += np.einsum("tef,tf->te", C * C, vq)
    # the keys' dK: sum_u P^2 (V_u - O_t)^2 (sum_f Q_t[f]^2 var_k[u,f]) / d
    W = P2 * ((q * q) @ vk_.T) / d
    out += W @ (v * v) - 2.0 * o * (W @ v) + o * o * W.sum(1)[:, None]
    return out


def right_var(var, y) -> np.ndarray:
    """Y^T-side product Z = V^T Y (a weight gradient) with V carrying errors
    of variance var and Y exact: SIGMAS standard deviations of each output."""
    y = np.asarray(y, dtype=np.float64)
    return SIGMAS * np.sqrt(np.asarray(var, dtype=np.float64).T @ (y * y))


def attention_prob_bounds(q, k, v, do):
    """Error terms of dQ, dK, dV of one (sequence, head) from the two 16-bit
    operands of the backward's second products: P rounded to bfloat16 for
    dV_u = sum_t P[t,u] dO_t, and dS = P (dP - delta) rounded to bfloat16 for
    dK_u = sum_t dS[t,u] q_t / sqrt(d) and dQ_t = sum_u dS[t,u] k_u / sqrt(d).
    Each rounding is an independent error of variance rounding_var at the
    oracle's P and dS.  Near one-hot rows (sharp scores) put P close to 1
    for many queries of one key, where these terms outgrow 1e-2 (|ref| + 1)."""
    q, k, v, do = (np.asarray(O._f64(a)) for a in (q, k, v, do))
    S, d = q.shape
    o, lse = O.attention_fwd(q, k, v)
    s = q @ k.T / np.sqrt(d)
    s[np.triu(np.ones((S, S), dtype=bool), 1)] = -np.inf
    P = np.exp(s - lse[:, None])
    dS = P * (do @ v.T - (do * o).sum(1)[:, None])
    var_p, var_ds = rounding_var(P), rounding_var(dS)
    var_p[P == 0] = 0.0
    var_ds[dS == 0] = 0.0
    bv = SIGMAS * np.sqrt(var_p.T @ (do * do))
    bk = SIGMAS / np.sqrt(d) * np.sqrt(var_ds.T @ (q * q))
    bq = SIGMAS / np.sqrt(d) * np.sqrt(var_ds @ (k * k))
    return bq, bk, bv
