"""Shared test helpers: tolerance check and device plumbing (no method arithmetic)."""
import numpy as np
import torch

DEV = "cuda:0"

# Tolerance for floating-point parity with the fp64 oracle (bf16 inputs,
# fp32 accumulation, bf16-rounded activations): elementwise
# |gpu - ref| <= 1e-2 * (|ref| + 1) and relative Frobenius error <= 5e-3.
ELEM_TOL = 1e-2
FROB_TOL = 5e-3


def to64(t) -> np.ndarray:
    if isinstance(t, np.ndarray):
        return t.astype(np.float64)
    return t.detach().to("cpu", torch.float64).numpy()


def assert_close(gpu, ref, what="", elem_tol=ELEM_TOL, frob_tol=FROB_TOL):
    g = to64(gpu)
    r = to64(ref)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    assert np.all(np.isfinite(g)), f"{what}: non-finite values"
    err = np.abs(g - r)
    bound = elem_tol * (np.abs(r) + 1.0)
    bad = err > bound
    if bad.any():
        idx = np.argwhere(bad)[0]
        raise AssertionError(f"{what}: {bad.sum()} elements out of tolerance, first at "
                             f"{tuple(idx)}: gpu={g[tuple(idx)]} ref={r[tuple(idx)]}")
    nr = np.linalg.norm(r)
    if nr > 0:
        rel = np.linalg.norm(g - r) / nr
        assert rel <= frob_tol, f"{what}: relative Frobenius error {rel:.3e} > {frob_tol}"
    return float(err.max()) if err.size else 0.0


def dev(t: torch.Tensor) -> torch.Tensor:
    return t.to(DEV)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round fp64 values to bf16 (RNE) -- used only to build GPU inputs."""
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).to(torch.bfloat16).to(
        torch.float64).numpy()
