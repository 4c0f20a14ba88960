"""Shared checks for the GPU parity tests (test infrastructure).

Index acceptance (kNN): a row is accepted when its indices are in range, free
of duplicates, and at every output position p the oracle's float64 distance
of the GPU's index equals that of the oracle's index within 1e-5; so indices
are identical except inside near-tie windows narrower than 1e-5.

Outputs (pooling, MRConv): ||gpu - ref||_inf <= tol * ||ref||_inf with
tol = 1e-4 for fp32 and 2e-2 for bf16, where ref is the oracle evaluated on
the exact stored inputs the GPU saw (teacher forcing); the element-wise
relative error (floor tol * ||ref||_inf) is reported, and contractions are
also held element by element to their forward error bound (check_close).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle as O
from paper_2604_21290_amd import inputs as I

NEAR_TIE = 1e-5
TOL = {I.F32: 1e-4, I.BF16: 2e-2}


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2604_21290_amd import api
    api.lib()  # raises if the HIP library is missing: no silent fallback


def to_dev(s: I.Stored) -> torch.Tensor:
    if s.dtype == I.F32:
        return torch.from_numpy(np.ascontiguousarray(s.bits)).cuda()
    return torch.from_numpy(np.ascontiguousarray(s.bits).view(np.int16)).cuda().view(torch.bfloat16)


def from_dev(t: torch.Tensor) -> I.Stored:
    if t.dtype == torch.float32:
        return I.from_bits(t.detach().cpu().numpy(), I.F32)
    if t.dtype == torch.bfloat16:
        return I.from_bits(t.detach().view(torch.int16).cpu().numpy().view(np.uint16), I.BF16)
    raise TypeError(t.dtype)


def check_idx(gpu_idx: np.ndarray, D: np.ndarray, k: int, d: int, rows=None, label="") -> dict:
    """gpu_idx [B, N, k]; D = oracle.knn_distances [B, len(rows) or N, M].  The
    reference lists are oracle.dilated_lists(D, k, d) (both pinned)."""
    g = gpu_idx if rows is None else gpu_idx[:, rows]
    M = D.shape[-1]
    assert g.shape == D.shape[:2] + (k,), (label, g.shape, D.shape)
    assert g.min() >= 0 and g.max() < M, (label, "index out of range")
    s = np.sort(g, -1)
    dup = (s[..., 1:] == s[..., :-1]).any(-1)
    assert not dup.any(), (label, "duplicate neighbours", np.argwhere(dup)[:5])
    ref = O.dilated_lists(D, k, d)
    dg = np.take_along_axis(D, g.astype(np.int64), -1)
    dr = np.take_along_axis(D, ref, -1)
    diff = np.abs(dg - dr)
    bad = diff >= NEAR_TIE
    assert not bad.any(), (label, "index mismatch beyond the near-tie window",
                           np.argwhere(bad)[:5], diff.max())
    differ = (g != ref).any(-1)
    return {"rows": int(np.prod(g.shape[:2])), "near_tie_rows": int(differ.sum()),
            "max_dist_diff": float(diff.max())}


UNIT_ROUNDOFF = {I.F32: 2.0 ** -24, I.BF16: 2.0 ** -8}
ELEM_LOG = []   # (label, element-wise relative error) of every check_close call


def check_close(gpu: np.ndarray, ref: np.ndarray, dtype: str, label="", mag=None,
                n_terms: int = 0) -> float:
    """Norm-scaled bound ||gpu - ref||_inf <= tol ||ref||_inf (tol 1e-4 fp32,
    2e-2 bf16), plus the element-wise relative error
        e_i = |gpu_i - ref_i| / max(|ref_i|, tol ||ref||_inf),
    which is reported (printed, and kept in ELEM_LOG).

    With mag (per element, the sum of |products| the output is a contraction
    of, e.g. |x''| @ |W|^T) every element is also held to the forward error
    bound of one stored-type rounding of the contraction's operands and of the
    output plus an n_terms-long fp32 accumulation:
        |gpu_i - ref_i| <= 2u (|ref_i| + mag_i) + n_terms 2^-24 mag_i,
    with u the unit roundoff of the stored type (2^-8 bf16, 2^-24 fp32).  (A
    constant element-wise bound of tol cannot hold where the output cancels:
    the bf16 rounding of the max-relative half alone gives e_i of several tol
    there.)  Returns the norm-scaled relative error."""
    tol = TOL[dtype]
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (label, gpu.shape, ref.shape)
    assert np.isfinite(gpu).all(), (label, "non-finite output")
    d = np.abs(gpu - ref)
    err = float(d.max()) if d.size else 0.0
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    assert err <= tol * max(scale, 1e-30), (label, err, scale, err / max(scale, 1e-30))
    elem = float((d / np.maximum(np.abs(ref), max(tol * scale, 1e-30))).max()) if d.size else 0.0
    ELEM_LOG.append((label, elem))
    if mag is not None:
        u = UNIT_ROUNDOFF[dtype]
        mag = np.asarray(mag, dtype=np.float64)
        bound = 2 * u * (np.abs(ref) + mag) + n_terms * 2.0 ** -24 * mag
        over = d > bound
        assert not over.any(), (label, "element beyond its forward error bound",
                                np.argwhere(over)[:5], float((d / np.maximum(bound, 1e-300)).max()))
    print(f"[check] {label}: norm-scaled rel err {err / max(scale, 1e-30):.3e}, "
          f"element-wise rel err {elem:.3e}", flush=True)
    return err / max(scale, 1e-30)


def mrconv_mag(xcat: np.ndarray, W: np.ndarray) -> np.ndarray:
    """Per output element, sum_c |x''_c W_oc| (the oracle's concatenation and W)."""
    return np.abs(xcat) @ np.abs(np.asarray(W, dtype=np.float64)).T
