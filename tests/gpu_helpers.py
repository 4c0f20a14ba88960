"""Shared checks for the GPU parity tests (test infrastructure).

Index acceptance (kNN): a row is accepted when its indices are in range, free
of duplicates, and at every output position p the oracle's float64 distance
of the GPU's index equals that of the oracle's index within 1e-5; so indices
are identical except inside near-tie windows narrower than 1e-5.

Outputs (pooling, MRConv): ||gpu - ref||_inf <= tol * ||ref||_inf with
tol = 1e-4 for fp32 and 2e-2 for bf16, where ref is the oracle evaluated on
the exact stored inputs the GPU saw (teacher forcing).
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


def ref_from_dist(D: np.ndarray, k: int, d: int) -> np.ndarray:
    """Oracle dilated lists from oracle distances [B, rows, M]."""
    return np.stack([O.knn_order(D[b], k * d)[:, ::d][:, :k] for b in range(D.shape[0])])


def check_idx(gpu_idx: np.ndarray, D: np.ndarray, k: int, d: int, rows=None, label="") -> dict:
    """gpu_idx [B, N, k]; D oracle distances [B, len(rows) or N, M]."""
    g = gpu_idx if rows is None else gpu_idx[:, rows]
    M = D.shape[-1]
    assert g.shape == D.shape[:2] + (k,), (label, g.shape, D.shape)
    assert g.min() >= 0 and g.max() < M, (label, "index out of range")
    s = np.sort(g, -1)
    dup = (s[..., 1:] == s[..., :-1]).any(-1)
    assert not dup.any(), (label, "duplicate neighbours", np.argwhere(dup)[:5])
    ref = ref_from_dist(D, k, d)
    dg = np.take_along_axis(D, g.astype(np.int64), -1)
    dr = np.take_along_axis(D, ref, -1)
    diff = np.abs(dg - dr)
    bad = diff >= NEAR_TIE
    assert not bad.any(), (label, "index mismatch beyond the near-tie window",
                           np.argwhere(bad)[:5], diff.max())
    differ = (g != ref).any(-1)
    return {"rows": int(np.prod(g.shape[:2])), "near_tie_rows": int(differ.sum()),
            "max_dist_diff": float(diff.max())}


def check_close(gpu: np.ndarray, ref: np.ndarray, dtype: str, label="") -> float:
    tol = TOL[dtype]
    err = float(np.abs(gpu - ref).max())
    scale = float(np.abs(ref).max())
    assert np.isfinite(gpu).all(), (label, "non-finite output")
    assert err <= tol * max(scale, 1e-30), (label, err, scale, err / max(scale, 1e-30))
    return err / max(scale, 1e-30)
