"""GPU parity of gl_mrconv (fused gather-max + FC) against the CPU oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check_close, from_dev, mrconv_mag, require_gpu, to_dev
from paper_2604_21290_amd import inputs as I

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-test]", *a, flush=True)


def _mr_case(x, idx, Wt, bias=None, keys=None, label=""):
    from paper_2604_21290_amd import api
    _say("mrconv", label, tuple(x.shape), "k", idx.shape[2], "Cout", Wt.shape[0])
    out = api.mrconv(to_dev(x), torch.from_numpy(idx).cuda(), to_dev(Wt),
                     None if bias is None else to_dev(bias),
                     keys=None if keys is None else to_dev(keys))
    torch.cuda.synchronize()
    got = from_dev(out).value
    ref, xcat = O.mrconv_ref(x.value, idx, Wt.value, None if bias is None else bias.value,
                             keys=None if keys is None else keys.value, return_concat=True)
    return check_close(got, ref, x.dtype, label, mag=mrconv_mag(xcat, Wt.value),
                       n_terms=xcat.shape[-1])


@pytest.mark.parametrize("name", ["single", "vig_ti", "vig_b", "pyr_s1", "pyr_s2", "hires",
                                  "vig_ti_448", "vig_s", "pyr_s3", "pyr_s4"])
def test_mrconv_workload_full(name):
    """Full-size update with the workload's own graph (built by the oracle on
    a sample of images for speed; indices are inputs here)."""
    require_gpu()
    w = I.WORKLOADS[name]
    x = I.make_features(w)
    keys = None
    if w.pool_r > 1:
        keys = I.store(O.pool_keys_ref(x.value, w.H, w.W, w.pool_r), w.dtype)
    idx = I.random_indices(w.seed, w.B, w.N, w.k, w.M)
    # self-loop in slot 0 for the unpooled graphs, as the kNN graph has it
    if w.pool_r == 1:
        idx[:, :, 0] = np.arange(w.N)[None, :]
    Wt = I.make_weight(w, 0)
    rel = _mr_case(x, idx, Wt, I.make_bias(w, 0, zero=False), keys, label=name)
    _say(name, "max rel err", rel)


EDGE = [
    # label, B, N, M (None: keys = x), C, Cout, k, dtype, bias
    ("k1_self", 2, 30, None, 16, 16, 1, I.BF16, False),
    ("ragged_tile_rows", 3, 37, None, 24, 40, 5, I.BF16, True),
    ("cout_8", 1, 50, None, 32, 8, 3, I.BF16, True),
    ("cout_wide", 1, 20, None, 32, 200, 4, I.BF16, False),
    ("pooled_keys", 2, 64, 16, 40, 40, 9, I.BF16, True),
    ("fp32_small", 2, 21, None, 12, 20, 7, I.F32, True),
    ("fp32_vig", 1, 196, None, 192, 192, 9, I.F32, False),
    ("k_max_64", 1, 70, None, 16, 16, 64, I.BF16, True),
    ("wide_C_1024", 1, 40, None, 1024, 64, 9, I.BF16, True),
    # small grids: output columns split over workgroups (groups of 4 tiles, a
    # partial last group, ragged node tiles, fp32)
    ("cols_ragged_bf16", 2, 45, None, 64, 120, 7, I.BF16, True),
    ("cols_ragged_fp32", 1, 77, None, 48, 200, 9, I.F32, True),
    ("cols_pooled", 1, 100, 25, 96, 96, 9, I.BF16, False),
    # two-pass form (gather to [x | m], then the tiled GEMM): ragged node and
    # output tiles, a half contraction step at the end, fp32, pooled keys, k > 16
    ("split_ragged_R_Cout", 3, 70, None, 512, 300, 9, I.BF16, True),
    ("split_K_tail", 2, 45, None, 520, 264, 9, I.BF16, False),
    ("split_fp32", 2, 77, None, 320, 136, 7, I.F32, True),
    ("split_pooled", 2, 196, 49, 576, 576, 9, I.BF16, True),
    ("split_k20", 1, 150, None, 512, 512, 20, I.BF16, False),
    # 8 K nodes and more (at least 256 node tiles; C and Cout <= 256 take the
    # lean tile, on 64-node tiles when they fit 64 KB of LDS): ragged last
    # tile, a half contraction step (C % 16 == 8), narrow and wide Cout,
    # pooled keys, k = 1 and k = 16, fp32
    ("large_R_ragged", 3, 5471, None, 64, 64, 9, I.BF16, True),
    ("large_R_C72_half_step", 2, 8200, None, 72, 72, 9, I.BF16, True),
    ("large_R_cout_40", 1, 16384, None, 48, 40, 5, I.BF16, False),
    ("large_R_cout_200", 1, 16390, None, 32, 200, 9, I.BF16, True),
    ("large_R_k7_pooled", 2, 8250, 100, 32, 32, 7, I.BF16, True),
    ("large_R_k1", 1, 16384, None, 16, 16, 1, I.BF16, False),
    ("large_R_k16", 1, 16384, None, 64, 64, 16, I.BF16, True),
    ("large_R_fp32_lean", 1, 16400, None, 40, 56, 9, I.F32, True),
    ("large_R_C192_lean64", 1, 8200, None, 192, 192, 9, I.BF16, True),
    ("large_R_C256_lean32_cout200", 1, 8300, None, 256, 200, 9, I.BF16, False),
    ("large_R_fp32_C160_lean32", 1, 8300, None, 160, 96, 7, I.F32, True),
    ("large_R_C264_not_lean", 1, 8300, None, 264, 64, 9, I.BF16, True),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_mrconv_edges(case):
    require_gpu()
    label, B, N, M, C, Cout, k, dt, with_bias = case
    g = np.random.default_rng(C * 7 + N)
    x = I.store(g.standard_normal((B, N, C)), dt)
    keys = None if M is None else I.store(g.standard_normal((B, M, C)), dt)
    Mk = N if M is None else M
    idx = g.integers(0, Mk, (B, N, k)).astype(np.int32)
    if label == "k1_self":
        idx[:, :, 0] = np.arange(N)
    Wt = I.store(g.uniform(-0.2, 0.2, (Cout, 2 * C)), dt)
    bias = I.store(g.uniform(-1, 1, Cout), dt) if with_bias else None
    _mr_case(x, idx, Wt, bias, keys, label=label)


def test_mrconv_self_only_is_x_times_Wx():
    """k = 1 with each node its own neighbour: m = 0, out = x W_x^T (exact parts)."""
    require_gpu()
    from paper_2604_21290_amd import api
    g = np.random.default_rng(3)
    x = I.store(g.standard_normal((1, 32, 16)), I.BF16)
    idx = np.arange(32, dtype=np.int32)[None, :, None]
    Wi = I.store(np.hstack([np.eye(16), g.standard_normal((16, 16))]), I.BF16)
    out = api.mrconv(to_dev(x), torch.from_numpy(idx).cuda(), to_dev(Wi))
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(out).value, x.value)


def test_mrconv_deterministic():
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.with_batch(I.WORKLOADS["vig_ti"], 4)
    x = to_dev(I.make_features(w))
    idx = torch.from_numpy(I.random_indices(1, 4, w.N, w.k, w.M)).cuda()
    Wt = to_dev(I.make_weight(w, 0))
    a = api.mrconv(x, idx, Wt)
    b = api.mrconv(x, idx, Wt)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# -- multi-head update (gl_mrconv_heads) --------------------------------------------
HEADS = [
    # label, workload, batch, heads   (hd = C / heads)
    ("vig_ti_h16", "vig_ti", 4, 16),             # hd 12: steps straddle heads
    ("vig_ti_h16_b1_ragged", "vig_ti", 1, 16),   # 196 nodes: ragged node tile
    ("vig_ti_h4", "vig_ti", 4, 4),               # hd 48
    ("vig_ti_h1", "vig_ti", 2, 1),               # hd 192: one head, 6 steps a half
    ("pyr_s2_h8", "pyr_s2", 2, 8),               # hd 20, pooled keys
    ("pyr_s2_h4", "pyr_s2", 2, 4),               # hd 40
    ("pyr_s1_h20_hd4", "pyr_s1", 1, 20),         # hd 4, r = 4 pooled keys
    ("vig_b_h16", "vig_b", 2, 16),               # hd 40 at C = 640
    ("vig_b_h8", "vig_b", 4, 8),                 # hd 80
    ("single_fp32_h16", "single", 1, 16),        # fp32, hd 12
    ("single_fp32_h3", "single", 1, 3),          # fp32, hd 64
    # Wh expanded into the dense block-diagonal W in the workspace: heads of
    # a width that is no multiple of 4, or wider than 8 steps, take the fused
    # multi-head tile over it; channels too wide for the fused tile's LDS rows
    # take the two-pass update
    ("vig_ti_h32_hd6_expand", "vig_ti", 2, 32),
    ("vig_b_h2_hd320_expand", "vig_b", 1, 2),
    ("single_fp32_h48_hd4", "single", 1, 48),
    ("wide_bf16_h16_expand", I.Workload("wide_bf16", 1, 14, 14, 2560, 9, (1,), I.BF16, seed=11), 1, 16),
    ("wide_fp32_h10_expand", I.Workload("wide_fp32", 1, 7, 7, 1280, 9, (1,), I.F32, seed=12), 1, 10),
]


def _block_diag(Wh: np.ndarray) -> np.ndarray:
    """Dense [C, 2C] = [W_x | W_m] from per-head [H, hd, 2hd]."""
    H, hd = Wh.shape[0], Wh.shape[1]
    C = H * hd
    W = np.zeros((C, 2 * C))
    for h in range(H):
        W[h * hd:(h + 1) * hd, h * hd:(h + 1) * hd] = Wh[h][:, :hd]
        W[h * hd:(h + 1) * hd, C + h * hd:C + (h + 1) * hd] = Wh[h][:, hd:]
    return W


@pytest.mark.parametrize("case", HEADS, ids=[c[0] for c in HEADS])
def test_mrconv_heads(case):
    """gl_mrconv_heads with per-head Wh [H, hd, 2hd] against the oracle's
    multi-head update, each element held to the forward error bound of the
    2hd-term contraction (the dense block-diagonal W gives the same |x''||W|)."""
    require_gpu()
    from paper_2604_21290_amd import api
    label, name, B, H = case
    w = I.with_batch(name if isinstance(name, I.Workload) else I.WORKLOADS[name], B)
    x = I.make_features(w)
    keys = None
    if w.pool_r > 1:
        keys = I.store(O.pool_keys_ref(x.value, w.H, w.W, w.pool_r), w.dtype)
    idx = I.random_indices(w.seed, w.B, w.N, w.k, w.M)
    hd = w.C // H
    g = np.random.default_rng(H * 1000 + w.C)
    Wh = I.store(g.uniform(-1, 1, (H, hd, 2 * hd)) / np.sqrt(2 * hd), w.dtype)
    b = I.make_bias(w, 0, zero=False)
    _say("mrconv heads", label, "B", w.B, "N", w.N, "C", w.C, "H", H, "hd", hd)
    xd, idd = to_dev(x), torch.from_numpy(idx).cuda()
    kd = None if keys is None else to_dev(keys)
    out = api.mrconv_heads(xd, idd, to_dev(Wh), to_dev(b), keys=kd)
    torch.cuda.synchronize()
    kv = None if keys is None else keys.value
    ref = O.mrconv_heads_ref(x.value, idx, Wh.value, b.value, keys=kv)
    _, xcat = O.mrconv_ref(x.value, idx, _block_diag(Wh.value), b.value, keys=kv,
                           return_concat=True)
    check_close(from_dev(out).value, ref, w.dtype, label,
                mag=mrconv_mag(xcat, _block_diag(Wh.value)), n_terms=2 * w.C)
