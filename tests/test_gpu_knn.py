"""GPU parity of gl_knn_graph and gl_pool_keys against the CPU oracle."""
import zlib

import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check_close, check_idx, from_dev, require_gpu, to_dev
from paper_2604_21290_amd import inputs as I

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-test]", *a, flush=True)


def _knn_case(x: I.Stored, k, d, keys: I.Stored | None = None, rows=None, label=""):
    from paper_2604_21290_amd import api
    xd = to_dev(x)
    kd = to_dev(keys) if keys is not None else None
    _say("knn", label, tuple(x.shape), "M", None if keys is None else keys.shape[1], "k", k, "d", d)
    idx = api.knn_graph(xd, k, d, keys=kd)
    torch.cuda.synchronize()
    D = O.knn_distances(x.value, None if keys is None else keys.value, rows=rows)
    return check_idx(idx.cpu().numpy(), D, k, d, rows=rows, label=label)


# -- the workloads at full size (sampled rows where N = 3136) -----------------
@pytest.mark.parametrize("name", ["single", "vig_ti", "vig_b", "hires", "vig_ti_448", "vig_s",
                                  "pyr_s3", "pyr_s4"])
def test_knn_workload_full(name):
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.WORKLOADS[name]
    x = I.make_features(w)
    rows = None
    if w.N > 500:
        rows = np.sort(np.random.default_rng(99).choice(w.N, 384, replace=False))
    xd = to_dev(x)
    D = O.knn_distances(x.value, rows=rows)
    for d in sorted(set(w.dilations)):
        _say("knn", name, "d", d)
        idx = api.knn_graph(xd, w.k, d)
        torch.cuda.synchronize()
        st = check_idx(idx.cpu().numpy(), D, w.k, d, rows=rows, label=f"{name} d={d}")
        _say(name, "d", d, st)


@pytest.mark.parametrize("name", ["pyr_s1", "pyr_s2"])
def test_knn_pooled_workload_full(name):
    """Pooled keys: the pool is checked against the oracle pool, and the graph
    against the oracle evaluated on the GPU's stored keys (teacher forcing)."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.WORKLOADS[name]
    x = I.make_features(w)
    xd = to_dev(x)
    _say("pool", name)
    keys = api.pool_keys(xd, w.H, w.W, w.pool_r)
    torch.cuda.synchronize()
    ks = from_dev(keys)
    check_close(ks.value, O.pool_keys_ref(x.value, w.H, w.W, w.pool_r), w.dtype, f"pool {name}")
    rows = np.sort(np.random.default_rng(98).choice(w.N, min(w.N, 512), replace=False))
    idx = api.knn_graph(xd, w.k, w.dilations[0], keys=keys)
    torch.cuda.synchronize()
    D = O.knn_distances(x.value, ks.value, rows=rows)
    _say(name, check_idx(idx.cpu().numpy(), D, w.k, w.dilations[0], rows=rows, label=name))


# -- edge cases -------------------------------------------------------------------
EDGE = [
    # label, B, N, M (None = keys are x), C, k, d, dtype, features
    ("ragged_rows_k1", 2, 37, None, 8, 1, 1, I.BF16, "unit"),
    ("k_equals_M_fp32", 1, 5, None, 4, 5, 1, I.F32, "unit"),
    ("k_equals_M_bf16", 1, 16, None, 16, 16, 1, I.BF16, "unit"),
    ("pooled_like_small_M", 2, 50, 13, 16, 4, 3, I.BF16, "unit"),
    ("chunk_boundary_257_maxKK", 1, 70, 257, 32, 16, 4, I.BF16, "unit"),
    ("three_chunks", 2, 100, 600, 24, 9, 2, I.BF16, "normal"),
    ("max_M_4096", 1, 48, 4096, 16, 16, 4, I.BF16, "unit"),
    ("max_M_fp32", 1, 33, 4096, 8, 8, 8, I.F32, "unit"),
    ("C_tail_bf16", 2, 60, None, 40, 9, 1, I.BF16, "unit"),
    ("C_tail_fp32", 2, 60, None, 12, 9, 3, I.F32, "unit"),
    ("wide_C_bf16", 1, 40, None, 1024, 9, 4, I.BF16, "unit"),
    ("unnormalised_fp32", 3, 196, None, 192, 9, 2, I.F32, "normal"),
    ("KK_33_R4", 1, 196, None, 64, 11, 3, I.BF16, "normal"),
    # streamed-key kernel (M > 256): ragged last chunk, widest rows, fp32
    ("stream_ragged_M333", 2, 90, 333, 96, 16, 2, I.BF16, "normal"),
    ("stream_wide_C768_bf16", 1, 70, 300, 768, 9, 1, I.BF16, "unit"),
    ("stream_wide_C384_fp32", 1, 70, 300, 384, 9, 2, I.F32, "normal"),
    ("stream_C160_R4", 2, 64, 784, 160, 16, 4, I.BF16, "unit"),
    ("stream_fp32_C96", 1, 130, 3136, 96, 16, 2, I.F32, "normal"),
    # more than 256 workgroups of 128 rows: the four-wave form of the narrow rows
    ("stream_four_waves_B33", 33, 1000, 400, 64, 9, 2, I.BF16, "normal"),
    # LDS-staged wide kernel (bf16, C >= 256, M <= 256): key-row buckets 64 / 128 /
    # 224 / 256, a partial last stage (C = 520), K' = 64, one query row
    ("wide_M64_bucket", 2, 50, 64, 512, 9, 2, I.BF16, "unit"),
    ("wide_M65_C520_KK64", 1, 33, 65, 520, 16, 4, I.BF16, "normal"),
    ("wide_M200_ragged", 3, 97, 200, 512, 9, 3, I.BF16, "unit"),
    ("wide_M256_max", 1, 70, 256, 640, 16, 2, I.BF16, "unit"),
    ("wide_self_unnormalised", 2, 196, None, 640, 9, 1, I.BF16, "normal"),
    ("wide_N1", 2, 1, 30, 512, 3, 1, I.BF16, "unit"),
    ("wide_C264_partial", 2, 45, 100, 264, 9, 2, I.BF16, "normal"),
]


@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_knn_edges(case):
    require_gpu()
    label, B, N, M, C, k, d, dt, feat = case
    seed = zlib.crc32(label.encode()) % 10000
    x = I.random_features(seed, B, N, C, dt, unit=(feat == "unit"))
    keys = None if M is None else I.random_features(seed + 1, B, M, C, dt, unit=(feat == "unit"))
    _say(label, _knn_case(x, k, d, keys, label=label))


# Keys resident in LDS, 64 query rows per workgroup (bf16, M <= 256, 32 < C <=
# 160, at least 384 workgroups): every key-tile bucket (4 / 8 / 13 / 16 tiles),
# two to five contraction steps' worth of channels with partial last steps,
# both norm orders (below and from C = 128), K' up to 64, ragged last row
# tiles.  Sampled rows keep the oracle fast.
RESIDENT = [
    # label, B, N, M, C, k, d
    ("res_pyr_like_ragged", 16, 2049, 196, 80, 9, 1),
    ("res_C40_M100_KK18", 32, 1000, 100, 40, 9, 2),
    ("res_C128_M256_KK64", 8, 4100, 256, 128, 16, 4),
    ("res_C72_M64", 16, 2048, 64, 72, 9, 3),
    ("res_C56_M209", 16, 2048, 209, 56, 9, 1),
    ("res_C96_M17_k1", 16, 2047, 17, 96, 1, 1),
    ("res_C128_wide_order", 16, 1600, 196, 128, 9, 1),
    ("res_C136_M150_KK18", 32, 800, 150, 136, 9, 2),
    ("res_C160_M256_KK64", 8, 3100, 256, 160, 16, 4),
    # 8-wave workgroups of 128 rows (at most 256 of them), a 12-row last tile
    ("res_8_waves_tail12", 2, 12300, 200, 64, 9, 2),
]


@pytest.mark.parametrize("case", RESIDENT, ids=[c[0] for c in RESIDENT])
def test_knn_resident(case):
    require_gpu()
    label, B, N, M, C, k, d = case
    seed = zlib.crc32(label.encode()) % 10000
    x = I.random_features(seed, B, N, C, I.BF16, unit=False)
    keys = I.random_features(seed + 1, B, M, C, I.BF16, unit=False)
    rows = np.sort(np.random.default_rng(seed).choice(N, 256, replace=False))
    _say(label, _knn_case(x, k, d, keys, rows=rows, label=label))


def test_knn_resident_duplicates_and_zero_rows():
    """Zero query rows, zero key rows and duplicated key rows on the
    resident-key kernel: ties resolve to the lower key index."""
    require_gpu()
    g = np.random.default_rng(11)
    B, N, M, C = 8, 4096, 150, 64
    a = g.standard_normal((B, N, C))
    kv = g.standard_normal((B, M, C))
    a[:, ::7] = 0.0
    kv[:, 10] = 0.0
    kv[:, 20:40] = kv[:, 0:20]
    x = I.store(a, I.BF16)
    keys = I.store(kv, I.BF16)
    rows = np.sort(np.concatenate([np.arange(0, 70, 7), g.choice(N, 246, replace=False)]))
    rows = np.unique(rows)
    for d in (1, 3):
        _say("resident dup/zero", _knn_case(x, 9, d, keys, rows=rows, label=f"res dup d={d}"))


@pytest.mark.parametrize("C", [32, 512])
def test_knn_duplicates_and_zero_rows(C):
    require_gpu()
    g = np.random.default_rng(5)
    a = g.standard_normal((2, 64, C))
    a[:, 40] = a[:, 3]          # exact duplicate: row 40's nearest must be 3
    a[:, 50] = a[:, 3]
    a[:, 10] = 0.0              # zero rows
    a[:, 20] = 0.0
    for dt in (I.BF16, I.F32):
        x = I.store(a, dt)
        st = _knn_case(x, 6, 1, label=f"dups {dt}")
        from paper_2604_21290_amd import api
        idx = api.knn_graph(to_dev(x), 6, 1).cpu().numpy()
        assert (idx[:, 40, :3] == [3, 40, 50]).all() and (idx[:, 3, :3] == [3, 40, 50]).all()
        assert set(idx[0, 10, :2]) == {10, 20}
        _say("dups", dt, st)


def test_knn_clustered_mixture_small():
    require_gpu()
    w = I.Workload("mix", 2, 20, 20, 32, 16, (2,), I.BF16, seed=77, features="mixture")
    x = I.make_features(w)
    _say(_knn_case(x, 16, 2, label="mixture 20x20"))


def test_knn_deterministic():
    require_gpu()
    from paper_2604_21290_amd import api
    x = to_dev(I.make_features(I.with_batch(I.WORKLOADS["hires"], 2)))
    a = api.knn_graph(x, 16, 2)
    b = api.knn_graph(x, 16, 2)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_pool_edges():
    require_gpu()
    from paper_2604_21290_amd import api
    # windows of r = 2 and 4 take the kernels that issue the whole window at
    # once (both storage types); r = 1 and 3 take the loop
    for (B, H, W, C, r, dt) in [(2, 8, 12, 16, 4, I.BF16), (1, 6, 6, 8, 3, I.F32),
                                (3, 10, 10, 24, 1, I.BF16), (1, 28, 28, 160, 2, I.F32),
                                (2, 8, 16, 12, 4, I.F32), (3, 6, 10, 40, 2, I.BF16)]:
        x = I.random_features(H * W + C, B, H * W, C, dt, unit=False)
        _say("pool", B, H, W, C, r, dt)
        k = api.pool_keys(to_dev(x), H, W, r)
        torch.cuda.synchronize()
        got = from_dev(k).value
        check_close(got, O.pool_keys_ref(x.value, H, W, r), dt, "pool edge")
        if r == 1:
            assert np.array_equal(got, x.value)
