"""Pins for the CPU oracle: checks against closed forms, hand-derived cases,
invariants and independent pure-Python brute force.

Each pin takes an oracle-like namespace `ref` (with knn_ref, max_relative_ref,
mrconv_ref, pool_keys_ref, max_pool_nodes_ref, stack_ref, gelu_ref, linear_ref,
vig_block_ref, vig_stack_ref) and raises AssertionError on failure, so
the same pins run against the oracle (test_oracle_pins.py) and against copies
of it with planted mistakes (test_oracle_mutants.py), which every mistake must
fail at least one pin.
"""
from __future__ import annotations

import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def circle5():
    with open(os.path.join(GOLDEN, "circle5.json")) as f:
        g = json.load(f)
    ang = [math.radians(a) for a in g["angles_deg"]]
    # exact coordinates where they exist
    pts = []
    for a, deg in zip(ang, g["angles_deg"]):
        if deg == 0:
            pts.append((1.0, 0.0))
        elif deg == 90:
            pts.append((0.0, 1.0))
        elif deg == 180:
            pts.append((-1.0, 0.0))
        else:
            pts.append((math.cos(a), math.sin(a)))
    return g, ang, np.array(pts)[None]  # [1, 5, 2]


# ---------------------------------------------------------------------------
# pure-Python brute force (no numpy arithmetic), tiny inputs only
# ---------------------------------------------------------------------------
def _bf_unit(row):
    n = math.sqrt(math.fsum(v * v for v in row))
    n = max(n, 1e-12)
    return [v / n for v in row]


def bf_knn(x, k, d, keys=None):
    """Brute-force dilated kNN: explicit loops, (distance, index) tuples sorted
    lexicographically, ranks 0, d, ..., (k-1)d."""
    x = np.asarray(x).tolist()
    keys = x if keys is None else np.asarray(keys).tolist()
    out = []
    for b in range(len(x)):
        Ks = [_bf_unit(r) for r in keys[b]]
        rows = []
        for q in x[b]:
            qu = _bf_unit(q)
            cand = []
            for j, kv in enumerate(Ks):
                s = math.fsum((a - c) ** 2 for a, c in zip(qu, kv))
                cand.append((s, j))
            cand.sort()
            rows.append([cand[t * d][1] for t in range(k)])
        out.append(rows)
    return np.array(out)


def bf_mrconv(x, idx, W, bias, keys=None):
    x = np.asarray(x).tolist()
    keys = x if keys is None else np.asarray(keys).tolist()
    W = np.asarray(W).tolist()
    idx = np.asarray(idx).tolist()
    B, N, C = len(x), len(x[0]), len(x[0][0])
    Cout = len(W)
    out = np.zeros((B, N, Cout))
    for b in range(B):
        for i in range(N):
            m = []
            for c in range(C):
                m.append(max(keys[b][j][c] - x[b][i][c] for j in idx[b][i]))
            cat = list(x[b][i]) + m
            for o in range(Cout):
                s = math.fsum(cat[c] * W[o][c] for c in range(2 * C))
                out[b, i, o] = s + (0.0 if bias is None else bias[o])
    return out


# ---------------------------------------------------------------------------
# kNN pins
# ---------------------------------------------------------------------------
def pin_circle_closed_form_fixture(ref):
    """The fixture's lists equal the closed form 2 - 2cos(dtheta), sorted."""
    g, ang, _ = circle5()
    n = len(ang)
    for key, k, d in (("knn_k3_d1", 3, 1), ("knn_k2_d2", 2, 2), ("knn_k2_d1", 2, 1)):
        rows = []
        for i in range(n):
            cand = sorted((round(2 - 2 * math.cos(ang[i] - ang[j]), 12), j) for j in range(n))
            rows.append([cand[t * d][1] for t in range(k)])
        assert rows == g[key], key


def pin_circle_knn(ref):
    g, _, x = circle5()
    for key, k, d in (("knn_k3_d1", 3, 1), ("knn_k2_d2", 2, 2), ("knn_k2_d1", 2, 1)):
        got = ref.knn_ref(x, k, d)[0].tolist()
        assert got == g[key], (key, got)


def pin_knn_bruteforce(ref):
    rng = np.random.default_rng(11)
    for trial in range(6):
        B, N, C = 2, int(rng.integers(3, 14)), int(rng.integers(1, 7))
        x = rng.standard_normal((B, N, C))
        if trial % 2 == 0:
            x[:, N // 2] = x[:, 0]          # exact duplicate rows -> exact ties
        k = int(rng.integers(1, 4))
        d = int(rng.integers(1, 3))
        if k * d > N:
            k, d = 1, 1
        assert np.array_equal(ref.knn_ref(x, k, d), bf_knn(x, k, d)), trial
        # pooled-style: keys different from queries, M != N
        M = int(rng.integers(k * d, 12)) if k * d < 12 else k * d
        keys = rng.standard_normal((B, M, C))
        assert np.array_equal(ref.knn_ref(x, k, d, keys=keys), bf_knn(x, k, d, keys)), trial


def pin_knn_self_first(ref):
    rng = np.random.default_rng(12)
    x = rng.standard_normal((3, 40, 8))
    idx, D = ref.knn_ref(x, 5, 1, return_dist=True)
    assert np.array_equal(idx[:, :, 0], np.broadcast_to(np.arange(40), (3, 40)))
    assert np.allclose(np.take_along_axis(D, idx[:, :, :1], 2), 0.0, atol=1e-12)


def pin_knn_duplicates_lower_index(ref):
    rng = np.random.default_rng(13)
    x = rng.standard_normal((1, 30, 6))
    x[0, 17] = x[0, 4]
    idx = ref.knn_ref(x, 3, 1)
    assert idx[0, 17, 0] == 4 and idx[0, 17, 1] == 17
    assert idx[0, 4, 0] == 4 and idx[0, 4, 1] == 17


def _near_tie_free(D, kk, gap=1e-9):
    s = np.sort(D, axis=-1)
    return np.all(np.abs(s[..., kk] - s[..., kk - 1]) > gap) if s.shape[-1] > kk else True


def pin_knn_permutation_equivariant(ref):
    rng = np.random.default_rng(14)
    x = rng.standard_normal((2, 50, 12))
    k = 6
    perm = rng.permutation(50)
    inv = np.argsort(perm)
    a = ref.knn_ref(x, k, 1)
    b = ref.knn_ref(x[:, perm], k, 1)          # row p of b is node perm[p]
    # map b's neighbour ids back to original ids and rows back to original order
    b_mapped = perm[b][:, inv]
    assert np.array_equal(np.sort(a, -1), np.sort(b_mapped, -1))
    assert np.array_equal(a, b_mapped)         # same order too (no near ties here)


def pin_knn_scale_invariant(ref):
    rng = np.random.default_rng(15)
    x = rng.standard_normal((2, 45, 10))
    assert np.array_equal(ref.knn_ref(x, 7, 2), ref.knn_ref(3.0 * x, 7, 2))
    assert np.array_equal(ref.knn_ref(x, 7, 2), ref.knn_ref(0.125 * x, 7, 2))


def pin_knn_dilation_consistency(ref):
    rng = np.random.default_rng(16)
    x = rng.standard_normal((2, 60, 9))
    for k, d in ((4, 2), (3, 3), (9, 4)):
        full = ref.knn_ref(x, k * d, 1)
        assert np.array_equal(ref.knn_ref(x, k, d), full[:, :, ::d])


def pin_knn_full_is_permutation(ref):
    rng = np.random.default_rng(17)
    x = rng.standard_normal((2, 23, 5))
    idx = ref.knn_ref(x, 23, 1)
    assert np.array_equal(np.sort(idx, -1), np.broadcast_to(np.arange(23), idx.shape))


def pin_knn_zero_rows(ref):
    x = np.zeros((1, 4, 3))
    x[0, 1] = (1.0, 0.0, 0.0)
    x[0, 2] = (0.0, 2.0, 0.0)
    x[0, 3] = (0.0, 0.0, 0.0)
    idx, D = ref.knn_ref(x, 4, 1, return_dist=True)
    # zero row 0: distance 0 to the other zero row 3 and to itself, 1 to unit rows
    assert idx[0, 0].tolist() == [0, 3, 1, 2]
    assert np.allclose(D[0, 0], [0, 1, 1, 0])
    assert idx[0, 1].tolist() == [1, 0, 3, 2]   # d(1,0)=1=d(1,3) < d(1,2)=2


def pin_knn_sorted_by_distance(ref):
    rng = np.random.default_rng(18)
    x = rng.standard_normal((2, 64, 16))
    idx, D = ref.knn_ref(x, 12, 1, return_dist=True)
    dsel = np.take_along_axis(D, idx, 2)
    assert np.all(np.diff(dsel, axis=-1) >= 0)
    # the k-th selected is no farther than every unselected node
    mask = np.ones_like(D, dtype=bool)
    np.put_along_axis(mask, idx, False, 2)
    assert np.all(dsel[..., -1:] <= np.where(mask, D, np.inf).min(-1, keepdims=True))


# ---------------------------------------------------------------------------
# distances and dilated lists on their own (what the GPU parity tests rank
# against): knn_distances and dilated_lists
# ---------------------------------------------------------------------------
def bf_sq_dist(x, keys=None, rows=None):
    """Pure-Python squared distances between the normalised query rows `rows`
    of x and every normalised key row, [B, len(rows), M]."""
    xl = np.asarray(x).tolist()
    kl = xl if keys is None else np.asarray(keys).tolist()
    rows = list(range(len(xl[0]))) if rows is None else [int(r) for r in rows]
    out = []
    for b in range(len(xl)):
        Ks = [_bf_unit(r) for r in kl[b]]
        out.append([[math.fsum((a - c) ** 2 for a, c in zip(_bf_unit(xl[b][i]), kv)) for kv in Ks]
                    for i in rows])
    return np.array(out)


def _dist_cases(seed, zero_query=True):
    """Tiny inputs with zero rows, duplicate rows, keys of unequal norms
    (pooled-style, M != N) and query-row subsets.  (A zero query row is at
    distance |k|^2 = 1 from every key up to rounding, so its order is a
    near-tie everywhere; the list pin leaves it out.)"""
    rng = np.random.default_rng(seed)
    for trial in range(4):
        B, N, C = 2, int(rng.integers(5, 12)), int(rng.integers(2, 6))
        x = rng.standard_normal((B, N, C)) * rng.uniform(0.2, 4.0, (B, N, 1))
        if zero_query:
            x[:, 1] = 0.0
        x[:, N - 1] = x[:, 2]
        M = int(rng.integers(4, 10))
        keys = rng.standard_normal((B, M, C)) * rng.uniform(0.2, 4.0, (B, M, 1))
        keys[:, M - 1] = 0.0
        rows = np.sort(rng.choice(N, int(rng.integers(2, N)), replace=False))
        yield trial, x, keys, rows


def pin_knn_distances_bruteforce(ref):
    for trial, x, keys, rows in _dist_cases(31):
        for kk, rr in ((None, None), (keys, None), (None, rows), (keys, rows)):
            got = ref.knn_distances(x, kk, rows=rr)
            want = bf_sq_dist(x, kk, rr)
            assert got.shape == want.shape, (trial, got.shape, want.shape)
            assert np.allclose(got, want, rtol=0, atol=1e-12), (trial, np.abs(got - want).max())


def pin_knn_distances_circle(ref):
    """Unit vectors at angles a_i: D[i, j] = 2 - 2 cos(a_i - a_j), exactly 0 on
    the diagonal; scaling a row does not change it."""
    g, ang, x = circle5()
    want = np.array([[2 - 2 * math.cos(a - b) for b in ang] for a in ang])
    got = ref.knn_distances(x * np.array([1.0, 3.0, 0.5, 2.0, 7.0])[None, :, None])[0]
    assert np.allclose(got, want, rtol=0, atol=1e-12)
    assert np.all(np.diag(got) == 0.0)


def pin_dilated_lists_bruteforce(ref):
    """Lists by a (distance, index) tuple sort, on distances with many exact ties."""
    rng = np.random.default_rng(32)
    D = rng.integers(0, 4, size=(2, 7, 13)).astype(np.float64)
    for k, d in ((1, 1), (3, 1), (4, 2), (3, 4), (13, 1), (2, 6)):
        want = [[[sorted((D[b, i, j], j) for j in range(13))[t * d][1] for t in range(k)]
                 for i in range(7)] for b in range(2)]
        assert np.array_equal(ref.dilated_lists(D, k, d), np.array(want)), (k, d)


def pin_distance_lists_are_knn_ref(ref):
    """dilated_lists(knn_distances(...)) is the graph knn_ref and the loop
    brute force give, for pooled-style keys, row subsets and d = 1..4; the
    distances knn_ref returns are the brute-force ones."""
    for trial, x, keys, rows in _dist_cases(33, zero_query=False):
        M = keys.shape[1]
        for d in (1, 2, 3, 4):
            k = max(1, min(3, M // d))
            for kk, rr in ((keys, rows), (None, rows), (keys, None)):
                idx, D = ref.knn_ref(x, k, d, keys=kk, rows=rr, return_dist=True)
                lists = ref.dilated_lists(ref.knn_distances(x, kk, rows=rr), k, d)
                assert np.array_equal(lists, idx), (trial, d)
                bf = bf_knn(x, k, d, kk)
                assert np.array_equal(idx, bf if rr is None else bf[:, rr]), (trial, d)
                assert np.allclose(D, bf_sq_dist(x, kk, rr), rtol=0, atol=1e-12), (trial, d)


# ---------------------------------------------------------------------------
# MRConv pins
# ---------------------------------------------------------------------------
def pin_circle_mrconv(ref):
    g, _, x = circle5()
    idx = np.array(g["knn_k3_d1"])[None]
    m = ref.max_relative_ref(x, idx)
    assert np.allclose(m[0, 0], g["mrconv_k3_m0"], atol=1e-15)
    assert np.allclose(m[0, 3], g["mrconv_k3_m3"], atol=1e-15)
    # W = [0 | I]: the output is the max-relative part; W = [I | 0]: the input
    W = np.hstack([np.zeros((2, 2)), np.eye(2)])
    assert np.allclose(ref.mrconv_ref(x, idx, W)[0, 0], [0.0, 1.0], atol=1e-15)
    W = np.hstack([np.eye(2), np.zeros((2, 2))])
    assert np.allclose(ref.mrconv_ref(x, idx, W), x, atol=0)


def pin_mrconv_bruteforce(ref):
    rng = np.random.default_rng(21)
    for trial in range(4):
        B, N, C, Cout, k = 2, 7, 3, 4, 3
        x = rng.standard_normal((B, N, C))
        idx = rng.integers(0, N, (B, N, k))
        W = rng.standard_normal((Cout, 2 * C))
        bias = rng.standard_normal(Cout)
        assert np.allclose(ref.mrconv_ref(x, idx, W, bias), bf_mrconv(x, idx, W, bias),
                           rtol=0, atol=1e-12), trial
        M = 5
        keys = rng.standard_normal((B, M, C))
        idk = rng.integers(0, M, (B, N, k))
        assert np.allclose(ref.mrconv_ref(x, idk, W, bias, keys=keys),
                           bf_mrconv(x, idk, W, bias, keys), rtol=0, atol=1e-12), trial


def pin_mrconv_self_only(ref):
    rng = np.random.default_rng(22)
    x = rng.standard_normal((2, 9, 4))
    idx = np.broadcast_to(np.arange(9)[None, :, None], (2, 9, 1)).copy()
    assert np.array_equal(ref.max_relative_ref(x, idx), np.zeros_like(x))
    W = rng.standard_normal((5, 8))
    bias = rng.standard_normal(5)
    want = np.einsum("bnc,oc->bno", x, W[:, :4]) + bias
    assert np.allclose(ref.mrconv_ref(x, idx, W, bias), want, atol=1e-12)


def pin_mrconv_translation(ref):
    rng = np.random.default_rng(23)
    x = rng.standard_normal((2, 11, 5))
    idx = rng.integers(0, 11, (2, 11, 4))
    v = rng.standard_normal(5)
    assert np.allclose(ref.max_relative_ref(x + v, idx), ref.max_relative_ref(x, idx), atol=1e-12)


def pin_mrconv_max_minus(ref):
    """max_t (y_t - x) == (max_t y_t) - x exactly (rounding is monotone)."""
    rng = np.random.default_rng(24)
    x = rng.standard_normal((1, 13, 6))
    idx = rng.integers(0, 13, (1, 13, 5))
    nb = x[0][idx[0]]                      # [13, 5, 6]
    want = nb.max(axis=1) - x[0]
    assert np.array_equal(ref.max_relative_ref(x, idx)[0], want)


def pin_mrconv_bias_only(ref):
    rng = np.random.default_rng(25)
    x = rng.standard_normal((1, 6, 3))
    idx = rng.integers(0, 6, (1, 6, 2))
    bias = np.array([0.5, -2.0])
    out = ref.mrconv_ref(x, idx, np.zeros((2, 6)), bias)
    assert np.array_equal(out, np.broadcast_to(bias, (1, 6, 2)))


# ---------------------------------------------------------------------------
# key pooling pins
# ---------------------------------------------------------------------------
def pin_pool_closed_form(ref):
    H, W, r, C = 8, 12, 4, 3
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    x = np.zeros((2, H * W, C))
    x[..., 0] = yy.ravel()
    x[..., 1] = xx.ravel()
    x[..., 2] = 5.0
    k = ref.pool_keys_ref(x, H, W, r)
    Wr = W // r
    for p in range(H // r):
        for q in range(Wr):
            assert np.allclose(k[:, p * Wr + q], [p * r + (r - 1) / 2, q * r + (r - 1) / 2, 5.0])
    assert np.array_equal(ref.pool_keys_ref(x, H, W, 1), x)


# ---------------------------------------------------------------------------
# stack pins
# ---------------------------------------------------------------------------
def pin_stack_single_layer(ref):
    rng = np.random.default_rng(31)
    x = rng.standard_normal((2, 16, 4))
    W = rng.standard_normal((4, 8))
    out = ref.stack_ref(x, [W], [None], (1,), 3, 4, 4)
    assert np.allclose(out, ref.mrconv_ref(x, ref.knn_ref(x, 3, 1), W), atol=1e-12)


def pin_stack_identity_weights(ref):
    rng = np.random.default_rng(32)
    x = rng.standard_normal((2, 16, 4))
    Wi = np.hstack([np.eye(4), np.zeros((4, 4))])
    a = ref.stack_ref(x, [Wi] * 4, None, (1, 1, 2, 2), 3, 4, 4, schedule="lookahead")
    b = ref.stack_ref(x, [Wi] * 4, None, (1, 1, 2, 2), 3, 4, 4, schedule="standard")
    assert np.array_equal(a, x) and np.array_equal(b, x)


def pin_stack_circle_two_blocks(ref):
    """Two blocks on the circle with W = [0 | I], k = 2, d = 1, worked by hand.

    Block 0 uses G(X^0): neighbours {0,1}, {1,0}, {2,1}, {3,4}, {4,3}, so
    X^1 = max(0, x_nb - x_i) = (0, 1/2), (1 - c30, 0), (c30, 0), (1 - c20, 0), (0, s20).
    Lookahead block 1 reuses G(X^0):
    X^2 = (1 - c30, 0), (0, 1/2), (0, 0), (0, s20), (1 - c20, 0).
    The standard schedule rebuilds G(X^1).  Normalised, rows 0 and 4 are (0, 1)
    and rows 1-3 are (1, 0) exactly, so distances are exact 0/2 ties and the
    lower index wins: neighbours {0,4}, {1,2}, {1,2}, {1,2}, {0,4} (node 3 is
    not its own neighbour), giving
    X^2 = (0, 0), (2c30 - 1, 0), (0, 0), (c30 + c20 - 1, 0), (0, 1/2 - s20).
    """
    _, _, x = circle5()
    c30, c20, s20 = math.cos(math.pi / 6), math.cos(math.pi / 9), math.sin(math.pi / 9)
    W = np.hstack([np.zeros((2, 2)), np.eye(2)])
    la = ref.stack_ref(x, [W, W], None, (1, 1), 2, 1, 5, schedule="lookahead")[0]
    want_la = np.array([(1 - c30, 0), (0, 0.5), (0, 0), (0, s20), (1 - c20, 0)])
    assert np.allclose(la, want_la, atol=1e-12), la
    st = ref.stack_ref(x, [W, W], None, (1, 1), 2, 1, 5, schedule="standard")[0]
    want_st = np.array([(0, 0), (2 * c30 - 1, 0), (0, 0), (c30 + c20 - 1, 0),
                        (0, 0.5 - s20)])
    assert np.allclose(st, want_st, atol=1e-12), st


def pin_stack_pooled_graph_source(ref):
    """With pooling, block l's graph ranks pooled keys of its source features
    and MRConv gathers keys pooled from its own input."""
    rng = np.random.default_rng(33)
    H = W = 4
    x = rng.standard_normal((1, 16, 3))
    Wt = rng.standard_normal((3, 6))
    xs, graphs = ref.stack_ref(x, [Wt, Wt], None, (1, 1), 2, H, W, pool_r=2,
                               return_all=True)
    k0 = ref.pool_keys_ref(x, H, W, 2)
    assert np.array_equal(graphs[0], ref.knn_ref(x, 2, 1, keys=k0))
    assert np.array_equal(graphs[1], graphs[0])          # lookahead: both from X^0
    assert np.allclose(xs[2], ref.mrconv_ref(xs[1], graphs[1], Wt,
                                             keys=ref.pool_keys_ref(xs[1], H, W, 2)))


# ---------------------------------------------------------------------------
# multi-head MRConv pins (Sec. II-A, Sec. IV-C2)
# ---------------------------------------------------------------------------
def bf_mrconv_heads(x, idx, Wh, bias=None):
    """Pure-Python per-head loops."""
    x = np.asarray(x).tolist()
    idx = np.asarray(idx).tolist()
    Wh = np.asarray(Wh).tolist()
    H, hd = len(Wh), len(Wh[0])
    B, N, C = len(x), len(x[0]), len(x[0][0])
    out = np.zeros((B, N, C))
    for b in range(B):
        for i in range(N):
            m = [max(x[b][j][c] - x[b][i][c] for j in idx[b][i]) for c in range(C)]
            for h in range(H):
                xs = x[b][i][h * hd:(h + 1) * hd]
                ms = m[h * hd:(h + 1) * hd]
                for o in range(hd):
                    s = math.fsum(a * w for a, w in zip(xs + ms, Wh[h][o]))
                    out[b, i, h * hd + o] = s + (0.0 if bias is None else bias[h * hd + o])
    return out


def pin_mrconv_heads_bruteforce(ref):
    rng = np.random.default_rng(51)
    x = rng.standard_normal((2, 7, 6))
    idx = rng.integers(0, 7, (2, 7, 3))
    Wh = rng.standard_normal((3, 2, 4))
    b = rng.standard_normal(6)
    assert np.allclose(ref.mrconv_heads_ref(x, idx, Wh, b), bf_mrconv_heads(x, idx, Wh, b),
                       atol=1e-12)


def pin_mrconv_heads_one_head_is_dense(ref):
    """H = 1 is the dense update with W = [W_x | W_m]."""
    rng = np.random.default_rng(52)
    x = rng.standard_normal((2, 9, 5))
    idx = rng.integers(0, 9, (2, 9, 4))
    W = rng.standard_normal((5, 10))
    assert np.allclose(ref.mrconv_heads_ref(x, idx, W[None]), ref.mrconv_ref(x, idx, W),
                       atol=1e-12)


def pin_mrconv_heads_locality(ref):
    """Changing head h's input channels changes only head h's outputs."""
    rng = np.random.default_rng(53)
    x = rng.standard_normal((1, 8, 8))
    idx = np.tile(np.arange(8)[None, :, None], (1, 1, 2))
    idx[..., 1] = (idx[..., 1] + 3) % 8
    Wh = rng.standard_normal((4, 2, 4))
    a = ref.mrconv_heads_ref(x, idx, Wh)
    x2 = x.copy()
    x2[..., 4:6] += rng.standard_normal((1, 8, 2))   # head 2
    c = ref.mrconv_heads_ref(x2, idx, Wh)
    assert np.array_equal(a[..., :4], c[..., :4]) and np.array_equal(a[..., 6:], c[..., 6:])
    assert not np.allclose(a[..., 4:6], c[..., 4:6])


# ---------------------------------------------------------------------------
# full ViG block pins (Eq. 11-15, Alg. 1)
# ---------------------------------------------------------------------------
PHI1 = 0.8413447460685429   # standard normal CDF at 1 (printed tables)
PHI2 = 0.9772498680518208   # standard normal CDF at 2


def _bf_gelu(v):
    return 0.5 * v * (1.0 + math.erf(v / math.sqrt(2.0)))


def bf_linear(x, W, b=None):
    """Pure-Python x W^T + b over the last axis (W[out, in])."""
    x = np.asarray(x).tolist()
    W = np.asarray(W).tolist()
    B, N = len(x), len(x[0])
    out = np.zeros((B, N, len(W)))
    for bb in range(B):
        for i in range(N):
            for o, wrow in enumerate(W):
                s = math.fsum(a * w for a, w in zip(x[bb][i], wrow))
                out[bb, i, o] = s + (0.0 if b is None else float(b[o]))
    return out


def bf_pool(x, H, W, r):
    """Pure-Python means over the r x r windows of the row-major H x W grid."""
    xl = np.asarray(x).tolist()
    B, C, Wr = len(xl), len(xl[0][0]), W // r
    out = np.zeros((B, (H // r) * Wr, C))
    for b in range(B):
        for p in range(H // r):
            for q in range(Wr):
                for c in range(C):
                    vals = [xl[b][(p * r + u) * W + q * r + v][c] for u in range(r) for v in range(r)]
                    out[b, p * Wr + q, c] = math.fsum(vals) / (r * r)
    return out


def bf_vig_block(x, idx, p, H=None, W=None, r=1):
    gel = np.vectorize(_bf_gelu)
    u = bf_linear(x, p["W_in"], p.get("b_in"))
    keys = bf_pool(u, H, W, r) if r > 1 else None
    ut = bf_mrconv(u, idx, p["W_upd"], p.get("b_upd"), keys=keys)
    y = bf_linear(gel(ut), p["W_out"], p.get("b_out")) + np.asarray(x)
    h = gel(bf_linear(y, p["W_1"], p.get("b_1")))
    return bf_linear(h, p["W_2"], p.get("b_2")) + y


def _vig_params(rng, C, bias=True):
    p = {"W_in": rng.standard_normal((C, C)), "W_upd": rng.standard_normal((C, 2 * C)),
         "W_out": rng.standard_normal((C, C)), "W_1": rng.standard_normal((4 * C, C)),
         "W_2": rng.standard_normal((C, 4 * C)) * 0.5}
    if bias:
        for n, o in (("b_in", C), ("b_upd", C), ("b_out", C), ("b_1", 4 * C), ("b_2", C)):
            p[n] = rng.standard_normal(o)
    return p


def pin_gelu_closed_form(ref):
    """sigma(x) = x Phi(x): table values of Phi, and sigma(x) - sigma(-x) = x."""
    x = np.array([0.0, 1.0, -1.0, 2.0, -2.0, 30.0, -30.0])
    want = np.array([0.0, PHI1, -(1.0 - PHI1), 2 * PHI2, -2 * (1.0 - PHI2), 30.0, 0.0])
    assert np.allclose(ref.gelu_ref(x), want, rtol=0, atol=1e-15), ref.gelu_ref(x)
    z = np.linspace(-5, 5, 41)
    assert np.allclose(ref.gelu_ref(z) - ref.gelu_ref(-z), z, rtol=0, atol=1e-14)


def pin_linear_bruteforce(ref):
    rng = np.random.default_rng(41)
    x = rng.standard_normal((2, 5, 3))
    W = rng.standard_normal((4, 3))
    b = rng.standard_normal(4)
    assert np.allclose(ref.linear_ref(x, W, b), bf_linear(x, W, b), atol=1e-12)
    assert np.allclose(ref.linear_ref(x, W), bf_linear(x, W), atol=1e-12)


def pin_vig_block_bruteforce(ref):
    rng = np.random.default_rng(42)
    x = rng.standard_normal((1, 6, 3))
    idx = rng.integers(0, 6, (1, 6, 2))
    p = _vig_params(rng, 3)
    assert np.allclose(ref.vig_block_ref(x, idx, p), bf_vig_block(x, idx, p), atol=1e-10)


def pin_vig_block_residual_identity(ref):
    """W_out = 0 and W_2 = 0 (no biases): both residual paths return X exactly."""
    rng = np.random.default_rng(43)
    x = rng.standard_normal((2, 7, 4))
    p = _vig_params(rng, 4, bias=False)
    p["W_out"] = np.zeros((4, 4))
    p["W_2"] = np.zeros((4, 16))
    idx = rng.integers(0, 7, (2, 7, 3))
    assert np.array_equal(ref.vig_block_ref(x, idx, p), x)


def pin_vig_block_hand(ref):
    """Worked by hand, self-only graph (m = 0):
    (a) W_in = I, W_upd = [I | 0], W_out = I, W_1 = 0: U = Ut = X,
        Y = sigma(X) + X, FFN = sigma(0) W_2 = 0, so X' = X + sigma(X);
    (b) W_out = 0 (Y = X), W_1 = [I; 0], b_1 = (1, -1, 0, ...), W_2 = [I | 0]:
        X' = sigma(X + b_1[:2]) + X, at X = 0 that is (Phi(1), -(1 - Phi(1)))."""
    C = 2
    idx = np.arange(2)[None, :, None]
    I2 = np.eye(C)
    x = np.array([[[1.0, -1.0], [2.0, 0.0]]])
    pa = {"W_in": I2, "W_upd": np.hstack([I2, np.zeros((C, C))]), "W_out": I2,
          "W_1": np.zeros((4 * C, C)), "W_2": np.ones((C, 4 * C))}
    want = np.array([[[1 + PHI1, -1 - (1 - PHI1)], [2 + 2 * PHI2, 0.0]]])
    assert np.allclose(ref.vig_block_ref(x, idx, pa), want, rtol=0, atol=1e-14)
    W1 = np.zeros((4 * C, C))
    W1[:C] = I2
    W2 = np.zeros((C, 4 * C))
    W2[:, :C] = I2
    b1 = np.zeros(4 * C)
    b1[:2] = (1.0, -1.0)
    pb = {"W_in": I2, "W_upd": np.hstack([I2, np.zeros((C, C))]), "W_out": np.zeros((C, C)),
          "W_1": W1, "b_1": b1, "W_2": W2}
    x0 = np.zeros((1, 2, C))
    want = np.array([[[PHI1, -(1 - PHI1)], [PHI1, -(1 - PHI1)]]])
    assert np.allclose(ref.vig_block_ref(x0, idx, pb), want, rtol=0, atol=1e-14)


def pin_vig_stack_graph_source(ref):
    """Lookahead: blocks 0 and 1 use G(U^0), block 2 uses G(U^1); standard:
    block l uses G(U^l), with U^l = X^l W_in^l^T computed here."""
    rng = np.random.default_rng(44)
    x = rng.standard_normal((1, 12, 3))
    ps = [_vig_params(rng, 3) for _ in range(3)]
    for p in ps:
        p["W_2"] = p["W_2"] * 0.1
    dil = (1, 2, 1)
    xs, us, graphs = ref.vig_stack_ref(x, ps, dil, 3, schedule="lookahead", return_all=True)
    u = [xs[l] @ ps[l]["W_in"].T + ps[l]["b_in"] for l in range(3)]
    for l in range(3):
        assert np.allclose(us[l], u[l], atol=1e-12)
    assert np.array_equal(graphs[0], ref.knn_ref(u[0], 3, 1))
    assert np.array_equal(graphs[1], ref.knn_ref(u[0], 3, 2))
    assert np.array_equal(graphs[2], ref.knn_ref(u[1], 3, 1))
    assert np.allclose(xs[3], ref.vig_block_ref(xs[2], graphs[2], ps[2]), atol=1e-12)
    xs, us, graphs = ref.vig_stack_ref(x, ps, dil, 3, schedule="standard", return_all=True)
    for l in range(3):
        ul = xs[l] @ ps[l]["W_in"].T + ps[l]["b_in"]
        assert np.array_equal(graphs[l], ref.knn_ref(ul, 3, dil[l]))


def pin_vig_block_pooled_bruteforce(ref):
    """Pyramid stages: the keys are U pooled 2 x 2 on a 4 x 6 grid, and MRConv
    gathers those pooled rows."""
    rng = np.random.default_rng(45)
    H, W, r = 4, 6, 2
    x = rng.standard_normal((2, H * W, 3))
    idx = rng.integers(0, 6, (2, H * W, 3))
    p = _vig_params(rng, 3)
    got = ref.vig_block_ref(x, idx, p, H=H, W=W, pool_r=r)
    assert np.allclose(got, bf_vig_block(x, idx, p, H, W, r), atol=1e-10)


def pin_vig_block_single_key(ref):
    """One pooled key (2 x 2 grid, r = 2): m_i = mean(U) - u_i, worked by hand
    with W_in = I, W_upd = [0 | I], W_out = I, W_1 = 0 and no biases, so
    X' = X + sigma(mean(X) - X)."""
    C = 2
    I2 = np.eye(C)
    x = np.array([[[1.0, -1.0], [3.0, 0.0], [-1.0, 2.0], [1.0, 3.0]]])   # mean (1, 1)
    p = {"W_in": I2, "W_upd": np.hstack([np.zeros((C, C)), I2]), "W_out": I2,
         "W_1": np.zeros((4 * C, C)), "W_2": np.ones((C, 4 * C))}
    idx = np.zeros((1, 4, 1), dtype=np.int64)
    g = {0.0: 0.0, 1.0: PHI1, -1.0: -(1 - PHI1), 2.0: 2 * PHI2, -2.0: -2 * (1 - PHI2)}
    m = np.array([1.0, 1.0]) - x[0]
    want = x[0] + np.array([[g[v] for v in row] for row in m])
    got = ref.vig_block_ref(x, idx, p, H=2, W=2, pool_r=2)
    assert np.allclose(got[0], want, rtol=0, atol=1e-14), got


def pin_vig_stack_pooled_graph_source(ref):
    """Pooled lookahead stack: graph l ranks the keys pooled from its source U
    (U^0 for blocks 0 and 1, U^(l-1) after), and block l gathers keys pooled
    from its own U."""
    rng = np.random.default_rng(46)
    H, W, r = 4, 4, 2
    x = rng.standard_normal((1, H * W, 3))
    ps = [_vig_params(rng, 3) for _ in range(3)]
    for p in ps:
        p["W_2"] = p["W_2"] * 0.1
    dil = (1, 2, 1)
    xs, us, graphs = ref.vig_stack_ref(x, ps, dil, 2, schedule="lookahead", return_all=True,
                                       H=H, W=W, pool_r=r)
    u = [bf_linear(xs[l], ps[l]["W_in"], ps[l]["b_in"]) for l in range(3)]
    for l, s in enumerate((0, 0, 1)):
        assert np.array_equal(graphs[l], ref.knn_ref(u[s], 2, dil[l], keys=bf_pool(u[s], H, W, r)))
    assert np.allclose(xs[3], bf_vig_block(xs[2], graphs[2], ps[2], H, W, r), atol=1e-10)


def pin_vig_stack_pooled_all_keys(ref):
    """k equal to the number of pooled keys (d = 1): every graph row holds all
    of them, so the max-relative part ignores which U built the graph and the
    lookahead and standard schedules give the same X^L."""
    rng = np.random.default_rng(47)
    H, W, r = 4, 4, 2
    x = rng.standard_normal((2, H * W, 3))
    ps = [_vig_params(rng, 3) for _ in range(3)]
    for p in ps:
        p["W_2"] = p["W_2"] * 0.1
    la, _, g = ref.vig_stack_ref(x, ps, (1, 1, 1), 4, schedule="lookahead", return_all=True,
                                 H=H, W=W, pool_r=r)
    st = ref.vig_stack_ref(x, ps, (1, 1, 1), 4, schedule="standard", H=H, W=W, pool_r=r)
    for gl in g:
        assert np.array_equal(np.sort(gl, axis=-1), np.broadcast_to(np.arange(4), gl.shape))
    assert np.allclose(la[-1], st, rtol=0, atol=1e-12)


# ---------------------------------------------------------------------------
# inter-stage max pooling pins
# ---------------------------------------------------------------------------
def pin_max_pool_closed_form(ref):
    """On a non-square grid whose channel 0 increases along rows and channel 1
    along columns, each window's maximum sits at its bottom-right node."""
    H, W, r = 6, 10, 2
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    x = np.zeros((2, H * W, 3))
    x[..., 0] = yy.ravel() * W + xx.ravel()
    x[..., 1] = -(xx.ravel() * 100.0) + yy.ravel()     # largest at the window's left column
    x[..., 2] = -7.5
    out = ref.max_pool_nodes_ref(x, H, W, r)
    Wr = W // r
    assert out.shape == (2, (H // r) * Wr, 3)
    for p in range(H // r):
        for q in range(Wr):
            assert out[0, p * Wr + q, 0] == (p * r + r - 1) * W + q * r + r - 1
            assert out[1, p * Wr + q, 1] == -(q * r) * 100.0 + p * r + r - 1
            assert out[0, p * Wr + q, 2] == -7.5
    assert np.array_equal(ref.max_pool_nodes_ref(x, H, W, 1), x)


def pin_max_pool_bruteforce(ref):
    """Pure-Python maxima over each window of a random 4 x 6 grid, r = 2."""
    g = np.random.default_rng(5)
    H, W, r, C = 4, 6, 2, 3
    x = g.standard_normal((1, H * W, C))
    out = ref.max_pool_nodes_ref(x, H, W, r)
    for p in range(H // r):
        for q in range(W // r):
            for c in range(C):
                vals = [float(x[0, (p * r + u) * W + q * r + v, c]) for u in range(r) for v in range(r)]
                assert out[0, p * (W // r) + q, c] == max(vals)


def pin_max_pool_dominates_mean(ref):
    """max >= mean over every window, with equality exactly where the window
    is constant."""
    g = np.random.default_rng(6)
    H, W, r = 8, 8, 4
    x = g.standard_normal((2, H * W, 4))
    # channel 3 constant per window
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    x[..., 3] = ((yy // r) * 10 + (xx // r)).ravel()
    mx = ref.max_pool_nodes_ref(x, H, W, r)
    mean = ref.pool_keys_ref(x, H, W, r)
    assert np.all(mx[..., :3] > mean[..., :3])
    assert np.array_equal(mx[..., 3], mean[..., 3])


PINS = [
    pin_circle_closed_form_fixture, pin_circle_knn, pin_knn_bruteforce, pin_knn_self_first,
    pin_knn_duplicates_lower_index, pin_knn_permutation_equivariant, pin_knn_scale_invariant,
    pin_knn_dilation_consistency, pin_knn_full_is_permutation, pin_knn_zero_rows,
    pin_knn_sorted_by_distance, pin_circle_mrconv, pin_mrconv_bruteforce, pin_mrconv_self_only,
    pin_mrconv_translation, pin_mrconv_max_minus, pin_mrconv_bias_only, pin_pool_closed_form,
    pin_stack_single_layer, pin_stack_identity_weights, pin_stack_circle_two_blocks,
    pin_stack_pooled_graph_source, pin_gelu_closed_form, pin_linear_bruteforce,
    pin_vig_block_bruteforce, pin_vig_block_residual_identity, pin_vig_block_hand,
    pin_vig_stack_graph_source, pin_vig_block_pooled_bruteforce, pin_vig_block_single_key,
    pin_vig_stack_pooled_graph_source, pin_vig_stack_pooled_all_keys,
    pin_mrconv_heads_bruteforce, pin_mrconv_heads_one_head_is_dense,
    pin_mrconv_heads_locality, pin_max_pool_closed_form, pin_max_pool_bruteforce,
    pin_max_pool_dominates_mean, pin_knn_distances_bruteforce, pin_knn_distances_circle,
    pin_dilated_lists_bruteforce, pin_distance_lists_are_knn_ref,
]


def failing_pins(ref):
    bad = []
    for p in PINS:
        try:
            p(ref)
        except Exception as e:  # noqa: BLE001 - any failure counts
            bad.append((p.__name__, repr(e)[:200]))
    return bad
