"""CPU float64 oracle for the GraphLeap graph-convolution hot path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this module.  The product path (the
HIP library and its Python binding) never imports, links or calls it, and it
shares no code with that path.

Everything here is the plain definition, written for a reader to check against
the paper by eye: no blocking, fusion or reordering beyond what the definition
states.  Inputs are float64 arrays holding the exact values of the stored
(fp32 or bf16) tensors.

Pins (what ties each function to something other than itself) are in
tests/oracle_pins.py, run by tests/test_oracle_pins.py; every function below
has at least one, and tests/test_oracle_mutants.py plants mistakes in copies of
each that the pins must catch.

Readings of points the paper leaves open (each is also listed in the design
notes):
  * G(.) ranks by squared Euclidean distance between L2-normalised rows
    (eps 1e-12); the square root of Alg. 2 is monotone and is dropped.
  * Ties are broken by the lower key index; the k output indices are ordered by
    (distance, index) ascending, so position 0 is the nearest node.
  * Dilated kNN with dilation d keeps the k*d nearest and returns ranks
    0, d, 2d, ..., (k-1)d.  Self-loops are kept.
  * MRConv concatenates [x_i, max_j(x_j - x_i)] and applies W[Cout, 2C]
    (columns 0..C-1 act on x_i, columns C..2C-1 on the max-relative part),
    plus a bias.
  * With key pooling (pyramid stages) the graph connects each node to pooled
    key nodes and MRConv gathers the pooled (unnormalised) key rows.
  * The lookahead stack uses G(X^0) for blocks 0 and 1 and G(X^(l-1)) for
    block l >= 2; each graph gets the dilation of the block that consumes it.
  * Multi-head MRConv splits the channels into H equal contiguous heads; head
    h's outputs see only head h's channels of x_i and of m_i.
  * The full ViG block (Eq. 11-15, Alg. 1): sigma is the exact GELU
    x Phi(x); fully connected layers are x W^T + b with W[out, in] and an
    optional bias; there is no normalisation layer (the equations have none);
    MRConv is single-head; the FFN is C -> 4C -> C.  Its lookahead graph comes
    from the projected features U^(l-1) (U^0 for blocks 0 and 1).  At pyramid
    stages its keys are pooled from U, as the reduced block's are from X.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

EPS = 1e-12


# ----------------------------------------------------------------------------
# kNN graph  (Sec. II-B, Eq. 4; Sec. IV-B; Alg. 2)
# ----------------------------------------------------------------------------
def l2_normalize(v: np.ndarray) -> np.ndarray:
    """Rows divided by max(||row||_2, eps).  Zero rows stay zero."""
    v = np.asarray(v, dtype=np.float64)
    n = np.sqrt((v * v).sum(axis=-1, keepdims=True))
    return v / np.maximum(n, EPS)


def pairwise_sq_dist(Q: np.ndarray, K: np.ndarray, row_chunk: int = 64) -> np.ndarray:
    """D[i, j] = sum_c (Q[i, c] - K[j, c])^2 by direct differences (Alg. 2,
    the accumulated squared difference before its square root).  Rows are
    processed in chunks only to bound memory; each entry is the same sum."""
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    D = np.empty((Q.shape[0], K.shape[0]))
    for s in range(0, Q.shape[0], row_chunk):
        diff = Q[s:s + row_chunk, None, :] - K[None, :, :]
        D[s:s + row_chunk] = (diff * diff).sum(axis=-1)
    return D


def knn_order(D: np.ndarray, kk: int) -> np.ndarray:
    """For each row, the kk key indices of smallest distance, ordered by
    (distance, index).  A stable sort over increasing j gives the lower index
    first among equal distances."""
    return np.argsort(D, axis=1, kind="stable")[:, :kk]


def knn_ref(x: np.ndarray, k: int, dilation: int = 1, keys: np.ndarray | None = None,
            rows: np.ndarray | None = None, return_dist: bool = False):
    """Dilated kNN graph G(x) (Eq. 4 with the dilation of Sec. IV-B).

    x: [B, N, C] features; keys: [B, M, C] or None (keys = x).
    rows: optional subset of query rows (same for every image) to evaluate.
    Returns idx [B, len(rows) or N, k] int64 (and D [B, rows, M] if asked).
    """
    x = np.asarray(x, dtype=np.float64)
    keys = x if keys is None else np.asarray(keys, dtype=np.float64)
    B, N, _ = x.shape
    M = keys.shape[1]
    kk = k * dilation
    if k < 1 or dilation < 1 or kk > M:
        raise ValueError("need 1 <= k, 1 <= dilation, k*dilation <= M")
    rows = np.arange(N) if rows is None else np.asarray(rows)
    idx = np.empty((B, len(rows), k), dtype=np.int64)
    dist = np.empty((B, len(rows), M)) if return_dist else None
    for b in range(B):
        Q = l2_normalize(x[b, rows])
        K = l2_normalize(keys[b])
        D = pairwise_sq_dist(Q, K)
        order = knn_order(D, kk)
        idx[b] = order[:, ::dilation][:, :k]
        if return_dist:
            dist[b] = D
    return (idx, dist) if return_dist else idx


def knn_distances(x: np.ndarray, keys: np.ndarray | None = None,
                  rows: np.ndarray | None = None) -> np.ndarray:
    """The distances G(x) ranks by (Eq. 4 on L2-normalised rows; Alg. 2 before
    its square root): D[b, i, j] = || x[b, rows[i]]/|x| - keys[b, j]/|keys_j| ||^2,
    [B, len(rows) or N, M].  Query rows are selected first, then normalised;
    every key row is normalised on its own (keys = x when None)."""
    x = np.asarray(x, dtype=np.float64)
    keys = x if keys is None else np.asarray(keys, dtype=np.float64)
    rows = np.arange(x.shape[1]) if rows is None else np.asarray(rows)
    return np.stack([pairwise_sq_dist(l2_normalize(x[b, rows]), l2_normalize(keys[b]))
                     for b in range(x.shape[0])])


def dilated_lists(D: np.ndarray, k: int, dilation: int = 1) -> np.ndarray:
    """Dilated kNN lists from distances D [B, rows, M] (the dilated kNN of
    Sec. IV-B): per row, the k*dilation keys of smallest (distance, index),
    of which ranks 0, d, 2d, ..., (k-1)d are kept.  Returns [B, rows, k] int64."""
    D = np.asarray(D, dtype=np.float64)
    kk = k * dilation
    if k < 1 or dilation < 1 or kk > D.shape[-1]:
        raise ValueError("need 1 <= k, 1 <= dilation, k*dilation <= M")
    return np.stack([knn_order(D[b], kk)[:, ::dilation][:, :k] for b in range(D.shape[0])])


# ----------------------------------------------------------------------------
# key pooling for pyramid stages (workload recipe; the paper reduces nodes
# between stages with pooling in Sec. IV-E, here keys are averaged r x r)
# ----------------------------------------------------------------------------
def pool_keys_ref(x: np.ndarray, H: int, W: int, r: int) -> np.ndarray:
    """keys[b, p*(W/r) + q, c] = mean_{u,v < r} x[b, (p*r + u)*W + (q*r + v), c]."""
    x = np.asarray(x, dtype=np.float64)
    B, N, C = x.shape
    if N != H * W or H % r or W % r:
        raise ValueError("bad pooling shape")
    Hr, Wr = H // r, W // r
    out = np.zeros((B, Hr * Wr, C))
    for p in range(Hr):
        for q in range(Wr):
            acc = np.zeros((B, C))
            for u in range(r):
                for v in range(r):
                    acc += x[:, (p * r + u) * W + (q * r + v), :]
            out[:, p * Wr + q, :] = acc / (r * r)
    return out


def max_pool_nodes_ref(x: np.ndarray, H: int, W: int, r: int) -> np.ndarray:
    """Inter-stage node reduction of pyramid models (Sec. IV-E: node counts are
    reduced between stages by max pooling): r x r windows of the row-major
    H x W node grid, stride r,
        out[b, p*(W/r) + q, c] = max_{u,v < r} x[b, (p*r + u)*W + (q*r + v), c].
    """
    x = np.asarray(x, dtype=np.float64)
    B, N, C = x.shape
    if N != H * W or H % r or W % r:
        raise ValueError("bad pooling shape")
    Hr, Wr = H // r, W // r
    out = np.empty((B, Hr * Wr, C))
    for p in range(Hr):
        for q in range(Wr):
            best = np.full((B, C), -np.inf)
            for u in range(r):
                for v in range(r):
                    best = np.maximum(best, x[:, (p * r + u) * W + (q * r + v), :])
            out[:, p * Wr + q, :] = best
    return out


# ----------------------------------------------------------------------------
# MRConv  (Sec. II-A, Eq. 2 and Eq. 3; split W_x / W_m of Sec. IV-C2)
# ----------------------------------------------------------------------------
def max_relative_ref(x: np.ndarray, idx: np.ndarray, keys: np.ndarray | None = None) -> np.ndarray:
    """m[b, i, c] = max_t (keys[b, idx[b, i, t], c] - x[b, i, c])   (Eq. 2)."""
    x = np.asarray(x, dtype=np.float64)
    keys = x if keys is None else np.asarray(keys, dtype=np.float64)
    B, N, C = x.shape
    k = idx.shape[2]
    m = np.full((B, N, C), -np.inf)
    for t in range(k):
        nb = np.take_along_axis(keys, idx[:, :, t][:, :, None].astype(np.int64), axis=1)
        m = np.maximum(m, nb - x)
    return m


def mrconv_ref(x: np.ndarray, idx: np.ndarray, W: np.ndarray, b: np.ndarray | None = None,
               keys: np.ndarray | None = None, return_concat: bool = False):
    """x'_i = [x_i, max_j (x_j - x_i)] W^T + b   (Eq. 2-3, bias kept).

    W: [Cout, 2C]; the first C columns multiply x_i, the last C the max-relative
    part (the W_x / W_m split).  Returns [B, N, Cout]."""
    x = np.asarray(x, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    m = max_relative_ref(x, idx, keys)
    xcat = np.concatenate([x, m], axis=-1)
    out = xcat @ W.T
    if b is not None:
        out = out + np.asarray(b, dtype=np.float64)
    return (out, xcat) if return_concat else out


def mrconv_heads_ref(x: np.ndarray, idx: np.ndarray, Wh: np.ndarray, b: np.ndarray | None = None,
                     keys: np.ndarray | None = None) -> np.ndarray:
    """Multi-head MRConv update (Sec. II-A; the per-head W_x,h / W_m,h of
    Sec. IV-C2): channels split into H equal contiguous heads of hd = C/H;
    output head h is  x_h W_x,h^T + m_h W_m,h^T  (+ b), with x_h and m_h the
    head's channels of x_i and of the max-relative m_i.

    Wh: [H, hd, 2 hd], row o of head h = [W_x,h[o, :] | W_m,h[o, :]].
    Returns [B, N, C]."""
    x = np.asarray(x, dtype=np.float64)
    Wh = np.asarray(Wh, dtype=np.float64)
    H, hd = Wh.shape[0], Wh.shape[1]
    m = max_relative_ref(x, idx, keys)
    outs = []
    for h in range(H):
        sl = slice(h * hd, (h + 1) * hd)
        cat = np.concatenate([x[..., sl], m[..., sl]], axis=-1)
        outs.append(cat @ Wh[h].T)
    out = np.concatenate(outs, axis=-1)
    if b is not None:
        out = out + np.asarray(b, dtype=np.float64)
    return out


# ----------------------------------------------------------------------------
# stacks: GraphLeap lookahead (Eq. 10-12, bootstrap, Alg. 1) and the
# standard same-layer schedule (Eq. 5-7) for comparison
# ----------------------------------------------------------------------------
def graph_source_blocks(L: int, schedule: str = "lookahead") -> list:
    """Index of the feature tensor X^s each block's graph is built from."""
    if schedule == "standard":
        return list(range(L))
    if schedule != "lookahead":
        raise ValueError(schedule)
    # block 0 bootstraps from its own input; block l >= 1 uses X^(l-1)
    return [0] + list(range(L - 1))


def stack_ref(x0: np.ndarray, Ws: list, bs: list, dilations, k: int, H: int, W: int,
              pool_r: int = 1, schedule: str = "lookahead", return_all: bool = False):
    """Run L blocks of X^(l+1) = MRConv(X^l; Ghat^l) in float64.

    Ghat^l = G(X^src(l)) with the dilation of block l (the consumer), keys
    pooled r x r from the same X^src(l) when pool_r > 1; MRConv gathers keys
    pooled from its own input X^l."""
    L = len(dilations)
    src = graph_source_blocks(L, schedule)
    xs = [np.asarray(x0, dtype=np.float64)]
    graphs = []
    for l in range(L):
        xg = xs[src[l]]
        kg = pool_keys_ref(xg, H, W, pool_r) if pool_r > 1 else None
        idx = knn_ref(xg, k, dilations[l], keys=kg)
        graphs.append(idx)
        ku = pool_keys_ref(xs[l], H, W, pool_r) if pool_r > 1 else None
        xs.append(mrconv_ref(xs[l], idx, Ws[l], bs[l] if bs is not None else None, keys=ku))
    if return_all:
        return xs, graphs
    return xs[-1]


# ----------------------------------------------------------------------------
# the full GraphLeap ViG block (Sec. III Eq. 11-15; Alg. 1): FC1, the
# leap-ahead graph, MRConv, FC2 + residual, FFN + residual
# ----------------------------------------------------------------------------
VIG_PARAMS = ("W_in", "b_in", "W_upd", "b_upd", "W_out", "b_out", "W_1", "b_1", "W_2", "b_2")


def gelu_ref(x: np.ndarray) -> np.ndarray:
    """sigma(x) = x Phi(x) = x/2 (1 + erf(x / sqrt 2)), the exact GELU."""
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def linear_ref(x: np.ndarray, W: np.ndarray, b: np.ndarray | None = None) -> np.ndarray:
    """A fully connected layer over the channel axis: x W^T + b, W[out, in]."""
    out = np.asarray(x, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
    if b is not None:
        out = out + np.asarray(b, dtype=np.float64)
    return out


def vig_block_ref(x: np.ndarray, idx: np.ndarray, p: dict, return_all: bool = False,
                  H: int | None = None, W: int | None = None, pool_r: int = 1):
    """Block l of Alg. 1 given the graph it uses:
        U  = X W_in^T + b_in                        (FC1, Eq. 11)
        Ut = MRConv(U; idx)  with W_upd [C, 2C]     (Eq. 13)
        Y  = sigma(Ut) W_out^T + b_out + X          (FC2 + residual, Eq. 14)
        X' = sigma(Y W_1^T + b_1) W_2^T + b_2 + Y   (FFN + residual, Eq. 15)
    idx indexes U's rows, or with pool_r > 1 the rows of U's r x r key
    pooling over the H x W grid, which MRConv then gathers (the pyramid
    stages' pooled keys).  Missing biases are zero.  Returns X' (or X', U,
    Ut, Y)."""
    x = np.asarray(x, dtype=np.float64)
    u = linear_ref(x, p["W_in"], p.get("b_in"))
    keys = pool_keys_ref(u, H, W, pool_r) if pool_r > 1 else None
    ut = mrconv_ref(u, idx, p["W_upd"], p.get("b_upd"), keys=keys)
    y = linear_ref(gelu_ref(ut), p["W_out"], p.get("b_out")) + x
    h = gelu_ref(linear_ref(y, p["W_1"], p.get("b_1")))
    xn = linear_ref(h, p["W_2"], p.get("b_2")) + y
    return (xn, u, ut, y) if return_all else xn


def vig_stack_ref(x0: np.ndarray, params: list, dilations, k: int,
                  schedule: str = "lookahead", return_all: bool = False,
                  H: int | None = None, W: int | None = None, pool_r: int = 1):
    """L full blocks.  Lookahead (Eq. 12 and the bootstrap of Alg. 1): block 0
    uses G(U^0) and block l >= 1 uses G(U^(l-1)); standard (Eq. 6): block l
    uses G(U^l).  Each graph gets the dilation of the block that consumes it.
    With pool_r > 1 every graph ranks the r x r pooled keys of the U it is
    built from, and each block's MRConv gathers the keys pooled from its own
    U.  Returns X^L, or (xs, us, graphs) with return_all."""
    if schedule not in ("lookahead", "standard"):
        raise ValueError(schedule)
    L = len(dilations)
    xs = [np.asarray(x0, dtype=np.float64)]
    us, graphs = [], []
    for l in range(L):
        u = linear_ref(xs[l], params[l]["W_in"], params[l].get("b_in"))
        us.append(u)
        src = u if (schedule == "standard" or l == 0) else us[l - 1]
        keys = pool_keys_ref(src, H, W, pool_r) if pool_r > 1 else None
        idx = knn_ref(src, k, dilations[l], keys=keys)
        graphs.append(idx)
        xs.append(vig_block_ref(xs[l], idx, params[l], H=H, W=W, pool_r=pool_r))
    if return_all:
        return xs, us, graphs
    return xs[-1]
