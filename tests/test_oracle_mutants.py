"""Planted mistakes in copies of the oracle must each fail at least one pin.

Each mutant replaces one oracle function with a version carrying a plausible
bug (a dropped normalisation, a wrong sign, a transposed operand, an index off
by one, the other tie-break, ...).  CPU only; the real oracle is untouched.
"""
import types

import numpy as np
import pytest

import oracle
from oracle import graphleap_ref as R
from oracle_pins import failing_pins


def _ns(**over):
    base = {n: getattr(oracle, n) for n in dir(oracle) if not n.startswith("_")}
    base.update(over)
    ns = types.SimpleNamespace(**base)
    return ns


def _knn_factory(normalize=True, descending=False, dil_offset=0, tie_high=False,
                 dist="sq"):
    def knn(x, k, dilation=1, keys=None, rows=None, return_dist=False):
        x = np.asarray(x, dtype=np.float64)
        ks = x if keys is None else np.asarray(keys, dtype=np.float64)
        B, N, _ = x.shape
        rows_ = np.arange(N) if rows is None else np.asarray(rows)
        kk = k * dilation
        idx = np.empty((B, len(rows_), k), dtype=np.int64)
        dist_all = np.empty((B, len(rows_), ks.shape[1]))
        for b in range(B):
            Q = R.l2_normalize(x[b, rows_]) if normalize else x[b, rows_]
            K = R.l2_normalize(ks[b]) if normalize else ks[b]
            diff = Q[:, None, :] - K[None, :, :]
            D = (diff * diff).sum(-1) if dist == "sq" else np.abs(diff).sum(-1)
            if descending:
                order = np.argsort(-D, axis=1, kind="stable")
            elif tie_high:
                order = (D.shape[1] - 1 - np.argsort(D[:, ::-1], axis=1, kind="stable"))
            else:
                order = np.argsort(D, axis=1, kind="stable")
            sel = order[:, :kk + dil_offset][:, dil_offset::dilation][:, :k]
            idx[b] = sel
            dist_all[b] = D
        return (idx, dist_all) if return_dist else idx
    return knn


def _maxrel_factory(sign=1, use_min=False):
    def maxrel(x, idx, keys=None):
        x = np.asarray(x, dtype=np.float64)
        ks = x if keys is None else np.asarray(keys, dtype=np.float64)
        out = None
        for t in range(idx.shape[2]):
            nb = np.take_along_axis(ks, idx[:, :, t][:, :, None].astype(np.int64), axis=1)
            v = sign * (nb - x)
            out = v if out is None else (np.minimum(out, v) if use_min else np.maximum(out, v))
        return out
    return maxrel


def _mrconv_factory(maxrel=None, swap_halves=False, transpose_w=False, drop_bias=False):
    mr = maxrel or R.max_relative_ref

    def mrconv(x, idx, W, b=None, keys=None, return_concat=False):
        x = np.asarray(x, dtype=np.float64)
        W = np.asarray(W, dtype=np.float64)
        m = mr(x, idx, keys)
        cat = np.concatenate([m, x] if swap_halves else [x, m], axis=-1)
        Wt = W.reshape(W.shape[1], W.shape[0]) if transpose_w else W.T
        out = cat @ Wt
        if b is not None and not drop_bias:
            out = out + np.asarray(b, dtype=np.float64)
        return (out, cat) if return_concat else out
    return mrconv


def _pool_transposed(x, H, W, r):
    x = np.asarray(x, dtype=np.float64)
    B, N, C = x.shape
    Hr, Wr = H // r, W // r
    out = np.zeros((B, Hr * Wr, C))
    for p in range(Hr):
        for q in range(Wr):
            acc = 0.0
            for u in range(r):
                for v in range(r):
                    acc = acc + x[:, (p * r + v) * W + (q * r + u), :]   # u/v swapped
            out[:, q * Hr + p, :] = acc / (r * r)                      # output transposed
    return out


def _stack_factory(schedule_override=None, knn=None, mrconv=None, pool=None):
    knn = knn or R.knn_ref
    mrconv = mrconv or R.mrconv_ref
    pool = pool or R.pool_keys_ref

    def stack(x0, Ws, bs, dilations, k, H, W, pool_r=1, schedule="lookahead",
              return_all=False):
        L = len(dilations)
        sched = schedule_override or schedule
        src = R.graph_source_blocks(L, sched)
        xs = [np.asarray(x0, dtype=np.float64)]
        graphs = []
        for l in range(L):
            xg = xs[src[l]]
            kg = pool(xg, H, W, pool_r) if pool_r > 1 else None
            idx = knn(xg, k, dilations[l], keys=kg)
            graphs.append(idx)
            ku = pool(xs[l], H, W, pool_r) if pool_r > 1 else None
            xs.append(mrconv(xs[l], idx, Ws[l], bs[l] if bs is not None else None, keys=ku))
        return (xs, graphs) if return_all else xs[-1]
    return stack


def _gelu_tanh(x):
    x = np.asarray(x, dtype=np.float64)
    return 0.5 * x * (1 + np.tanh(np.sqrt(2 / np.pi) * (x + 0.044715 * x ** 3)))


def _linear_untransposed(x, W, b=None):
    out = np.asarray(x, dtype=np.float64) @ np.asarray(W, dtype=np.float64).reshape(
        np.asarray(W).shape[1], np.asarray(W).shape[0])
    return out if b is None else out + b


def _block_factory(fc2_residual=True, ffn_residual="y", gelu_after_wout=False,
                   drop_b1=False, linear=None, pool_from="u"):
    lin = linear or R.linear_ref

    def block(x, idx, p, return_all=False, H=None, W=None, pool_r=1):
        x = np.asarray(x, dtype=np.float64)
        u = lin(x, p["W_in"], p.get("b_in"))
        keys = None
        if pool_r > 1 and pool_from != "none":
            keys = R.pool_keys_ref(u if pool_from == "u" else x, H, W, pool_r)
        ut = R.mrconv_ref(u, idx, p["W_upd"], p.get("b_upd"), keys=keys)
        if gelu_after_wout:
            y = R.gelu_ref(lin(ut, p["W_out"], p.get("b_out")))
        else:
            y = lin(R.gelu_ref(ut), p["W_out"], p.get("b_out"))
        if fc2_residual:
            y = y + x
        h = R.gelu_ref(lin(y, p["W_1"], None if drop_b1 else p.get("b_1")))
        xn = lin(h, p["W_2"], p.get("b_2")) + (y if ffn_residual == "y" else x)
        return (xn, u, ut, y) if return_all else xn
    return block


def _vig_stack_factory(graph_from="u", lag=1, block=None, graph_keys="pooled"):
    blk = block or R.vig_block_ref

    def stack(x0, params, dilations, k, schedule="lookahead", return_all=False, H=None,
              W=None, pool_r=1):
        L = len(dilations)
        xs = [np.asarray(x0, dtype=np.float64)]
        us, graphs = [], []
        for l in range(L):
            u = R.linear_ref(xs[l], params[l]["W_in"], params[l].get("b_in"))
            us.append(u)
            feats = us if graph_from == "u" else xs
            j = l if (schedule == "standard" or l == 0) else max(l - lag, 0)
            keys = None
            if pool_r > 1 and graph_keys != "unpooled":
                # "own": keys pooled from the consuming block's U, not the source's
                keys = R.pool_keys_ref(us[l] if graph_keys == "own" else feats[j], H, W, pool_r)
            idx = R.knn_ref(feats[j], k, dilations[l], keys=keys)
            graphs.append(idx)
            xs.append(blk(xs[l], idx, params[l], H=H, W=W, pool_r=pool_r))
        return (xs, us, graphs) if return_all else xs[-1]
    return stack


def _heads_factory(shift_m=False, swap=False):
    def mh(x, idx, Wh, b=None, keys=None):
        x = np.asarray(x, dtype=np.float64)
        Wh = np.asarray(Wh, dtype=np.float64)
        H, hd = Wh.shape[0], Wh.shape[1]
        m = R.max_relative_ref(x, idx, keys)
        outs = []
        for h in range(H):
            sl = slice(h * hd, (h + 1) * hd)
            hm = ((h + 1) % H) if shift_m else h
            slm = slice(hm * hd, (hm + 1) * hd)
            parts = [m[..., slm], x[..., sl]] if swap else [x[..., sl], m[..., slm]]
            outs.append(np.concatenate(parts, axis=-1) @ Wh[h].T)
        out = np.concatenate(outs, axis=-1)
        return out if b is None else out + b
    return mh


def _max_pool_factory(offset=0, transposed=False, mean=False):
    def mp(x, H, W, r):
        x = np.asarray(x, dtype=np.float64)
        B, N, C = x.shape
        Hr, Wr = H // r, W // r
        out = np.empty((B, Hr * Wr, C))
        for p in range(Hr):
            for q in range(Wr):
                rows = [min((p * r + u + offset) * W + (q * r + v), N - 1) for u in range(r) for v in range(r)]
                vals = x[:, rows, :]
                o = q * Hr + p if transposed else p * Wr + q
                out[:, o, :] = vals.mean(1) if mean else vals.max(1)
        return out
    return mp


def _dist_factory(norm_keys=True, rows_on_keys=False, ignore_rows=False, norm_after_rows=True):
    def dist(x, keys=None, rows=None):
        x = np.asarray(x, dtype=np.float64)
        ks = x if keys is None else np.asarray(keys, dtype=np.float64)
        rows_ = np.arange(x.shape[1]) if (rows is None or ignore_rows) else np.asarray(rows)
        out = []
        for b in range(x.shape[0]):
            Q = R.l2_normalize(x[b])[rows_] if norm_after_rows else R.l2_normalize(x[b, rows_])
            K = ks[b, rows_] if rows_on_keys else ks[b]
            K = R.l2_normalize(K) if norm_keys else K
            out.append(R.pairwise_sq_dist(Q, K))
        return np.stack(out)
    return dist


def _lists_factory(offset=0, tie_high=False):
    def lists(D, k, dilation=1):
        D = np.asarray(D, dtype=np.float64)
        out = []
        for b in range(D.shape[0]):
            if tie_high:
                order = D.shape[-1] - 1 - np.argsort(D[b][:, ::-1], axis=1, kind="stable")
            else:
                order = np.argsort(D[b], axis=1, kind="stable")
            out.append(order[:, offset:k * dilation + offset][:, ::dilation][:, :k])
        return np.stack(out)
    return lists


MUTANTS = {
    "knn_no_normalisation": dict(knn_ref=_knn_factory(normalize=False)),
    "knn_descending": dict(knn_ref=_knn_factory(descending=True)),
    "knn_dilation_offset": dict(knn_ref=_knn_factory(dil_offset=1)),
    "knn_tie_higher_index": dict(knn_ref=_knn_factory(tie_high=True)),
    "knn_l1_distance": dict(knn_ref=_knn_factory(dist="l1")),
    "maxrel_sign_flipped": dict(max_relative_ref=_maxrel_factory(sign=-1),
                                mrconv_ref=_mrconv_factory(_maxrel_factory(sign=-1))),
    "maxrel_min_not_max": dict(max_relative_ref=_maxrel_factory(use_min=True),
                               mrconv_ref=_mrconv_factory(_maxrel_factory(use_min=True))),
    "mrconv_halves_swapped": dict(mrconv_ref=_mrconv_factory(swap_halves=True)),
    "mrconv_weight_transposed": dict(mrconv_ref=_mrconv_factory(transpose_w=True)),
    "mrconv_bias_dropped": dict(mrconv_ref=_mrconv_factory(drop_bias=True)),
    "pool_transposed": dict(pool_keys_ref=_pool_transposed),
    "stack_standard_not_lookahead": dict(stack_ref=_stack_factory(schedule_override="standard")),
    "stack_pool_transposed": dict(stack_ref=_stack_factory(pool=_pool_transposed)),
    "gelu_tanh_approximation": dict(gelu_ref=_gelu_tanh),
    "linear_weight_not_transposed": dict(linear_ref=_linear_untransposed),
    "block_no_fc2_residual": dict(vig_block_ref=_block_factory(fc2_residual=False)),
    "block_ffn_residual_from_x": dict(vig_block_ref=_block_factory(ffn_residual="x")),
    "block_gelu_after_wout": dict(vig_block_ref=_block_factory(gelu_after_wout=True)),
    "block_ffn_bias_dropped": dict(vig_block_ref=_block_factory(drop_b1=True)),
    "vig_stack_graph_from_x": dict(vig_stack_ref=_vig_stack_factory(graph_from="x")),
    "vig_stack_no_lookahead": dict(vig_stack_ref=_vig_stack_factory(lag=0)),
    "block_keys_pooled_from_x": dict(vig_block_ref=_block_factory(pool_from="x")),
    "block_gathers_unpooled_rows": dict(vig_block_ref=_block_factory(pool_from="none")),
    "vig_stack_graph_keys_unpooled": dict(vig_stack_ref=_vig_stack_factory(graph_keys="unpooled")),
    "vig_stack_graph_keys_from_own_u": dict(vig_stack_ref=_vig_stack_factory(graph_keys="own")),
    "heads_m_from_next_head": dict(mrconv_heads_ref=_heads_factory(shift_m=True)),
    "heads_halves_swapped": dict(mrconv_heads_ref=_heads_factory(swap=True)),
    "max_pool_window_shifted": dict(max_pool_nodes_ref=_max_pool_factory(offset=1)),
    "max_pool_output_transposed": dict(max_pool_nodes_ref=_max_pool_factory(transposed=True)),
    "max_pool_is_mean": dict(max_pool_nodes_ref=_max_pool_factory(mean=True)),
    "dist_keys_not_normalised": dict(knn_distances=_dist_factory(norm_keys=False)),
    "dist_rows_applied_to_keys": dict(knn_distances=_dist_factory(rows_on_keys=True)),
    "dist_rows_ignored": dict(knn_distances=_dist_factory(ignore_rows=True)),
    "dilated_lists_offset": dict(dilated_lists=_lists_factory(offset=1)),
    "dilated_lists_tie_higher_index": dict(dilated_lists=_lists_factory(tie_high=True)),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    bad = failing_pins(_ns(**MUTANTS[name]))
    assert bad, f"mutant {name} passed every pin"


def test_real_oracle_passes_all():
    assert failing_pins(oracle) == []
