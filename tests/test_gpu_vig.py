"""GPU parity of the full GraphLeap ViG block (gl_linear, gl_vig_block,
gl_vig_stack) against the CPU oracle (Eq. 11-15, Alg. 1).

Blocks are teacher-forced: each block's projected features U, the graph built
from them and its output are checked against the oracle evaluated on the exact
stored tensors the GPU saw; the stack entry must then reproduce the
block-by-block run bit for bit."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check_close, check_idx, from_dev, require_gpu, to_dev
from paper_2604_21290_amd import inputs as I

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-test]", *a, flush=True)


def _dev_params(p: dict) -> dict:
    return {n: to_dev(v) for n, v in p.items()}


def _host_params(p: dict) -> dict:
    return {n: v.value for n, v in p.items()}


# -- gl_linear --------------------------------------------------------------------
LIN = [
    # label, R, K, Cout, act_in, act_out, residual, bias, dtype
    ("fc1_vig_ti", 6272, 192, 192, 0, 0, False, True, I.BF16),
    ("fc2_gelu_in_residual", 1000, 192, 192, 1, 0, True, True, I.BF16),
    ("ffn1_gelu_out", 777, 192, 768, 0, 1, False, True, I.BF16),
    ("ffn2_residual", 777, 768, 192, 0, 0, True, False, I.BF16),
    ("ragged_k_tail", 131, 40, 70, 1, 1, True, True, I.BF16),
    ("fp32_all", 257, 36, 130, 1, 1, True, True, I.F32),
    ("one_row", 1, 8, 1, 0, 0, False, False, I.BF16),
    # the 128 x 128, 8-wave tile: ragged rows, columns and last K stage; GELU on
    # either side; fp32
    ("big128_ragged", 33000, 520, 200, 0, 0, True, True, I.BF16),
    ("big128_gelu_out", 16384, 640, 640, 0, 1, False, True, I.BF16),
    ("big128_gelu_in_fp32", 33000, 256, 260, 1, 0, True, True, I.F32),
    # one-stage tiles (257..384 bytes of K per row): a partly filled stage,
    # ragged rows and columns, GELU on either side, fp32
    ("one_stage_k160_ragged", 999, 160, 72, 0, 0, True, True, I.BF16),
    ("one_stage_k136_gelu_in_out", 515, 136, 200, 1, 1, False, True, I.BF16),
    ("one_stage_fp32_k96", 300, 96, 100, 1, 0, True, False, I.F32),
    ("one_stage_fp32_k68", 77, 68, 33, 0, 1, True, True, I.F32),
    # 192-byte stages and one-stage tiles in half the LDS (the first pyramid
    # stage's C = 80 layers)
    ("k80_ffn1_gelu_out", 20000, 80, 320, 0, 1, False, True, I.BF16),
    ("k80_fc2_gelu_in_residual", 20001, 80, 80, 1, 0, True, True, I.BF16),
    ("k96_ragged_cols", 3001, 96, 99, 0, 0, True, False, I.BF16),
    ("k128_one_stage_8_waves", 4097, 128, 200, 0, 1, True, True, I.BF16),
    # GELU on A over one to six k-steps, channels past K in the last one,
    # ragged rows
    ("k8_gelu_in", 16400, 8, 48, 1, 0, True, False, I.BF16),
    ("k40_gelu_in_cout16", 20000, 40, 16, 1, 0, False, True, I.BF16),
    ("k192_gelu_in_out", 16500, 192, 192, 1, 1, True, True, I.BF16),
]


@pytest.mark.parametrize("case", LIN, ids=[c[0] for c in LIN])
def test_linear_parity(case):
    require_gpu()
    from paper_2604_21290_amd import api
    label, R, K, Co, ai, ao, with_res, with_bias, dt = case
    g = np.random.default_rng(R + 7 * K + Co)
    x = I.store(g.standard_normal((R, K)), dt)
    W = I.store(g.uniform(-1, 1, (Co, K)) / np.sqrt(K), dt)
    b = I.store(g.uniform(-0.5, 0.5, Co), dt) if with_bias else None
    r = I.store(g.standard_normal((R, Co)), dt) if with_res else None
    _say("linear", label)
    out = api.linear(to_dev(x), to_dev(W), None if b is None else to_dev(b), ai, ao,
                     None if r is None else to_dev(r))
    torch.cuda.synchronize()
    xa = O.gelu_ref(x.value) if ai else x.value
    ref = O.linear_ref(xa, W.value, None if b is None else b.value)
    if ao:
        ref = O.gelu_ref(ref)
    if r is not None:
        ref = ref + r.value
    check_close(from_dev(out).value, ref, dt, label)


def test_linear_residual_in_place():
    require_gpu()
    from paper_2604_21290_amd import api
    g = np.random.default_rng(5)
    x = I.store(g.standard_normal((300, 64)), I.BF16)
    W = I.store(g.uniform(-0.2, 0.2, (64, 64)), I.BF16)
    r = I.store(g.standard_normal((300, 64)), I.BF16)
    rd = to_dev(r)
    out = api.linear(to_dev(x), to_dev(W), residual=rd, out=rd)
    torch.cuda.synchronize()
    assert out.data_ptr() == rd.data_ptr()
    check_close(from_dev(out).value, O.linear_ref(x.value, W.value) + r.value, I.BF16, "in place")


# -- full blocks ------------------------------------------------------------------
# pyramid stages run three blocks with dilations (1, 2, 1), so that both graphs
# built inside blocks (from U^0 with d = 2, from U^1 with d = 1) rank pooled keys
PYR_DIL = (1, 2, 1)


def _workload(name, B):
    """name[:opt] at batch B; ":f32" runs the workload in fp32, ":pool2" pools
    its keys 2 x 2 (at C = 640 the update then takes the two-pass form with
    pooled keys and the GELU in its GEMM's epilogue)."""
    base, _, opt = name.partition(":")
    w = I.with_batch(I.WORKLOADS[base], B)
    if opt == "pool2":
        w = dataclasses.replace(w, pool_r=2)
    if w.pool_r > 1:
        w = dataclasses.replace(w, dilations=PYR_DIL)
    if opt == "f32":
        w = dataclasses.replace(w, dtype=I.F32)
    return w


def _grid(w):
    return dict(H=w.H, W=w.W, pool_r=w.pool_r)


def _run_blocks(w, L, x0d, params_d, same_stream=False):
    """Drive L full blocks through gl_vig_block; return xs, us, graphs used."""
    from paper_2604_21290_amd import api
    B, N, C = x0d.shape
    dil = w.dilations
    s_up = torch.cuda.current_stream()
    la = api.Lookahead(s_up, s_up if same_stream else torch.cuda.Stream())
    ws = api.vig_workspace(x0d, w.k, **_grid(w))
    bufs = [torch.empty((B, N, w.k), dtype=torch.int32, device="cuda") for _ in range(2)]
    u0 = api.linear(x0d, params_d[0]["W_in"], params_d[0].get("b_in"))
    keys0 = api.pool_keys(u0, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
    api.knn_graph(u0, w.k, dil[0], keys=keys0, out=bufs[0])
    xs, us, graphs, cur = [x0d], [], [], 0
    for l in range(L):
        idx_next, nxt = None, cur
        if l + 1 < L and not (l == 0 and dil[1] == dil[0]):
            nxt = 1 - cur
            idx_next = bufs[nxt]
        torch.cuda.synchronize()
        graphs.append(bufs[cur].clone())
        x_out, u_out = la.vig_block(xs[-1], bufs[cur], params_d[l], ws, idx_next=idx_next,
                                    dilation_next=dil[l + 1] if idx_next is not None else 1,
                                    **_grid(w))
        torch.cuda.synchronize()
        us.append(u_out.clone())
        xs.append(x_out)
        cur = nxt
    torch.cuda.synchronize()
    la.close()
    return xs, us, graphs


@pytest.mark.parametrize("name,B,L", [("vig_ti", 4, 6), ("vig_b", 2, 5), ("single", 1, 1),
                                      ("pyr_s1", 2, 3), ("pyr_s2", 2, 3), ("pyr_s2:f32", 1, 3),
                                      ("vig_b:pool2", 2, 3)])
def test_vig_blocks_teacher_forced(name, B, L):
    require_gpu()
    from paper_2604_21290_amd import api
    w = _workload(name, B)
    x0 = I.make_features(w)
    ps = [I.make_vig_params(w, l) for l in range(L)]
    pd = [_dev_params(p) for p in ps]
    ph = [_host_params(p) for p in ps]
    _say("vig blocks", name, "B", B, "L", L)
    xs, us, graphs = _run_blocks(w, L, to_dev(x0), pd)
    hx = [from_dev(x).value for x in xs]
    hu = [from_dev(u).value for u in us]
    for l in range(L):
        # U^l = X^l W_in^T + b_in on the stored X^l
        check_close(hu[l], O.linear_ref(hx[l], ph[l]["W_in"], ph[l]["b_in"]), w.dtype,
                    f"{name} U^{l}")
        # the graph used by block l: G(U^0) for l <= 1, else G(U^(l-1)), on stored U
        # and, at pyramid stages, on the stored keys pooled from it
        s_l = 0 if l == 0 else l - 1
        src = hu[s_l]
        keys = None
        if w.pool_r > 1:
            keys = from_dev(api.pool_keys(us[s_l], w.H, w.W, w.pool_r)).value
            check_close(keys, O.pool_keys_ref(src, w.H, w.W, w.pool_r), w.dtype,
                        f"{name} keys of U^{s_l}")
        g = graphs[l].cpu().numpy()
        check_idx(g, O.knn_distances(src, keys), w.k, w.dilations[l], label=f"{name} graph {l}")
        # X^(l+1) from the stored X^l and the GPU's graph
        ref = O.vig_block_ref(hx[l], g, ph[l], **_grid(w))
        rel = check_close(hx[l + 1], ref, w.dtype, f"{name} block {l}")
        _say(name, "block", l, "rel", rel)


@pytest.mark.parametrize("name,B,L", [("vig_ti", 4, 6), ("vig_b", 2, 5), ("pyr_s1", 2, 3),
                                      ("pyr_s2", 2, 3), ("pyr_s2:f32", 1, 3), ("vig_b:pool2", 2, 3)])
def test_vig_stack_matches_blocks(name, B, L):
    require_gpu()
    from paper_2604_21290_amd import api
    w = _workload(name, B)
    x0d = to_dev(I.make_features(w))
    pd = [_dev_params(I.make_vig_params(w, l)) for l in range(L)]
    dil = list(w.dilations[:L])
    xs, _, _ = _run_blocks(w, L, x0d, pd)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    outs = {}
    for name_s, sc in (("fused", api.GL_SCHED_LOOKAHEAD_FUSED), ("two_stream", api.GL_SCHED_LOOKAHEAD)):
        _say("vig stack", name, name_s)
        outs[name_s] = la.vig_stack(x0d, pd, dil, w.k, schedule=sc, **_grid(w))
    torch.cuda.synchronize()
    la.close()
    for k_, v in outs.items():
        assert torch.equal(v, xs[-1]), f"{name}: stack ({k_}) differs from block-by-block"


@pytest.mark.parametrize("name", ["vig_ti", "pyr_s2"])
def test_vig_standard_schedule_teacher_forced(name):
    require_gpu()
    from paper_2604_21290_amd import api
    w = _workload(name, 2)
    L = 3
    x0d = to_dev(I.make_features(w))
    ps = [I.make_vig_params(w, l) for l in range(L)]
    pd = [_dev_params(p) for p in ps]
    dil = list(w.dilations[:L])
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.current_stream())
    ws = api.vig_workspace(x0d, w.k, **_grid(w))
    # block by block: graph from this block's own U (and its pooled keys)
    xs = [x0d]
    for l in range(L):
        u = api.linear(xs[-1], pd[l]["W_in"], pd[l]["b_in"])
        keys = api.pool_keys(u, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
        idx = api.knn_graph(u, w.k, dil[l], keys=keys)
        x_out, u_out = la.vig_block(xs[-1], idx, pd[l], ws, **_grid(w))
        torch.cuda.synchronize()
        assert torch.equal(u, u_out)
        ref = O.vig_block_ref(from_dev(xs[-1]).value, idx.cpu().numpy(), _host_params(ps[l]),
                              **_grid(w))
        check_close(from_dev(x_out).value, ref, w.dtype, f"{name} standard block {l}")
        check_idx(idx.cpu().numpy(),
                  O.knn_distances(from_dev(u).value, None if keys is None else from_dev(keys).value),
                  w.k, dil[l], label=f"{name} standard graph {l}")
        xs.append(x_out)
    st = la.vig_stack(x0d, pd, dil, w.k, schedule=api.GL_SCHED_STANDARD, **_grid(w))
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(st, xs[-1])


@pytest.mark.parametrize("name", ["vig_ti", "pyr_s2"])
def test_vig_zero_branches_are_identity(name):
    """W_out = 0 and W_2 = 0, no biases: every schedule returns X^0 bit for bit."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = _workload(name, 2)
    L = min(4, w.L)
    x0d = to_dev(I.make_features(w))
    pd = []
    for l in range(L):
        p = _dev_params(I.make_vig_params(w, l, bias=False))
        p["W_out"] = torch.zeros_like(p["W_out"])
        p["W_2"] = torch.zeros_like(p["W_2"])
        pd.append(p)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    for sc in (api.GL_SCHED_LOOKAHEAD_FUSED, api.GL_SCHED_LOOKAHEAD, api.GL_SCHED_STANDARD):
        out = la.vig_stack(x0d, pd, list(w.dilations[:L]), w.k, schedule=sc, **_grid(w))
        torch.cuda.synchronize()
        assert torch.equal(out, x0d), sc
    la.close()


def test_vig_pooled_shape_errors():
    """Pooling windows that do not divide the grid or leave fewer keys than k,
    a grid that does not match N, and a short workspace are refused before
    anything is enqueued."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = _workload("pyr_s2", 1)
    x0d = to_dev(I.make_features(w))
    pd = [_dev_params(I.make_vig_params(w, 0))]
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    ws = api.vig_workspace(x0d, w.k, w.H, w.W, w.pool_r)
    idx = torch.zeros((1, w.N, w.k), dtype=torch.int32, device="cuda")
    with pytest.raises(api.GraphLeapError, match="BAD_SHAPE"):
        la.vig_block(x0d, idx, pd[0], ws, H=w.H, W=w.W, pool_r=3)      # 3 does not divide 28
    with pytest.raises(api.GraphLeapError, match="BAD_SHAPE"):
        la.vig_stack(x0d, pd, [1], w.k, ws=ws, H=w.H, W=w.W, pool_r=0)
    with pytest.raises(api.GraphLeapError, match="grid"):
        la.vig_stack(x0d, pd, [1], w.k, ws=ws, H=w.H, W=w.W + 1, pool_r=1)  # H*W != N
    with pytest.raises(api.GraphLeapError, match="BAD_K"):
        la.vig_stack(x0d, pd, [1], w.k, ws=ws, H=w.H, W=w.W, pool_r=14)     # M = 4 < k = 9
    small = ws[: ws.numel() // 2]
    with pytest.raises(api.GraphLeapError, match="BAD_SHAPE"):
        la.vig_stack(x0d, pd, [1], w.k, ws=small, H=w.H, W=w.W, pool_r=w.pool_r)
    torch.cuda.synchronize()
    la.close()


@pytest.mark.parametrize("name,B", [("vig_ti", 4), ("pyr_s2", 2)])
def test_vig_stack_hip_graph_replay(name, B):
    """The fused-schedule full-block stack captured in a HIP graph: every
    replay, with eager work and synchronisations between replays, equals the
    eager run.  Everything lives in the caller's workspace (at the pyramid
    stage the pooled keys too), so the capture holds no allocation."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = _workload(name, B)
    L = min(4, w.L)
    x0d = to_dev(I.make_features(w))
    pd = [_dev_params(I.make_vig_params(w, l)) for l in range(L)]
    dil = list(w.dilations[:L])
    s = torch.cuda.Stream()
    la = api.Lookahead(s, s)
    ws = api.vig_workspace(x0d, w.k, **_grid(w))
    ref = torch.empty_like(x0d)
    with torch.cuda.stream(s):
        la.vig_stack(x0d, pd, dil, w.k, schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws, x_out=ref,
                     **_grid(w))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    out = torch.empty_like(x0d)
    with torch.cuda.graph(g, stream=s):
        la.vig_stack(x0d, pd, dil, w.k, schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws, x_out=out,
                     **_grid(w))
    for r in range(4):
        out.zero_()
        junk = api.linear(x0d, pd[0]["W_in"])      # eager work between replays
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        _say(name, "graph replay", r)
        assert torch.equal(out, ref), f"{name}: replay {r} differs"
        del junk
    la.close()


@pytest.mark.parametrize("name", ["vig_ti", "vig_b", "pyr_s1", "pyr_s2"])
def test_vig_block_full_size_sampled(name):
    """One full block at the workload's full batch (the grids the benchmark
    launches), teacher-forced: the GPU's graph of U^0 goes in, and the first
    two images of X^1 and of the next graph G(U^0, d_1) are checked against
    the oracle on the stored tensors."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.WORKLOADS[name]
    d1 = 2
    x0 = I.make_features(w)
    p = I.make_vig_params(w, 0)
    x0d, pd = to_dev(x0), _dev_params(p)
    _say("vig full size", name, "B", w.B)
    u0 = api.linear(x0d, pd["W_in"], pd["b_in"])
    keys = api.pool_keys(u0, w.H, w.W, w.pool_r) if w.pool_r > 1 else None
    idx0 = api.knn_graph(u0, w.k, 1, keys=keys)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    ws = api.vig_workspace(x0d, w.k, **_grid(w))
    idx1 = torch.empty_like(idx0)
    x1, u_out = la.vig_block(x0d, idx0, pd, ws, idx_next=idx1, dilation_next=d1, **_grid(w))
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(u_out, u0)
    nb = 2
    hx0 = from_dev(x0d[:nb]).value
    hu0 = from_dev(u0[:nb]).value
    ph = _host_params(p)
    g0 = idx0[:nb].cpu().numpy()
    ref = O.vig_block_ref(hx0, g0, ph, **_grid(w))
    check_close(from_dev(x1[:nb]).value, ref, w.dtype, f"{name} full-size block, 2 images")
    hk = None if keys is None else from_dev(keys[:nb]).value
    check_idx(idx1[:nb].cpu().numpy(), O.knn_distances(hu0, hk), w.k, d1,
              label=f"{name} full-size next graph")


@pytest.mark.parametrize("name", ["vig_ti", "vig_b", "vig_s", "pyr_s1", "pyr_s3"])
def test_vig_stack_fused_equals_two_stream_full_size(name):
    """At the workload's full batch and depth (the launch configurations the
    benchmark times: one-launch blocks, build and gather sharing a launch,
    separate launches), the fused schedule's full-block stack equals the
    two-stream lookahead bit for bit."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.WORKLOADS[name]
    x0d = to_dev(I.make_features(w))
    pd = [_dev_params(I.make_vig_params(w, l)) for l in range(w.L)]
    dil = list(w.dilations)
    _say("vig stack full size", name, "B", w.B, "L", w.L)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    ws = api.vig_workspace(x0d, w.k, **_grid(w))
    fused = la.vig_stack(x0d, pd, dil, w.k, schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws,
                         **_grid(w))
    two = la.vig_stack(x0d, pd, dil, w.k, schedule=api.GL_SCHED_LOOKAHEAD, ws=ws, **_grid(w))
    torch.cuda.synchronize()
    la.close()
    assert torch.isfinite(fused.float()).all()
    assert torch.equal(fused, two), f"{name}: fused full-block stack differs from two-stream"
