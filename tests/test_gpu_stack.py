"""GPU parity of the GraphLeap lookahead (gl_lookahead_bootstrap,
gl_graphleap_block, gl_graphleap_stack) and of the standard schedule.

Every block is teacher-forced: the graph it used is checked against the oracle
kNN of the exact stored features (and pooled keys) it was built from, and its
output against the oracle MRConv of its exact stored inputs.  Free-running
fp64 stacks are not compared (near-tie flips may legitimately diverge)."""
import zlib

import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check_close, check_idx, from_dev, mrconv_mag, require_gpu, to_dev
from paper_2604_21290_amd import inputs as I

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-test]", *a, flush=True)


def _weights(w, L, zero_bias=True):
    Ws = [I.make_weight(w, l) for l in range(L)]
    bs = [I.make_bias(w, l, zero=zero_bias) for l in range(L)]
    Wst = I.Stored(np.stack([s.bits for s in Ws]), np.stack([s.value for s in Ws]), w.dtype)
    bst = I.Stored(np.stack([s.bits for s in bs]), np.stack([s.value for s in bs]), w.dtype)
    return Wst, bst


def run_blocks(w, x0d, Wd, bd, same_stream=False):
    """Drive the lookahead block by block; return (features, graphs used)."""
    from paper_2604_21290_amd import api
    B, N, C = x0d.shape
    L, dil = w.L, w.dilations
    s_up = torch.cuda.current_stream()
    la = api.Lookahead(s_up, s_up if same_stream else torch.cuda.Stream())
    bufs = [torch.empty((B, N, w.k), dtype=torch.int32, device="cuda") for _ in range(2)]
    keys_ws = (torch.empty((B, w.M, C), dtype=x0d.dtype, device="cuda") if w.pool_r > 1 else None)
    la.bootstrap(x0d, w.H, w.W, w.k, dil[0], w.pool_r, keys_ws, bufs[0])
    xs, graphs, cur = [x0d], [], 0
    for l in range(L):
        idx_next, nxt = None, cur
        if l + 1 < L:
            if not (l == 0 and dil[1] == dil[0]):
                nxt = 1 - cur
                idx_next = bufs[nxt]
        torch.cuda.synchronize()
        graphs.append(bufs[cur].clone())
        x_out = torch.empty_like(x0d)
        la.block(xs[-1], w.H, w.W, bufs[cur], Wd[l], bd[l], w.pool_r, keys_ws, x_out,
                 idx_next, dil[l + 1] if idx_next is not None else 1)
        xs.append(x_out)
        cur = nxt
    torch.cuda.synchronize()
    la.close()
    return xs, graphs


def teacher_forced_checks(w, xs, graphs, Wst, bst, schedule="lookahead", n_img=None,
                          rows=None):
    """xs: GPU features X^0..X^L; graphs: GPU graph used by each block."""
    from paper_2604_21290_amd import api
    src = O.graph_source_blocks(w.L, schedule)
    sl = slice(None) if n_img is None else slice(0, n_img)
    # only the checked images travel to the host
    host = [from_dev(x[sl]) for x in xs]
    sl = slice(None)
    stats = []
    for l in range(w.L):
        xg = host[src[l]].value[sl]
        keys_g = keys_u = None
        if w.pool_r > 1:
            nb = xg.shape[0]
            kg = from_dev(api.pool_keys(xs[src[l]], w.H, w.W, w.pool_r)[:nb])
            check_close(kg.value, O.pool_keys_ref(xg, w.H, w.W, w.pool_r), w.dtype,
                        f"pool block {l}")
            keys_g = kg.value
            keys_u = from_dev(api.pool_keys(xs[l], w.H, w.W, w.pool_r)[:nb]).value
        g = graphs[l][:xg.shape[0]].cpu().numpy()
        D = O.knn_distances(xg, keys_g, rows=rows)
        st = check_idx(g, D, w.k, w.dilations[l], rows=rows, label=f"{w.name} graph {l}")
        ref, xcat = O.mrconv_ref(host[l].value[sl], g, Wst.value[l], bst.value[l], keys=keys_u,
                                 return_concat=True)
        rel = check_close(host[l + 1].value[sl], ref, w.dtype, f"{w.name} block {l}",
                          mag=mrconv_mag(xcat, Wst.value[l]), n_terms=2 * w.C)
        stats.append((l, st["near_tie_rows"], rel))
    _say(w.name, schedule, "per-block (block, near-tie rows, rel err):", stats)


CASES = [
    # name, batch used on the GPU (None: the workload's full batch), images
    # checked against the oracle, sampled rows
    ("single", None, None, None),
    ("vig_ti", None, None, None),
    ("vig_b", None, 4, None),
    ("pyr_s1", None, 4, 384),
    ("pyr_s2", None, 4, None),
    ("hires", None, 2, 384),
    ("vig_ti_448", None, 2, 256),
    ("vig_s", None, 4, None),
    ("pyr_s3", None, 4, None),
    ("pyr_s4", None, 4, None),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_lookahead_blocks_teacher_forced(case):
    require_gpu()
    name, B, n_img, nrows = case
    w = I.WORKLOADS[name] if B is None else I.with_batch(I.WORKLOADS[name], B)
    rows = None
    if nrows is not None:
        rows = np.sort(np.random.default_rng(7).choice(w.N, nrows, replace=False))
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L)
    x0d, Wd, bd = to_dev(x0), to_dev(Wst), to_dev(bst)
    _say("lookahead blocks", name, "B", w.B)
    xs, graphs = run_blocks(w, x0d, Wd, bd)
    teacher_forced_checks(w, xs, graphs, Wst, bst, n_img=n_img, rows=rows)


@pytest.mark.parametrize("name", ["single", "vig_ti", "vig_b", "pyr_s1", "pyr_s2", "hires",
                                  "vig_ti_448", "vig_s", "pyr_s3", "pyr_s4"])
def test_stack_entry_matches_blocks_and_serial(name):
    """gl_graphleap_stack at the full workload size (the launch configuration
    the benchmark times) equals the block-by-block run bit for bit, and the
    overlapped run equals the same kernels on one stream."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.WORKLOADS[name]
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L)
    x0d, Wd, bd = to_dev(x0), to_dev(Wst), to_dev(bst)
    _say("stack entry", name)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    out = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r)
    out2 = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r)
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(out, out2), "stack not deterministic"
    xs, _ = run_blocks(w, x0d, Wd, bd)
    assert torch.equal(out, xs[-1]), "stack entry differs from block-by-block"
    xs1, _ = run_blocks(w, x0d, Wd, bd, same_stream=True)
    assert torch.equal(xs1[-1], xs[-1]), "one-stream run differs from overlapped run"
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    ws = api.make_stack_workspace(x0d, w.H, w.W, w.k, w.pool_r)
    fused = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r,
                     schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws)
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(fused, out), "one-launch blocks differ from the two-stream schedule"


@pytest.mark.parametrize("name", ["pyr_s1", "pyr_s2"])
def test_pooled_builds_agree_across_kernels(name):
    """At the pyramid's first two stages the standalone build keeps the keys
    resident in LDS, while the one-launch block builds with the in-register
    tile (stage 1, C = 80) or the LDS-staged wide tile (stage 2, C = 160).
    Both must rank the same packed keys.  With the dilation changing from
    block to block, the fused schedule builds every next graph inside the
    block and the two-stream schedule builds it standalone; the two stacks
    must be equal bit for bit, and the graphs are teacher-forced."""
    require_gpu()
    import dataclasses
    from paper_2604_21290_amd import api
    w = dataclasses.replace(I.WORKLOADS[name], dilations=(1, 2, 3, 1))
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L)
    x0d, Wd, bd = to_dev(x0), to_dev(Wst), to_dev(bst)
    _say("pooled builds", w.name, "dilations", w.dilations)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    two = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r)
    ws = api.make_stack_workspace(x0d, w.H, w.W, w.k, w.pool_r)
    fused = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r,
                     schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws)
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(fused, two), "block-built graphs differ from standalone-built graphs"
    xs, graphs = run_blocks(w, x0d, Wd, bd)
    assert torch.equal(xs[-1], two)
    rows = np.sort(np.random.default_rng(8).choice(w.N, 256, replace=False))
    teacher_forced_checks(w, xs, graphs, Wst, bst, n_img=2, rows=rows)


def _fused_graph_buffer(dil, Lp):
    """Which of the two graph buffers holds the graph the last block of an
    Lp-block fused-schedule stack used (the stack's own buffer rotation)."""
    cur = used = 0
    for l in range(Lp):
        used = cur
        if l + 1 < Lp and not (l == 0 and dil[1] == dil[0]):
            cur = 1 - cur
    return used


@pytest.mark.parametrize("name", ["vig_ti", "pyr_s2"])
def test_fused_schedule_teacher_forced(name):
    """The timed schedule (one launch per block) checked against the oracle
    directly: the stack's first l+1 blocks give X^(l+1) and leave the graph
    block l used in the workspace; each is graded on the GPU's own inputs."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.WORKLOADS[name]
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L, zero_bias=False)
    x0d, Wd, bd = to_dev(x0), to_dev(Wst), to_dev(bst)
    dil = list(w.dilations)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    full = la.stack(x0d, w.H, w.W, Wd, bd, dil, w.k, w.pool_r,
                    schedule=api.GL_SCHED_LOOKAHEAD_FUSED)
    xs, graphs = [x0d], []
    for l in range(w.L):
        ws = api.make_stack_workspace(x0d, w.H, w.W, w.k, w.pool_r)
        _say("fused prefix", name, "blocks", l + 1)
        out = la.stack(x0d, w.H, w.W, Wd[:l + 1], bd[:l + 1], dil[:l + 1], w.k, w.pool_r,
                       schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws)
        torch.cuda.synchronize()
        xs.append(out)
        graphs.append(ws["idx"][_fused_graph_buffer(dil, l + 1)].clone())
    la.close()
    assert torch.equal(xs[-1], full), "prefix run differs from the full stack"
    teacher_forced_checks(w, xs, graphs, Wst, bst, schedule="lookahead")


@pytest.mark.parametrize("name", ["vig_ti", "pyr_s2"])
def test_standard_schedule_teacher_forced(name):
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.with_batch(I.WORKLOADS[name], 8)
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L)
    x0d, Wd, bd = to_dev(x0), to_dev(Wst), to_dev(bst)
    xs, graphs = [x0d], []
    for l in range(w.L):
        keys = api.pool_keys(xs[l], w.H, w.W, w.pool_r) if w.pool_r > 1 else None
        idx = api.knn_graph(xs[l], w.k, w.dilations[l], keys=keys)
        graphs.append(idx)
        xs.append(api.mrconv(xs[l], idx, Wd[l], bd[l], keys=keys))
    torch.cuda.synchronize()
    teacher_forced_checks(w, xs, graphs, Wst, bst, schedule="standard")
    la = api.Lookahead()
    out = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r,
                   schedule=api.GL_SCHED_STANDARD)
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(out, xs[-1])


def test_identity_weights_schedules_agree():
    """W = [I | 0], b = 0 keeps every block's features equal to X^0, so the
    lookahead and standard schedules give X^0 back bit for bit."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.with_batch(I.WORKLOADS["vig_ti"], 4)
    x0d = to_dev(I.make_features(w))
    eye = np.hstack([np.eye(w.C), np.zeros((w.C, w.C))])
    Wd = to_dev(I.store(np.stack([eye] * w.L), w.dtype))
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    a = la.stack(x0d, w.H, w.W, Wd, None, list(w.dilations), w.k)
    b = la.stack(x0d, w.H, w.W, Wd, None, list(w.dilations), w.k, schedule=api.GL_SCHED_STANDARD)
    c = la.stack(x0d, w.H, w.W, Wd, None, list(w.dilations), w.k,
                 schedule=api.GL_SCHED_LOOKAHEAD_FUSED)
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(a, x0d) and torch.equal(b, x0d) and torch.equal(c, x0d)


def test_profiling_records_builds():
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.with_batch(I.WORKLOADS["vig_ti"], 4)
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    la.set_profiling(64)
    la.stack(to_dev(x0), w.H, w.W, to_dev(Wst), to_dev(bst), list(w.dilations), w.k)
    torch.cuda.synchronize()
    times = la.kernel_times_ms(api.GL_TIME_BUILD)
    upd = la.kernel_times_ms(api.GL_TIME_UPDATE)
    la.close()
    assert len(times) == w.L - 1          # bootstrap + L-2 lookahead builds (d_1 == d_0)
    assert len(upd) == w.L
    assert all(t > 0 for t in times) and all(t > 0 for t in upd)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    la.set_profiling(64)
    la.stack(to_dev(x0), w.H, w.W, to_dev(Wst), to_dev(bst), list(w.dilations), w.k,
             schedule=api.GL_SCHED_LOOKAHEAD_FUSED)
    torch.cuda.synchronize()
    b = la.kernel_times_ms(api.GL_TIME_BUILD)
    u = la.kernel_times_ms(api.GL_TIME_UPDATE)
    f = la.kernel_times_ms(api.GL_TIME_FUSED)
    la.close()
    # bootstrap build; blocks 0 and L-1 are plain updates; blocks 1..L-2 one launch each
    assert (len(b), len(u), len(f)) == (1, 2, w.L - 2)


@pytest.mark.parametrize("name", ["vig_ti", "vig_b"])
def test_stack_hip_graph_replay(name):
    """The fused-schedule stack captured in a HIP graph: every replay, with
    eager work and synchronisations between replays, equals the eager run.
    At ViG-B the updates take the two-pass form through the caller's
    workspace, so the capture holds no allocation."""
    require_gpu()
    from paper_2604_21290_amd import api
    w = I.with_batch(I.WORKLOADS[name], 4)
    x0d = to_dev(I.make_features(w))
    Wst, bst = _weights(w, w.L, zero_bias=False)
    Wd, bd = to_dev(Wst), to_dev(bst)
    s = torch.cuda.Stream()
    la = api.Lookahead(s, s)
    ws = api.make_stack_workspace(x0d, w.H, w.W, w.k)
    ref = torch.empty_like(x0d)
    with torch.cuda.stream(s):
        la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k,
                 schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws, x_out=ref)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    out = torch.empty_like(x0d)
    with torch.cuda.graph(g, stream=s):
        la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k,
                 schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws, x_out=out)
    for r in range(4):
        out.zero_()
        junk = api.knn_graph(x0d, w.k, 2)          # eager work between replays
        torch.cuda.synchronize()
        with torch.cuda.stream(s):
            g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {r} differs"
        del junk
    la.close()


# Two-pass updates (wide W) whose gather shares the fused schedule's launch
# with the next build: both key-row buckets of the LDS-staged build (M <= 128
# and up to 224), ragged node counts (R not a multiple of the 32-node gather
# tile, query rows not a multiple of 32), k = 16 and dilations up to 3.
TWO_PASS = [
    # label, B, H, W, C, k, dilations
    ("two_pass_M100_k16", 3, 10, 10, 320, 16, (1, 2, 3)),
    ("two_pass_M196_ragged", 2, 14, 14, 384, 9, (1, 1, 2, 2)),
    ("two_pass_M221_C640", 1, 13, 17, 640, 9, (1, 3)),
]


@pytest.mark.parametrize("case", TWO_PASS, ids=[c[0] for c in TWO_PASS])
def test_two_pass_shared_launch(case):
    require_gpu()
    from paper_2604_21290_amd import api
    label, B, H, W, C, k, dil = case
    w = I.Workload(label, B, H, W, C, k, dil, I.BF16, seed=zlib.crc32(label.encode()) % 1000)
    x0 = I.make_features(w)
    Wst, bst = _weights(w, w.L, zero_bias=False)
    x0d, Wd, bd = to_dev(x0), to_dev(Wst), to_dev(bst)
    _say("two-pass shared launch", label)
    xs, graphs = run_blocks(w, x0d, Wd, bd)
    teacher_forced_checks(w, xs, graphs, Wst, bst)
    la = api.Lookahead(torch.cuda.current_stream(), torch.cuda.Stream())
    ws = api.make_stack_workspace(x0d, w.H, w.W, w.k, w.pool_r)
    fused = la.stack(x0d, w.H, w.W, Wd, bd, list(w.dilations), w.k, w.pool_r,
                     schedule=api.GL_SCHED_LOOKAHEAD_FUSED, ws=ws)
    torch.cuda.synchronize()
    la.close()
    assert torch.equal(fused, xs[-1]), f"{label}: fused schedule differs from block-by-block"
