"""GPU parity of the pyramid stage transition: gl_max_pool_nodes (bit-exact,
a maximum of stored values needs no rounding) and max pooling followed by the
gl_linear width projection, against the CPU oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from gpu_helpers import check_close, from_dev, require_gpu, to_dev
from paper_2604_21290_amd import inputs as I

pytestmark = pytest.mark.gpu


def _say(*a):
    print("[gpu-test]", *a, flush=True)


MAX_POOL = [
    # label, B, H, W, C, r, dtype
    ("stage1_to_2", 32, 56, 56, 80, 2, I.BF16),      # ViG-Py-S widths (paper's model table)
    ("stage2_to_3", 32, 28, 28, 160, 2, I.BF16),
    ("stage3_to_4", 32, 14, 14, 400, 2, I.BF16),
    ("fp32", 3, 10, 14, 12, 2, I.F32),
    ("non_square_r4", 2, 8, 12, 16, 4, I.BF16),
    ("r1_identity", 2, 5, 7, 8, 1, I.BF16),
    ("single_window", 1, 2, 2, 8, 2, I.BF16),
    ("r3_fp32", 1, 9, 6, 4, 3, I.F32),
]


@pytest.mark.parametrize("case", MAX_POOL, ids=[c[0] for c in MAX_POOL])
def test_max_pool_nodes(case):
    require_gpu()
    from paper_2604_21290_amd import api
    label, B, H, W, C, r, dt = case
    x = I.random_features(H * W * 7 + C, B, H * W, C, dt, unit=False)
    _say("max_pool", label, (B, H, W, C), "r", r, dt)
    out = api.max_pool_nodes(to_dev(x), H, W, r)
    torch.cuda.synchronize()
    got = from_dev(out).value
    ref = O.max_pool_nodes_ref(x.value, H, W, r)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref), (label, float(np.abs(got - ref).max()))


@pytest.mark.parametrize("dt", [I.BF16, I.F32])
def test_stage_transition_pool_then_project(dt):
    """Stage 1 -> 2 of the pyramid: 2 x 2 max pooling of the 56 x 56 grid, then
    the 80 -> 160 width projection (gl_linear), on 4 images."""
    require_gpu()
    from paper_2604_21290_amd import api
    B, H, W, C, Cn = 4, 56, 56, 80, 160
    g = np.random.default_rng(21)
    x = I.random_features(77, B, H * W, C, dt, unit=False)
    Wp = I.store(g.uniform(-0.1, 0.1, (Cn, C)), dt)
    bp = I.store(g.uniform(-0.5, 0.5, Cn), dt)
    _say("stage transition", (B, H, W, C), "->", Cn, dt)
    pooled = api.max_pool_nodes(to_dev(x), H, W, 2)
    y = api.linear(pooled, to_dev(Wp), to_dev(bp))
    torch.cuda.synchronize()
    ref = O.linear_ref(O.max_pool_nodes_ref(x.value, H, W, 2), Wp.value, bp.value)
    check_close(from_dev(y).value, ref, dt, "stage transition")
