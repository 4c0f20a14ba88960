"""Seeded input generators: storage rounding and workload shapes.  CPU only."""
import math

import numpy as np
import torch

from paper_2604_21290_amd import inputs as I


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    a = np.concatenate([g.standard_normal(20000) * 10.0 ** g.integers(-6, 6, 20000),
                        [0.0, -0.0, 1.0, -1.0, 3.0e38, 1e-40]])
    mine = I.f64_to_bf16_bits(a)
    ref = torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy()
    assert np.array_equal(mine, ref.view(np.uint16))
    back = I.bf16_bits_to_f64(mine)
    assert np.array_equal(back, torch.from_numpy(ref).view(torch.bfloat16).double().numpy())


def test_workloads_shapes():
    W = I.WORKLOADS
    assert (W["vig_ti"].B, W["vig_ti"].N, W["vig_ti"].C, W["vig_ti"].L) == (32, 196, 192, 12)
    assert W["vig_ti"].dilations == (1, 1, 1, 1, 2, 2, 2, 2, 3, 3, 3, 3)
    assert W["vig_b"].dilations == (1,) * 4 + (2,) * 4 + (3,) * 4 + (4,) * 4
    assert (W["pyr_s1"].N, W["pyr_s1"].M) == (3136, 196)
    assert (W["pyr_s2"].N, W["pyr_s2"].M) == (784, 196)
    assert (W["hires"].N, W["hires"].M, W["hires"].k) == (3136, 3136, 16)
    assert (W["vig_ti_448"].N, W["vig_s"].C, W["pyr_s3"].C, W["pyr_s4"].N) == (784, 320, 400, 49)
    for w in W.values():
        assert w.k * max(w.dilations) <= w.M


def test_generators_deterministic_and_stored_exactly():
    w = I.with_batch(I.WORKLOADS["vig_ti"], 2)
    a, b = I.make_features(w), I.make_features(w)
    assert np.array_equal(a.bits, b.bits) and a.bits.dtype == np.uint16
    assert a.shape == (2, 196, 192)
    assert np.allclose(np.linalg.norm(a.value, axis=-1), 1.0, atol=1e-2)
    Wt = I.make_weight(w, 3)
    assert Wt.shape == (192, 384)
    assert np.abs(Wt.value).max() <= math.sqrt(6 / 384) * (1 + 2 ** -8)
    h = I.make_features(I.with_batch(I.WORKLOADS["hires"], 1))
    assert h.shape == (1, 3136, 96)
    s = I.make_features(I.WORKLOADS["single"])
    assert s.bits.dtype == np.float32 and np.array_equal(s.value, s.bits.astype(np.float64))
