"""Input generators: seeded, reproducible, and the bf16 conversion is round-to-nearest-even."""
import numpy as np
import torch

import workloads as W


def test_bf16_conversion_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000, dtype=np.float32) * s for s in (1e-30, 1e-3, 1, 1e3, 1e30)])
    # ties: mantissa low half exactly 0x8000
    ties = (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = W.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_configs_reproducible_and_shaped():
    c1 = W.CONFIGS[1]
    a, b = W.fwd_inputs(c1), W.fwd_inputs(c1)
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert a["x"].shape == (1, 1024, 64) and a["x"].dtype == np.float32
    assert a["gamma"].shape == (64, 4) and a["gamma"].dtype == np.float32
    assert a["gamma"].min() >= 1e-3 and a["gamma"].max() <= 0.5
    assert a["omega"].min() >= 0 and a["omega"].max() <= np.float32(np.pi)
    r = W.fwd_inputs(W.CONFIGS[3], L=64)
    assert r["x"].dtype == np.uint16 and r["x"].shape == (4, 64, 256)
    assert r["gamma"].min() >= 1e-5 * 0.999 and r["gamma"].max() <= 1.0


def test_decode_stream_is_one_sequence():
    c4 = W.CONFIGS[4]
    s1 = W.DecodeInputs(c4, B=2, L=8, D=4)
    a = np.concatenate([s1.steps(3), s1.steps(5)])
    s2 = W.DecodeInputs(c4, B=2, L=8, D=4)
    b = s2.steps(8)
    assert np.array_equal(a, b)
    assert np.array_equal(s1.prompt, s2.prompt)


def test_train_layers_independent_streams():
    c5 = W.CONFIGS[5]
    l2a = W.train_layer_inputs(c5, 2, B=1, L=16, D=8)
    l2b = W.train_layer_inputs(c5, 2, B=1, L=16, D=8)
    l3 = W.train_layer_inputs(c5, 3, B=1, L=16, D=8)
    assert np.array_equal(l2a["x"], l2b["x"]) and not np.array_equal(l2a["x"], l3["x"])
