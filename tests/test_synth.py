"""The seeded input generators (CPU only)."""

import numpy as np
import torch

import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -1e-40], dtype=np.float32)])
    # ties: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 (rounds to even = 1.0)
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_draws_are_seeded_and_independent():
    a = synth.normal_bf16((4, 8, 128), 2, 0, 3, synth.TAG_K)
    b = synth.normal_bf16((4, 8, 128), 2, 0, 3, synth.TAG_K)
    c = synth.normal_bf16((4, 8, 128), 2, 0, 4, synth.TAG_K)
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    p = synth.page_permutation(100, 2, 1)
    assert sorted(p.tolist()) == list(range(100))


def test_workload_shapes():
    w = synth.decode_b64()
    assert w.ns == 64 and all(1024 <= c <= 32768 for c in w.prefix) and w.new == [1] * 64
    w = synth.stack70_decode()
    assert w.layers.count(synth.FULL) == 10 and w.layers[6] == synth.FULL and w.layers[69] == synth.FULL
    w = synth.mixed_step()
    assert w.ns == 264 and all(0 <= p <= 65536 for p in w.prefix[:8])
    assert all(2048 <= c <= 65536 for c in w.prefix[8:])
    med = np.median(w.prefix[8:])
    assert 5000 < med < 13000
    assert synth.cu_seqlens([3, 0, 2]).tolist() == [0, 3, 3, 5]
