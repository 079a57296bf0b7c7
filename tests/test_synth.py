"""The seeded input generator gives the same bits on every backend."""
import numpy as np
import torch

import synth


def test_numpy_and_torch_streams_agree():
    key = synth.w_key(0, "tiny", 3)
    for dtype, std in (("bf16", 1 / 64), ("f32", 1.0)):
        a = synth.normal_np(key, (37, 129), std, dtype)
        b = synth.normal_torch(key, (37, 129), std, dtype, "cpu")
        if dtype == "bf16":
            assert np.array_equal(a.view(np.int16), b.view(torch.int16).numpy())
        else:
            assert np.array_equal(a, b.numpy())


def test_rows_and_distribution():
    key = synth.x_key(0, "fork4-8b", 0)
    full = synth.normal_np(key, (300, 64), 1.0, "bf16")
    rows = synth.normal_rows_np(key, 64, [0, 17, 299], 1.0, "bf16")
    assert np.array_equal(rows, full[[0, 17, 299]])
    v = synth.to_f64(synth.normal_np(key, (200000,), 1.0, "f32"), "f32")
    assert abs(v.mean()) < 0.01 and abs(v.std() - 1) < 0.01
    assert np.abs(v).max() < 4.4


def test_streams_differ_and_bf16_rounding():
    a = synth.normal_np((0, 1, 2), (1000,), 1.0, "f32")
    b = synth.normal_np((0, 1, 3), (1000,), 1.0, "f32")
    assert np.mean(a == b) < 0.01
    # round-to-nearest-even at the halfway point of two bf16 neighbours
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5], dtype=np.float32)
    assert list(synth.f32_to_bf16_bits(x)) == [0x3F80, 0x3F82, 0xC020]
    assert synth.to_f64(np.array([0x3F80, 0xC020], np.uint16), "bf16").tolist() == [1.0, -2.5]


def test_offset_streams_and_f64():
    key = synth.w_key(0, "tiny", 0)
    full = synth.normal_np(key, (10, 33), 0.5, "bf16")
    part = synth.normal_torch(key, (4, 33), 0.5, "bf16", "cpu", start=5 * 33)
    assert np.array_equal(part.view(torch.int16).numpy(), full[5:9].view(np.int16))
    f = synth.normal_f64(key, (4, 33), 0.5, "bf16", start=5 * 33)
    assert np.array_equal(f, synth.to_f64(full[5:9], "bf16"))
