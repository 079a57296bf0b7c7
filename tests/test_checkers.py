"""Pins of the tolerance checks the GPU parity tests apply to re-rotated keys.

A composition rotates stored keys by the position shift of their segment.
The GPU tests compare the device's result with the oracle's re-rotation of
the device's own stored source keys and allow one rounding to the storage
type plus float32 arithmetic noise (``twin.close_one_rounding``).  These CPU
tests model the device's arithmetic in NumPy and show that the check accepts
a correct float32 rotation rounded once, and rejects the mistakes it is there
to catch: an angle formed in float32 at a large shift, a wrong sign of the
sine, a rotation by the wrong shift, and the double rounding of comparing
against a key rounded before the rotation.
"""
import numpy as np
import pytest

import synth
from oracle import apply_rope, inv_freq, rerotate
from twin import close_one_rounding, close_rerotated

DH, BASE = 128, 500000.0


def _bf16(x):
    return synth.bf16_bits_to_f64(synth.f32_to_bf16_bits(np.asarray(x, dtype=np.float32)))


def _keys(n=512, seed=0):
    rng = np.random.default_rng(seed)
    return _bf16(rng.standard_normal((2, n, DH)) * 2.0)   # stored bf16 keys, |k| ~ 2


def _device_rotation(k, delta, angle32=False, sign=1.0):
    """A float32 rotation of stored keys as the compose kernel computes it:
    cos / sin of |delta| theta_i from a double table rounded to float32 (or,
    with angle32, of an angle formed in float32), products and sums in
    float32, then one rounding to bf16."""
    th = inv_freq(DH, BASE)
    ad = abs(delta)
    if angle32:
        ang = (np.float32(ad) * th.astype(np.float32)).astype(np.float64)
    else:
        ang = ad * th
    c = np.cos(ang).astype(np.float32)
    s = (np.sin(ang) * (1 if delta >= 0 else -1) * sign).astype(np.float32)
    k32 = k.astype(np.float32)
    x, y = k32[..., :DH // 2], k32[..., DH // 2:]
    out = np.concatenate([x * c - y * s, x * s + y * c], axis=-1)
    return _bf16(out)


@pytest.mark.parametrize("delta", [1, 4096, -29960, 30200, 34500])
def test_one_rounding_accepts_a_correct_rotation(delta):
    k = _keys()
    close_one_rounding(_device_rotation(k, delta), rerotate(k, delta, BASE), "bf16")


def test_one_rounding_rejects_a_float32_angle():
    """An angle p * theta formed in float32 is off by up to ~2e-3 rad at
    p ~ 3e4: far inside the old two-rounding bound, caught here."""
    k = _keys()
    got = _device_rotation(k, 30200, angle32=True)
    want = rerotate(k, 30200, BASE)
    close_rerotated(got, want, "bf16")                  # the loose bound lets it through
    with pytest.raises(AssertionError):
        close_one_rounding(got, want, "bf16")


@pytest.mark.parametrize("mistake", ["sign", "shift"])
def test_one_rounding_rejects_wrong_rotations(mistake):
    k = _keys(seed=1)
    if mistake == "sign":
        got = _device_rotation(k, 4096, sign=-1.0)
    else:
        got = _device_rotation(k, 4097)
    with pytest.raises(AssertionError):
        close_one_rounding(got, rerotate(k, 4096, BASE), "bf16")


def test_double_rounding_is_not_one_rounding():
    """Against the unrounded oracle (projected key rotated straight to its new
    position) the device result carries two roundings, which the one-rounding
    bound does not allow: that is why the check re-rotates the stored key."""
    rng = np.random.default_rng(3)
    u = rng.standard_normal((2, 4096, DH)) * 2.0               # projected keys, float64
    p, delta = 100, 30000
    stored = _bf16(apply_rope(u, np.full(u.shape[1], p), BASE))   # rounded once at p
    got = _device_rotation(stored, delta)                          # rounded again
    with pytest.raises(AssertionError):
        close_one_rounding(got, apply_rope(u, np.full(u.shape[1], p + delta), BASE), "bf16")
    close_one_rounding(got, rerotate(stored, delta, BASE), "bf16")
