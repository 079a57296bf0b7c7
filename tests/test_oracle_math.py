"""Pins for the oracle's arithmetic (RoPE, attention, projection), CPU only.

Each check compares the oracle with something other than itself: a closed
form, an independent formulation (complex rotation, blockwise online softmax,
explicit loops), or a library routine (torch's scaled_dot_product_attention
and linear in float64).
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import apply_rope, causal_gqa_attention, inv_freq, project_qkv, rerotate

RNG = np.random.default_rng(1234)


# ------------------------------------------------------------------ RoPE

def test_inv_freq_closed_form():
    th = inv_freq(8, 10000.0)
    assert th[0] == 1.0
    np.testing.assert_allclose(th, [1.0, 0.1, 0.01, 0.001], rtol=1e-15)


def test_rope_hand_example_dh4():
    # dh=4, base=1e4: theta = (1, 0.01); pairs (u0,u2) and (u1,u3); p=1.
    # cos 1 = 0.5403023058681398, sin 1 = 0.8414709848078965,
    # cos .01 = 0.9999500004166653, sin .01 = 0.009999833334166664
    u = np.array([[1.0, 2.0, 3.0, 4.0]])
    got = apply_rope(u, [1], 10000.0)[0]
    want = [1 * 0.5403023058681398 - 3 * 0.8414709848078965,
            2 * 0.9999500004166653 - 4 * 0.009999833334166664,
            1 * 0.8414709848078965 + 3 * 0.5403023058681398,
            2 * 0.009999833334166664 + 4 * 0.9999500004166653]
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)


@pytest.mark.parametrize("dh,base", [(64, 10000.0), (128, 10000.0), (128, 500000.0)])
def test_rope_matches_complex_rotation(dh, base):
    # independent formulation: z_i = u_i + i u_{i+dh/2} multiplied by e^{i p theta_i}
    u = RNG.standard_normal((7, dh))
    pos = np.array([0, 1, 5, 100, 4095, 32767, 35071])
    half = dh // 2
    z = u[:, :half] + 1j * u[:, half:]
    theta = np.array([base ** (-2.0 * i / dh) for i in range(half)])
    zr = z * np.exp(1j * pos[:, None] * theta[None, :])
    want = np.concatenate([zr.real, zr.imag], axis=1)
    # angles reach 3.5e4 rad: float64 argument rounding is ~1e-11 there
    np.testing.assert_allclose(apply_rope(u, pos, base), want, rtol=0, atol=1e-10)


def test_rope_group_properties():
    dh, base = 128, 10000.0
    u = RNG.standard_normal((5, dh))
    pos = np.array([0, 3, 17, 4096, 30000])
    r = apply_rope(u, pos, base)
    # R(0) = I
    np.testing.assert_array_equal(apply_rope(u, np.zeros(5, int), base), u)
    # norm preserved
    np.testing.assert_allclose(np.linalg.norm(r, axis=1), np.linalg.norm(u, axis=1), rtol=1e-13)
    # R(delta) R(p) = R(p + delta), for positive and negative shifts
    for d in (1, 32, 4096, 28672, -3):
        np.testing.assert_allclose(rerotate(r, d, base), apply_rope(u, pos + d, base),
                                   rtol=0, atol=1e-10)
    # R(-delta) R(delta) = I
    np.testing.assert_allclose(rerotate(rerotate(u, 4096, base), -4096, base), u, atol=1e-12)


def test_rope_relative_position_property():
    # <R(p) q, R(s) k> depends only on p - s
    dh, base = 64, 10000.0
    q, k = RNG.standard_normal(dh), RNG.standard_normal(dh)
    a = apply_rope(q[None], [130], base)[0] @ apply_rope(k[None], [100], base)[0]
    b = apply_rope(q[None], [30], base)[0] @ apply_rope(k[None], [0], base)[0]
    assert abs(a - b) < 1e-10


def test_rope_not_applied_to_wrong_pairs():
    # a vector with energy in one pair only stays in that pair
    dh = 16
    u = np.zeros((1, dh))
    u[0, 3] = 1.0
    r = apply_rope(u, [7], 10000.0)[0]
    nz = set(np.nonzero(np.abs(r) > 1e-15)[0].tolist())
    assert nz <= {3, 3 + dh // 2}


# ------------------------------------------------------------------ attention

def _sdpa_ref(q, k, v):
    qt = torch.from_numpy(q)[None]
    kt = torch.from_numpy(k)[None]
    vt = torch.from_numpy(v)[None]
    return F.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True)[0].numpy()


@pytest.mark.parametrize("hq,hkv,t,dh", [(4, 2, 9, 16), (8, 8, 5, 8), (32, 8, 33, 128), (8, 1, 17, 64)])
def test_attention_matches_torch_sdpa(hq, hkv, t, dh):
    q = RNG.standard_normal((hq, t, dh))
    k = RNG.standard_normal((hkv, t, dh))
    v = RNG.standard_normal((hkv, t, dh))
    pos = np.arange(t) + 11
    got = causal_gqa_attention(q, k, v, pos, pos)
    np.testing.assert_allclose(got, _sdpa_ref(q, k, v), rtol=0, atol=1e-12)


def test_attention_explicit_loops():
    hq, hkv, dh = 4, 2, 3
    tq, tk = 3, 5
    q = RNG.standard_normal((hq, tq, dh))
    k = RNG.standard_normal((hkv, tk, dh))
    v = RNG.standard_normal((hkv, tk, dh))
    kpos = np.arange(tk)
    qpos = np.array([2, 3, 4])
    got = causal_gqa_attention(q, k, v, qpos, kpos)
    for h in range(hq):
        g = h // (hq // hkv)
        for t in range(tq):
            w = []
            for s in range(tk):
                if kpos[s] <= qpos[t]:
                    d = sum(q[h, t, i] * k[g, s, i] for i in range(dh)) / math.sqrt(dh)
                    w.append((math.exp(d), s))
            z = sum(e for e, _ in w)
            for i in range(dh):
                o = sum(e * v[g, s, i] for e, s in w) / z
                assert abs(o - got[h, t, i]) < 1e-12


def test_attention_two_token_closed_form():
    # q = (1, 0); k0 = (0, 0), k1 = (1, 0); at t=1 weights are 1 : e^{1/sqrt 2}
    q = np.array([[[0.0, 0.0], [1.0, 0.0]]])
    k = np.array([[[0.0, 0.0], [1.0, 0.0]]])
    v = np.array([[[1.0, 2.0], [3.0, -1.0]]])
    o = causal_gqa_attention(q, k, v, [0, 1], [0, 1])
    e = math.exp(1 / math.sqrt(2))
    np.testing.assert_allclose(o[0, 0], [1.0, 2.0], atol=1e-15)
    np.testing.assert_allclose(o[0, 1], [(1 + 3 * e) / (1 + e), (2 - e) / (1 + e)], atol=1e-15)


def test_attention_special_cases():
    dh = 8
    # one visible key -> o = v
    q = RNG.standard_normal((2, 1, dh))
    k = RNG.standard_normal((1, 1, dh))
    v = RNG.standard_normal((1, 1, dh))
    o = causal_gqa_attention(q, k, v, [0], [0])
    np.testing.assert_allclose(o[0, 0], v[0, 0], atol=1e-15)
    np.testing.assert_allclose(o[1, 0], v[0, 0], atol=1e-15)
    # identical keys -> running mean of the visible values
    t = 6
    k = np.repeat(RNG.standard_normal((1, 1, dh)), t, axis=1)
    v = RNG.standard_normal((1, t, dh))
    q = RNG.standard_normal((1, t, dh))
    o = causal_gqa_attention(q, k, v, np.arange(t), np.arange(t))
    for i in range(t):
        np.testing.assert_allclose(o[0, i], v[0, :i + 1].mean(axis=0), atol=1e-13)
    # keys after the query are invisible: appending future keys changes nothing
    k2 = np.concatenate([k, RNG.standard_normal((1, 3, dh))], axis=1)
    v2 = np.concatenate([v, RNG.standard_normal((1, 3, dh))], axis=1)
    o2 = causal_gqa_attention(q, k2, v2, np.arange(t), np.arange(t + 3))
    np.testing.assert_allclose(o2, o, atol=1e-13)


def test_attention_blockwise_online_softmax_form():
    # an independent blockwise formulation with running max / sum
    hq, hkv, tq, tk, dh = 4, 2, 7, 41, 16
    q = RNG.standard_normal((hq, tq, dh)) * 3
    k = RNG.standard_normal((hkv, tk, dh))
    v = RNG.standard_normal((hkv, tk, dh))
    qpos = np.arange(tk - tq, tk)
    kpos = np.arange(tk)
    want = causal_gqa_attention(q, k, v, qpos, kpos)
    g = hq // hkv
    for h in range(hq):
        for t in range(tq):
            m, l, acc = -np.inf, 0.0, np.zeros(dh)
            for c0 in range(0, tk, 8):
                sl = slice(c0, min(c0 + 8, tk))
                s = k[h // g, sl] @ q[h, t] / math.sqrt(dh)
                s = np.where(kpos[sl] <= qpos[t], s, -np.inf)
                mn = max(m, s.max())
                if mn == -np.inf:
                    continue
                p = np.exp(s - mn)
                acc = acc * math.exp(m - mn) + p @ v[h // g, sl]
                l = l * math.exp(m - mn) + p.sum()
                m = mn
            np.testing.assert_allclose(acc / l, want[h, t], atol=1e-12)


# ------------------------------------------------------------------ projection

def test_projection_matches_torch_linear():
    hq, hkv, dh, d, t = 4, 2, 8, 24, 5
    x = RNG.standard_normal((t, d))
    w = RNG.standard_normal(((hq + 2 * hkv) * dh, d))
    q, k, v = project_qkv(x, w, hq, hkv, dh)
    y = F.linear(torch.from_numpy(x), torch.from_numpy(w)).numpy()   # [t, cols]
    # column layout: Hq query heads, then Hkv key heads, then Hkv value heads
    for h in range(hq):
        np.testing.assert_allclose(q[h], y[:, h * dh:(h + 1) * dh], atol=1e-12)
    for h in range(hkv):
        np.testing.assert_allclose(k[h], y[:, (hq + h) * dh:(hq + h + 1) * dh], atol=1e-12)
        np.testing.assert_allclose(v[h], y[:, (hq + hkv + h) * dh:(hq + hkv + h + 1) * dh],
                                   atol=1e-12)


def test_oracle_exports():
    for name in ("OraclePool", "OracleError", "Status", "PACK_MAGIC"):
        assert hasattr(oracle, name)


def test_partial_projections_agree_with_full():
    from oracle import project_kv, project_q
    hq, hkv, dh, d, t = 4, 2, 8, 24, 5
    x = RNG.standard_normal((t, d))
    w = RNG.standard_normal(((hq + 2 * hkv) * dh, d))
    q, k, v = project_qkv(x, w, hq, hkv, dh)
    k2, v2 = project_kv(x, w, hq, hkv, dh)
    q2 = project_q(x[[1, 4]], w, hq, hkv, dh)
    np.testing.assert_allclose(k2, k, atol=1e-13)
    np.testing.assert_allclose(v2, v, atol=1e-13)
    np.testing.assert_allclose(q2, q[:, [1, 4]].transpose(1, 0, 2), atol=1e-13)
