"""Pins of the row-wise attention checker used by the full-size GPU tests.

At the benchmark's full sizes the GPU tests cannot run the oracle pool, so
they evaluate attention row by row: ``oracle.attention_rows`` for selected
(query row, KV head) pairs and ``tests/fullsize.ref_rows``, which projects
and rotates the query rows and maps query head h to KV head h // G.  Both are
pinned here against the dense ``causal_gqa_attention`` (itself pinned against
torch's SDPA and explicit loops) and against the oracle pool's materialize and
attend outputs, at G = 4 and G = 8, with position offsets, rows on both sides
of each visibility boundary and a row that sees a single key.
"""
import numpy as np
import pytest

import synth
from fullsize import ref_kv, ref_rows
from oracle import OraclePool, apply_rope, attention_rows, causal_gqa_attention
from oracle.pool import PoolShape


@pytest.mark.parametrize("hq,hkv", [(8, 2), (16, 2), (8, 1)])
def test_attention_rows_equals_dense_causal_gqa(hq, hkv):
    rng = np.random.default_rng(11)
    dh, tk, p0 = 16, 23, 1000
    g = hq // hkv
    k = rng.standard_normal((hkv, tk, dh))
    v = rng.standard_normal((hkv, tk, dh))
    k_pos = p0 + np.arange(tk)
    # queries at every key position (the first sees one key) and one past the end
    q_pos = np.concatenate([k_pos, [p0 + tk]])
    q = rng.standard_normal((hq, q_pos.size, dh))
    dense = causal_gqa_attention(q, k, v, q_pos, k_pos)
    for t in range(q_pos.size):
        heads = np.arange(hq) // g
        got = attention_rows(q[:, t], k, v, np.full(hq, q_pos[t]), k_pos, heads)
        np.testing.assert_allclose(got, dense[:, t], rtol=0, atol=1e-12)
    # the row at the first key position is that key's value, whatever q is
    one = attention_rows(q[:, 0], k, v, np.full(hq, p0), k_pos, np.arange(hq) // g)
    np.testing.assert_allclose(one, v[np.arange(hq) // g, 0], rtol=0, atol=1e-12)


def test_attention_rows_visibility_boundary():
    """A row at position p sees exactly the keys at positions <= p: its output
    changes when the key at p changes and not when the key at p + 1 does."""
    rng = np.random.default_rng(5)
    hkv, tk, dh, p0 = 1, 9, 8, 40
    k = rng.standard_normal((hkv, tk, dh))
    v = rng.standard_normal((hkv, tk, dh))
    k_pos = p0 + np.arange(tk)
    q = rng.standard_normal((1, dh))
    for t in range(tk - 1):
        base = attention_rows(q, k, v, [p0 + t], k_pos, [0])
        v2 = v.copy()
        v2[0, t] += 1.0                      # the key at the row's own position
        assert np.abs(attention_rows(q, k, v2, [p0 + t], k_pos, [0]) - base).max() > 1e-3
        v3 = v.copy()
        v3[0, t + 1] += 1.0                  # the first key after it
        np.testing.assert_array_equal(attention_rows(q, k, v3, [p0 + t], k_pos, [0]), base)
        # brute force over the t + 1 visible keys
        s = (k[0, :t + 1] @ q[0]) / np.sqrt(dh)
        w = np.exp(s - s.max())
        np.testing.assert_allclose(base[0], (w / w.sum()) @ v[0, :t + 1], rtol=0, atol=1e-12)


class _Rows:
    """The two attributes ``ref_kv`` / ``ref_rows`` read from a device twin."""

    def __init__(self, shape, weights):
        self.s = shape
        self._w = weights

    def w64(self, layer):
        return self._w[layer]


def _pool(hq, hkv, rope_base=10000.0):
    s = synth.ModelShape("rows", 2, 64, hq, hkv, 16, 4, "f32", rope_base)
    w = [synth.to_f64(synth.normal_np(synth.w_key(3, "rows", l), (s.qkv_cols, s.d_model),
                                      s.w_std, "f32"), "f32") for l in range(s.n_layers)]
    pshape = PoolShape(s.n_layers, s.d_model, hq, hkv, s.head_dim, s.block_size, "f32",
                       s.rope_base, 4096, 8, 1)
    return s, w, OraclePool(pshape, 64, weights=w)


def _x(shape, rows, tag):
    key = synth.x_key(3, "rows", tag)
    return synth.to_f64(synth.normal_np(key, (rows, shape.d_model), 1.0, "f32"), "f32")


@pytest.mark.parametrize("hq,hkv", [(8, 2), (8, 1)])
def test_ref_rows_equals_oracle_materialize_and_attend(hq, hkv):
    """ref_rows over ref_kv keys reproduces the pool's outputs row by row:
    a materialize at an offset position, then a 5-token append and a decode
    step of a forked child (all of the child's keys, query rows at the end)."""
    s, w, orc = _pool(hq, hkv)
    mt = _Rows(s, w)
    pos0, T = 1234, 21
    x0 = _x(s, T, 0)
    root, o0 = orc.materialize(x0, pos0=pos0)
    kid = orc.fork(root, 1)[0]
    x1 = _x(s, 5, 1)
    o1 = orc.attend([kid], x1[None])
    x2 = _x(s, 1, 2)
    o2 = orc.attend([kid], x2[None])
    xs = np.concatenate([x0, x1, x2])
    pos = pos0 + np.arange(xs.shape[0])
    for layer in range(s.n_layers):
        k, v = ref_kv(mt, layer, xs, pos)
        # materialize rows: row t sees keys 0..t (the first row one key)
        rows = np.array([0, 1, 2, 7, T - 2, T - 1])
        got = ref_rows(mt, layer, x0[rows], pos[rows], k, v, pos, rows + 1)
        np.testing.assert_allclose(got, o0[layer][rows], rtol=0, atol=1e-11)
        # append rows over the forked prefix
        r1 = np.arange(5)
        got = ref_rows(mt, layer, x1, pos[T + r1], k, v, pos, T + r1 + 1)
        np.testing.assert_allclose(got, o1[layer, 0], rtol=0, atol=1e-11)
        got = ref_rows(mt, layer, x2, pos[T + 5:], k, v, pos, [T + 6])
        np.testing.assert_allclose(got, o2[layer, 0], rtol=0, atol=1e-11)


def test_ref_rows_head_grouping_matters():
    """With G = 4 the rows of query heads 0..3 use KV head 0 and 4..7 KV head
    1: mapping head h to KV head h % Hkv instead changes the output."""
    s, w, orc = _pool(8, 2)
    mt = _Rows(s, w)
    x = _x(s, 6, 9)
    pos = np.arange(6)
    sid, o = orc.materialize(x)
    k, v = ref_kv(mt, 0, x, pos)
    got = ref_rows(mt, 0, x, pos, k, v, pos, np.arange(6) + 1)
    np.testing.assert_allclose(got, o[0], rtol=0, atol=1e-11)
    q = apply_rope(np.asarray(x @ w[0][:8 * 16].T).reshape(6, 8, 16).transpose(1, 0, 2),
                   pos, s.rope_base)
    wrong = np.stack([attention_rows(q[:, t], k, v, np.full(8, t), pos, np.arange(8) % 2)
                      for t in range(6)])
    assert np.abs(wrong.reshape(6, -1) - o[0]).max() > 1e-3
