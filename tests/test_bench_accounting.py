"""The algorithmic work that bench.py divides by measured time, pinned to
closed forms evaluated independently here (no GPU).

Projection: 2 T d (Hq + 2 Hkv) dh flops per layer.  Causal attention of T new
queries over n cached keys: 4 Hq dh flops per (query, key) pair with key
position <= query position, i.e. T n + T (T + 1) / 2 pairs per head and layer
(attention section of the KV-Materialize / KV-Resume algorithms).  KV bytes:
K and V rows of Hkv heads x dh channels per layer.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402

S8 = synth.LLAMA8B_SHAPE
S70 = synth.LLAMA70B_SHAPE


def test_shapes_are_the_llama_attention_stacks():
    assert (S8.n_layers, S8.d_model, S8.n_q_heads, S8.n_kv_heads, S8.head_dim) == (32, 4096, 32, 8, 128)
    assert (S70.n_layers, S70.d_model, S70.n_q_heads, S70.n_kv_heads, S70.head_dim) == (80, 8192, 64, 8, 128)
    assert S8.qkv_cols == 6144 and S70.qkv_cols == 10240


@pytest.mark.parametrize("shape,tokens,expect", [
    (S8, 8192, 1.32e13),      # [8192, 4096] x [4096, 6144], 32 layers
    (S8, 32768, 5.28e13),
    (S70, 16384, 2.20e14),    # [16384, 8192] x [8192, 10240], 80 layers
])
def test_projection_flops(shape, tokens, expect):
    got = bench.proj_flops(shape, tokens)
    assert got == 2 * tokens * shape.d_model * shape.qkv_cols * shape.n_layers
    assert abs(got - expect) / expect < 0.01


@pytest.mark.parametrize("shape,n_before,T,expect", [
    (S8, 0, 8192, 1.76e13),       # materialize of the 8192-token context
    (S8, 0, 32768, 2.82e14),
    (S8, 32768, 2048, 3.63e13),   # 2048-token append over a 32768-token cache
    (S8, 8192, 512, 9.07e12 / 4),  # one agent's 512-token append
    (S70, 0, 16384, 3.52e14),
])
def test_causal_attention_flops(shape, n_before, T, expect):
    got = bench.attn_flops(shape, n_before, T)
    # brute-force pair count on a reduced case with the same formula shape
    pairs = sum(n_before + t + 1 for t in range(T))
    assert got == 4.0 * shape.n_q_heads * shape.head_dim * pairs * shape.n_layers
    assert abs(got - expect) / expect < 0.01


def test_attention_pairs_brute_force_tiny():
    tiny = synth.TINY_SHAPE
    for n_before, T in [(0, 1), (0, 5), (3, 4), (16, 1)]:
        pairs = sum(1 for t in range(T) for k in range(n_before + T) if k <= n_before + t)
        assert bench.attn_flops(tiny, n_before, T) == \
            4.0 * tiny.n_q_heads * tiny.head_dim * pairs * tiny.n_layers


def test_kv_bytes_per_token_and_blocks():
    assert bench.kv_bytes_per_token(S8) == 128 * 1024
    assert bench.kv_bytes_per_token(S70) == 320 * 1024
    assert S8.block_bytes == 16 * 128 * 1024        # 2 MiB blocks of 16 tokens
    assert S70.block_bytes == 32 * 320 * 1024       # 10 MiB blocks of 32 tokens


def test_decode_step_unique_kv_bytes():
    # four agents over an 8192-token context with 512-token suffixes: the
    # shared context counts once per step, each agent's own keys once
    kvb = bench.kv_bytes_per_token(S8)
    first = kvb * (8192 + 4 * (512 + 1))
    assert abs(first - 1.34e9) / 1.34e9 < 0.01
    last = kvb * (8192 + 4 * (512 + 128))
    assert abs(last - 1.41e9) / 1.41e9 < 0.01
    # the weights every decode step streams: L (Hq + 2 Hkv) dh d bf16 values
    assert S8.n_layers * S8.qkv_cols * S8.d_model * 2 == 1610612736
