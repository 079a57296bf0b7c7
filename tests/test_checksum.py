"""The payload checksum (oracle) against closed forms, and the oracle's
checked unpack; CPU only."""
import numpy as np
import pytest

from oracle import OracleError, OraclePool, Status, payload_checksum
from oracle.pool import PACK_CHECKSUM, PoolShape

M64 = 1 << 64


def words(arr):
    return np.asarray(arr, dtype="<u4").tobytes()


def test_all_ones():
    for n in (1, 2, 7, 1000):
        assert payload_checksum(words([1] * n)) == (n, n * (n + 1) // 2)


def test_single_word_position_weight():
    for n, k, w in [(4, 0, 5), (4, 3, 0xFFFFFFFF), (100, 37, 123456789)]:
        a = [0] * n
        a[k] = w
        assert payload_checksum(words(a)) == (w, (k + 1) * w)


def test_little_endian_words():
    assert payload_checksum(b"\x01\x00\x00\x00\x00\x01\x00\x00") == (1 + 256, 1 + 2 * 256)
    assert payload_checksum(b"\x00\x00\x00\x80") == (1 << 31, 1 << 31)


def test_wraps_modulo_2_64():
    n = 1 << 17                                   # (2^32 - 1) n (n + 1) / 2 > 2^64
    m = 0xFFFFFFFF
    s1, s2 = payload_checksum(words(np.full(n, m, dtype=np.uint64)))
    assert s1 == (m * n) % M64
    assert s2 == (m * n * (n + 1) // 2) % M64
    assert m * n * (n + 1) // 2 >= M64


def test_exchange_changes_s2_by_the_closed_form():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 1 << 32, 64, dtype=np.uint64)
    i, j = 3, 41
    b = a.copy()
    b[i], b[j] = a[j], a[i]
    s1a, s2a = payload_checksum(words(a))
    s1b, s2b = payload_checksum(words(b))
    assert s1a == s1b
    assert (s2b - s2a) % M64 == ((j - i) * (int(a[i]) - int(a[j]))) % M64


def test_linear_in_words_without_overflow():
    rng = np.random.default_rng(6)
    a = rng.integers(0, 1 << 31, 50, dtype=np.uint64)
    b = rng.integers(0, 1 << 31, 50, dtype=np.uint64)
    ca, cb, cab = (payload_checksum(words(x)) for x in (a, b, a + b))
    assert cab == ((ca[0] + cb[0]) % M64, (ca[1] + cb[1]) % M64)


def test_rejects_ragged_length():
    with pytest.raises(ValueError):
        payload_checksum(b"\x00" * 6)


def _pool():
    shape = PoolShape(n_layers=1, d_model=4, n_q_heads=2, n_kv_heads=1, head_dim=4,
                      block_size=2, max_pos=64, max_states=8)
    return OraclePool(shape, 8, store_kv=False), shape


def _hdr(shape, nb, nt, raw):
    return dict(magic=0x5453564B, version=2, model_id=shape.model_id,
                compat=shape.compat_key(), pos_begin=0, n_tokens=nt, blk_begin=0,
                n_blocks=nb, block_bytes=shape.block_bytes,
                payload_bytes=nb * shape.block_bytes, lineage=0, src_state_id=9,
                flags=PACK_CHECKSUM, checksum=payload_checksum(raw))


def test_checked_unpack_accepts_and_rolls_back():
    p, shape = _pool()
    raw = bytes(range(256))[: 2 * shape.block_bytes]           # 2 blocks of 64 bytes
    h = _hdr(shape, 2, 3, raw)
    s0 = p.unpack(h, raw=raw)
    assert p.table(s0) == [0, 1]
    bad = bytearray(raw)
    bad[70] ^= 0x10
    with pytest.raises(OracleError) as e:
        p.unpack(h, raw=bytes(bad))
    assert e.value.status == Status.CHECKSUM
    # blocks 2, 3 were drawn and went back to the ring tail; id 1 is used up
    rc, ring, head, tail = p.allocator()
    assert (head, tail) == (4, 10) and list(ring[:2]) == [2, 3]
    assert list(rc[:4]) == [1, 1, 0, 0]
    s2 = p.unpack(h, raw=raw)
    assert s2 == 2 and p.table(s2) == [4, 5]
    # a checked header needs the bytes; unknown flags are a bad header
    with pytest.raises(OracleError) as e:
        p.unpack(h)
    assert e.value.status == Status.ARG
    with pytest.raises(OracleError) as e:
        p.unpack(dict(h, flags=2), raw=raw)
    assert e.value.status == Status.BAD_HEADER
