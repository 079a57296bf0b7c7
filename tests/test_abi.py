"""The C-ABI library loads and exports every function the header declares.

CPU only: no compute call is made (there is no GPU here).
"""
import ctypes
import os

from paper_2607_10987_amd import kvstate as kv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_header_symbols():
    lib = kv.lib()
    names = kv.header_functions()
    assert len(names) >= 20
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_covers_header():
    for n in kv.header_functions():
        assert callable(getattr(kv, n)), n


def test_struct_layouts_match_header():
    # kv_model_cfg: 10 int32 + double + uint64
    assert ctypes.sizeof(kv.kv_model_cfg) == 56
    assert ctypes.sizeof(kv.kv_segment) == 24
    # ... + flags, reserved (2 uint32) + checksum (2 uint64)
    assert ctypes.sizeof(kv.kv_pack_header) == 8 + 8 + 56 + 4 * 8 + 3 * 8 + 8 + 8 + 16


def test_host_only_calls():
    c = kv.make_cfg(32, 4096, 32, 8, 128, 16, "bf16", 35072, 64)
    pool_b, meta_b = kv.kv_pool_bytes(c, 4096)
    assert pool_b == 4096 * 32 * 2 * 8 * 16 * 128 * 2
    assert meta_b > 4096 * 8
    assert kv.kv_scratch_bytes(c, 8192, 1, 8192) >= 32 * 8192 * 4096 * 2
    assert kv.kv_strerror(kv.KV_ERR_OOM) == "KV_ERR_OOM"
    bad = kv.make_cfg(32, 4096, 30, 8, 128, 16, "bf16", 1024, 4)   # Hq not a multiple of Hkv
    try:
        kv.kv_pool_bytes(bad, 16)
        raise AssertionError("accepted a bad configuration")
    except kv.KVError as e:
        assert e.status == kv.KV_ERR_ARG


def test_library_path_in_tree():
    assert os.path.dirname(kv.LIB_PATH).endswith("paper_2607_10987_amd")


def test_bench_refuses_several_gpus():
    """bench.py measures one GPU; asking for more exits with a message."""
    import json
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]


def test_scratch_bound_covers_decode_partials():
    """kv_scratch_bytes bounds the decode split-key partials for every batch
    up to the one asked for: fp32 (m, l, pad, pad, o[dh]) per (layer, member,
    query head, chunk), chunks of 1024 keys, or of 512 for a batch of one."""
    c = kv.make_cfg(32, 4096, 32, 8, 128, 16, "bf16", 35072, 64)
    q_bytes = 32 * 1 * 32 * 128 * 2                # one token row of Q per layer
    for batch in (1, 2, 4, 16):
        for keys in (1, 511, 513, 8704, 34816):
            need = 0
            for b in range(1, batch + 1):
                ck = 512 if b == 1 else 1024
                chunks = -(-keys // ck)
                need = max(need, 32 * b * 32 * chunks * (4 + 128) * 4)
            got = kv.kv_scratch_bytes(c, 1, batch, keys)
            assert got >= need + q_bytes, (batch, keys, got, need)


class _FakeCuda:
    """Stands in for a CUDA tensor in the binding's argument checks (CPU)."""

    def __init__(self, numel, dtype, contiguous=True):
        self.is_cuda = True
        self.dtype = dtype
        self._n = numel
        self._c = contiguous

    def numel(self):
        return self._n

    def is_contiguous(self):
        return self._c

    def data_ptr(self):
        raise AssertionError("the library was called with a bad tensor")


def test_binding_rejects_bad_tensors_before_calling():
    """x, o and w handed to kv_materialize / kv_attend / kv_set_weights must
    be contiguous CUDA tensors of the pool's dtype, large enough for the
    call; anything else raises KVError before the library is called."""
    import pytest
    import torch
    c = kv.make_cfg(2, 64, 4, 2, 16, 4, "bf16", 128, 4)
    handle = 0x5EED
    kv._CFGS[handle] = c
    bf = torch.bfloat16
    try:
        T, cols = 5, (4 + 2 * 2) * 16
        for batch in (1, 3):
            nx, no = batch * T * 64, 2 * batch * T * 4 * 16   # x [b][T][d], o [L][b][T][Hq dh]
            cases = [
                (torch.zeros(nx, dtype=bf), _FakeCuda(no, bf), kv.KV_ERR_ARG),       # CPU x
                (_FakeCuda(nx, torch.float32), _FakeCuda(no, bf), kv.KV_ERR_ARG),   # dtype
                (_FakeCuda(nx, bf, False), _FakeCuda(no, bf), kv.KV_ERR_ARG),       # strided
                (_FakeCuda(nx - 1, bf), _FakeCuda(no, bf), kv.KV_ERR_BUFSIZE),
                (_FakeCuda(nx, bf), _FakeCuda(no - 1, bf), kv.KV_ERR_BUFSIZE),
                (_FakeCuda(nx, bf), torch.zeros(no, dtype=bf), kv.KV_ERR_ARG),      # CPU o
            ]
            for x, o, code in cases:
                with pytest.raises(kv.KVError) as e:
                    if batch == 1:
                        kv.kv_materialize(handle, x, T, 0, o)
                    else:
                        kv.kv_attend(handle, [1, 2, 3], x, T, o)
                assert e.value.status == code, (batch, code)
        stride = 11 * cols * 64
        with pytest.raises(kv.KVError) as e:
            kv.kv_set_weights(handle, _FakeCuda(stride + cols * 64 - 1, bf), stride)
        assert e.value.status == kv.KV_ERR_BUFSIZE
    finally:
        kv._CFGS.pop(handle, None)
