"""Checked transfers and file checkpoints on the device, against the oracle.

The payloads are seeded synthetic block contents: the device copy is
generated on the GPU, and the expected bytes and checksums come from the
same stream generated on the CPU (``synth.normal_np``) and from
``oracle.payload_checksum``, never from the device.  Allocator metadata is
compared with the oracle after every call (``Twin``).
"""
import ctypes
import os

import numpy as np
import pytest
import torch

import synth
from oracle import payload_checksum
from oracle.pool import PACK_CHECKSUM
from paper_2607_10987_amd import kvstate as kv
from twin import Twin, close

pytestmark = pytest.mark.gpu

HDR = ctypes.sizeof(kv.kv_pack_header)


def small(dtype="bf16"):
    return synth.ModelShape("ck", 2, 32, 4, 2, 16, 4, dtype)


def raw_payload(tw, nb, nt, tag):
    """CPU storage values of the synthetic payload, slots past nt zeroed."""
    s = tw.s
    shp = (nb, s.n_layers, 2, s.n_kv_heads, s.block_size, s.head_dim)
    raw = synth.normal_np(synth.payload_key(tw.seed, tw.wl, tag), shp, 1.0, tw.dt).copy()
    last = nt - (nb - 1) * s.block_size
    raw[-1, :, :, :, last:] = 0
    return raw


def checked(hdr, ohdr, raw_bytes):
    """Copies of both headers carrying the CPU checksum of raw_bytes."""
    h = kv.kv_pack_header.from_buffer_copy(bytes(hdr))
    cs = payload_checksum(raw_bytes)
    h.flags, h.checksum[0], h.checksum[1] = PACK_CHECKSUM, cs[0], cs[1]
    return h, dict(ohdr, flags=PACK_CHECKSUM, checksum=cs)


def zero_tail(buf, tw, nb, nt):
    s = tw.s
    v = buf.view(tw.tdt).view(nb, s.n_layers, 2, s.n_kv_heads, s.block_size, s.head_dim)
    v[-1, :, :, :, nt - (nb - 1) * s.block_size:] = 0


def test_checked_pack_matches_cpu_checksum(gpu_available):
    tw = Twin(small(), n_blocks=64, max_pos=256, wl="ck-pack")
    nb, nt = 9, 34                                   # ragged: 2 tokens in the last block
    hdr, ohdr, buf, pay = tw.synthetic_transfer(nb, nt, 5, tag=1)
    u = tw.unpack(hdr, ohdr, buf, pay)
    raw = raw_payload(tw, nb, nt, tag=1)
    for b0, b1 in [(0, nb), (0, 1), (3, 7), (nb - 1, nb)]:
        out = torch.empty((b1 - b0) * tw.s.block_bytes, dtype=torch.uint8, device="cuda")
        h = kv.kv_pack_checked(tw.gpu.h, u, b0, b1, out)
        tw.orc.pack(tw.sid[u], b0, b1)
        want = raw[b0:b1].tobytes()
        assert h.flags == PACK_CHECKSUM
        assert (h.checksum[0], h.checksum[1]) == payload_checksum(want), (b0, b1)
        assert out.cpu().numpy().tobytes() == want, (b0, b1)
        tw.check_meta()
    # the unchecked pack leaves the checksum fields empty
    out = torch.empty(nb * tw.s.block_bytes, dtype=torch.uint8, device="cuda")
    h = kv.kv_pack(tw.gpu.h, u, 0, nb, out)
    tw.orc.pack(tw.sid[u], 0, nb)
    assert h.flags == 0 and tuple(h.checksum) == (0, 0)
    tw.close()


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_checked_unpack_accepts_and_rolls_back(gpu_available, dtype):
    tw = Twin(small(dtype), n_blocks=48, max_pos=256, wl="ck-unpack")
    nb, nt = 6, 23
    hdr, ohdr, buf, pay = tw.synthetic_transfer(nb, nt, 0, tag=2)
    zero_tail(buf, tw, nb, nt)
    raw = raw_payload(tw, nb, nt, tag=2).tobytes()
    hc, ohc = checked(hdr, ohdr, raw)
    u = kv.kv_unpack(tw.gpu.h, hc, buf)
    tw.sid[u] = tw.orc.unpack(ohc, pay, raw=raw)
    tw.check_meta()
    tw.check_state_kv(u)
    # one flipped bit anywhere in the payload is refused; the blocks drawn
    # for it go back to the ring on both sides
    for pos in (0, 1234, len(raw) - 1):
        bad = buf.clone()
        bad[pos] ^= 0x10
        badraw = bytearray(raw)
        badraw[pos] ^= 0x10
        with pytest.raises(kv.KVError) as e:
            kv.kv_unpack(tw.gpu.h, hc, bad)
        assert e.value.status == kv.KV_ERR_CHECKSUM
        with pytest.raises(Exception) as eo:
            tw.orc.unpack(ohc, pay, raw=bytes(badraw))
        assert eo.value.status == kv.KV_ERR_CHECKSUM
        tw.check_meta()
    # unknown flag bits: a bad header, nothing allocated
    hb = kv.kv_pack_header.from_buffer_copy(bytes(hc))
    hb.flags = 2
    with pytest.raises(kv.KVError) as e:
        kv.kv_unpack(tw.gpu.h, hb, buf)
    assert e.value.status == kv.KV_ERR_BAD_HEADER
    tw.check_meta()
    # the accepted state still works
    tw.attend([u], 3)
    tw.close()


def test_checkpoint_round_trip_and_errors(gpu_available, tmp_path):
    tw = Twin(small(), n_blocks=64, max_pos=256, wl="ck-file")
    nb, nt = 7, 26
    hdr, ohdr, buf, pay = tw.synthetic_transfer(nb, nt, 3, tag=3)
    zero_tail(buf, tw, nb, nt)
    u = tw.unpack(hdr, ohdr, buf, pay)
    tw.attend([u], 5)                            # 31 tokens, 8 blocks, device-computed tail
    path = str(tmp_path / "state.kvck")
    kv.kv_checkpoint_save(tw.gpu.h, u, path)
    _, want = tw.orc.pack(tw.sid[u], 0, 8)
    tw.check_meta()
    data = open(path, "rb").read()
    fh = kv.kv_pack_header.from_buffer_copy(data[:HDR])
    assert fh.magic == kv.KV_PACK_MAGIC and fh.version == kv.KV_PACK_VERSION
    assert (fh.pos_begin, fh.n_tokens, fh.blk_begin, fh.n_blocks) == (3, 31, 0, 8)
    assert fh.src_state_id == tw.sid[u] and fh.flags == PACK_CHECKSUM
    assert len(data) == HDR + fh.payload_bytes
    payload = data[HDR:]
    # the blocks the transfer brought in are the CPU stream, byte for byte
    head = raw_payload(tw, nb, nt, tag=3)[: nb - 1].tobytes()
    assert payload[: len(head)] == head
    assert (fh.checksum[0], fh.checksum[1]) == payload_checksum(payload)
    # the oracle's K/V of the state agree with the file's (bf16 tolerance)
    got = np.frombuffer(payload, dtype=np.uint16).reshape(
        8, tw.s.n_layers, 2, tw.s.n_kv_heads, tw.s.block_size, tw.s.head_dim)
    close(synth.to_f64(got, "bf16"), want, "bf16", "checkpoint payload")

    v = kv.kv_checkpoint_load(tw.gpu.h, path)
    ohdr_f = dict(magic=fh.magic, version=fh.version, model_id=tw.orc.shape.model_id,
                  compat=tw.orc.shape.compat_key(), pos_begin=3, n_tokens=31, blk_begin=0,
                  n_blocks=8, block_bytes=fh.block_bytes, payload_bytes=fh.payload_bytes,
                  lineage=fh.lineage, src_state_id=fh.src_state_id, flags=fh.flags,
                  checksum=(fh.checksum[0], fh.checksum[1]))
    tw.sid[v] = tw.orc.unpack(ohdr_f, want, raw=payload)
    tw.check_meta()
    out = torch.empty(fh.payload_bytes, dtype=torch.uint8, device="cuda")
    kv.kv_pack(tw.gpu.h, v, 0, 8, out)
    tw.orc.pack(tw.sid[v], 0, 8)
    assert out.cpu().numpy().tobytes() == payload

    # corrupted payload: refused after the whole file is read, rolled back
    bad = bytearray(data)
    bad[HDR + 777] ^= 0x01
    bpath = str(tmp_path / "bad.kvck")
    open(bpath, "wb").write(bytes(bad))
    with pytest.raises(kv.KVError) as e:
        kv.kv_checkpoint_load(tw.gpu.h, bpath)
    assert e.value.status == kv.KV_ERR_CHECKSUM
    with pytest.raises(Exception):
        tw.orc.unpack(ohdr_f, want, raw=bytes(bad[HDR:]))
    tw.check_meta()
    # short file, missing file, damaged header: nothing allocated
    spath = str(tmp_path / "short.kvck")
    open(spath, "wb").write(data[:-16])
    for p, status in [(spath, kv.KV_ERR_IO), (str(tmp_path / "none.kvck"), kv.KV_ERR_IO)]:
        with pytest.raises(kv.KVError) as e:
            kv.kv_checkpoint_load(tw.gpu.h, p)
        assert e.value.status == status
    hpath = str(tmp_path / "hdr.kvck")
    hb = bytearray(data)
    hb[4] ^= 0xFF                                 # version
    open(hpath, "wb").write(bytes(hb))
    with pytest.raises(kv.KVError) as e:
        kv.kv_checkpoint_load(tw.gpu.h, hpath)
    assert e.value.status == kv.KV_ERR_BAD_HEADER
    with pytest.raises(kv.KVError) as e:
        kv.kv_checkpoint_save(tw.gpu.h, u, str(tmp_path / "no_dir" / "x.kvck"))
    assert e.value.status == kv.KV_ERR_IO
    tw.check_meta()
    tw.attend([v, u], 2)
    tw.close()


def test_checkpoint_in_several_chunks(gpu_available, tmp_path):
    """A state larger than the 64 MiB staging buffer: 135 blocks of 512 KiB
    (128 per chunk), ragged last block."""
    shape = synth.ModelShape("ck-big", 8, 64, 16, 8, 128, 16, "bf16")
    assert shape.block_bytes == 512 * 1024
    tw = Twin(shape, n_blocks=300, max_pos=4096, wl="ck-big", check_kv=False)
    tw.orc.store_kv, tw.orc.kv = False, None      # metadata only on the oracle side
    nb, nt = 135, 134 * 16 + 5
    hdr, ohdr, buf, pay = tw.synthetic_transfer(nb, nt, 0, tag=4)
    zero_tail(buf, tw, nb, nt)
    u = kv.kv_unpack(tw.gpu.h, hdr, buf)
    tw.sid[u] = tw.orc.unpack(ohdr, None)
    raw = raw_payload(tw, nb, nt, tag=4).tobytes()
    path = str(tmp_path / "big.kvck")
    kv.kv_checkpoint_save(tw.gpu.h, u, path)
    tw.orc.pack(tw.sid[u], 0, nb)
    with open(path, "rb") as f:
        fh = kv.kv_pack_header.from_buffer_copy(f.read(HDR))
        assert f.read() == raw
    assert (fh.checksum[0], fh.checksum[1]) == payload_checksum(raw)
    v = kv.kv_checkpoint_load(tw.gpu.h, path)
    ohdr_f = dict(ohdr, pos_begin=0, src_state_id=tw.sid[u], lineage=fh.lineage,
                  flags=fh.flags, checksum=(fh.checksum[0], fh.checksum[1]))
    tw.sid[v] = tw.orc.unpack(ohdr_f, None, raw=raw)
    tw.check_meta()
    out = torch.empty(nb * shape.block_bytes, dtype=torch.uint8, device="cuda")
    h = kv.kv_pack_checked(tw.gpu.h, v, 0, nb, out)
    tw.orc.pack(tw.sid[v], 0, nb)
    assert (h.checksum[0], h.checksum[1]) == (fh.checksum[0], fh.checksum[1])
    assert torch.equal(out, buf)
    os.remove(path)
    tw.close()
