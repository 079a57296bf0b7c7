"""Payload checksum of a packed KV transfer (oracle; test infrastructure).

The paper lists durable storage and recovery of KV state as open work and
recovers a lost or unusable state by recomputation from a valid prefix; it
defines no integrity check.  The device library adds one to pack / unpack
and to its file checkpoints so that a corrupted transfer is refused instead
of being resumed from; this module is its definition, written out plainly:

  the payload is read as little-endian 32-bit words w_0 .. w_{N-1};
  s1 = sum of w_i          (mod 2^64)
  s2 = sum of (i + 1) w_i  (mod 2^64)

so a changed word changes s1, and exchanging two unequal words i < j changes
s2 by (j - i) (w_i - w_j).
"""
from __future__ import annotations

import numpy as np

MASK64 = (1 << 64) - 1


def payload_checksum(data) -> tuple[int, int]:
    """(s1, s2) of a byte payload whose length is a multiple of 4."""
    b = np.ascontiguousarray(np.frombuffer(memoryview(data).cast("B"), dtype=np.uint8))
    if b.size % 4:
        raise ValueError("payload length is not a multiple of 4")
    w = b.view("<u4").astype(np.uint64)
    # numpy uint64 arithmetic wraps modulo 2^64
    i1 = np.arange(1, w.size + 1, dtype=np.uint64)
    s1 = int(np.sum(w, dtype=np.uint64))
    s2 = int(np.sum(i1 * w, dtype=np.uint64))
    return s1 & MASK64, s2 & MASK64
