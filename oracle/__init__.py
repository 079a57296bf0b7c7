"""Float64 CPU oracle of the stateful KV operators (test infrastructure).

This package is the plain, slow, obviously-correct statement of what the
device library computes.  It is test infrastructure: only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The product path never calls it, and it shares no code with the
HIP library (its only common dependency is the ``synth`` input generator).

Modules
  rope       rotary position encoding and re-rotation by a position shift
  attention  causal grouped-query attention (dense, max-subtracted softmax)
  model      the per-layer QKV projection of one shared hidden-state matrix
  pool       the paged block pool: FIFO free ring, refcounts, block tables,
             catalog, and the seven operators (materialize, fork, attend,
             compose, pack, unpack, evict) plus release and pin
  policy     the transfer-vs-recompute decision of the scheduling rule
  checksum   the payload checksum of checked packs and file checkpoints

Operator semantics follow the paper's stateful-operator section (state object
S_KV = (M, Theta, B, Pi, Lambda, Gamma), Compat predicate, operator
signatures) and its KV-operator algorithms appendix (KV-Materialize, KV-Fork,
KV-Transfer, KV-Resume, Restricted-KV-Merge, KV-Evict).  The transformer
arithmetic (projection, RoPE, attention) is not defined by the paper; the
readings used are listed in each module.
"""
from .rope import inv_freq, rope_angles, apply_rope, rerotate  # noqa: F401
from .attention import causal_gqa_attention, attention_rows  # noqa: F401
from .model import project_qkv, project_kv, project_q, split_w  # noqa: F401
from .pool import (OraclePool, OracleError, Status, Lineage,  # noqa: F401
                   PACK_MAGIC, PACK_VERSION)
from .policy import kv_bytes, prefill_flops, plan_transfer  # noqa: F401
from .checksum import payload_checksum  # noqa: F401
