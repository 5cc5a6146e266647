"""CPU oracle for the EMU Split/Merge reshard and its transfer buckets.

TEST INFRASTRUCTURE ONLY. This package is the plain, slow, obviously correct definition that the GPU
path is checked against. Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it. The GPU library never calls it, and it shares no code with the GPU library.

What it computes (paper section 5 and section 6.2):

* An EMU is one model-stage replica ``<M, T_tp x pp, R, theta, omega>``; its parameter shards
  ``theta = {theta_i}, i = 1..tp*pp`` and its optimizer shards ``omega`` share one layout, and neither is
  sharded across data-parallel replicas (section 5, EMU definition).
* Split and Merge change the TP/PP layout of that state without changing the logical model state
  (section 5.2 primitives (a) and (b); section 6.2, preserving training semantics). The plain definition
  of that change is: rebuild the full logical tensors from the source shards, then cut them again for
  the destination layout: ``dst = shard(unshard(src, L_src), L_dst)``.
* Each shard travels as one contiguous buffer (section 6.2, transport): a destination rank's shards are
  concatenated in canonical order into a byte stream, and the stream is cut into buckets of ``B`` bytes.

The paper fixes neither the per-tensor sharding rules nor the fused-weight formats. The readings taken
here (column/row/vocab-parallel Megatron-style sharding, head-interleaved fused QKV per KV group, block
fused gate/up, norms replicated on every TP rank and read from TP rank 0, KV heads replicated when tp
exceeds their count, contiguous PP layer ranges with the first L mod pp stages holding one more layer,
rank = p * tp + t, vocab padding to a multiple of tp * m) are stated where they are used.

Modules:
  model    -- model shapes, layout validity, padded vocabulary, per-rank tensor inventory
  sharding -- logical tensors, shard, unshard, reshard (whole model or one tensor group at a time)
  buckets  -- per-rank byte streams, bucket pack and unpack
  coords   -- per-element coordinate formulas (pure Python) used by the brute-force pins
  convert  -- fp32 <-> bf16 conversion for the weight-synchronising reshard (round to nearest even)
"""

from .model import (  # noqa: F401
    Model, Layout, LayoutError, check_layout, padded_vocab, stage_layers, stage_of_layer, kv_local,
    rank_of, rank_inventory, TensorSpec, groups, DTYPE_BYTES,
)
from .sharding import (  # noqa: F401
    logical_tensors, shard, unshard, reshard, shard_group, unshard_group, reshard_group,
)
from .buckets import stream_bytes, bucket_count, pack, unpack  # noqa: F401
from .convert import convert, f32_to_bf16, bf16_to_f32  # noqa: F401
