"""CPU oracle for the memory-slice hot path.  TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct restatement of what the hot path computes:

* ``slice_state``: the bookkeeping of one memory slice and the local paged
  cache -- one owner per segment, guarded by a mapping table (EMA section 4,
  "Memory Slice"); allocation that first tries free memory (section 4.1);
  block copies driven by block tables (prefetch before use, section 4.2 and
  section 5.1's slice process); reclaim that preempts logically owned regions
  and releases a victim's whole dependency chain (section 4.1).
* ``attention``: float64 paged decode attention (textbook scaled dot-product
  attention; the paper uses vLLM's attention and gives no formula).
* ``layout``: the byte layout of one layer-block in each pool.
* ``invariants``: the properties the paper fixes (exactly-once ownership,
  static-dynamic symmetry after reclaim) plus conservation and the logical
  view of every block.
* ``slab``: the slab allocator of section 4.2.1 (slabs uniform across layers,
  one user each, freed slabs returned, reclaim of the slab with the fewest
  active requests) with the layer-major, slab-major and layer-group-major
  placements of sections 4.2.1-4.2.3 and the run structure of a layer-group
  swap.
* ``sched``: placement of slice units across GPU pairs by Greedy-Least-Loaded
  (section 5.2, Appendix C) and the cap after bursty preemptions (section 5.3).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package. It shares no code with the HIP library and never
imports it; the product path never imports this package.

Parity status: attention, layouts and block copies are pinned against
independent routines (tests/test_oracle_*.py); the invariant checks by
hand-built states that break each invariant and must be rejected
(tests/test_oracle_invariants.py); scheduling by hand-worked
placements and by the competitive bound of Appendix C checked against
brute-force optima (tests/test_sched.py). The reclaim policy details that
the paper leaves open (which slots the lender takes back, how the victim is
chosen, the order of compaction) are pinned only by hand-worked examples and
the invariants: parity unpinned by the paper for those choices.
"""
from .layout import LAYOUT_ATTN, LAYOUT_NHD, block_bytes, decode_block, encode_block, convert_block, to_float64
from .slice_state import (SliceOracle, OracleError, FREE, STAGING, LENDER, LOCAL, SLICE,
                          ERR_INVAL, ERR_NOMEM, ERR_OWNER)
from .attention import paged_decode_attention, contiguous_decode_attention
from .invariants import (InvariantError, check_ownership, check_conservation, check_sd_symmetry,
                         logical_view)
from .sched import SchedOracle
from .slab import (SlabSliceOracle, LAYER_MAJOR, SLAB_MAJOR, GROUP_MAJOR, BORROWED,
                   check_slab_tags, check_slab_sd_symmetry)

__all__ = [
    "LAYOUT_ATTN", "LAYOUT_NHD", "block_bytes", "decode_block", "encode_block", "convert_block",
    "to_float64", "SliceOracle", "OracleError", "FREE", "STAGING", "LENDER", "LOCAL", "SLICE",
    "ERR_INVAL", "ERR_NOMEM", "ERR_OWNER", "paged_decode_attention",
    "contiguous_decode_attention", "check_ownership", "check_conservation",
    "check_sd_symmetry", "logical_view", "InvariantError", "SchedOracle",
    "SlabSliceOracle", "LAYER_MAJOR", "SLAB_MAJOR", "GROUP_MAJOR", "BORROWED", "check_slab_tags",
    "check_slab_sd_symmetry",
]
