"""Synthetic workloads of the memory-slice hot path, driven through the
library: the seeded KV caches of the benchmark configurations
(``synthetic.Workload``), the bursty elastic trace (``bursty``), the
large-block copy stress (``stress``) and the slab step sweep (``slabs``).
Used by the GPU tests and the bench; values and placements come from
``synth``'s seeded generators."""
