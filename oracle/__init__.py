"""Oracle for the Seer hot path: plain, slow, fp64 CPU reference.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package;
only the tests, the smoke check and the CPU-baseline leg of the benchmark call
it.  It shares no code with the HIP library: its only inputs are the arrays
built by the seeded generators in ``workloads``.

Modules (each function cites the passage of the paper it follows):
  layer     -- one bidirectional transformer layer over packed sequences
               (denoising step, Sec. 3.1; attention, Sec. 3.6 equations)
  sparsity  -- per-position near-zero MLP activation count (Sec. 3.2-3.3)
  detect    -- SNR jump/plateau boundary criterion (Sec. 3.3)
  route     -- static micro-buckets, padding waste ratio, three-tier routing
               and the compaction layout (Sec. 3.4-3.5)
  pipeline  -- step 0 detection, one-shot truncation, truncated steps
  kvcache   -- truncated steps on the window rows with the prefix's keys and
               values cached (Appendix D, KV-cache compatibility)
  rope      -- rotary position embedding of queries and keys (the paper is
               silent on positions; RoFormer's definition, rotate-half pairs)

Parity status: every function here is pinned by CPU tests against values
fixed by the mathematics (brute force, closed forms, invariants, planted
inputs).  The paper prints no worked numeric example, so no value is pinned
to a printed table.
"""
from .layer import rms_norm, attention_seq, layer_forward, layer_forward_rows, silu
from .sparsity import near_zero_count
from .detect import detect_boundary, detect_batch
from .route import (bucket_set, bucket_of, padding_waste_ratio, coarse_class,
                    route_batch, repack_rows, RouteResult)
from .pipeline import run_pipeline, PipelineResult
from .kvcache import prefix_kv, layer_forward_cached_rows, layer_forward_cached
from .rope import rope_angles, apply_rope
