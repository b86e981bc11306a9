"""CPU oracle for the sparsity-aware fused attention forward (test infrastructure).

This package is test infrastructure.  Only the tests, the smoke check and the
CPU-baseline leg of the benchmark may import or run it; the library never
does, and the library's product path has no CPU fallback of any kind.

It is written from the paper's definitions, independently of the GPU code:

* ``attention``   -- the plain definition of attention (Section II-A, Eq. 1)
  with a block mask and the causal structure applied as -inf entries of the
  score matrix, in float64 with every score row materialised in full;
* ``block_index`` -- the tile classification of Section IV-A (a tile is
  skipped, processed as is, or masked locally), written as a compressed
  per-query-block list, plus the heaviest-first work order that stands in for
  the sparsity-aware placement of Section IV-C;
* ``block_select`` -- the mask producer that runs before the pass: top-k key
  blocks per query block by mean-pooled query/key score, plus the diagonal;
* ``lse_merge``   -- the per-row log-sum-exp of the scores and the rule that
  merges partial results computed over disjoint key chunks;
* ``fp8_attention`` -- a float64 model of the library's fp8 (E4M3) form:
  Algorithm 1's online recurrence with both products taking E4M3 operands
  under power-of-two scales (an extension of Section II-C's bf16 datapath).

Every function is pinned by tests against things other than itself: brute
force on tiny inputs, closed forms, invariants and an independent library
routine (see the module docstrings).
"""
from .masked_attention import attention, attention_rows, element_visibility, kv_head  # noqa: F401
from .block_index import N_BINS, build_index, count_bin, tile_classes, work_order  # noqa: F401
from .block_select import block_means, block_scores, keep_count, topk_meanpool_mask  # noqa: F401
from .lse_merge import attention_lse, merge_partials  # noqa: F401
from .fp8_attention import attention_fp8, e4m3_round, pow2_scale  # noqa: F401
