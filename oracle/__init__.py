"""Plain float64 CPU oracle for the ParallelVLM verify + UV-Prune + accept path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(``paper_2603_19610_amd``) never imports, calls or links it, and the oracle
imports nothing from the product path: the two share only the seeded input
generators in ``workloads``.

Each function is the operation's plain definition written out in float64 with
explicit loops over the indices the paper sums over, following the paper:

* ``verify_attn``      -- target verification forward over the cache (Sec. 2.2,
                          Sec. 4.2 Parallel Decoding) with the per-token
                          attention mass used by attention-guided pruning
                          (Sec. 3, Challenge 2).
* ``cos_similarity``   -- Eq. (similarity).
* ``criterion_cossim`` -- sum over text tokens of Eq. (similarity) for one layer.
* ``prefill_epilogue`` -- a prefill layer's residual add with that criterion
                          computed from the stored result (Sec. 4.1, 4.2).
* ``uvprune_score_*``  -- Eq. (average_similarity): layer-to-layer variation
                          summed over text tokens and layers 1..L.
* ``topk_select``      -- Eq. (topk_selection), keep ratio 1 - alpha (Sec. 4.2).
* ``gather_kv``        -- the draft's compact cache [V*, X] (Sec. 4.2, Stage I).
* ``spec_accept``      -- speculative-sampling accept/reject with residual
                          resampling (Sec. 2.2) and the bonus token (Suppl. B).
* ``window``           -- draft window size, Eq. (Prefill), and the speedup
                          model of Thm. (paravlm_speedup) and the supplement's
                          theorems and Lemma 1.
* ``rope``             -- rotary position embedding (1-D or M-RoPE) of the
                          verify rows and their append to the KV cache.
* ``pipeline``         -- the parallel decoding pipeline's scheduling: pre- and
                          post-verify modes and draft rollback (Suppl.
                          "Parallel Pipeline Details").
* ``paged``            -- verify attention, rope append and the compact-cache
                          gather over a paged cache, every row read or
                          written through the page table.

Parity status: every function here is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle_*.py`` against brute force, closed forms, library routines
or hand-computed fixtures; none is "parity unpinned".
"""
from .attention import verify_attn, verify_attn_rows
from .uvprune import (cos_similarity, criterion_cossim, prefill_epilogue, uvprune_score_cossim,
                      uvprune_score_mass)
from .select import topk_keys, topk_select, gather_kv
from .accept import spec_accept, softmax_t, NEAR_TIE_REL
from . import paged, pipeline, rope, window

__all__ = [
    "verify_attn", "verify_attn_rows", "cos_similarity", "criterion_cossim", "prefill_epilogue",
    "uvprune_score_cossim", "uvprune_score_mass", "topk_keys", "topk_select",
    "gather_kv", "spec_accept", "softmax_t", "NEAR_TIE_REL",
]
