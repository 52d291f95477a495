"""CPU oracle for batch super-tree verification.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, deliberately
unoptimised restatement of what the verification path computes, written from
the paper's definitions.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import it; the GPU library never does, and
the two share no code.

Stages (each module cites the passage it follows):

* ``gate``   -- path scores (eq. 5) and the budgeted global selection under the
               batch-level verification cap (eq. 4; budget-exchange argument of
               Theorem 2 and Proposition 1); ``gate_sparse`` first truncates
               each request at its first failed checkpoint depth (layer
               confidence eq. 6, gating signal eq. 7, Alg. 1 phase 1).
* ``elastic``-- Alg. 1's elastic budget scheduler (phase 1 depth extension
               with checkpoint gating, phase 2 width expansion) as a selection
               policy over the drafted pool.
* ``mask``   -- flatten & pack of the selected super-tree into per-request
               verify slots, position ids and ancestor bitmasks (Fig. 3, stage 3).
* ``attn``   -- tree-masked grouped-query attention of every verify slot over
               its request's KV prefix plus its in-tree ancestors, in float64
               (the single parallel verification forward of Section 3.1).
* ``serve``  -- the serving step around the path: target argmax feeding
               acceptance, KV commit of the accepted path into a paged cache,
               verification attention over that paged cache.
* ``accept`` -- greedy (temperature 0) acceptance of the longest draft path
               matching the target argmax (Section 2, standard SD).

Data-dependent problems never raise: they are OR-ed into an integer status
word (bit values in ``status``) and the offending value is clamped as each
function documents.
"""
from . import status
from .gate import path_scores, select_top_b, gate, gate_sparse
from .elastic import elastic_schedule
from .mask import build_tree_mask
from .attn import tree_verify_attn
from .accept import accept
from .serve import target_argmax, accept_from_logits, tree_verify_attn_paged, commit_kv
