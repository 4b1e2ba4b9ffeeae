"""CPU oracle for the Sirius hot path (arXiv 2409.03856). TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 NumPy statement of what the GPU library computes:

  * ffn      -- dense SwiGLU FFN, CATS-style threshold sparsity and the
                paper's per-token top-k variant (FSparse),
                Griffin-style prompt-chosen top-k neurons (CSparse) with
                condensed weights, threshold calibration, RMSNorm layer stack;
  * verify   -- the full model's likelihood check of drafted tokens:
                per-row softmax probability of the drafted token, first
                rejection below threshold r, corrected (argmax) token;
  * tree     -- the pruned tree drafting step (fixed treewidth, cumulative
                log-likelihood ranking) and the verification of a drafted tree
                (longest advance over its complete paths), Sec. 4;
  * kv       -- attention over the KV cache shared by the sparse and the full
                model, with the full model's direct rewrite of the drafted chunk's
                rows and the rollback after the check (Algorithm 1);
  * loop     -- the generation loop of Algorithm 1 on a small random-weight
                decoder: drafting by the sparse model, the full model's
                check with the direct cache rewrite, rollback and
                interleaving of the corrected token;
  * apu      -- the efficiency bookkeeping of Sec. 2.2 and Sec. 2.3
                (APU, effective density, speculative-decoding AAL).

Only the test suite, the package's smoke check and the benchmark's
CPU-baseline leg may import this package. The GPU library never calls it,
and it shares no code with the GPU library: it reads the same stored input
values (bf16 weights widened exactly, fp32 activations widened) and states
each definition directly.

Parity status: every function here is pinned by tests that do not go
through the oracle itself (hand-computed cases, closed forms printed in the
paper, brute-force loops on tiny inputs, invariants). None is "parity
unpinned".
"""

from .ffn import (  # noqa: F401
    widen_bf16,
    silu,
    ffn_dense,
    gate_activations,
    cats_active_sets,
    topk_active_sets,
    ffn_topk,
    ffn_masked,
    ffn_cats,
    calibrate_threshold,
    griffin_scores,
    griffin_topk,
    condense,
    ffn_condensed,
    rmsnorm,
    stack_layer,
)
from .verify import softmax_row_stats, verify_accept  # noqa: F401
from .tree import log_softmax, tree_build_step, tree_paths, tree_verify  # noqa: F401
from .apu import sd_aal, apu, effective_density  # noqa: F401
from .kv import attn_kv, kv_rollback  # noqa: F401
from . import loop  # noqa: F401
