"""fp64 CPU oracle for the sparse-prefill evidence probe -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package. The product path (the HIP library and its binding) never
calls it, and it imports nothing from the product: it shares only the seeded
input generator in ``workloads``.

What it computes (each function cites the passage it follows):

* ``layout``    -- the prefill context X = [X_sys; X_vis; X_Q], region-relative
                   blocks, and the token-level visibility predicate (appendix,
                   "Detailed Sparse Prefilling": context layout, frame-aligned
                   partition, always-visible system prefix, causal prefix of the
                   current block).
* ``attention`` -- masked-softmax attention over the allowed keys, the per-row
                   log-sum-exp, and the query-row softmax mass reduced onto
                   anchor frames (Evidence Decomposition: the query-frame cue
                   A_qf from the complete query-token group).
* ``aggregate`` -- head/query mean per layer (Evidence Decomposition: average
                   over heads, layer kept), the layer mean and the per-video
                   top-k frames.
* ``blocks``    -- the block-level active set implied by the token predicate.
* ``brute``     -- pure-Python loops over tiny inputs (an independent pin).
* ``topp``      -- the paper's adaptive top-p block retention (mean-key block
                   representative, block affinity over the history H_i,
                   softmax, smallest subset reaching tau_p) and the attention
                   and evidence it induces (appendix, "Detailed Sparse
                   Prefilling").
* ``cues``      -- the cross-frame cue A_ff and its timestamp-aligned E_ff,
                   and the intra-frame cue A_if (Evidence Decomposition).
* ``coarse``    -- the paper's coarse map (block affinity on retained blocks,
                   exact logits on E_i; appendix, coarse-map equation) and the
                   sparse-vs-dense alignment metrics.

Parity pins live in ``tests/`` (brute force, closed forms, a library attention
routine, invariants, planted ranking). No function here is "parity unpinned".
"""
from . import layout, attention, aggregate, blocks, brute, topp, cues, coarse  # noqa: F401
from .layout import Layout, Rule  # noqa: F401
from .attention import run_layer, attend  # noqa: F401
from .aggregate import frame_evidence, topk_per_video  # noqa: F401
