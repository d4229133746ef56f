"""CPU oracle for the speculative verification step (test infrastructure only).

A plain, slow, float64 implementation of what the GPU path computes, written
from the paper (SpecRoll, arXiv 2608.04962):

* ``heads``     -- future-token heads on the corrected hidden state
                   (Sec. 3.2, Eq. (heads); App. C, "Future-token proposer").
* ``tree``      -- ordered, without-replacement child lists per node
                   (App. B.1, Eq. (slotq), Eq. (childlist)).
* ``attention`` -- target attention of every tree node over its trajectory's
                   prefix plus its own root path (App. B.1, Eq. (nodep)).
* ``accept``    -- exact node-wise verification with full-vocabulary
                   residuals (App. B.2, Eq. (nodeaccept), Eq. (noderesidual),
                   Alg. "Exact node-wise tree verification").
* ``engine``    -- the concurrency-aware node budget and the tree it allows
                   (Sec. 3.2, Eq. (verification-budget), Eq. (tree-budget)) and
                   the accepted-path cache extraction.
* ``reflex``    -- verifier feedback directions, the trajectory-local
                   memory update, delayed-alignment reliability and the gated
                   head-state correction (Sec. 3.3; Sec. 3.4 Eq. (support) to
                   Eq. (reflex-correction); App. A.1; App. C).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may use this package. It shares no code with the HIP library and
does not import it; the product path never calls it.
"""
from .numerics import round_bf16, softmax, logsumexp  # noqa: F401
from .heads import clip_correction, layer_norm, silu, heads_forward  # noqa: F401
from .tree import tree_structure, top_m, sample_ordered_children, tree_build  # noqa: F401
from .attention import gather_prefix, tree_attention, tree_attention_node  # noqa: F401
from .accept import inverse_cdf, tree_accept, tree_accept_one, FALLBACK, BONUS  # noqa: F401
from .engine import tree_budget, commit_path  # noqa: F401
from .reflex import (feedback, reflex_feedback, ema_update, build_support, top_list, sketch,  # noqa: F401
                     moments_update, reliability, correction)
