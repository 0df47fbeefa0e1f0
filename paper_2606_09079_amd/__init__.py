"""MI355X (gfx950) decode hot path of Lookahead Sparse Attention.

score every compressed chunk (Memory Indexer dot product) -> keep the top-k
chunks -> sparse decode attention over the kept chunks, and the recall path
(full gated multi-head Memory Indexer, sigmoid threshold, OR over indexer
layers, K_max bound) in front of the same attention, the two-level selection
(recall, native top-k inside it, always-resident window) and the host tier
(pinned host mirror, GPU reserve of chunk slots, residency plan, copies,
attention over the reserve), the re-layout of a token-major cache into the
paged blocks the attention reads, and the golden-label pipeline (softmax, top-p,
votes across layers, union over the window), as hand-written HIP
kernels behind the C ABI of ``include/lsa.h``.  The Python layer is the thin
ctypes binding in :mod:`.lsa`; importing it loads ``liblsa.so`` and raises if
that is not possible.
"""
from .lsa import (LIB, Golden, Indexer, LsaError, Problem, Tier, TwoLevel, lsa_decode_step,  # noqa: F401
                  lsa_decode_step_noalloc, lsa_kv_pack,
                  lsa_golden_labels, lsa_golden_sizes, lsa_max_keep, lsa_max_sel, lsa_recall_scores,
                  lsa_recall_select, lsa_recall_step, lsa_score_chunks, lsa_sparse_decode_attn, lsa_tier_attend,
                  lsa_tier_fetch, lsa_tier_fetch_dma, lsa_tier_plan, lsa_tier_reset, lsa_tier_sizes, lsa_tier_step,
                  lsa_topk_chunks, lsa_two_level_sizes, lsa_two_level_step, lsa_validate, lsa_workspace_init,
                  lsa_workspace_size, last_error)
