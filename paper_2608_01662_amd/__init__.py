"""LongCat Sparse Attention (LSA) hot path for AMD Instinct MI355X (gfx950).

HIP kernels behind a C-ABI (include/lsa.h, built into liblsa.so) and a thin ctypes binding:
indexer (mean keys, coarse page scores, page top-M, fine token scores, token top-K with sink and
window merge, runs), and sparse attention over the resulting index list, reused across layers.
"""
from .lsa import (AttnParams, IndexParams, LSAError, MLA, MQA, attn_workspace_size,  # noqa: F401
                  block_means, index_decode, index_prefill, index_workspace_size, lib, sparse_attn,
                  version)
