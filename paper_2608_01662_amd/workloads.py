"""Workload presets: the shapes the LSA hot path is measured and checked on.

Each preset names its sizes; none holds any of the method's arithmetic. The five full-size
workloads mirror the paper's settings (Table 6 model shapes, Sec. 3.1 / 3.3 budgets) at one GPU's
share; the reduced ones keep every structural feature (several tiles, ragged tails, hierarchical
mode active) at sizes the float64 oracle finishes in seconds.
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    # indexer
    n_heads: int
    head_dim: int
    fp8: bool
    page: int
    sub_block: int
    keep_pages: int
    k_sparse: int
    k_sink: int
    k_swa: int
    run_align: int
    # attention
    attn: str                    # "mqa" (16 x 128) or "mla" (64 x 576/512)
    sm_scale: float
    layers: int = 1              # layers sharing one index list (cross-layer indexing)
    # sequence
    seq_len: int = 0             # prefill: tokens of the single sequence
    chunk: int = 0               # prefill: query rows per call (0 = all rows at once)
    batch: int = 0               # decode: sequences (one new token each)
    ctx_lo: int = 0
    ctx_hi: int = 0
    kv_page: int = 0             # decode: tokens per cache page
    pooling: str = "mean"        # coarse-stage block summary: "mean" (Eq. 9) or "minmax" (Eq. 13)
    hi_min_kv: int = 0           # adaptive dispatch: caches of at most this many tokens indexed flat

    @property
    def k_cap(self) -> int:
        return self.k_sink + self.k_swa + self.k_sparse

    @property
    def decode(self) -> bool:
        return self.batch > 0

    def index_params(self):
        from .lsa import IndexParams
        return IndexParams(self.n_heads, self.head_dim, self.fp8, self.page, self.sub_block, self.keep_pages,
                           self.k_sparse, self.k_sink, self.k_swa, self.run_align, self.pooling, self.hi_min_kv)

    def attn_params(self):
        from .lsa import MLA, MQA, AttnParams
        return AttnParams(sm_scale=self.sm_scale, **(MLA if self.attn == "mla" else MQA))

    @property
    def attn_dims(self):
        return (16, 128, 128) if self.attn == "mqa" else (64, 576, 512)


MLA_SCALE = 192 ** -0.5          # MLA query/key head: 128 nope + 64 rope dims (Table 6)
MQA_SCALE = 128 ** -0.5

# 1. single-sequence prefill, L = 2048, MQA attention
L2K_MQA = Workload("prefill_L2048_mqa", seed=0, n_heads=8, head_dim=64, fp8=False, page=64, sub_block=64,
                   keep_pages=16, k_sparse=256, k_sink=4, k_swa=128, run_align=64, attn="mqa",
                   sm_scale=MQA_SCALE, seq_len=2048)
# 2. single-sequence prefill, L = 32K, fp8 indexer keys, MLA attention
L32K_MLA = Workload("prefill_L32768_mla", seed=1, n_heads=32, head_dim=128, fp8=True, page=64, sub_block=64,
                    keep_pages=128, k_sparse=2048, k_sink=4, k_swa=512, run_align=64, attn="mla",
                    sm_scale=MLA_SCALE, seq_len=32768)
# 3. single-sequence prefill, L = 128K, one index list shared by 4 layers
L128K_CLI4 = Workload("prefill_L131072_cli4_mla", seed=2, n_heads=32, head_dim=128, fp8=True, page=128,
                      sub_block=128, keep_pages=64, k_sparse=2048, k_sink=4, k_swa=1024, run_align=128,
                      attn="mla", sm_scale=MLA_SCALE, layers=4, seq_len=131072)
# 4. batched decode, 64 sequences of 16K..128K tokens in permuted 64-token pages
DECODE64 = Workload("decode_b64_ctx16k_128k_mla", seed=3, n_heads=32, head_dim=128, fp8=True, page=64,
                    sub_block=64, keep_pages=128, k_sparse=2048, k_sink=4, k_swa=256, run_align=64, attn="mla",
                    sm_scale=MLA_SCALE, batch=64, ctx_lo=16384, ctx_hi=131072, kv_page=64)
# 5. chunked prefill of a 1M-token sequence, 8192-row chunks, 4 layers sharing each index list
L1M_CHUNKED = Workload("prefill_L1048576_chunk8192_cli4_mla", seed=4, n_heads=32, head_dim=128, fp8=True,
                       page=128, sub_block=128, keep_pages=256, k_sparse=4096, k_sink=4, k_swa=2048,
                       run_align=128, attn="mla", sm_scale=MLA_SCALE, layers=4, seq_len=1048576, chunk=8192)

# 6. the paper's chosen hierarchical setting at scale: 16 mean keys per 128-token page (B = 8) and
#    M = 1024 recalled pages (131072 fine candidates per row), on the 1M-token chunked prefill
L1M_HI_B8 = replace(L1M_CHUNKED, name="prefill_L1048576_chunk8192_cli4_hi_b8_m1024", sub_block=8, keep_pages=1024)

FULL = [L2K_MQA, L32K_MLA, L128K_CLI4, DECODE64, L1M_CHUNKED, L1M_HI_B8]
BY_NAME = {w.name: w for w in FULL}

# Reduced shapes for oracle parity at full-row coverage (same structure, smaller L and budgets).
SMALL_MLA = replace(L32K_MLA, name="small_L4096_mla", seq_len=4096, keep_pages=16, k_sparse=256, k_swa=128)
SMALL_CLI = replace(L128K_CLI4, name="small_L8192_cli4", seq_len=8192, keep_pages=8, k_sparse=384, k_swa=512,
                    layers=2)
SMALL_SUBBLOCK = replace(L128K_CLI4, name="small_L8192_B8", seq_len=8192, sub_block=8, keep_pages=8,
                         k_sparse=384, k_swa=512, layers=1)
SMALL_FLAT = replace(L2K_MQA, name="small_L2048_flat", keep_pages=0)
# min-max pooling of the coarse stage (Eq. 13), with one and with 16 sub-blocks per page
SMALL_MINMAX = replace(SMALL_CLI, name="small_L8192_cli4_minmax", pooling="minmax")
SMALL_MINMAX_B8 = replace(SMALL_SUBBLOCK, name="small_L8192_B8_minmax", pooling="minmax")
SMALL_DECODE = replace(DECODE64, name="small_decode_b8", batch=8, ctx_lo=2048, ctx_hi=6000, keep_pages=16,
                       k_sparse=256, k_swa=128)
SMALL_DECODE_MINMAX = replace(SMALL_DECODE, name="small_decode_b8_minmax", pooling="minmax")
SMALL_CHUNKED = replace(L1M_CHUNKED, name="small_L16384_chunk1000", seq_len=16384, chunk=1000, keep_pages=16,
                        k_sparse=512, k_swa=256, layers=2)
