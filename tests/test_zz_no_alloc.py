"""lsa_index_decode_static (the decode indexer whose scratch is the library's fixed device array,
for callers that cannot allocate) against lsa_index_decode with a caller workspace, through the
C-ABI: integer outputs (index lists, counts, runs, recalled pages) must be bit-identical.

Two calls in a row share the array, the second with a smaller input (fewer sequences, shorter
contexts), so a stale entry left by the first call would show in the second; a flat-mode call over
128K-token contexts needs more than the array holds for all rows at once and runs in two row
passes."""
from __future__ import annotations

from dataclasses import replace

import numpy as np
import pytest
import torch

from paper_2608_01662_amd import lsa, synth
from paper_2608_01662_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _case(w, batch=None, seed_shift=0, table_cols=None):
    ctx, table, n_phys = synth.decode_layout(w.seed + seed_shift, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    if batch is not None:
        ctx, table = ctx[:batch], table[:batch]
    if table_cols is not None:          # a wider page table (unused entries -1) raises max_pages
        wide = np.full((table.shape[0], table_cols), -1, np.int32)
        wide[:, :table.shape[1]] = table
        table = wide
    n_tok = n_phys * w.kv_page
    B = ctx.shape[0]
    qI = synth.device_normal_bf16((B, w.n_heads, w.head_dim), w.seed + seed_shift, synth.T_QI, DEV,
                                  scale=float(w.head_dim) ** -0.5)
    wI = synth.device_uniform_f32((B, w.n_heads), w.seed + seed_shift, synth.T_W, DEV)
    kI, ks = synth.device_fp8_keys(n_tok, w.head_dim, w.seed + seed_shift, DEV)
    prm = w.index_params()
    bk = lsa.block_keys(prm, kI, ks) if w.keep_pages > 0 else None
    return dict(prm=prm, ctx=P.to_dev(ctx), table=P.to_dev(table), n_phys=n_phys, q=qI, w=wI, k=kI, ks=ks, bk=bk)


def _outputs(prm, B, pages):
    o = dict(idx=torch.full((B, prm.k_cap), -7, dtype=torch.int32, device=DEV),
             count=torch.full((B,), -7, dtype=torch.int32, device=DEV),
             runs=torch.full((B, prm.k_cap, 2), -7, dtype=torch.int32, device=DEV),
             run_count=torch.full((B,), -7, dtype=torch.int32, device=DEV))
    if pages:
        o["pages"] = torch.full((B, prm.keep_pages), -7, dtype=torch.int32, device=DEV)
    return o


def _both(c, kv_page):
    prm, B = c["prm"], c["ctx"].shape[0]
    pages = prm.keep_pages > 0
    ref = lsa.index_decode(prm, c["ctx"], c["table"], kv_page, c["n_phys"], c["q"], c["w"], c["k"], c["ks"], c["bk"],
                           runs=True, pages=pages, out=_outputs(prm, B, pages))
    got = lsa.index_decode_static(prm, c["ctx"], c["table"], kv_page, c["n_phys"], c["q"], c["w"], c["k"], c["ks"],
                                  c["bk"], out=_outputs(prm, B, pages))
    torch.cuda.synchronize()
    assert set(got) == set(ref)
    for key in ref:
        assert torch.equal(got[key], ref[key]), key
    return ref


def test_static_decode_two_calls_second_smaller():
    """The 64-sequence decode workload (16K..128K contexts, hierarchical), then 5 sequences of the
    reduced one (2K..6K contexts): both equal the workspace call bit for bit."""
    big = _both(_case(W.DECODE64), W.DECODE64.kv_page)
    assert int(big["count"].min()) > 0
    small = _both(_case(W.SMALL_DECODE, batch=5, seed_shift=1), W.SMALL_DECODE.kv_page)
    assert small["idx"].shape[0] == 5


def test_static_decode_row_passes():
    """Flat indexing of the 64 sequences with a page table of 4096 entries per sequence (a 256K
    capacity): 1 MB of fine-score keys per row, so the 32 MB array takes the rows in three passes
    of 31; equal to the workspace call bit for bit."""
    w = replace(W.DECODE64, keep_pages=0)
    cols = 4096
    per_row = cols * w.page * 4 + 768
    assert -(-w.batch // (((32 << 20) - 768) // (per_row - 768))) == 3   # three passes, one row fits
    _both(_case(w, table_cols=cols), w.kv_page)
