"""Sharded decode emulated on one GPU. The paper's key-value parallel layout (App. B) puts page i
of every sequence on rank i mod N. Here each virtual rank sees only its own pages (the page-table
entries of the other pages are -1, which the kernels skip), and the host merges the ranks:

* indexing (flat, as under KVP): the union of the ranks' local sparse selections, re-ranked by
  score with the (score desc, position asc) rule, must give the global top-K_sparse of the
  unsharded call, up to score ties;
* attention: the ranks' (o, lse) partials over their shares of S_t, merged by log-sum-exp, must
  equal the unsharded output within bf16 rounding.
"""
from __future__ import annotations

from dataclasses import replace

import numpy as np
import pytest
import torch

import oracle.lsa_oracle as orc
from paper_2608_01662_amd import lsa, synth
from paper_2608_01662_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu

N_RANKS = 4


def _rank_table(table: np.ndarray, r: int) -> np.ndarray:
    """Page table of virtual rank r: logical pages i with i mod N_RANKS != r are not held (-1)."""
    t = table.copy()
    t[:, np.arange(t.shape[1]) % N_RANKS != r] = -1
    return t


def test_kvp_index_rerank_equals_unsharded():
    w = replace(W.SMALL_DECODE, keep_pages=0)
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    inp = synth.indexer_inputs(w.seed, w.batch, n_phys * w.kv_page, w.n_heads, w.head_dim, w.fp8)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    dctx = P.to_dev(ctx)
    full = lsa.index_decode(prm, dctx, P.to_dev(table), w.kv_page, n_phys, q, wt, k, ks, None, runs=False)
    local = [lsa.index_decode(prm, dctx, P.to_dev(_rank_table(table, r)), w.kv_page, n_phys, q, wt, k, ks, None,
                              runs=False) for r in range(N_RANKS)]
    torch.cuda.synchronize()
    full = {key: v.cpu().numpy() for key, v in full.items()}
    local = [{key: v.cpu().numpy() for key, v in out.items()} for out in local]
    k_pool = P.oracle_keys(inp).reshape(n_phys, w.kv_page, -1)
    qf = orc.bf16_bits_to_f64(inp["q"])
    ties = 0
    for b in range(w.batch):
        t = int(ctx[b]) - 1
        fixed = set(range(min(w.k_sink, t + 1))) | set(range(max(0, t - w.k_swa + 1), t + 1))
        S = full["idx"][b, :full["count"][b]].tolist()
        assert fixed <= set(S)
        union = []
        for r, out in enumerate(local):
            Sr = out["idx"][b, :out["count"][b]].tolist()
            assert fixed <= set(Sr), "every rank's list carries sink and window"
            sparse_r = [s for s in Sr if s not in fixed]
            assert all((s // w.kv_page) % N_RANKS == r for s in sparse_r), f"rank {r} selected a page it does not hold"
            assert len(sparse_r) <= w.k_sparse
            union += sparse_r
        # the re-rank on the host, scored by the oracle over the logical keys
        k_log = orc.logical_rows(k_pool, table[b], t + 1, w.kv_page)
        elig = np.arange(w.k_sink, t - w.k_swa + 1, dtype=np.int64)
        scores = orc.indexer_scores(qf[b], inp["w"][b], k_log[elig]) if elig.size else np.zeros(0)
        score_of = dict(zip(elig.tolist(), scores.tolist()))
        ids = np.array(sorted(union), np.int64)
        merged = orc.arg_top(np.array([score_of[s] for s in ids.tolist()]), ids, w.k_sparse)
        sparse_full = [s for s in S if s not in fixed]
        ties += P.tie_equivalent(sparse_full, merged, elig, scores, w.k_sparse)
    print(f"KVP index re-rank over {N_RANKS} virtual ranks: {w.batch} sequences, {ties} tie swaps")


def test_kvp_attention_combine_equals_unsharded():
    w = W.SMALL_DECODE
    H, dqk, dv = w.attn_dims
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    a = synth.attention_inputs(w.seed, 0, w.batch, n_phys * w.kv_page, H, dqk, dv, latent=True)
    g = np.random.default_rng(4)
    idx = np.full((w.batch, w.k_cap), -1, np.int32)
    cnt = np.zeros(w.batch, np.int32)
    for b in range(w.batch):
        t = int(ctx[b]) - 1
        S = np.unique(np.concatenate([np.arange(w.k_sink), g.choice(t + 1, w.k_sparse, replace=False),
                                      np.arange(t - w.k_swa + 1, t + 1)]))
        idx[b, :S.size] = S
        cnt[b] = S.size
    kv = P.bf16_dev(a["kv"]).view(n_phys, w.kv_page, dqk)
    q = P.bf16_dev(a["q"])
    didx, dcnt = P.to_dev(idx), P.to_dev(cnt)
    o, lse = lsa.sparse_attn(w.attn_params(), q, kv, None, didx, dcnt, page_table=P.to_dev(table),
                             kv_page_size=w.kv_page)
    parts = [lsa.sparse_attn(w.attn_params(), q, kv, None, didx, dcnt, page_table=P.to_dev(_rank_table(table, r)),
                             kv_page_size=w.kv_page) for r in range(N_RANKS)]
    torch.cuda.synchronize()
    o_r = np.stack([p[0].float().cpu().numpy().astype(np.float64) for p in parts])   # [N, batch, H, dv]
    l_r = np.stack([p[1].cpu().numpy().astype(np.float64) for p in parts])           # [N, batch, H]
    l_m = np.logaddexp.reduce(l_r, axis=0)
    o_m = (np.exp(l_r - l_m[None])[..., None] * o_r).sum(axis=0)
    o_full = o.float().cpu().numpy().astype(np.float64)
    err = np.abs(o_m - o_full)
    assert err.max() <= 2e-2, f"merged output differs by {err.max():.3e}"
    rel = np.linalg.norm(o_m - o_full) / np.linalg.norm(o_full)
    assert rel <= 1e-2, f"merged output relative difference {rel:.3e}"
    assert np.abs(l_m - lse.cpu().numpy()).max() <= 2e-3
    print(f"KVP attention combine over {N_RANKS} virtual ranks: max|d| {err.max():.2e}, rel {rel:.2e}")
