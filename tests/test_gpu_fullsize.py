"""GPU parity at the full sizes of the five workloads (paper-like shapes), through the C-ABI and in
the launch configuration the library uses for them (the benchmark's for L = 128K), on sampled
rows that the float64 oracle computes one by one: the boundary rows of the streaming split and
of pages, the last rows, and seeded random rows. Inputs are drawn on the device (seeded torch
Philox streams, paper_2608_01662_amd.synth) and the oracle reads the exact same buffers copied
back. Each test checks the indexer stage-wise (recalled pages, then tokens) and the sparse
attention of every checked row, given the GPU's own index list, against Eq. (3)."""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import oracle.lsa_oracle as orc
from paper_2608_01662_amd import lsa, synth
from paper_2608_01662_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _sample_positions(w, t_lo, t_hi, n_random, seed):
    """Positions in [t_lo, t_hi]: where E_t becomes non-empty, where the eligible range crosses a
    page edge, where the recalled pages stop covering all eligible ones, the last rows, plus
    seeded random rows."""
    first = w.k_sink + w.k_swa                      # first t with a non-empty eligible range
    c = {first - 1, first, first + 1, first + w.page - 1, first + w.page,
         first + w.keep_pages * w.page - 1, first + w.keep_pages * w.page + 1, t_hi - 1, t_hi}
    c |= set(np.random.default_rng(seed).integers(t_lo, t_hi + 1, n_random).tolist())
    return sorted(t for t in c if t_lo <= t <= t_hi)


def _indexer_oracle(w, q_rows, w_rows, codes, scales, rows_t, n_kv):
    """Oracle index rows for positions rows_t; q_rows / w_rows are the rows' own inputs."""
    prm = P.oracle_params(w)
    k_hat = orc.dequantized_keys(codes[:n_kv], scales[:n_kv])
    k_mean = P.oracle_block_cache(w, k_hat)
    qf = orc.bf16_bits_to_f64(q_rows)
    return [P.oracle_index_row(t, qf[i], w_rows[i], k_hat, k_mean, prm) for i, t in enumerate(rows_t)]


def _bits(t: torch.Tensor) -> np.ndarray:
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _check_attention(w, Q, KV, rows, idx, cnt, o, lse):
    """Attention of rows (indices into Q/o) over their GPU index lists against the oracle; the
    gathered latent rows are copied back, so the oracle sees exactly the cache's bytes."""
    H, dqk, dv = w.attn_dims
    worst = (0.0, 0.0)
    for i, r in enumerate(rows):
        S = idx[i][: cnt[i]]
        kv_rows = _bits(KV[torch.from_numpy(S.astype(np.int64)).to(DEV)])
        oref, lref = orc.attention_for_set(_bits(Q[r]), kv_rows, None, np.arange(S.size), dv, w.sm_scale)
        mx, rel = P.check_attention_row(o[i], lse[i], oref, lref, f"row {r}")
        worst = (max(worst[0], mx), max(worst[1], rel))
    return worst


def _prefill_case(w, q_start, n_q, n_kv, layers, n_random, seed, split_attn=False, runs_layers=()):
    """Indexer + sparse attention for query rows [q_start, q_start + n_q) of one sequence with
    n_kv cached tokens, as the library runs them; checks the sampled rows against the oracle. For
    the layers in runs_layers, attention over the run encoding must equal the list form on every
    row, bit for bit."""
    H, dqk, dv = w.attn_dims
    prm = w.index_params()
    qI = synth.device_normal_bf16((n_q, w.n_heads, w.head_dim), w.seed, synth.T_QI, DEV,
                                  scale=1.0 / math.sqrt(w.head_dim))
    wI = synth.device_uniform_f32((n_q, w.n_heads), w.seed, synth.T_W, DEV)
    kI, ks = synth.device_fp8_keys(n_kv, w.head_dim, w.seed, DEV)
    bk = lsa.block_keys(prm, kI, ks)
    out = lsa.index_prefill(prm, qI, wI, kI, ks, bk, q_start, n_kv=n_kv, runs=True, pages=True)
    rows_t = _sample_positions(w, q_start, q_start + n_q - 1, n_random, seed)
    rows = [t - q_start for t in rows_t]
    sel = torch.tensor(rows, device=DEV)
    g_idx, g_cnt = out["idx"][sel].cpu().numpy(), out["count"][sel].cpu().numpy()
    g_pages = out["pages"][sel].cpu().numpy()
    res = _indexer_oracle(w, _bits(qI[sel]), wI[sel].cpu().numpy(), kI.cpu().numpy(), ks.cpu().numpy(),
                          rows_t, n_kv)
    stats = P.check_index_rows(w, rows_t, g_idx, g_cnt, g_pages, res)
    P.check_runs(out["runs"][sel].cpu().numpy(), out["run_count"][sel].cpu().numpy(), g_idx, g_cnt, w.run_align)
    del qI, wI, bk
    # the same index list feeds every layer of the group (only the layers' inputs differ)
    for layer in layers:
        Q = synth.device_normal_bf16((n_q, H, dqk), w.seed, synth.T_Q + layer, DEV, rows_per_chunk=2048)
        KV = synth.device_normal_bf16((n_kv, dqk), w.seed, synth.T_KV + layer, DEV)
        if split_attn:   # listed part and contiguous window on two streams, merged by LSE
            o, lse = lsa.hfa_attn(w.attn_params(), Q, KV, out["idx"], out["count"], q_start, w.k_swa)
        else:
            o, lse = lsa.sparse_attn(w.attn_params(), Q, KV, None, out["idx"], out["count"])
        if layer in runs_layers:
            o2, lse2 = lsa.sparse_attn_runs(w.attn_params(), Q, KV, out["runs"], out["run_count"])
            torch.cuda.synchronize()
            assert torch.equal(o, o2) and torch.equal(lse, lse2), f"{w.name} layer {layer}: run form differs"
            del o2, lse2
        worst = _check_attention(w, Q, KV, rows, g_idx, g_cnt, o[sel].float().cpu().numpy(),
                                 lse[sel].cpu().numpy())
        print(f"{w.name} layer {layer}: index {stats}, attention worst max|d| {worst[0]:.2e} rel {worst[1]:.2e}")
        del Q, KV, o, lse
    torch.cuda.empty_cache()


def test_fullsize_prefill_L32768():
    w = W.L32K_MLA
    _prefill_case(w, 0, w.seq_len, w.seq_len, layers=[0], n_random=40, seed=101)


def test_fullsize_prefill_L131072_cross_layer():
    w = W.L128K_CLI4
    _prefill_case(w, 0, w.seq_len, w.seq_len, layers=[0, w.layers - 1], n_random=32, seed=102, runs_layers=[0])


def test_fullsize_split_attention_L131072():
    """The split attention (Sec. 4.1.1) at the benchmark's size: 131072 rows in 8 passes of 16384,
    sampled rows against the oracle's Eq. (3) over the GPU's own index lists."""
    w = W.L128K_CLI4
    _prefill_case(w, 0, w.seq_len, w.seq_len, layers=[0], n_random=24, seed=106, split_attn=True)


def test_fullsize_prefill_L1M_last_chunk():
    """The last 8192-row chunk of the 1M-token prefill, against the whole 1M-token prefix."""
    w = W.L1M_CHUNKED
    q_start = w.seq_len - w.chunk
    _prefill_case(w, q_start, w.chunk, w.seq_len, layers=[0], n_random=16, seed=103, runs_layers=[0])


def test_fullsize_prefill_L1M_paper_hi_setting():
    """The paper's chosen hierarchical setting at scale (B = 8, P = 128, M = 1024: 131072 fine
    candidates per row, selected with the candidate keys read from global memory), on the last
    8192-row chunk of the 1M-token prefill."""
    w = W.L1M_HI_B8
    q_start = w.seq_len - w.chunk
    _prefill_case(w, q_start, w.chunk, w.seq_len, layers=[0], n_random=12, seed=104)


def test_fullsize_flat_L131072_row_passes():
    """Flat indexing (Eq. 7 over every eligible token) of the last 20000 rows of the 128K prefill:
    512 KB of candidate scores per row, so the library scores the rows in two passes over its
    workspace (16384 rows, then 3616), each selecting from global memory. Rows on both sides of
    the pass boundary, the last row and seeded random rows against the oracle."""
    from dataclasses import replace
    w = replace(W.L128K_CLI4, keep_pages=0)
    n, n_q = w.seq_len, 20000
    q_start = n - n_q
    prm = w.index_params()
    qI = synth.device_normal_bf16((n_q, w.n_heads, w.head_dim), w.seed, synth.T_QI, DEV,
                                  scale=1.0 / math.sqrt(w.head_dim))
    wI = synth.device_uniform_f32((n_q, w.n_heads), w.seed, synth.T_W, DEV)
    kI, ks = synth.device_fp8_keys(n, w.head_dim, w.seed, DEV)
    out = lsa.index_prefill(prm, qI, wI, kI, ks, None, q_start, n_kv=n, runs=True)
    rows = sorted({0, 1, 16383, 16384, 16385, n_q - 1} |
                  set(np.random.default_rng(105).integers(0, n_q, 6).tolist()))
    sel = torch.tensor(rows, device=DEV)
    rows_t = [q_start + r for r in rows]
    g_idx, g_cnt = out["idx"][sel].cpu().numpy(), out["count"][sel].cpu().numpy()
    res = _indexer_oracle(w, _bits(qI[sel]), wI[sel].cpu().numpy(), kI.cpu().numpy(), ks.cpu().numpy(), rows_t, n)
    stats = P.check_index_rows(w, rows_t, g_idx, g_cnt, None, res)
    P.check_runs(out["runs"][sel].cpu().numpy(), out["run_count"][sel].cpu().numpy(), g_idx, g_cnt, w.run_align)
    print(f"flat L=131072 rows {rows_t[0]}..{rows_t[-1]}: index {stats}")


def test_fullsize_decode_b64():
    """64 sequences of 16K..128K tokens in randomly permuted 64-token pages, one new token each;
    every sequence is checked."""
    w = W.DECODE64
    H, dqk, dv = w.attn_dims
    prm = w.index_params()
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    n_tok = n_phys * w.kv_page
    qI = synth.device_normal_bf16((w.batch, w.n_heads, w.head_dim), w.seed, synth.T_QI, DEV,
                                  scale=1.0 / math.sqrt(w.head_dim))
    wI = synth.device_uniform_f32((w.batch, w.n_heads), w.seed, synth.T_W, DEV)
    kI, ks = synth.device_fp8_keys(n_tok, w.head_dim, w.seed, DEV)
    bk = lsa.block_keys(prm, kI, ks)
    ctx_d, table_d = P.to_dev(ctx), P.to_dev(table)
    out = lsa.index_decode(prm, ctx_d, table_d, w.kv_page, n_phys, qI, wI, kI, ks, bk, runs=True, pages=True)
    g = {k: v.cpu().numpy() for k, v in out.items()}
    batch_rows = list(range(w.batch))  # every sequence
    codes = kI.cpu().numpy().reshape(n_phys, w.kv_page, -1)
    scales = ks.cpu().numpy().reshape(n_phys, w.kv_page)
    qb, wb = _bits(qI), wI.cpu().numpy()
    prmo = P.oracle_params(w)
    rows_t, res = [], []
    for b in batch_rows:
        t = int(ctx[b]) - 1
        k_log = orc.dequantized_keys(orc.logical_rows(codes, table[b], t + 1, w.kv_page),
                                     orc.logical_rows(scales, table[b], t + 1, w.kv_page))
        k_mean = P.oracle_block_cache(w, k_log)
        res.append(P.oracle_index_row(t, orc.bf16_bits_to_f64(qb[b]), wb[b], k_log, k_mean, prmo))
        rows_t.append(t)
    stats = P.check_index_rows(w, rows_t, g["idx"][batch_rows], g["count"][batch_rows], g["pages"][batch_rows], res)
    P.check_runs(g["runs"][batch_rows], g["run_count"][batch_rows], g["idx"][batch_rows], g["count"][batch_rows],
                 w.run_align)
    del qI, wI, kI, ks, bk
    # paged attention: logical positions go through the same page table
    Q = synth.device_normal_bf16((w.batch, H, dqk), w.seed, synth.T_Q, DEV)
    KV = synth.device_normal_bf16((n_tok, dqk), w.seed, synth.T_KV, DEV)
    o, lse = lsa.sparse_attn(w.attn_params(), Q, KV.view(n_phys, w.kv_page, dqk), None, out["idx"], out["count"],
                             page_table=table_d, kv_page_size=w.kv_page)
    o, lse = o.float().cpu().numpy(), lse.cpu().numpy()
    worst = (0.0, 0.0)
    for b in batch_rows:
        S = g["idx"][b][: g["count"][b]]
        phys = table[b][S // w.kv_page].astype(np.int64) * w.kv_page + S % w.kv_page
        kv_rows = _bits(KV[torch.from_numpy(phys).to(DEV)])
        oref, lref = orc.attention_for_set(_bits(Q[b]), kv_rows, None, np.arange(S.size), dv, w.sm_scale)
        mx, rel = P.check_attention_row(o[b], lse[b], oref, lref, f"sequence {b}")
        worst = (max(worst[0], mx), max(worst[1], rel))
    print(f"{w.name}: index {stats}, attention worst max|d| {worst[0]:.2e} rel {worst[1]:.2e}")
