"""GPU parity of lsa_sparse_attn (MQA-128 and MLA-576/512, contiguous and paged caches) against the
oracle's Eq. (3) through the C-ABI. The GPU and the oracle always get the same index list (built
by the oracle or by the test), so the comparison isolates the attention kernel."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import oracle.lsa_oracle as orc
from paper_2608_01662_amd import lsa, synth
from paper_2608_01662_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def _oracle_index(w, rows_t, n_kv):
    inp = P.prefill_inputs(w, n_kv)
    prm = P.oracle_params(w)
    k_hat = P.oracle_keys(inp)
    k_mean = orc.sub_block_mean_keys(k_hat, w.sub_block) if w.keep_pages > 0 else None
    qf = orc.bf16_bits_to_f64(inp["q"])
    idx = np.full((len(rows_t), w.k_cap), -1, np.int32)
    cnt = np.zeros(len(rows_t), np.int32)
    for i, t in enumerate(rows_t):
        S = orc.index_row(t, qf[t], inp["w"][t], k_hat, k_mean, prm)["S"]
        idx[i, :S.size] = S
        cnt[i] = S.size
    return idx, cnt


def _attn_inputs(w, layer, n_q, n_kv):
    H, dqk, dv = w.attn_dims
    return synth.attention_inputs(w.seed, layer, n_q, n_kv, H, dqk, dv, latent=(w.attn == "mla"))


def _gpu_attn(w, a, rows, idx, cnt, lse=True):
    q = P.bf16_dev(a["q"][rows])
    kv = P.bf16_dev(a["kv"])
    v = P.bf16_dev(a["v"]) if a["v"] is not None else None
    o, l = lsa.sparse_attn(w.attn_params(), q, kv, v, P.to_dev(idx), P.to_dev(cnt), lse=lse)
    torch.cuda.synchronize()
    o = o.float().cpu().numpy()
    return o, (l.cpu().numpy() if l is not None else None)


def _check_rows(w, a, rows, idx, cnt, o, l):
    H, dqk, dv = w.attn_dims
    worst = (0.0, 0.0)
    for i, t in enumerate(rows):
        S = idx[i][: cnt[i]]
        S = S[(S >= 0) & (S < a["kv"].shape[0])]
        oref, lref = orc.attention_for_set(a["q"][t], a["kv"], a["v"], S, dv, w.sm_scale)
        mx, rel = P.check_attention_row(o[i], None if l is None else l[i], oref, lref, f"row {t}")
        worst = (max(worst[0], mx), max(worst[1], rel))
    return worst


@pytest.mark.parametrize("w", [W.L2K_MQA, W.SMALL_MLA], ids=lambda w: w.name)
def test_attention_parity_oracle_index(w):
    n = w.seq_len
    rows = list(range(0, n, 3 if w.attn == "mqa" else 13)) + [n - 1, w.k_sink + w.k_swa + 1, 5]
    idx, cnt = _oracle_index(w, rows, n)
    a = _attn_inputs(w, 0, n, n)
    o, l = _gpu_attn(w, a, rows, idx, cnt)
    print(w.name, "worst (max|d|, rel)", _check_rows(w, a, rows, idx, cnt, o, l))


@pytest.mark.parametrize("attn", ["mqa", "mla"])
def test_dense_causal_equals_sdpa(attn):
    """K >= t+1: the index list is [0, t] and sparse attention is causal softmax attention
    (torch's scaled_dot_product_attention in float64 on the CPU)."""
    from dataclasses import replace
    w = replace(W.L2K_MQA if attn == "mqa" else W.SMALL_MLA, seq_len=200)
    T = w.seq_len
    H, dqk, dv = w.attn_dims
    a = _attn_inputs(w, 0, T, T)
    idx = np.full((T, T), -1, np.int32)
    for t in range(T):
        idx[t, :t + 1] = np.arange(t + 1)
    cnt = np.arange(1, T + 1, dtype=np.int32)
    o, l = _gpu_attn(w, a, list(range(T)), idx, cnt)
    q = torch.from_numpy(orc.bf16_bits_to_f64(a["q"])).permute(1, 0, 2)[None]
    kf = torch.from_numpy(orc.bf16_bits_to_f64(a["kv"]))
    vf = kf[:, :dv] if a["v"] is None else torch.from_numpy(orc.bf16_bits_to_f64(a["v"]))
    ref = torch.nn.functional.scaled_dot_product_attention(
        q, kf[None, None].expand(1, H, T, dqk), vf.contiguous()[None, None].expand(1, H, T, dv),
        is_causal=True, scale=w.sm_scale)[0].permute(1, 0, 2).numpy()
    for t in range(T):
        P.check_attention_row(o[t], None, ref[t], None, f"t={t}")


@pytest.mark.parametrize("attn", ["mqa", "mla"])
def test_closed_forms_and_edge_lists(attn):
    from dataclasses import replace
    w = replace(W.L2K_MQA if attn == "mqa" else W.SMALL_MLA, seq_len=300)
    H, dqk, dv = w.attn_dims
    n_kv = w.seq_len
    a = _attn_inputs(w, 0, 8, n_kv)
    k_cap = 96
    g = np.random.default_rng(1)
    idx = np.full((8, k_cap), -1, np.int32)
    cnt = np.zeros(8, np.int32)
    idx[0, 0] = 17; cnt[0] = 1                                       # one token: o = v_17
    idx[1, :70] = g.choice(n_kv, 70, replace=False); cnt[1] = 70     # unsorted, ragged (70 = 2 tiles + 6)
    idx[2, :70] = idx[1, :70][::-1]; cnt[2] = 70                     # same set, reversed order
    cnt[3] = 0                                                       # empty set: o = 0, lse = -inf
    idx[4, :40] = np.arange(40); idx[4, 10] = -1; idx[4, 20] = n_kv + 5; cnt[4] = 40   # bad entries skipped
    idx[5, :k_cap] = np.arange(k_cap) * 3; cnt[5] = k_cap            # full capacity
    idx[6, :33] = np.arange(33); cnt[6] = 33                         # one past a tile
    idx[7, :5] = [0, 0, 1, 1, 2]; cnt[7] = 5                         # duplicates attend twice
    rows = list(range(8))
    a["q"] = a["q"][:8].copy()
    a["q"][2] = a["q"][1]                                            # rows 1 and 2: same query, same set
    o, l = _gpu_attn(w, a, rows, idx, cnt)
    vbits = a["kv"][:, :dv] if a["v"] is None else a["v"]
    assert np.array_equal(o[0], np.repeat(orc.bf16_bits_to_f64(vbits[17])[None], H, 0))
    assert np.abs(o[1] - o[2]).max() <= 2e-2 and np.allclose(l[1], l[2], atol=1e-4)
    assert np.all(o[3] == 0) and np.all(np.isneginf(l[3]))
    for i in (1, 4, 5, 6, 7):
        S = idx[i][: cnt[i]]
        S = S[(S >= 0) & (S < n_kv)]
        oref, lref = orc.attention_for_set(a["q"][i], a["kv"], a["v"], S, dv, w.sm_scale)
        P.check_attention_row(o[i], l[i], oref, lref, f"row {i}")


# Rows whose scores jump far above everything before them at chosen list positions: (list length,
# [(list position, log2 margin of the jump over the largest background score of every head)]).
# Position 32 t + x lies in tile t, token half x // 16 of the MLA kernel's tiles. A margin above 8
# moves the lazy reference maximum of the half that holds the jump; the other half then differs
# for a tile (or to the end of the list, when the jump is in the last tile).
_SPIKE_ROWS = [
    (300, [(2 * 32 + 20, 9.5)]),                      # mid-list, second half
    (300, [(4 * 32 + 3, 9.5)]),                       # mid-list, first half
    (310, [(9 * 32 + 18, 9.5)]),                      # last (partial) tile, second half
    (300, [(32 + 5, 9.5), (6 * 32 + 24, 19.0)]),      # two jumps, one per half
    (300, [(3 * 32 + 5, 9.5), (3 * 32 + 25, 9.5)]),   # both halves of one tile
    (300, [(0, 9.5)]),                                # the first entry
    (20, [(18, 9.5)]),                                # one partial tile
    (300, [(7 * 32 + 10, 9.5), (7 * 32 + 11, 12.0)]),  # two in one half of one tile
]


def _spike_inputs(w, k_cap=320):
    """Queries q_h = q0 + 0.1 noise per row (every head scores a vector along q0 alike), background
    cache rows N(0, 0.25), and per jump a cache row c * q0 / |q0| with c chosen so that every head's
    score of it exceeds that head's largest background score of the row by the listed margin (log2
    units). Returns bf16 bits of Q [rows, H, 576] and of the cache, and the index lists."""
    H, dqk, dv = w.attn_dims
    g = np.random.default_rng(11)
    n_kv, n_rows = w.seq_len, len(_SPIKE_ROWS)
    n_bg = n_kv - 2 * n_rows  # the last 2 rows per test row hold its jumps
    q0 = g.standard_normal((n_rows, dqk))
    q_bits = orc.f64_to_bf16_bits(q0[:, None, :] + 0.1 * g.standard_normal((n_rows, H, dqk)))
    kv_bits = orc.f64_to_bf16_bits(0.5 * g.standard_normal((n_kv, dqk)))
    qf = orc.bf16_bits_to_f64(q_bits)
    idx = np.full((n_rows, k_cap), -1, np.int32)
    cnt = np.zeros(n_rows, np.int32)
    to_log2 = w.sm_scale / np.log(2.0)
    for i, (n, spikes) in enumerate(_SPIKE_ROWS):
        bg = g.choice(n_bg, n - len(spikes), replace=False)
        bgmax = (qf[i] @ orc.bf16_bits_to_f64(kv_bits[bg]).T).max(axis=1) * to_log2  # per head
        u = q0[i] / np.linalg.norm(q0[i])
        d = (qf[i] @ u) * to_log2  # per head, per unit of c
        lst = [int(r) for r in bg]
        for j, (pos, margin) in enumerate(spikes):
            r = n_bg + 2 * i + j
            kv_bits[r] = orc.f64_to_bf16_bits(np.max((bgmax + margin) / d) * u)
            lst.insert(pos, r)
        idx[i, :n] = lst
        cnt[i] = n
    return q_bits, kv_bits, idx, cnt


@pytest.mark.parametrize("copies", [1, 32], ids=["8_rows_split", "256_rows_one_pass"])
def test_softmax_reference_jumps(copies):
    """Scores that jump by more than 2^8 mid-list, in either token half of a tile, in both, twice,
    at the first entry and in the last partial tile: the lazy reference maxima of the two token
    halves then differ for a tile (or to the end), and the output must still equal Eq. 3 (oracle).
    8 rows are planned as 32-entry pieces merged by log-sum-exp; 256 rows (each row 32 times) as
    one pass per row, where the halves' maxima are reconciled across the tiles of the row."""
    from dataclasses import replace
    w = replace(W.SMALL_MLA, seq_len=2048)
    H, dqk, dv = w.attn_dims
    q_bits, kv_bits, idx, cnt = _spike_inputs(w)
    n = len(cnt)
    a = dict(q=np.tile(q_bits, (copies, 1, 1)), kv=kv_bits, v=None)
    idx_c, cnt_c = np.tile(idx, (copies, 1)), np.tile(cnt, copies)
    o, l = _gpu_attn(w, a, list(range(n * copies)), idx_c, cnt_c)
    for i in range(n):
        oref, lref = orc.attention_for_set(q_bits[i], kv_bits, None, idx[i, :cnt[i]], dv, w.sm_scale)
        P.check_attention_row(o[i], l[i], oref, lref, f"row {i} ({_SPIKE_ROWS[i]})")
        for c in range(1, copies):  # same row, same result
            assert np.array_equal(o[c * n + i], o[i]) and np.array_equal(l[c * n + i], l[i]), f"row {i} copy {c}"


def test_long_lists_beyond_one_staging_pass():
    """MLA index lists longer than the 8192 entries the kernel stages in LDS at a time: the list is
    walked in several passes (8192 = exactly one pass, 8193 = one entry into the second, and two
    longer ones), against the oracle."""
    from dataclasses import replace
    w = replace(W.SMALL_MLA, seq_len=20000)
    n_kv = w.seq_len
    a = _attn_inputs(w, 0, 4, n_kv)
    k_cap = 16448
    counts = [8192, 8193, 12345, 16448]
    g = np.random.default_rng(5)
    idx = np.full((4, k_cap), -1, np.int32)
    cnt = np.array(counts, np.int32)
    for i, c in enumerate(counts):
        idx[i, :c] = np.sort(g.choice(n_kv, c, replace=False))
    o, l = _gpu_attn(w, a, list(range(4)), idx, cnt)
    H, dqk, dv = w.attn_dims
    for i in range(4):
        oref, lref = orc.attention_for_set(a["q"][i], a["kv"], a["v"], idx[i, :cnt[i]], dv, w.sm_scale)
        P.check_attention_row(o[i], l[i], oref, lref, f"row {i} ({cnt[i]} entries)")


def test_many_rows_mixed_lists():
    """Calls of 256 rows or more run one pass over each row's whole list (no split into pieces):
    259 rows mixing short lists, empty lists, one exact tile and lists longer than one staging pass
    (8192 entries, so the list is staged in two passes), against the oracle."""
    from dataclasses import replace
    w = replace(W.SMALL_MLA, seq_len=12000)
    n_kv, n_rows, k_cap = w.seq_len, 259, 9000
    H, dqk, dv = w.attn_dims
    a = _attn_inputs(w, 0, n_rows, n_kv)
    g = np.random.default_rng(7)
    counts = g.integers(1, 400, n_rows)
    for i in (0, 5, 6, 11, 255, 258):
        counts[i] = 0                       # empty lists, also first and last of a group
    for i in (1, 4, 7, 12, 257):
        counts[i] = 8193 if i % 2 else 9000  # two staging passes
    counts[2] = 32                           # exactly one tile
    idx = np.full((n_rows, k_cap), -1, np.int32)
    for i, c in enumerate(counts):
        idx[i, :c] = g.choice(n_kv, c, replace=False)
    cnt = counts.astype(np.int32)
    o, l = _gpu_attn(w, a, list(range(n_rows)), idx, cnt)
    for i in range(n_rows):
        if cnt[i] == 0:
            assert np.all(o[i] == 0) and np.all(np.isneginf(l[i])), f"row {i}"
            continue
        oref, lref = orc.attention_for_set(a["q"][i], a["kv"], a["v"], idx[i, :cnt[i]], dv, w.sm_scale)
        P.check_attention_row(o[i], l[i], oref, lref, f"row {i} ({cnt[i]} entries)")


def test_mqa_long_lists():
    """MQA (16 x 128, separate K and V) over lists far longer than the L = 2048 workload's (1, 31,
    32, 33, 4097 and 9000 entries, the last tile partial), against the oracle."""
    from dataclasses import replace
    w = replace(W.L2K_MQA, seq_len=12000)
    n_kv = w.seq_len
    counts = [1, 31, 32, 33, 4097, 9000]
    a = _attn_inputs(w, 0, len(counts), n_kv)
    k_cap = max(counts)
    g = np.random.default_rng(11)
    idx = np.full((len(counts), k_cap), -1, np.int32)
    cnt = np.array(counts, np.int32)
    for i, c in enumerate(counts):
        idx[i, :c] = np.sort(g.choice(n_kv, c, replace=False))
    o, l = _gpu_attn(w, a, list(range(len(counts))), idx, cnt)
    H, dqk, dv = w.attn_dims
    for i in range(len(counts)):
        oref, lref = orc.attention_for_set(a["q"][i], a["kv"], a["v"], idx[i, :cnt[i]], dv, w.sm_scale)
        P.check_attention_row(o[i], l[i], oref, lref, f"row {i} ({cnt[i]} entries)")


@pytest.mark.parametrize("n_rows", [None, 8], ids=["all_rows", "split_8_rows"])
def test_run_form_equals_list_form(n_rows):
    """Attention over the indexer's run encoding equals attention over its index lists, bit for bit
    (the kernel expands the runs while staging a row's list); with 8 rows the call takes the split
    path (partials merged by log-sum-exp)."""
    w = W.SMALL_CLI
    inp = synth.indexer_inputs(w.seed, w.seq_len, w.seq_len, w.n_heads, w.head_dim, w.fp8)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_keys(prm, k, ks)
    out = lsa.index_prefill(prm, q, wt, k, ks, bk, 0, n_kv=w.seq_len, runs=True)
    rows = slice(None) if n_rows is None else slice(w.seq_len - n_rows, w.seq_len)
    a = _attn_inputs(w, 0, w.seq_len, w.seq_len)
    qa, kv = P.bf16_dev(a["q"][rows]), P.bf16_dev(a["kv"])
    o1, l1 = lsa.sparse_attn(w.attn_params(), qa, kv, None, out["idx"][rows].contiguous(), out["count"][rows].contiguous())
    o2, l2 = lsa.sparse_attn_runs(w.attn_params(), qa, kv, out["runs"][rows].contiguous(), out["run_count"][rows].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_run_form_edge_runs():
    """Hand-made runs: out-of-range starts and runs crossing the cache end (those entries are
    skipped), a negative length (counts as 0), an empty row, and lists longer than the capacity
    (cut at k_cap, also after a run of 2^31 - 1 entries); each row equals the list form over the
    same expanded list."""
    from dataclasses import replace
    w = replace(W.SMALL_MLA, seq_len=600)
    n_kv, k_cap, B = w.seq_len, 96, 7
    a = _attn_inputs(w, 0, B, n_kv)
    runs = np.zeros((B, k_cap, 2), np.int32)
    rc = np.zeros(B, np.int32)
    spec = [[(0, 4), (100, 30), (590, 20)],             # the last run crosses the cache end
            [(-5, 10), (40, 1), (41, 7)],                # starts below 0
            [(10, 3), (20, -4), (30, 5)],                # a negative length
            [],                                          # empty row
            [(0, 50), (200, 50), (400, 50)],             # 150 entries: cut at k_cap = 96
            [(i * 7, 1) for i in range(90)],             # many single-entry runs
            [(3, 2 ** 31 - 1), (10, 5)]]                 # a length beyond any capacity: cut at k_cap
    idx = np.full((B, k_cap), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for b, rs in enumerate(spec):
        rc[b] = len(rs)
        lst = []
        for j, (st, ln) in enumerate(rs):
            runs[b, j] = (st, ln)
            lst += list(range(st, st + min(max(ln, 0), k_cap)))
        lst = lst[:k_cap]
        cnt[b] = len(lst)
        idx[b, :len(lst)] = lst
    qa, kv = P.bf16_dev(a["q"][:B]), P.bf16_dev(a["kv"])
    o1, l1 = lsa.sparse_attn(w.attn_params(), qa, kv, None, P.to_dev(idx), P.to_dev(cnt))
    o2, l2 = lsa.sparse_attn_runs(w.attn_params(), qa, kv, P.to_dev(runs), P.to_dev(rc))
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert torch.all(o2[3] == 0) and torch.all(torch.isneginf(l2[3]))


def test_run_form_mqa_and_paged_equal_list_form():
    """Run form where the runs are expanded into a list first: MQA over the L = 2048 workload's
    indexer runs, and paged MLA decode over the decode indexer's runs (permuted page table);
    each equals the list form bit for bit."""
    w = W.L2K_MQA
    inp = synth.indexer_inputs(w.seed, w.seq_len, w.seq_len, w.n_heads, w.head_dim, w.fp8)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    out = lsa.index_prefill(prm, q, wt, k, ks, lsa.block_keys(prm, k, ks), 0, n_kv=w.seq_len, runs=True)
    a = _attn_inputs(w, 0, w.seq_len, w.seq_len)
    qa, kv, v = P.bf16_dev(a["q"]), P.bf16_dev(a["kv"]), P.bf16_dev(a["v"])
    o1, l1 = lsa.sparse_attn(w.attn_params(), qa, kv, v, out["idx"], out["count"])
    o2, l2 = lsa.sparse_attn_runs(w.attn_params(), qa, kv, out["runs"], out["run_count"], v=v)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2), "MQA run form differs"

    wd = W.SMALL_DECODE
    H, dqk, dv = wd.attn_dims
    ctx, table, n_phys = synth.decode_layout(wd.seed, wd.batch, wd.ctx_lo, wd.ctx_hi, wd.kv_page)
    inp = synth.indexer_inputs(wd.seed, wd.batch, n_phys * wd.kv_page, wd.n_heads, wd.head_dim, wd.fp8)
    prm = wd.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, wd)
    dtab = P.to_dev(table)
    out = lsa.index_decode(prm, P.to_dev(ctx), dtab, wd.kv_page, n_phys, q, wt, k, ks, lsa.block_keys(prm, k, ks))
    a = synth.attention_inputs(wd.seed, 0, wd.batch, n_phys * wd.kv_page, H, dqk, dv, latent=True)
    qa, kv = P.bf16_dev(a["q"]), P.bf16_dev(a["kv"]).view(n_phys, wd.kv_page, dqk)
    o1, l1 = lsa.sparse_attn(wd.attn_params(), qa, kv, None, out["idx"], out["count"], page_table=dtab,
                             kv_page_size=wd.kv_page)
    o2, l2 = lsa.sparse_attn_runs(wd.attn_params(), qa, kv, out["runs"], out["run_count"], page_table=dtab,
                                  kv_page_size=wd.kv_page)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2), "paged run form differs"


def test_run_expansion_edge_runs_mqa():
    """The run expansion (MQA path) on hand-made runs: out-of-range starts, negative lengths, an
    empty row, a length of 2^31 - 1 and a run count above k_cap; equal to the list form."""
    from dataclasses import replace
    w = replace(W.L2K_MQA, seq_len=600)
    n_kv, k_cap, B = w.seq_len, 96, 6
    a = _attn_inputs(w, 0, B, n_kv)
    spec = [[(0, 4), (100, 30), (590, 20)],
            [(-5, 10), (40, 1), (41, 7)],
            [(10, 3), (20, -4), (30, 5)],
            [],
            [(3, 2 ** 31 - 1), (10, 5)],
            [(i * 5, 1) for i in range(k_cap)]]
    runs = np.zeros((B, k_cap, 2), np.int32)
    rc = np.zeros(B, np.int32)
    idx = np.full((B, k_cap), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for b, rs in enumerate(spec):
        rc[b] = len(rs) if b != B - 1 else k_cap + 7     # the last row claims more runs than fit
        lst = []
        for j, (st, ln) in enumerate(rs):
            runs[b, j] = (st, ln)
            lst += list(range(st, st + min(max(ln, 0), k_cap)))
        lst = lst[:k_cap]
        cnt[b] = len(lst)
        idx[b, :len(lst)] = lst
    qa, kv, v = P.bf16_dev(a["q"][:B]), P.bf16_dev(a["kv"]), P.bf16_dev(a["v"])
    o1, l1 = lsa.sparse_attn(w.attn_params(), qa, kv, v, P.to_dev(idx), P.to_dev(cnt))
    o2, l2 = lsa.sparse_attn_runs(w.attn_params(), qa, kv, P.to_dev(runs), P.to_dev(rc), v=v)
    torch.cuda.synchronize()
    for b in range(B):
        assert torch.equal(o1[b], o2[b]) and torch.equal(l1[b], l2[b]), f"row {b}"


def test_run_form_long_and_many_runs():
    """Run form over lists of up to 16448 entries (several LDS staging passes, runs straddling a
    pass boundary), with thousands of runs per row (several batches per thread), more long runs
    than the block-wide queue holds, run lengths around the short-run cut, and one run cut at
    k_cap that crosses the cache end; each row equals the list form bit for bit."""
    from dataclasses import replace
    w = replace(W.SMALL_MLA, seq_len=20000)
    n_kv, k_cap = w.seq_len, 16448
    spec = [[(13 * i, 6) for i in range(1500)],
            [(2 * i, 1) for i in range(2500)] + [(6000, 9000)],
            [],
            [(5000, 20000)],
            [(6 * i, 5) for i in range(3000)]]
    st = 0
    while sum(n for _, n in spec[2]) < 12000:
        ln = 1 + len(spec[2]) % 9
        spec[2].append((st, ln))
        st += ln + 1
    B = len(spec)
    a = _attn_inputs(w, 0, B, n_kv)
    runs = np.zeros((B, k_cap, 2), np.int32)
    rc = np.zeros(B, np.int32)
    idx = np.full((B, k_cap), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    for b, rs in enumerate(spec):
        rc[b] = len(rs)
        runs[b, :len(rs)] = rs
        lst = np.concatenate([np.arange(s0, s0 + n) for s0, n in rs])[:k_cap]
        cnt[b] = len(lst)
        idx[b, :len(lst)] = np.where(lst < n_kv, lst, -1)
    assert cnt.tolist() == [9000, 11500, 12006, 16448, 15000]
    qa, kv = P.bf16_dev(a["q"][:B]), P.bf16_dev(a["kv"])
    o1, l1 = lsa.sparse_attn(w.attn_params(), qa, kv, None, P.to_dev(idx), P.to_dev(cnt))
    o2, l2 = lsa.sparse_attn_runs(w.attn_params(), qa, kv, P.to_dev(runs), P.to_dev(rc))
    torch.cuda.synchronize()
    for b in range(B):
        assert torch.equal(o1[b], o2[b]) and torch.equal(l1[b], l2[b]), f"row {b} ({cnt[b]} entries, {rc[b]} runs)"


def test_cross_layer_reuse():
    """One index list feeds several layers (Sec. 3.2): each layer's output matches the oracle on
    its own Q and KV, and the shared list is left byte-identical."""
    w = W.SMALL_CLI
    n = w.seq_len
    rows = list(range(0, n, 41)) + [n - 1]
    idx, cnt = _oracle_index(w, rows, n)
    didx, dcnt = P.to_dev(idx), P.to_dev(cnt)
    before = didx.clone()
    for layer in range(w.layers):
        a = _attn_inputs(w, layer, n, n)
        q = P.bf16_dev(a["q"][rows])
        o, l = lsa.sparse_attn(w.attn_params(), q, P.bf16_dev(a["kv"]), None, didx, dcnt)
        torch.cuda.synchronize()
        _check_rows(w, a, rows, idx, cnt, o.float().cpu().numpy(), l.cpu().numpy())
    assert torch.equal(before, didx)


def test_paged_equals_contiguous_and_oracle():
    """Decode over a permuted page table equals the same rows attended in a contiguous cache, and
    matches the oracle on the logical rows."""
    w = W.SMALL_DECODE
    H, dqk, dv = w.attn_dims
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    a = synth.attention_inputs(w.seed, 0, w.batch, n_phys * w.kv_page, H, dqk, dv, latent=True)
    g = np.random.default_rng(2)
    idx = np.full((w.batch, w.k_cap), -1, np.int32)
    cnt = np.zeros(w.batch, np.int32)
    for b in range(w.batch):
        t = int(ctx[b]) - 1
        S = np.unique(np.concatenate([np.arange(w.k_sink), g.choice(t + 1, w.k_sparse, replace=False),
                                      np.arange(t - w.k_swa + 1, t + 1)]))
        idx[b, :S.size] = S
        cnt[b] = S.size
    kv_paged = P.bf16_dev(a["kv"]).view(n_phys, w.kv_page, dqk)
    q = P.bf16_dev(a["q"])
    o_p, l_p = lsa.sparse_attn(w.attn_params(), q, kv_paged, None, P.to_dev(idx), P.to_dev(cnt),
                               page_table=P.to_dev(table), kv_page_size=w.kv_page)
    # contiguous equivalent: translate positions to pool rows on the host
    phys_idx = np.full_like(idx, -1)
    for b in range(w.batch):
        S = idx[b, :cnt[b]]
        phys_idx[b, :cnt[b]] = table[b][S // w.kv_page] * w.kv_page + S % w.kv_page
    o_c, l_c = lsa.sparse_attn(w.attn_params(), q, P.bf16_dev(a["kv"]), None, P.to_dev(phys_idx), P.to_dev(cnt))
    torch.cuda.synchronize()
    assert torch.equal(o_p, o_c) and torch.equal(l_p, l_c)
    pool = a["kv"].reshape(n_phys, w.kv_page, dqk)
    for b in range(w.batch):
        t = int(ctx[b]) - 1
        kv_log = orc.logical_rows(pool, table[b], t + 1, w.kv_page)
        oref, lref = orc.attention_for_set(a["q"][b], kv_log, None, idx[b, :cnt[b]], dv, w.sm_scale)
        P.check_attention_row(o_p[b].float().cpu().numpy(), l_p[b].cpu().numpy(), oref, lref, f"seq {b}")


def test_attention_determinism():
    w = W.SMALL_MLA
    n = w.seq_len
    rows = list(range(0, n, 17))
    idx, cnt = _oracle_index(w, rows, n)
    a = _attn_inputs(w, 0, n, n)
    o1, l1 = _gpu_attn(w, a, rows, idx, cnt)
    o2, l2 = _gpu_attn(w, a, rows, idx, cnt)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


@pytest.mark.parametrize("w,q0,n_q", [(W.SMALL_MLA, 0, 1536), (W.SMALL_CLI, 0, 1536), (W.SMALL_CLI, 777, 999)],
                         ids=["small_mla", "small_cli", "small_cli_odd_chunk"])
def test_split_attention_parity(w, q0, n_q):
    """Split attention (listed non-window part and contiguous window on two streams, merged by
    log-sum-exp; the window part runs in the query-tiled kernel, two consecutive rows per
    workgroup sharing each window tile): every seventh row of a chunk against the oracle's Eq. (3)
    over the whole list, and every row against the fused kernel. The lists come from the oracle's
    indexer (the window part is read from the cache, not from the list, so the lists must hold the
    whole window: they do). Chunks: from position 0 (first rows shorter than the window), and an
    odd count of rows from an odd position (the last row pair holds one row); one row's list is
    emptied (count 0: no window either, o = 0 and lse = -inf as in the fused kernel)."""
    n = w.seq_len
    n_q = min(n - q0, n_q)
    rows = list(range(q0, q0 + n_q))
    idx, cnt = _oracle_index(w, rows, n)
    skipped = n_q // 2
    cnt = cnt.copy()
    cnt[skipped] = 0
    a = _attn_inputs(w, 0, n, n)
    q = P.bf16_dev(a["q"][rows])
    kv = P.bf16_dev(a["kv"])
    o, l = lsa.hfa_attn(w.attn_params(), q, kv, P.to_dev(idx), P.to_dev(cnt), q0, w.k_swa)
    of, lf = lsa.sparse_attn(w.attn_params(), q, kv, None, P.to_dev(idx), P.to_dev(cnt))
    torch.cuda.synchronize()
    o, l, of, lf = o.float().cpu().numpy(), l.cpu().numpy(), of.float().cpu().numpy(), lf.cpu().numpy()
    assert np.all(o[skipped] == 0) and np.all(np.isneginf(l[skipped])), "an empty list attends to nothing"
    assert np.all(of[skipped] == 0) and np.all(np.isneginf(lf[skipped]))
    sel = [i for i in list(range(0, n_q, 7)) + [n_q - 2, n_q - 1] if i != skipped]
    worst = _check_rows(w, a, [rows[i] for i in sel], idx[sel], cnt[sel], o[sel], l[sel])
    # against the fused kernel: two bf16 roundings of the same value apart at most
    keep = np.arange(n_q) != skipped
    assert np.max(np.abs(o[keep] - of[keep])) <= 2e-2, np.max(np.abs(o[keep] - of[keep]))
    assert np.max(np.abs(l[keep] - lf[keep])) <= 2e-3, np.max(np.abs(l[keep] - lf[keep]))
    print(w.name, q0, n_q, "worst vs oracle", worst, "max |hfa - fused|", float(np.max(np.abs(o[keep] - of[keep]))))


def test_binding_rejects_mismatched_tensors():
    """The C ABI sees bare pointers, so the binding checks every tensor against the sizes it passes
    (dtype, device, contiguity, shape) and raises before anything is launched."""
    w = W.SMALL_MLA
    n, k_cap = 64, 96
    prm = w.attn_params()
    a = _attn_inputs(w, 0, n, 300)
    q, kv = P.bf16_dev(a["q"][:n]), P.bf16_dev(a["kv"])
    idx = torch.zeros((n, k_cap), dtype=torch.int32, device=q.device)
    cnt = torch.ones((n,), dtype=torch.int32, device=q.device)
    lsa.sparse_attn(prm, q, kv, None, idx, cnt)   # the well-formed call works
    bad = {
        "idx dtype": lambda: lsa.sparse_attn(prm, q, kv, None, idx.long(), cnt),
        "idx rows": lambda: lsa.sparse_attn(prm, q, kv, None, idx[: n - 1], cnt),
        "count rows": lambda: lsa.sparse_attn(prm, q, kv, None, idx, cnt[: n - 1]),
        "q not contiguous": lambda: lsa.sparse_attn(prm, q.transpose(0, 1).contiguous().transpose(0, 1), kv, None,
                                                    idx, cnt),
        "kv width": lambda: lsa.sparse_attn(prm, q, kv[:, :512].contiguous(), None, idx, cnt),
        "out shape": lambda: lsa.sparse_attn(prm, q, kv, None, idx, cnt,
                                             out=torch.empty((n - 1, 64, 512), dtype=torch.bfloat16, device=q.device)),
        "kv on host": lambda: lsa.sparse_attn(prm, q, kv.cpu(), None, idx, cnt),
        "runs shape": lambda: lsa.sparse_attn_runs(prm, q, kv, torch.zeros((n, k_cap), dtype=torch.int32,
                                                                           device=q.device), cnt),
    }
    for name, call in bad.items():
        with pytest.raises(ValueError):
            call()
            pytest.fail(name)
    wi = W.SMALL_CLI
    iprm = wi.index_params()
    inp = synth.indexer_inputs(wi.seed, 256, 256, wi.n_heads, wi.head_dim, wi.fp8)
    qi, wt, k, ks = P.gpu_index_inputs(inp, wi)
    bk = lsa.block_keys(iprm, k, ks)
    with pytest.raises(ValueError):   # more cached tokens claimed than the key tensor holds
        lsa.index_prefill(iprm, qi, wt, k, ks, bk, 0, n_kv=k.shape[0] + 1)
    with pytest.raises(ValueError):   # head weights of the wrong dtype
        lsa.index_prefill(iprm, qi, wt.double(), k, ks, bk, 0)
    torch.cuda.synchronize()
