"""GPU parity of the LSA indexer (lsa_block_means, lsa_index_prefill, lsa_index_decode) against
the oracle, through the C-ABI. Inputs are seeded and synthetic (paper_2608_01662_amd.synth)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from dataclasses import replace

import oracle.lsa_oracle as orc
from paper_2608_01662_amd import lsa, synth
from paper_2608_01662_amd import workloads as W
from tests import parity as P

pytestmark = pytest.mark.gpu


def _sample_rows(n, every, extra=()):
    rows = set(range(0, n, every)) | {n - 1} | {r for r in extra if 0 <= r < n}
    return sorted(rows)


def _run_prefill(w, inp, q_start=0, n_q=None, pages=True):
    n_kv = inp["k"].shape[0]
    n_q = n_kv - q_start if n_q is None else n_q
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_keys(prm, k, ks) if w.keep_pages > 0 else None
    out = lsa.index_prefill(prm, q[q_start:q_start + n_q], wt[q_start:q_start + n_q], k, ks, bk, q_start,
                            n_kv=n_kv, runs=True, pages=pages)
    torch.cuda.synchronize()
    return {key: v.cpu().numpy() for key, v in out.items()}, bk


def _oracle_rows(w, inp, rows_t):
    prm = P.oracle_params(w)
    k_hat = P.oracle_keys(inp)
    k_mean = P.oracle_block_cache(w, k_hat) if w.keep_pages > 0 else None
    qf = orc.bf16_bits_to_f64(inp["q"])
    return [P.oracle_index_row(t, qf[t], inp["w"][t], k_hat, k_mean, prm) for t in rows_t]


# ----------------------------------------------------------------------------- mean keys
@pytest.mark.parametrize("fp8,B", [(False, 64), (True, 64), (True, 128), (True, 8), (False, 1)])
def test_block_means_parity(fp8, B):
    w = W.L2K_MQA if not fp8 else W.L32K_MLA
    n = 4096 + 37  # ragged: the trailing partial sub-block is not written
    inp = synth.indexer_inputs(5, 1, n, 1, w.head_dim, fp8)
    page = 32 if B == 1 else (128 if B > 64 else 64)
    prm = lsa.IndexParams(8, w.head_dim, fp8, page, B, 0, 16, 4, 128, 64)
    _, _, k, ks = P.gpu_index_inputs(inp, w)
    got = lsa.block_means(prm, k, ks).view(torch.int16).cpu().numpy().view(np.uint16)
    ref = orc.f64_to_bf16_bits(orc.sub_block_mean_keys(P.oracle_keys(inp), B))
    assert got.shape == ref.shape
    # fp32 accumulation vs float64: a value next to a bf16 rounding boundary may land one ulp away
    diff = np.abs(got.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 1 and (diff > 0).mean() < 1e-3, (diff.max(), (diff > 0).mean())


@pytest.mark.parametrize("fp8,B", [(True, 64), (True, 8), (False, 64), (False, 1)])
def test_block_minmax_parity(fp8, B):
    """Min-max block cache (Eq. 13): exact extrema rounded once to bf16, bit-exact."""
    w = W.L2K_MQA
    inp = synth.indexer_inputs(5, 8, 1000, w.n_heads, w.head_dim, fp8)
    prm = lsa.IndexParams(w.n_heads, w.head_dim, fp8, 32 if B == 1 else 64, B, 16, 256, 4, 128, 64, "minmax")
    k = P.to_dev(inp["k"]) if fp8 else P.bf16_dev(inp["k"])
    ks = P.to_dev(inp["k_scale"]) if fp8 else None
    got = lsa.block_minmax(prm, k, ks).view(torch.int16).cpu().numpy().view(np.uint16)
    k_max, k_min = orc.sub_block_minmax_keys(P.oracle_keys(inp), B)
    ref = np.concatenate([orc.f64_to_bf16_bits(k_max), orc.f64_to_bf16_bits(k_min)], axis=1)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("pooling", ["mean", "minmax"])
@pytest.mark.parametrize("fp8", [True, False])
def test_block_keys_update_after_append(pooling, fp8):
    """Decode appends tokens to a cache whose block cache already exists: updating the sub-blocks
    of the appended rows (a list with repeats and out-of-range rows, which are skipped) gives the
    cache a full recomputation gives, bit for bit; untouched sub-blocks keep their values."""
    w = W.L2K_MQA
    n = 1024
    inp = synth.indexer_inputs(6, 8, n, w.n_heads, w.head_dim, fp8)
    prm = lsa.IndexParams(w.n_heads, w.head_dim, fp8, 64, 8, 16, 256, 4, 128, 64, pooling)
    k = P.to_dev(inp["k"]) if fp8 else P.bf16_dev(inp["k"])
    ks = P.to_dev(inp["k_scale"]) if fp8 else None
    full0 = lsa.block_keys(prm, k, ks)
    # overwrite rows [700, 713) (the "appended" tokens) with other keys, then update
    other = synth.indexer_inputs(7, 8, n, w.n_heads, w.head_dim, fp8)
    new_rows = np.arange(700, 713)
    sel = torch.from_numpy(new_rows).to(k.device)
    k2 = (P.to_dev(other["k"]) if fp8 else P.bf16_dev(other["k"]))
    k[sel] = k2[sel]
    if fp8:
        ks[sel] = P.to_dev(other["k_scale"])[sel]
    block = full0.clone()
    rows = torch.tensor(np.concatenate([new_rows, [705, -3, n, n + 100]]), dtype=torch.int64, device=k.device)
    lsa.block_keys_update(prm, rows, k, ks, block)
    full1 = lsa.block_keys(prm, k, ks)
    torch.cuda.synchronize()
    assert torch.equal(block.view(torch.int16), full1.view(torch.int16))
    touched = set((new_rows // 8).tolist())
    for b in range(n // 8):
        if b not in touched:
            assert torch.equal(block[b].view(torch.int16), full0[b].view(torch.int16))


def test_fp8_decode_all_codes():
    """Mean keys with B = 1 and unit scales are the decoded codes: all 256 e4m3fn codes, exactly."""
    codes = np.arange(256, dtype=np.uint32).astype(np.uint8)
    codes = codes[(codes & 0x7F) != 0x7F]                                   # drop the two NaN codes
    codes = np.concatenate([codes, codes[:2]]).reshape(-1, 64)             # 4 rows of 64 (d_I = 64)
    prm = lsa.IndexParams(8, 64, True, 32, 1, 0, 16, 4, 128, 64)
    out = lsa.block_means(prm, P.to_dev(codes), P.to_dev(np.ones(codes.shape[0], np.float32)))
    got = orc.bf16_bits_to_f64(out.view(torch.int16).cpu().numpy().view(np.uint16))
    ref = orc.e4m3fn_to_f64(codes)                     # every code is exact in bf16
    assert np.array_equal(got, ref)                    # value equality: the sum of one -0 is +0


# ----------------------------------------------------------------------------- prefill
@pytest.mark.parametrize("w", [W.L2K_MQA, W.SMALL_FLAT, W.SMALL_MLA, W.SMALL_CLI, W.SMALL_SUBBLOCK, W.SMALL_MINMAX,
                               W.SMALL_MINMAX_B8], ids=lambda w: w.name)
def test_index_prefill_parity(w):
    inp = P.prefill_inputs(w)
    out, _ = _run_prefill(w, inp)
    n = w.seq_len
    every = 1 if n <= 2048 else 5
    boundary = [w.k_sink + w.k_swa - 1, w.k_sink + w.k_swa, w.k_sink + w.k_swa + 1,
                w.k_sink + w.k_swa + w.page, w.keep_pages * w.page + w.k_swa, n - 2]
    rows = _sample_rows(n, every, boundary)
    res = _oracle_rows(w, inp, rows)
    stats = P.check_index_rows(w, rows, out["idx"][rows], out["count"][rows],
                               out["pages"][rows] if "pages" in out else None, res)
    P.check_runs(out["runs"][rows], out["run_count"][rows], out["idx"][rows], out["count"][rows], w.run_align)
    # every row (not only the sampled ones): structure
    for t in range(0, n, 97):
        P.check_structure(out["idx"][t][: out["count"][t]], t, w)
    print(w.name, stats)


def test_coarse_long_rows():
    """Calls whose rows hold more than 64 coarse tiles use the four-wave coarse_kernel over four
    query rows (keys read straight into the operand layout) instead of the staged one-wave kernel:
    d_I = 64, 2-token sub-blocks in 64-token pages (32 per page) and L = 8192 give the last rows
    128 tiles of 32 sub-blocks (coarse_kernel<64, 4, false, false, false>). Sampled rows against
    the oracle, stage-wise."""
    from dataclasses import replace
    w = replace(W.SMALL_MLA, name="small_L8192_d64_B2", head_dim=64, sub_block=2, seq_len=8192)
    assert (w.seq_len // w.page) * (w.page // w.sub_block) // 32 > 64
    inp = P.prefill_inputs(w)
    out, _ = _run_prefill(w, inp)
    boundary = [w.k_sink + w.k_swa, w.k_sink + w.k_swa + w.page, w.keep_pages * w.page + w.k_swa, w.seq_len - 2]
    rows = _sample_rows(w.seq_len, 157, boundary)
    res = _oracle_rows(w, inp, rows)
    stats = P.check_index_rows(w, rows, out["idx"][rows], out["count"][rows], out["pages"][rows], res)
    P.check_runs(out["runs"][rows], out["run_count"][rows], out["idx"][rows], out["count"][rows], w.run_align)
    print(w.name, stats)


@pytest.mark.parametrize("base", [W.SMALL_FLAT, W.SMALL_MLA], ids=lambda w: w.name)
def test_flat_short_window_partial_page(base):
    """Flat mode with K_swa < P and a cache that ends inside a page: the page holding a row's last
    eligible positions also holds positions past the cache, whose key rows the fine stage stages
    (re-reading the last cached key) but never scores. Every row against the oracle."""
    from dataclasses import replace
    w = replace(base, keep_pages=0, k_swa=16, k_sparse=192, seq_len=1000)
    assert w.k_swa < w.page and w.seq_len % w.page != 0
    inp = P.prefill_inputs(w)
    out, _ = _run_prefill(w, inp, pages=False)
    rows = list(range(w.seq_len))
    res = _oracle_rows(w, inp, rows)
    stats = P.check_index_rows(w, rows, out["idx"], out["count"], None, res)
    P.check_runs(out["runs"], out["run_count"], out["idx"], out["count"], w.run_align)
    print(w.name, stats)


@pytest.mark.parametrize("keep_pages,k_sink,k_swa,k_sparse", [
    (0, 0, 0, 1),       # flat, no sink, no window (E_t = [0, t]), one sparse token
    (0, 0, 0, 300),     # flat, a budget above the early rows' candidate count
    (1, 0, 64, 1),      # hierarchical with one recalled page, the shortest window (K_swa = P)
    (1, 0, 64, 64),     # the whole recalled page selected
    (2, 1, 64, 100),    # one sink token, two pages, a budget above one page
], ids=["flat_1", "flat_300", "hi_m1_k1", "hi_m1_kP", "hi_m2_sink1"])
def test_degenerate_budgets(keep_pages, k_sink, k_swa, k_sparse):
    """Smallest legal budgets and windows: no sink, no window (flat mode), one recalled page,
    one sparse token, and budgets at or above the candidate count; every row against the oracle."""
    from dataclasses import replace
    w = replace(W.L2K_MQA, name=f"degenerate_{keep_pages}_{k_sink}_{k_swa}_{k_sparse}", seq_len=700,
                keep_pages=keep_pages, k_sink=k_sink, k_swa=k_swa, k_sparse=k_sparse)
    inp = P.prefill_inputs(w)
    out, _ = _run_prefill(w, inp, pages=keep_pages > 0)
    rows = list(range(w.seq_len))
    res = _oracle_rows(w, inp, rows)
    stats = P.check_index_rows(w, rows, out["idx"], out["count"], out["pages"] if keep_pages > 0 else None, res)
    P.check_runs(out["runs"], out["run_count"], out["idx"], out["count"], w.run_align)
    print(w.name, stats)


@pytest.mark.parametrize("keep_pages", [0, 600])
def test_select_from_global_keys(keep_pages):
    """Rows with more candidates than the LDS holds (here 45056 in flat mode, 38400 with M = 600
    pages) are selected by the kernel that reads the candidate keys from global memory in every
    pass: the last 384 query rows of a 45056-token cache against the oracle, stage-wise."""
    from dataclasses import replace
    w = replace(W.L32K_MLA, seq_len=45056, keep_pages=keep_pages, k_sparse=1024)
    inp = P.prefill_inputs(w)
    q0 = w.seq_len - 384
    out, _ = _run_prefill(w, inp, q_start=q0, pages=keep_pages > 0)
    rows = sorted(set(range(q0, w.seq_len, 9)) | {w.seq_len - 1})
    res = _oracle_rows(w, inp, rows)
    sel = [t - q0 for t in rows]
    stats = P.check_index_rows(w, rows, out["idx"][sel], out["count"][sel],
                               out["pages"][sel] if "pages" in out else None, res)
    P.check_runs(out["runs"][sel], out["run_count"][sel], out["idx"][sel], out["count"][sel], w.run_align)
    print(w.name, keep_pages, stats)


def test_adaptive_dispatch():
    """hi_min_kv >= n_kv: the hierarchical parameters run flat (the same output as keep_pages = 0,
    pages_out all -1); hi_min_kv < n_kv: the hierarchical output, unchanged."""
    from dataclasses import replace
    w = W.SMALL_CLI
    inp = P.prefill_inputs(w)
    hi, _ = _run_prefill(w, inp)
    flat, _ = _run_prefill(replace(w, keep_pages=0), inp, pages=False)
    auto_flat, _ = _run_prefill(replace(w, hi_min_kv=w.seq_len), inp)
    auto_hi, _ = _run_prefill(replace(w, hi_min_kv=w.seq_len - 1), inp)
    P.assert_same_index_outputs({k: v for k, v in auto_flat.items() if k != "pages"}, flat)
    P.assert_same_index_outputs(auto_hi, hi)
    assert np.all(auto_flat["pages"] == -1)
    assert np.array_equal(auto_hi["pages"], hi["pages"])
    assert not np.array_equal(hi["idx"], flat["idx"])      # the two modes do differ here


@pytest.mark.parametrize("head_dim,fp8,keep_pages,pooling", [
    (128, False, 8, "mean"), (128, False, 0, "mean"), (64, True, 8, "mean"), (64, True, 0, "mean"),
    (64, True, 8, "minmax"), (64, False, 8, "minmax")],
    ids=["d128_bf16_hi", "d128_bf16_flat", "d64_fp8_hi", "d64_fp8_flat", "d64_fp8_minmax", "d64_bf16_minmax"])
def test_index_prefill_other_key_formats(head_dim, fp8, keep_pages, pooling):
    """The kernel instances the five workloads do not reach: bf16 keys with d_I = 128 and fp8 keys
    with d_I = 64, hierarchical (coarse_kernel<D, 4, false, false>, page select, fine_xcd_kernel)
    and flat (flat_dense_kernel), and min-max pooling at d_I = 64 (coarse_kernel<64, 2, false,
    true>), against the oracle on sampled rows."""
    from dataclasses import replace
    w = replace(W.SMALL_CLI, name=f"small_d{head_dim}_{'fp8' if fp8 else 'bf16'}_m{keep_pages}_{pooling}",
                head_dim=head_dim, fp8=fp8, keep_pages=keep_pages, pooling=pooling, seq_len=4096)
    inp = P.prefill_inputs(w)
    out, _ = _run_prefill(w, inp, pages=keep_pages > 0)
    rows = _sample_rows(w.seq_len, 11, [w.k_sink + w.k_swa, w.k_sink + w.k_swa + w.page, w.seq_len - 2])
    res = _oracle_rows(w, inp, rows)
    stats = P.check_index_rows(w, rows, out["idx"][rows], out["count"][rows],
                               out["pages"][rows] if "pages" in out else None, res)
    P.check_runs(out["runs"][rows], out["run_count"][rows], out["idx"][rows], out["count"][rows], w.run_align)
    print(w.name, stats)


@pytest.mark.parametrize("base,keep_pages", [(W.L2K_MQA, 16), (W.L2K_MQA, 0), (W.SMALL_CLI, 8),
                                             (W.SMALL_MINMAX, 8), (W.SMALL_CLI, 0)],
                         ids=["mqa_hi", "mqa_flat", "cli_hi", "cli_minmax", "cli_flat"])
def test_signed_head_weights(base, keep_pages):
    """Head weights of either sign (Eq. 1: w is a learned projection): w ~ U(-1, 1), and every
    fifth row with all weights <= 0, so that all of its scores are <= 0. This runs the sign-aware
    order keys of the page and token selections and the ReLU of the coarse and fine stages on
    negative sums. Every row (L = 2048) or every third row (L = 8192) against the oracle,
    stage-wise."""
    from dataclasses import replace
    w = replace(base, keep_pages=keep_pages)
    inp = P.prefill_inputs(w, signed_weights=True)
    assert (inp["w"] < 0).any() and (inp["w"][::5] <= 0).all()
    out, _ = _run_prefill(w, inp, pages=keep_pages > 0)
    n = w.seq_len
    rows = _sample_rows(n, 1 if n <= 2048 else 3, [w.k_sink + w.k_swa, n - 2])
    res = _oracle_rows(w, inp, rows)
    neg = [r for r in res if r["score"].size and r["score"].max() <= 0]
    assert len(neg) >= len(res) // 6, "rows whose scores are all <= 0 must be part of the check"
    stats = P.check_index_rows(w, rows, out["idx"][rows], out["count"][rows],
                               out["pages"][rows] if "pages" in out else None, res)
    P.check_runs(out["runs"][rows], out["run_count"][rows], out["idx"][rows], out["count"][rows], w.run_align)
    print(w.name, keep_pages, stats, "all-non-positive rows", len(neg))


def _slots(w, n_kv):
    """Candidate slots per row of the fine-score workspace: M * P, or every page in flat mode."""
    return (w.keep_pages if w.keep_pages > 0 else -(-n_kv // w.page)) * w.page


@pytest.mark.parametrize("seq_len,lo,hi", [(12288, 8192, 16384), (36000, 32768, 36900)],
                         ids=["reg_kpt32", "lds_staged"])
def test_selection_instances(seq_len, lo, hi):
    """The two selection kernels no workload reaches. Flat indexing (Eq. 7) with P = 128 and the
    L = 128K budget (K_cap = 4 + 1024 + 2048):
      * L = 12288: 96 pages = 12288 candidate slots per row, served by
        token_select_reg_kernel<512, 32> (keys in registers, 8193..16384 slots);
      * L = 36000: 282 pages = 36096 slots, served by token_select_kernel<512, false> (keys staged
        in LDS: more than the 32768 register slots, and slots + K_cap within the 156 KB of LDS).
    The last 256 rows of the cache, every third one against the oracle."""
    from dataclasses import replace
    w = replace(W.L128K_CLI4, name=f"flat_L{seq_len}", seq_len=seq_len, keep_pages=0, layers=1)
    slots = _slots(w, seq_len)
    assert lo < slots <= hi, slots
    if seq_len > 32768:
        assert (slots + w.k_cap) * 4 <= 160 * 1024 - 4096   # keys (reused for the run scratch) + list fit in LDS
    inp = P.prefill_inputs(w)
    q0 = seq_len - 256
    out, _ = _run_prefill(w, inp, q_start=q0, pages=False)
    rows = sorted(set(range(q0, seq_len, 3)) | {seq_len - 1})
    res = _oracle_rows(w, inp, rows)
    sel = [t - q0 for t in rows]
    stats = P.check_index_rows(w, rows, out["idx"][sel], out["count"][sel], None, res)
    P.check_runs(out["runs"][sel], out["run_count"][sel], out["idx"][sel], out["count"][sel], w.run_align)
    print(w.name, slots, stats)


def test_keep_all_equals_flat_on_gpu():
    """With M >= #pages the hierarchical kernels must return exactly the flat selection."""
    w = W.SMALL_MLA
    inp = P.prefill_inputs(w)
    from dataclasses import replace
    flat, _ = _run_prefill(replace(w, keep_pages=0), inp, pages=False)
    keep, _ = _run_prefill(replace(w, keep_pages=w.seq_len // w.page), inp, pages=False)
    assert np.array_equal(flat["count"], keep["count"])
    assert np.array_equal(flat["idx"], keep["idx"])


def test_designed_inputs_select_latest():
    """Designed case: every head's query is +e_0 and key s has component 0 equal to the bf16 value
    with bit pattern 0x3F80 + s (strictly increasing and exact), all other components 0: every
    eligible token's score grows with s, so the sparse part is the latest K_sparse eligible
    positions; with constant keys, ties go to the earliest."""
    from dataclasses import replace
    w = replace(W.L2K_MQA, keep_pages=0, seq_len=1024)
    n, H, d = w.seq_len, w.n_heads, w.head_dim
    for mode in ("increasing", "constant"):
        q = np.zeros((n, H, d), np.float32)
        q[:, :, 0] = 1.0
        kb = np.zeros((n, d), np.uint16)
        kb[:, 0] = (0x3F80 + np.arange(n)) if mode == "increasing" else 0x3F80
        inp = dict(q=synth.to_bf16_bits(q), w=np.ones((n, H), np.float32), k=kb, k_scale=None)
        out, _ = _run_prefill(w, inp, pages=False)
        for t in range(w.k_sink + w.k_swa, n, 13):
            elig = np.arange(w.k_sink, t - w.k_swa + 1)
            want = elig[-w.k_sparse:] if mode == "increasing" else elig[:w.k_sparse]
            S = out["idx"][t][: out["count"][t]]
            assert np.array_equal(S[w.k_sink:S.size - w.k_swa], want), (mode, t)


@pytest.mark.parametrize("mode", ["two_values_outliers", "dense_cluster_outliers"])
def test_selection_clustered_scores(mode):
    """Designed scores for the selection's range histograms (Eq. 7 then Eq. 6): every head's query
    is +e_0 and w = 1, so a token's score is H times component 0 of its key. Every 61st token is
    an outlier (key 32768), which stretches the key range so far that the other scores share one or
    a few of the first pass's 512 bins:
      * two_values_outliers: the rest alternate between 1.0 and 1.0078125; the boundary bin holds
        hundreds of keys, the next pass narrows to those two values and then to ties of one value
        (the direct pass, take = rank still missing);
      * dense_cluster_outliers: the rest take the 128 bf16 values of [1, 2) in turn; the first
        pass's boundary bin holds several values with 64 ties each, the next pass gives each value
        its own bin and ranks the boundary value's ties.
    Flat indexing at L = 8192 (K_sparse = 256, every row's candidates in registers); sampled rows
    against the oracle, ties to the earlier position."""
    from dataclasses import replace
    w = replace(W.L2K_MQA, name=f"clustered_{mode}", keep_pages=0, seq_len=8192)
    n, H, d = w.seq_len, w.n_heads, w.head_dim
    q = np.zeros((n, H, d), np.float32)
    q[:, :, 0] = 1.0
    kb = np.zeros((n, d), np.uint16)
    s = np.arange(n)
    kb[:, 0] = 0x3F80 + (s % 2) if mode == "two_values_outliers" else 0x3F80 + (s % 128)
    kb[s % 61 == 5, 0] = 0x4700
    inp = dict(q=synth.to_bf16_bits(q), w=np.ones((n, H), np.float32), k=kb, k_scale=None)
    out, _ = _run_prefill(w, inp, pages=False)
    rows = sorted(set(range(w.k_sink + w.k_swa + w.k_sparse, n, 151)) | {n - 1})
    res = _oracle_rows(w, inp, rows)
    stats = P.check_index_rows(w, rows, out["idx"][rows], out["count"][rows], None, res)
    P.check_runs(out["runs"][rows], out["run_count"][rows], out["idx"][rows], out["count"][rows], w.run_align)
    assert stats["exact"] == stats["rows"], stats   # exact ties: both sides take the earliest positions
    print(mode, stats)


def test_fine_scoring_orders_every_fp8_code():
    """The fine stage widens fp8 keys to bf16 on the GPU. Designed case: each eligible token carries
    one distinct e4m3fn code in component 0 (all 254 non-NaN codes, in seeded random positions),
    every head's query is +e_0 and the scales are 1, so a token's score is H * ReLU(code value).
    Sweeping K_sparse over 1..126 (the positive codes) makes the selected set at every threshold
    the K largest decoded values: a code decoded wrongly (or a flushed denormal) changes the set."""
    from dataclasses import replace
    w0 = replace(W.L2K_MQA, fp8=True, keep_pages=0)
    d, H = w0.head_dim, w0.n_heads
    n_elig = 256
    n_kv = w0.k_sink + n_elig + w0.k_swa
    t = n_kv - 1
    codes = np.arange(256, dtype=np.int64)
    codes = codes[(codes & 0x7F) != 0x7F]
    codes = np.concatenate([codes, [0, 0x80]]).astype(np.uint8)
    codes = np.random.default_rng(7).permutation(codes)
    k8 = np.zeros((n_kv, d), np.uint8)
    k8[w0.k_sink:w0.k_sink + n_elig, 0] = codes
    vals = orc.e4m3fn_to_f64(codes)
    order = np.lexsort((np.arange(n_elig), -vals))        # value desc, position asc
    q = np.zeros((1, H, d), np.float32)
    q[:, :, 0] = 1.0
    qd, wd = P.bf16_dev(synth.to_bf16_bits(q)), P.to_dev(np.ones((1, H), np.float32))
    kd, ksd = P.to_dev(k8), P.to_dev(np.ones(n_kv, np.float32))
    n_pos = int((vals > 0).sum())
    assert n_pos == 126
    for K in range(1, n_pos + 1):
        prm = replace(w0, k_sparse=K).index_params()
        out = lsa.index_prefill(prm, qd, wd, kd, ksd, None, t, n_kv=n_kv, runs=False)
        S = out["idx"][0][: int(out["count"][0])].cpu().numpy()
        sparse = S[w0.k_sink:S.size - w0.k_swa]
        want = np.sort(order[:K] + w0.k_sink)
        assert np.array_equal(sparse, want), K


def test_chunked_equals_single_call():
    """Rows of a chunked prefill equal the same rows of one call over the whole sequence."""
    w = W.SMALL_CHUNKED
    inp = P.prefill_inputs(w)
    whole, _ = _run_prefill(w, inp)
    for q0 in range(0, w.seq_len, w.chunk):
        nq = min(w.chunk, w.seq_len - q0)
        part, _ = _run_prefill(w, inp, q_start=q0, n_q=nq)
        P.assert_same_index_outputs(part, whole, slice(q0, q0 + nq))


def test_chunked_parity_sampled():
    w = W.SMALL_CHUNKED
    inp = P.prefill_inputs(w)
    q0 = 9000
    out, _ = _run_prefill(w, inp, q_start=q0, n_q=w.chunk)
    rows = list(range(0, w.chunk, 7)) + [w.chunk - 1]
    res = _oracle_rows(w, inp, [q0 + r for r in rows])
    P.check_index_rows(w, [q0 + r for r in rows], out["idx"][rows], out["count"][rows], out["pages"][rows], res)


def test_determinism():
    w = W.SMALL_MLA
    inp = P.prefill_inputs(w)
    a, _ = _run_prefill(w, inp)
    b, _ = _run_prefill(w, inp)
    P.assert_same_index_outputs(a, b)


def test_empty_and_tiny():
    w = W.L2K_MQA
    inp = synth.indexer_inputs(9, 40, 40, w.n_heads, w.head_dim, False)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_means(prm, k, ks)
    # zero rows: nothing launched, nothing written
    out = lsa.index_prefill(prm, q[:0], wt[:0], k, ks, bk, 0, n_kv=40)
    assert out["idx"].shape == (0, w.k_cap)
    # every row shorter than sink + window: S_t = [0, t]
    out = lsa.index_prefill(prm, q, wt, k, ks, bk, 0, n_kv=40)
    torch.cuda.synchronize()
    for t in range(40):
        assert out["count"][t].item() == t + 1
        assert np.array_equal(out["idx"][t, :t + 1].cpu().numpy(), np.arange(t + 1))


# ----------------------------------------------------------------------------- decode (paged)
def _decode_case(w, signed_weights=False):
    ctx, table, n_phys = synth.decode_layout(w.seed, w.batch, w.ctx_lo, w.ctx_hi, w.kv_page)
    inp = synth.indexer_inputs(w.seed, w.batch, n_phys * w.kv_page, w.n_heads, w.head_dim, w.fp8, signed_weights)
    return ctx, table, n_phys, inp


_DECODE_D64 = replace(W.SMALL_DECODE, name="small_decode_b8_d64_fp8", head_dim=64)
_DECODE_D64_MINMAX = replace(W.SMALL_DECODE_MINMAX, name="small_decode_b8_d64_bf16_minmax", head_dim=64, fp8=False)
_DECODE_BF16 = replace(W.SMALL_DECODE, name="small_decode_b8_bf16", fp8=False)
_DECODE_FLAT = replace(W.SMALL_DECODE, name="small_decode_b8_flat", keep_pages=0)


@pytest.mark.parametrize("w,signed", [(W.SMALL_DECODE, False), (W.SMALL_DECODE_MINMAX, False), (_DECODE_D64, False),
                                      (_DECODE_D64_MINMAX, False), (W.SMALL_DECODE, True), (_DECODE_BF16, False),
                                      (_DECODE_FLAT, False)],
                         ids=["mean", "minmax", "d64_fp8", "d64_bf16_minmax", "signed_w", "bf16", "flat"])
def test_index_decode_parity(w, signed):
    """Paged decode indexer against the oracle on every sequence. The d_I = 64 cases run the paged
    coarse instances coarse_kernel<64, 1, true, false / true> and fine_kernel<64, fp8 / bf16>;
    bf16 runs fine_kernel<128, bf16>; flat (keep_pages = 0) runs the fine kernel over every eligible
    page, looked up in the page table, and the selection over all of them; signed_w draws head
    weights of either sign (two of the eight sequences with all weights <= 0)."""
    ctx, table, n_phys, inp = _decode_case(w, signed)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    hier = w.keep_pages > 0
    bk = lsa.block_keys(prm, k, ks) if hier else None
    out = lsa.index_decode(prm, P.to_dev(ctx), P.to_dev(table), w.kv_page, n_phys, q, wt, k, ks, bk, pages=hier)
    torch.cuda.synchronize()
    out = {key: v.cpu().numpy() for key, v in out.items()}
    prmo = P.oracle_params(w)
    k_hat_pool = P.oracle_keys(inp).reshape(n_phys, w.kv_page, -1)
    qf = orc.bf16_bits_to_f64(inp["q"])
    rows_t, res = [], []
    for b in range(w.batch):
        t = int(ctx[b]) - 1
        k_log = orc.logical_rows(k_hat_pool, table[b], t + 1, w.kv_page)
        k_mean = P.oracle_block_cache(w, k_log)
        res.append(P.oracle_index_row(t, qf[b], inp["w"][b], k_log, k_mean, prmo))
        rows_t.append(t)
    P.check_index_rows(w, rows_t, out["idx"], out["count"], out.get("pages"), res)
    P.check_runs(out["runs"], out["run_count"], out["idx"], out["count"], w.run_align)


def test_decode_bad_rows_are_skipped():
    """Out-of-range context lengths give count 0 (no fault, nothing selected)."""
    w = W.SMALL_DECODE
    ctx, table, n_phys, inp = _decode_case(w)
    ctx = ctx.copy()
    ctx[0] = 0
    ctx[1] = table.shape[1] * w.kv_page + 1
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_keys(prm, k, ks)
    out = lsa.index_decode(prm, P.to_dev(ctx), P.to_dev(table), w.kv_page, n_phys, q, wt, k, ks, bk)
    torch.cuda.synchronize()
    assert out["count"][0].item() == 0 and out["count"][1].item() == 0
    assert out["count"][2].item() > 0


def test_decode_bad_page_table_entries():
    """Page-table entries outside [0, n_phys) (here -1 and n_phys) in one sequence's eligible range:
    the pages they name are scored 0 and never give a token to the sparse part (their key rows are
    never read), the row keeps its sink, its window and a full sparse part from its other pages,
    and every other sequence's output is unchanged. The paged attention over the result reads only
    mapped rows (finite output for the row)."""
    w = W.SMALL_DECODE
    ctx, table, n_phys, inp = _decode_case(w)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_keys(prm, k, ks)
    good = lsa.index_decode(prm, P.to_dev(ctx), P.to_dev(table), w.kv_page, n_phys, q, wt, k, ks, bk)
    r = 3
    t = int(ctx[r]) - 1
    hi_page = (t - w.k_swa) // w.kv_page
    bad = [hi_page // 3, (2 * hi_page) // 3]
    assert 0 < bad[0] < bad[1] < hi_page
    tab = table.copy()
    tab[r, bad[0]] = -1
    tab[r, bad[1]] = n_phys
    dtab = P.to_dev(tab)
    out = lsa.index_decode(prm, P.to_dev(ctx), dtab, w.kv_page, n_phys, q, wt, k, ks, bk)
    torch.cuda.synchronize()
    gi, gc = good["idx"].cpu().numpy(), good["count"].cpu().numpy()
    idx, cnt = out["idx"].cpu().numpy(), out["count"].cpu().numpy()
    for b in range(w.batch):
        if b != r:
            assert cnt[b] == gc[b] and np.array_equal(idx[b], gi[b]), f"sequence {b} changed"
    S = idx[r][: cnt[r]]
    assert cnt[r] == gc[r] == w.k_sink + w.k_swa + w.k_sparse
    for p in bad:
        assert not np.any((S >= p * w.kv_page) & (S < (p + 1) * w.kv_page)), f"token of unmapped page {p} selected"
    assert set(range(w.k_sink)) <= set(S.tolist()) and set(range(t - w.k_swa + 1, t + 1)) <= set(S.tolist())
    H, dqk, dv = w.attn_dims
    a = synth.attention_inputs(w.seed, 0, w.batch, n_phys * w.kv_page, H, dqk, dv, latent=True)
    qa, kv = P.bf16_dev(a["q"]), P.bf16_dev(a["kv"]).view(n_phys, w.kv_page, dqk)
    o, l = lsa.sparse_attn(w.attn_params(), qa, kv, None, out["idx"], out["count"], page_table=dtab,
                           kv_page_size=w.kv_page)
    torch.cuda.synchronize()
    assert torch.isfinite(o[r].float()).all() and torch.isfinite(l[r]).all()


@pytest.mark.parametrize("w", [W.SMALL_DECODE, W.SMALL_DECODE_MINMAX], ids=lambda w: w.name)
def test_decode_short_contexts(w):
    """Paged decode at the context lengths where the streaming split changes shape: one token,
    shorter than sink + window, exactly sink + window (E_t empty), one past it, page edges, and
    just above M * P eligible tokens (the first context whose pages are not all recalled). Indexer
    and paged attention against the oracle, row by row."""
    P_ = w.kv_page
    kw = w.k_sink + w.k_swa
    ctx = np.array([1, 2, w.k_sink + 1, kw - 1, kw, kw + 1, P_, P_ + 1, 2 * P_ + kw, 3 * P_,
                    w.keep_pages * P_ + kw, w.keep_pages * P_ + kw + P_ + 1], np.int32)
    B = ctx.size
    n_pages = (ctx + P_ - 1) // P_
    n_phys = int(n_pages.sum())
    perm = np.random.default_rng(11).permutation(n_phys).astype(np.int32)
    table = np.full((B, int(n_pages.max())), -1, np.int32)
    off = 0
    for b in range(B):
        table[b, :n_pages[b]] = perm[off:off + n_pages[b]]
        off += n_pages[b]
    inp = synth.indexer_inputs(w.seed + 7, B, n_phys * P_, w.n_heads, w.head_dim, w.fp8)
    prm = w.index_params()
    q, wt, k, ks = P.gpu_index_inputs(inp, w)
    bk = lsa.block_keys(prm, k, ks)
    out = lsa.index_decode(prm, P.to_dev(ctx), P.to_dev(table), P_, n_phys, q, wt, k, ks, bk, pages=True)
    torch.cuda.synchronize()
    res_dev = {key: v for key, v in out.items()}
    out = {key: v.cpu().numpy() for key, v in out.items()}
    prmo = P.oracle_params(w)
    k_hat_pool = P.oracle_keys(inp).reshape(n_phys, P_, -1)
    qf = orc.bf16_bits_to_f64(inp["q"])
    rows_t, res = [], []
    for b in range(B):
        t = int(ctx[b]) - 1
        k_log = orc.logical_rows(k_hat_pool, table[b], t + 1, P_)
        res.append(P.oracle_index_row(t, qf[b], inp["w"][b], k_log, P.oracle_block_cache(w, k_log), prmo))
        rows_t.append(t)
    P.check_index_rows(w, rows_t, out["idx"], out["count"], out["pages"], res)
    P.check_runs(out["runs"], out["run_count"], out["idx"], out["count"], w.run_align)
    assert out["count"][0] == 1 and out["idx"][0, 0] == 0
    # paged attention over those index lists
    H, dqk, dv = w.attn_dims
    a = synth.attention_inputs(w.seed + 7, 0, B, n_phys * P_, H, dqk, dv, latent=True)
    o, lse = lsa.sparse_attn(w.attn_params(), P.bf16_dev(a["q"]), P.bf16_dev(a["kv"]).view(n_phys, P_, dqk), None,
                             res_dev["idx"], res_dev["count"], page_table=P.to_dev(table), kv_page_size=P_)
    torch.cuda.synchronize()
    pool = a["kv"].reshape(n_phys, P_, dqk)
    for b in range(B):
        t = int(ctx[b]) - 1
        kv_log = orc.logical_rows(pool, table[b], t + 1, P_)
        oref, lref = orc.attention_for_set(a["q"][b], kv_log, None, out["idx"][b, :out["count"][b]], dv, w.sm_scale)
        P.check_attention_row(o[b].float().cpu().numpy(), lse[b].cpu().numpy(), oref, lref, f"seq {b} (ctx {ctx[b]})")
