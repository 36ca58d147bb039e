"""Comparison rules between the HIP path and the oracle, and shared test plumbing.

Index sets: the sink and window parts must match exactly. The selected parts must have the same
size, and every element of their symmetric difference must have an oracle score within
tol * |tau| of tau, the oracle's k-th largest score (a tie, up to the float32 rounding of the GPU
scores). The hierarchical indexer is checked stage by stage: recalled pages first (same rule on
page scores), then the final selection against the oracle's fine stage run on the pages the GPU
recalled (the oracle's own pages, or the GPU's where the two differ by a page-score tie).

Attention: per row max|delta| <= 2e-2 and ||delta||_F / ||o_ref||_F <= 1e-2 (bf16 output,
fp32 accumulation); log-sum-exp within 2e-3 absolute.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle.lsa_oracle as orc
from paper_2608_01662_amd import synth

TOL_SCORE = 1e-3
ATOL_O, RTOL_O, ATOL_LSE = 2e-2, 1e-2, 2e-3


def oracle_params(w) -> orc.IndexParams:
    return orc.IndexParams(page=w.page, sub_block=w.sub_block, keep_pages=w.keep_pages, k_sparse=w.k_sparse,
                           k_sink=w.k_sink, k_swa=w.k_swa, run_align=w.run_align, pooling=w.pooling)


def oracle_block_cache(w, k_hat):
    """The oracle's Stage 1 cache for workload w: mean keys, or (k_max, k_min) with min-max pooling."""
    if w.pooling == "minmax":
        return orc.sub_block_minmax_keys(k_hat, w.sub_block)
    return orc.sub_block_mean_keys(k_hat, w.sub_block)


def tie_equivalent(gpu_sel, orc_sel, ids, scores, k, tol=TOL_SCORE) -> int:
    """Returns the size of the symmetric difference; raises AssertionError if it is not made of
    near-ties of the oracle's k-th score."""
    g, o = set(np.asarray(gpu_sel).tolist()), set(np.asarray(orc_sel).tolist())
    assert len(g) == len(gpu_sel), "duplicate entries in the GPU selection"
    assert len(g) == len(o), f"selection sizes differ: gpu {len(g)} oracle {len(o)}"
    diff = g ^ o
    if not diff:
        return 0
    score_of = dict(zip(np.asarray(ids).tolist(), np.asarray(scores).tolist()))
    assert diff <= set(score_of), f"GPU selected non-candidates {sorted(diff - set(score_of))[:8]}"
    tau = float(np.sort(np.asarray(scores, np.float64))[::-1][k - 1])
    for x in diff:
        gap = abs(score_of[x] - tau)
        assert gap <= tol * abs(tau) if tau != 0 else gap == 0, \
            f"element {x} score {score_of[x]!r} is not a tie of threshold {tau!r}"
    return len(diff)


def check_structure(S, t, w):
    """Eq. (6): ascending, unique, within [0, t], sink and window present, right size."""
    S = np.asarray(S)
    assert np.all(np.diff(S) > 0), "index list not strictly ascending"
    assert S.size == 0 or (S[0] >= 0 and S[-1] <= t)
    n_elig = max(0, t - w.k_swa - w.k_sink + 1)
    cand = n_elig
    want = min(t + 1, w.k_sink + w.k_swa + min(w.k_sparse, cand))
    if w.keep_pages <= 0 or n_elig == 0:
        assert S.size == want, f"row t={t}: count {S.size} != {want}"
    else:
        assert S.size <= want
    sset = set(S.tolist())
    assert set(range(min(w.k_sink, t + 1))) <= sset, "sink missing"
    assert set(range(max(0, t - w.k_swa + 1), t + 1)) <= sset, "window missing"


def oracle_index_row(t, q_t, w_t, k_hat, k_mean, prm):
    """The oracle's index row for position t (Eq. 6-7, 9-12), with a `rerun` entry that repeats
    the fine stage (Eq. 11-12, oracle steps 5-8) on another page list, so that a row whose
    recalled pages differ from the oracle's by a tie can be checked on the pages the GPU recalled."""
    r = orc.index_row(t, q_t, w_t, k_hat, k_mean, prm)
    r["rerun"] = lambda pages: orc.index_row(t, q_t, w_t, k_hat, k_mean, prm, pages_override=pages)
    return r


def _check_fine_stage(w, t, S, r, k_sparse):
    """Fixed parts exact, sparse part tie-equivalent to the oracle's on the same candidates."""
    ks, kw_ = w.k_sink, w.k_swa
    assert S.size == r["S"].size, f"row t={t}: count {S.size} != oracle {r['S'].size}"
    assert np.array_equal(S[:ks], r["S"][:ks]), f"row t={t}: sink part differs"
    assert np.array_equal(S[S.size - kw_:], r["S"][r["S"].size - kw_:]), f"row t={t}: window part differs"
    tie_equivalent(S[ks:S.size - kw_], r["sparse"], r["cand"], r["score"], k_sparse)


def check_index_rows(w, rows_t, gpu_idx, gpu_cnt, gpu_pages, results, allow_page_tie_frac=0.02):
    """Stage-wise comparison of GPU index rows with oracle results (one dict per row, from
    oracle_index_row). Hierarchical rows: the recalled pages are compared first (tie rule on the
    page scores, Eq. 9-10); where they differ by a tie, the oracle's fine stage is run again on
    the GPU's pages and the final selection is compared with that (Eq. 11-12), so a tie at the
    page threshold cannot hide an error of the fine stage."""
    prm = oracle_params(w)
    stats = dict(rows=0, exact=0, page_tie_rows=0, token_tie_rows=0)
    for i, (t, r) in enumerate(zip(rows_t, results)):
        S = np.asarray(gpu_idx[i][: int(gpu_cnt[i])])
        assert np.all(np.asarray(gpu_idx[i][int(gpu_cnt[i]):]) == -1), f"row t={t}: padding not -1"
        check_structure(S, t, w)
        stats["rows"] += 1
        if r["pages"] is not None and gpu_pages is not None:
            gp = np.asarray(gpu_pages[i])
            gp = gp[gp >= 0]
            if not np.array_equal(gp, r["pages"]):
                tie_equivalent(gp, r["pages"], r["page_ids"], r["page_score"], w.keep_pages)
                assert "rerun" in r, f"row t={t}: recalled pages differ by a tie, and no oracle rerun is available"
                r = r["rerun"](gp)
                stats["page_tie_rows"] += 1
        if np.array_equal(S, r["S"]):
            stats["exact"] += 1
            continue
        _check_fine_stage(w, t, S, r, prm.k_sparse)
        stats["token_tie_rows"] += 1
    assert stats["page_tie_rows"] <= allow_page_tie_frac * max(1, stats["rows"]) + 1, stats
    return stats


def check_runs(gpu_runs, gpu_run_count, gpu_idx, gpu_cnt, C):
    """Runs must be exactly the oracle's re-encoding of the GPU's own index list (entries past the
    run count are not part of the output)."""
    for i in range(len(gpu_cnt)):
        S = np.asarray(gpu_idx[i][: int(gpu_cnt[i])])
        want = orc.runs_of(S, C)
        n = int(gpu_run_count[i])
        got = [tuple(x) for x in np.asarray(gpu_runs[i][:n]).tolist()]
        assert got == want, f"row {i}: runs differ"


def assert_same_index_outputs(a, b, rows=None):
    """Two index outputs (dicts of numpy arrays) are identical: every array exactly, except runs,
    which only count up to each row's run count (entries past it are not written)."""
    sel = slice(None) if rows is None else rows
    assert set(a) == set(b), (sorted(a), sorted(b))
    for key in a:
        if key == "runs":
            continue
        assert np.array_equal(a[key], b[key][sel]), key
    if "runs" in a:
        ra, rb, n = a["runs"], b["runs"][sel], a["run_count"]
        for i in range(len(n)):
            assert np.array_equal(ra[i][: n[i]], rb[i][: n[i]]), f"runs of row {i}"


def check_attention_row(o_gpu, lse_gpu, o_ref, lse_ref, where=""):
    o_gpu = np.asarray(o_gpu, np.float64)
    d = o_gpu - o_ref
    mx = float(np.abs(d).max())
    rel = float(np.linalg.norm(d) / max(np.linalg.norm(o_ref), 1e-30))
    assert mx <= ATOL_O and rel <= RTOL_O, f"{where}: max|d|={mx:.3g} rel={rel:.3g}"
    if lse_gpu is not None:
        dl = float(np.abs(np.asarray(lse_gpu, np.float64) - lse_ref).max())
        assert dl <= ATOL_LSE, f"{where}: lse error {dl:.3g}"
    return mx, rel


# ----------------------------------------------------------------------------- input plumbing
def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.view(dtype)
    return t.cuda()


def bf16_dev(bits):
    return to_dev(bits.view(np.int16), torch.bfloat16)


def oracle_keys(inp):
    return orc.dequantized_keys(inp["k"], inp["k_scale"])


def gpu_index_inputs(inp, w):
    q = bf16_dev(inp["q"])
    wt = to_dev(inp["w"])
    if w.fp8:
        k = to_dev(inp["k"])
        ks = to_dev(inp["k_scale"])
    else:
        k = bf16_dev(inp["k"])
        ks = None
    return q, wt, k, ks


def prefill_inputs(w, n_kv=None, signed_weights=False):
    n_kv = n_kv or w.seq_len
    return synth.indexer_inputs(w.seed, n_kv, n_kv, w.n_heads, w.head_dim, w.fp8, signed_weights)
