"""Oracle for the LongCat Sparse Attention (LSA) hot path: a plain, slow, float64 CPU reference.

TEST INFRASTRUCTURE ONLY. The tests, the smoke check and the benchmark's CPU-baseline leg are
the only code allowed to import this module. The product path (the HIP library and its Python
binding) never calls it, and this module imports nothing from the product path.

What it computes, following "LongCat Sparse Attention: Taming the Lightning via Streaming-aware
Hierarchical Cross-Layer Indexing" (arXiv 2608.01662):

  * Sec. 2.2, Eq. (1): lightning-indexer score  I_{t,s} = sum_j w_{t,j} ReLU(q_{t,j} . k_s)
    with one key shared by all indexer heads (MQA).
  * Sec. 2.2, Eq. (2)-(3): top-K selection and attention restricted to the selected set; the
    MLA latent vector c_s serves as key (all d_qk columns) and value (first d_v columns).
  * Sec. 3.1, Eq. (6)-(7): streaming-aware budget: S_t = S_sink u S_swa u S_sparse, with the
    sparse part chosen by top-K_sparse over positions outside sink and window.
  * Sec. 3.3, Eq. (9)-(12): hierarchical indexing: per-sub-block mean keys, coarse page score,
    top-M pages, fine token score over the recalled pages, final top-K_sparse.
  * Eq. (13), the pooling ablation of hierarchical indexing: min-max pooling, a block score from
    the per-dimension extrema of the sub-block's keys in place of the mean-key dot product.
  * Sec. 3.2 and Sec. 4.1: cross-layer indexing has nothing to compute: the owner layer's S_t is
    passed unchanged to every layer of the group.

Hierarchical indexing is an approximation of Eq. (7), so `index_row` takes the algorithm's steps
in the paper's order (Eq. 9 -> 10 -> 11 -> 12). With all pages kept (M >= #eligible pages, or
flat mode) the steps collapse to the plain definition, Eq. (7).

Readings taken where the paper is silent or 1-based:
  * positions are 0-based: sink = [0, K_sink), window = [t-K_swa+1, t], eligible range
    E_t = [K_sink, t-K_swa]; when E_t is empty, S_t = [0, t].
  * the sparse part selects K_sparse tokens (Eq. 12 names K_sparse); the index-list capacity is
    K_cap = K_sink + K_swa + K_sparse.
  * the coarse stage scores only pages holding at least one eligible token; other pages could
    contribute no candidate (Eq. 7 excludes sink and window).
  * the mean keys are the per-dimension mean of the dequantised keys of a sub-block, stored
    in bfloat16 with one round-to-nearest-even (Stage 1 caches them); the
    extrema of min-max pooling are stored the same way.
  * both top-K operations order by (score descending, position ascending).
  * fp8 keys are OCP e4m3fn codes times a per-token fp32 scale.
  * runs re-encode S_t: maximal stretches of consecutive positions, cut at multiples of C; the
    set itself is unchanged.
  * the log-sum-exp output uses the natural logarithm.

Every function here is pinned by a CPU test against something other than itself (a library
routine, a closed form, brute force, or an invariant); see tests/test_oracle_*.py.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

# ============================================================================ number formats


def bf16_bits_to_f64(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float64. Exact: a bfloat16 is the top half of a float32."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):          # NaN patterns stay NaN
        return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x) -> np.ndarray:
    """Round float64 values to bfloat16 (nearest, ties to even) in one step; return bit patterns.

    bfloat16 keeps 8 significant bits, exponent range of float32, subnormal quantum 2**-133.
    Rounding straight from float64 avoids the double rounding of a float32 detour.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.zeros(x.shape, dtype=np.uint16)
    finite = np.isfinite(x) & (x != 0)
    xf = x[finite]
    _, e = np.frexp(xf)                      # |x| = m * 2**e, 0.5 <= m < 1
    qe = np.maximum(e - 8, -133)             # exponent of one unit in the last place
    y = np.ldexp(np.rint(np.ldexp(xf, -qe)), qe)   # np.rint rounds half to even
    y32 = y.astype(np.float32)               # exact (or inf on overflow past the largest bf16)
    out[finite] = (y32.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    zeros = x == 0
    out[zeros] = np.where(np.signbit(x[zeros]), 0x8000, 0x0000).astype(np.uint16)
    infs = np.isinf(x)
    out[infs] = np.where(x[infs] > 0, 0x7F80, 0xFF80).astype(np.uint16)
    out[np.isnan(x)] = 0x7FC0
    return out


def e4m3fn_to_f64(codes) -> np.ndarray:
    """OCP 8-bit float E4M3 ("fn": no infinities) -> float64.

    1 sign bit, 4 exponent bits (bias 7), 3 mantissa bits; exponent 0 is subnormal
    (m * 2**-9); the code with all exponent and mantissa bits set is NaN.
    """
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & ((c & 0x7) == 7), np.nan, mag)
    return sign * mag


def dequantized_keys(k, k_scale=None) -> np.ndarray:
    """Indexer key cache -> float64 keys k_s [n, d].

    bfloat16 keys (uint16 bit patterns) decode directly; fp8 keys (uint8 e4m3fn codes) are
    multiplied by their per-token scale, an exact product in float64.
    """
    k = np.asarray(k)
    if k.dtype == np.uint16:
        return bf16_bits_to_f64(k)
    if k.dtype == np.uint8:
        if k_scale is None:
            raise ValueError("fp8 keys need a per-token scale")
        return e4m3fn_to_f64(k) * np.asarray(k_scale, dtype=np.float32).astype(np.float64)[:, None]
    raise TypeError(f"unsupported key storage {k.dtype}")


# ============================================================================ parameters


@dataclass(frozen=True)
class IndexParams:
    """Hyper-parameters of one LSA indexer (Sec. 3.1 and Sec. 3.3)."""
    page: int            # P, page size of the coarse stage
    sub_block: int       # B, sub-block size of the mean keys; B divides P
    keep_pages: int      # M, pages recalled by the coarse stage; <= 0 means flat (no coarse stage)
    k_sparse: int        # K_sparse
    k_sink: int          # K_sink
    k_swa: int           # K_swa
    run_align: int       # C, runs never cross a multiple of C
    pooling: str = "mean"  # coarse-stage block summary: "mean" (Eq. 9) or "minmax" (Eq. 13)

    @property
    def k_cap(self) -> int:
        return self.k_sink + self.k_swa + self.k_sparse


# ============================================================================ indexer steps


def indexer_scores(q_t, w_t, keys) -> np.ndarray:
    """Eq. (1) / Eq. (11): I_{t,s} = sum_j w_{t,j} ReLU(q_{t,j} . k_s) for every row k_s of `keys`.

    q_t [H_I, d], w_t [H_I], keys [n, d] -> [n].
    """
    dots = np.asarray(q_t, np.float64) @ np.asarray(keys, np.float64).T        # [H_I, n]
    return np.asarray(w_t, np.float64) @ np.maximum(dots, 0.0)


def sub_block_mean_keys(k_hat, sub_block: int) -> np.ndarray:
    """Sec. 3.3, Stage 1: k^mean_n = per-dimension mean of the keys of sub-block n.

    Only complete sub-blocks are formed; the cache stores them in bfloat16 (one rounding).
    k_hat [n_tok, d] float64 -> [n_tok // B, d] float64 (values representable in bfloat16).
    """
    k_hat = np.asarray(k_hat, np.float64)
    n_sub = k_hat.shape[0] // sub_block
    means = k_hat[: n_sub * sub_block].reshape(n_sub, sub_block, k_hat.shape[1]).mean(axis=1)
    return bf16_bits_to_f64(f64_to_bf16_bits(means))


def sub_block_minmax_keys(k_hat, sub_block: int):
    """Eq. (13) (the pooling ablation of hierarchical indexing): per-dimension maximum and minimum
    of the keys of each sub-block.

    Only complete sub-blocks are formed; like the mean keys they are stored in bfloat16, each
    extremum rounded once (rounding is monotone, so k_min <= k_max survives it).
    k_hat [n_tok, d] float64 -> (k_max, k_min), each [n_tok // B, d] float64.
    """
    k_hat = np.asarray(k_hat, np.float64)
    n_sub = k_hat.shape[0] // sub_block
    blocks = k_hat[: n_sub * sub_block].reshape(n_sub, sub_block, k_hat.shape[1])
    if n_sub == 0:  # a cache shorter than one sub-block has no block keys
        empty = np.zeros((0, k_hat.shape[1]))
        return empty, empty.copy()
    k_max = bf16_bits_to_f64(f64_to_bf16_bits(blocks.max(axis=1)))
    k_min = bf16_bits_to_f64(f64_to_bf16_bits(blocks.min(axis=1)))
    return k_max, k_min


def streaming_sets(t: int, prm: IndexParams):
    """Eq. (6): the fixed parts of S_t and the range left to the indexer (Eq. 7).

    Returns (S_sink, S_swa, eligible) where eligible is (lo, hi) inclusive, or None when sink
    and window already cover [0, t].
    """
    sink = np.arange(0, min(prm.k_sink, t + 1))
    swa = np.arange(max(0, t - prm.k_swa + 1), t + 1)
    lo, hi = prm.k_sink, t - prm.k_swa
    return sink, swa, ((lo, hi) if lo <= hi else None)


def page_scores(q_t, w_t, k_mean, pages, prm: IndexParams) -> np.ndarray:
    """Eq. (9): I^page_{t,p} = sum_j w_{t,j} sum_{n in page p} ReLU(q_{t,j} . k^mean_n).

    k_mean holds one row per sub-block; page p owns sub-blocks [p*P/B, (p+1)*P/B).
    """
    per_page = prm.page // prm.sub_block
    pages = np.asarray(pages, np.int64)
    sub = (pages[:, None] * per_page + np.arange(per_page)[None, :]).reshape(-1)
    dots = np.asarray(q_t, np.float64) @ k_mean[sub].T                       # [H_I, n_pages*per_page]
    relu = np.maximum(dots, 0.0).reshape(dots.shape[0], len(pages), per_page).sum(axis=2)
    return np.asarray(w_t, np.float64) @ relu                                 # [n_pages]


def page_scores_minmax(q_t, w_t, k_max, k_min, pages, prm: IndexParams) -> np.ndarray:
    """Eq. (13) in the coarse score: per head j and sub-block n,
    s~_{t,n,j} = sum_d max(q_{t,j,d} k^max_{n,d}, q_{t,j,d} k^min_{n,d}), then
    I^page_{t,p} = sum_j w_{t,j} sum_{n in page p} ReLU(s~_{t,n,j}).
    """
    per_page = prm.page // prm.sub_block
    pages = np.asarray(pages, np.int64)
    sub = (pages[:, None] * per_page + np.arange(per_page)[None, :]).reshape(-1)
    q = np.asarray(q_t, np.float64)                                          # [H_I, d]
    hi = q[:, None, :] * np.asarray(k_max, np.float64)[sub][None, :, :]       # [H_I, n, d]
    lo = q[:, None, :] * np.asarray(k_min, np.float64)[sub][None, :, :]
    s_tilde = np.maximum(hi, lo).sum(axis=2)                                 # [H_I, n]
    relu = np.maximum(s_tilde, 0.0).reshape(q.shape[0], len(pages), per_page).sum(axis=2)
    return np.asarray(w_t, np.float64) @ relu                                 # [n_pages]


def arg_top(scores, ids, k: int) -> np.ndarray:
    """arg topK (Eq. 2, 7, 10, 12): the k ids of largest score, ties to the smaller id.

    Returns the chosen ids in ascending order; all ids when there are at most k.
    """
    ids = np.asarray(ids, np.int64)
    if len(ids) <= k:
        return np.sort(ids)
    order = np.lexsort((ids, -np.asarray(scores, np.float64)))
    return np.sort(ids[order[:k]])


def eligible_pages(lo: int, hi: int, prm: IndexParams) -> np.ndarray:
    """Pages holding at least one eligible position of [lo, hi]."""
    return np.arange(lo // prm.page, hi // prm.page + 1)


def candidates_of_pages(pages, lo: int, hi: int, prm: IndexParams) -> np.ndarray:
    """Eq. (10)/(12): S^page_t restricted to the eligible range (ascending positions)."""
    pages = np.asarray(pages, np.int64)
    pos = (pages[:, None] * prm.page + np.arange(prm.page)[None, :]).reshape(-1)
    return pos[(pos >= lo) & (pos <= hi)]


def runs_of(S, align: int) -> list[tuple[int, int]]:
    """Re-encode an ascending position list as (start, length) runs.

    A run is a maximal stretch of consecutive positions that does not cross a multiple of
    `align` (a new run starts at every gap and at every position divisible by `align`).
    """
    runs: list[list[int]] = []
    for s in np.asarray(S, np.int64).tolist():
        if runs and s == runs[-1][0] + runs[-1][1] and s % align != 0:
            runs[-1][1] += 1
        else:
            runs.append([s, 1])
    return [(a, n) for a, n in runs]


def index_row(t: int, q_t, w_t, k_hat, k_mean, prm: IndexParams, pages_override=None) -> dict:
    """One query row of the LSA indexer: S_t and the intermediate quantities.

    t: 0-based position of the query; q_t [H_I, d]; w_t [H_I]; k_hat [>= t+1, d] float64 keys;
    k_mean: the Stage 1 block cache, unused in flat mode: the sub-block mean keys (Eq. 9), or
    with prm.pooling == "minmax" the pair (k_max, k_min) of sub_block_minmax_keys (Eq. 13).
    pages_override: run Eq. (11)-(12) on this page list instead of the coarse stage's own
    choice (used to check the fine stage on the pages another implementation recalled).

    Returns a dict with
      S          ascending int64 positions of S_t  (Eq. 6)
      sink, swa  the fixed parts
      pages      recalled pages P_t (ascending) or None in flat mode / when E_t is empty
      page_ids, page_score   every eligible page and its coarse score (Eq. 9), HI only
      cand, score            candidate positions S^page_t n E_t and their fine scores (Eq. 11)
      sparse     S_sparse (ascending)
    """
    sink, swa, elig = streaming_sets(t, prm)
    out = dict(t=t, sink=sink, swa=swa, pages=None, page_ids=None, page_score=None,
               cand=np.zeros(0, np.int64), score=np.zeros(0), sparse=np.zeros(0, np.int64))
    if elig is None:                                    # sink and window cover [0, t]
        out["S"] = np.arange(t + 1)
        return out
    lo, hi = elig
    all_pages = eligible_pages(lo, hi, prm)
    if prm.keep_pages > 0:
        # Stage 1: coarse page score (Eq. 9, or Eq. 13 with min-max pooling) and top-M pages (Eq. 10)
        if prm.pooling == "minmax":
            ps = page_scores_minmax(q_t, w_t, k_mean[0], k_mean[1], all_pages, prm)
        else:
            ps = page_scores(q_t, w_t, k_mean, all_pages, prm)
        out["page_ids"], out["page_score"] = all_pages, ps
        pages = arg_top(ps, all_pages, prm.keep_pages)
        if pages_override is not None:
            pages = np.sort(np.asarray(pages_override, np.int64))
        out["pages"] = pages
    else:
        pages = all_pages                               # flat: every eligible position
    # Stage 2: fine token score over the recalled pages (Eq. 11), final top-K_sparse (Eq. 12)
    cand = candidates_of_pages(pages, lo, hi, prm)
    score = indexer_scores(q_t, w_t, k_hat[cand])
    sparse = arg_top(score, cand, prm.k_sparse)
    out.update(cand=cand, score=score, sparse=sparse)
    out["S"] = np.concatenate([sink, sparse, swa])      # sink < E_t < window: already ascending
    return out


# ============================================================================ attention


def sparse_attention_row(q_t, keys, values, scale: float):
    """Eq. (3): attention of one query (all heads) over the selected tokens only.

    q_t [H, d_qk]; keys [n, d_qk]; values [n, d_v] (for an MLA latent cache both are slices of
    the same selected rows). Returns (o [H, d_v], lse [H]) with lse = log sum_s exp(z_s),
    z_s = scale * q . k_s (natural log).
    """
    z = float(scale) * (np.asarray(q_t, np.float64) @ np.asarray(keys, np.float64).T)   # [H, n]
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    l = e.sum(axis=1, keepdims=True)
    o = (e @ np.asarray(values, np.float64)) / l
    return o, m[:, 0] + np.log(l[:, 0])


def attention_for_set(q_t_bits, kv_bits, v_bits, S, d_v: int, scale: float):
    """Decode the bfloat16 inputs of one query and its selected rows, then apply Eq. (3).

    kv_bits: latent cache [n_kv, d_qk] (V = first d_v columns) when v_bits is None, else K.
    """
    S = np.asarray(S, np.int64)
    q = bf16_bits_to_f64(q_t_bits)
    k = bf16_bits_to_f64(kv_bits[S])
    v = k[:, :d_v] if v_bits is None else bf16_bits_to_f64(v_bits[S])
    return sparse_attention_row(q, k, v, scale)


# ============================================================================ paged caches


def logical_rows(paged, page_table_row, n_tokens: int, page_size: int) -> np.ndarray:
    """Rows 0..n_tokens-1 of one sequence whose cache lives in pages: logical row s is row
    s % page_size of physical page page_table_row[s // page_size]. paged: [n_phys, page_size, ...]."""
    s = np.arange(n_tokens)
    phys = np.asarray(page_table_row, np.int64)[s // page_size]
    return np.asarray(paged)[phys, s % page_size]
