"""Pins of the oracle against things other than itself.

Each `pin_*` takes the oracle module and raises AssertionError when the oracle disagrees with
a library routine (torch casts, torch SDPA, numpy reductions), a closed form worked out from the
paper's equations, a brute-force search, or an invariant of the method. The same pins run
against deliberately broken copies of the oracle (tests/test_oracle_pins.py) to show that a
plausible mistake fails at least one of them.
"""
from __future__ import annotations

import itertools
from fractions import Fraction

import numpy as np
import torch


def _prm(orc, **kw):
    base = dict(page=4, sub_block=4, keep_pages=0, k_sparse=3, k_sink=2, k_swa=4, run_align=4)
    base.update(kw)
    return orc.IndexParams(**base)


# ----------------------------------------------------------------------------- number formats
def pin_bf16_decode(orc):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64).numpy()
    got = orc.bf16_bits_to_f64(bits)
    assert np.array_equal(got, ref, equal_nan=True), "bf16 decode differs from torch"


def pin_bf16_round_vs_torch(orc):
    """On float32 inputs one RNE step to bf16 is torch's cast."""
    g = np.random.default_rng(7)
    mant = g.random(200000) + 1.0
    expo = g.integers(-140, 127, size=mant.size)
    x = (np.ldexp(mant, expo) * np.where(g.random(mant.size) < 0.5, -1, 1)).astype(np.float32)
    # exact halfway points and their float32 neighbours
    base = torch.from_numpy(g.standard_normal(5000).astype(np.float32)).to(torch.bfloat16)
    b32 = base.to(torch.float32).numpy().view(np.uint32)
    half = (b32 + np.uint32(0x8000)).view(np.float32)
    x = np.concatenate([x, half, np.nextafter(half, np.float32(np.inf)),
                        np.nextafter(half, np.float32(-np.inf)), np.float32([0.0, -0.0, 1e-45, 3e38])])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = orc.f64_to_bf16_bits(x.astype(np.float64))
    assert np.array_equal(got, ref), f"bf16 rounding differs from torch on {np.sum(got != ref)} values"


def _bf16_rne_exact(v: Fraction) -> Fraction:
    """Round a positive rational to 8 significant bits, ties to even (normal range only)."""
    e = 0
    while v >= 2:
        v /= 2
        e += 1
    while v < 1:
        v *= 2
        e -= 1
    n = v * 128                               # 128 <= n < 256
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return Fraction(fl, 128) * (Fraction(2) ** e)


def pin_bf16_round_exact(orc):
    """Float64 values within a float32 ulp of a bf16 halfway point round by exact arithmetic
    (a float32 detour would round them twice)."""
    g = np.random.default_rng(11)
    xs = []
    for _ in range(300):
        m = int(g.integers(128, 256))
        e = int(g.integers(-20, 20))
        mid = Fraction(2 * m + 1, 256) * Fraction(2) ** e            # halfway between two bf16
        for d in (Fraction(0), Fraction(1, 2 ** 40), -Fraction(1, 2 ** 40)):
            xs.append(mid + d * Fraction(2) ** e)
    got = orc.bf16_bits_to_f64(orc.f64_to_bf16_bits(np.array([float(x) for x in xs])))
    for x, y in zip(xs, got):
        assert Fraction(float(y)) == _bf16_rne_exact(Fraction(float(x))), f"bf16 rounding of {float(x)!r}"


def pin_e4m3fn_decode(orc):
    codes = np.arange(256, dtype=np.uint32).astype(np.uint8)
    ref = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(orc.e4m3fn_to_f64(codes), ref, equal_nan=True), "e4m3fn decode differs from torch"


def pin_dequant_fp8(orc):
    g = np.random.default_rng(3)
    codes = g.integers(0, 256, size=(9, 16)).astype(np.uint8)
    codes[(codes & 0x7F) == 0x7F] = 0x10          # avoid NaN codes
    scale = g.random(9).astype(np.float32) + 0.1
    ref = torch.from_numpy(codes.copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    ref = ref * scale.astype(np.float64)[:, None]
    assert np.array_equal(orc.dequantized_keys(codes, scale), ref)


# ----------------------------------------------------------------------------- Eq. (1)
def pin_score_closed_form(orc):
    """Eq. (1) with q_j = e_j and w = (1, 10, 100): I = max(0,k0) + 10 max(0,k1) + 100 max(0,k2)."""
    q = np.eye(3)
    w = np.array([1.0, 10.0, 100.0])
    keys = np.array([[2.0, -3.0, 0.5], [-1.0, 4.0, -2.0], [0.25, 0.0, 1.0], [-1, -1, -1.0]])
    want = np.array([2 + 0 + 50, 0 + 40 + 0, 0.25 + 0 + 100, 0.0])
    assert np.array_equal(orc.indexer_scores(q, w, keys), want)


def pin_score_single_head_dot(orc):
    """One head with weight 1: I_s = ReLU(q . k_s) with numpy's dot product, on non-square shapes."""
    g = np.random.default_rng(5)
    q = g.standard_normal((1, 5))
    keys = g.standard_normal((7, 5))
    want = np.array([max(0.0, float(np.dot(q[0], k))) for k in keys])
    assert np.allclose(orc.indexer_scores(q, np.ones(1), keys), want, rtol=1e-14, atol=1e-15)


def pin_score_heads_additive(orc):
    """Heads add (Eq. 1 is a sum over j) and reordering heads together with their weights is a no-op."""
    g = np.random.default_rng(6)
    q = g.standard_normal((6, 4))
    w = g.random(6)
    keys = g.standard_normal((11, 4))
    full = orc.indexer_scores(q, w, keys)
    parts = orc.indexer_scores(q[:2], w[:2], keys) + orc.indexer_scores(q[2:], w[2:], keys)
    perm = g.permutation(6)
    assert np.allclose(full, parts, rtol=1e-13) and np.allclose(full, orc.indexer_scores(q[perm], w[perm], keys), rtol=1e-13)


# ----------------------------------------------------------------------------- arg topK
def pin_topk_bruteforce(orc):
    """arg topK = the size-k subset with the largest score sum; among equal sums the
    lexicographically smallest sorted position list (ties go to earlier positions)."""
    g = np.random.default_rng(8)
    for trial in range(40):
        n = int(g.integers(1, 10))
        k = int(g.integers(1, 5))
        ids = np.sort(g.choice(50, size=n, replace=False))
        scores = g.integers(-2, 4, size=n).astype(np.float64)        # many exact ties
        if n <= k:
            best = tuple(ids.tolist())
        else:
            best, best_sum = None, None
            for c in itertools.combinations(range(n), k):
                s = scores[list(c)].sum()
                key = tuple(ids[list(c)].tolist())
                if best_sum is None or s > best_sum or (s == best_sum and key < best):
                    best, best_sum = key, s
        assert tuple(orc.arg_top(scores, ids, k).tolist()) == best, (trial, scores, ids, k)


# ----------------------------------------------------------------------------- Eq. (6)-(7) flat
def _flat_case(orc, d, keys_fn, L=40, H=1):
    prm = _prm(orc, page=4, sub_block=4, keep_pages=0, k_sparse=5, k_sink=3, k_swa=6)
    k_hat = np.array([keys_fn(s) for s in range(L)], dtype=np.float64).reshape(L, d)
    return prm, k_hat


def pin_flat_designed_orders(orc):
    """d_I = 1, q = +1, w = 1: increasing keys select the latest eligible tokens, decreasing
    keys the earliest, equal keys the earliest (tie rule)."""
    q, w = np.ones((1, 1)), np.ones(1)
    for keys_fn, pick in ((lambda s: s + 1.0, "late"), (lambda s: 100.0 - s, "early"), (lambda s: 1.0, "early")):
        prm, k_hat = _flat_case(orc, 1, keys_fn)
        for t in range(prm.k_sink + prm.k_swa, 40):
            lo, hi = prm.k_sink, t - prm.k_swa
            elig = np.arange(lo, hi + 1)
            want = elig[-prm.k_sparse:] if pick == "late" else elig[:prm.k_sparse]
            r = orc.index_row(t, q, w, k_hat, None, prm)
            assert np.array_equal(r["sparse"], want), (pick, t, r["sparse"], want)


def pin_streaming_structure(orc):
    """Eq. (6): S_t = sink u window u sparse, ascending, within [0, t], of size
    min(t+1, K_sink + K_swa + min(K_sparse, |E_t|)); [0, t] when sink and window meet."""
    g = np.random.default_rng(9)
    for prm in (_prm(orc, k_sparse=3, k_sink=2, k_swa=4), _prm(orc, k_sparse=7, k_sink=0, k_swa=1),
                _prm(orc, k_sparse=1, k_sink=5, k_swa=8, page=8, sub_block=4, keep_pages=2)):
        L = 48
        q, w = g.standard_normal((3, 4)), g.random(3)
        k_hat = g.standard_normal((L, 4))
        k_mean = orc.sub_block_mean_keys(k_hat, prm.sub_block)
        for t in range(L):
            S = orc.index_row(t, q, w, k_hat, k_mean, prm)["S"]
            n_elig = max(0, t - prm.k_swa - prm.k_sink + 1)
            assert np.all(np.diff(S) > 0) and S[0] >= 0 and S[-1] == t
            assert len(S) == min(t + 1, prm.k_sink + prm.k_swa + min(prm.k_sparse, n_elig)), (t, S)
            assert set(range(min(prm.k_sink, t + 1))) <= set(S.tolist())
            assert set(range(max(0, t - prm.k_swa + 1), t + 1)) <= set(S.tolist())
            if n_elig == 0:
                assert np.array_equal(S, np.arange(t + 1))


def pin_flat_bruteforce_rows(orc):
    """Flat selection equals a brute-force search, over all subsets of the eligible range, for the
    K_sparse positions with the largest total score (ties: lexicographically smallest)."""
    g = np.random.default_rng(10)
    prm = _prm(orc, k_sparse=3, k_sink=2, k_swa=3, keep_pages=0)
    L, H, d = 16, 2, 3
    q, w = g.standard_normal((H, d)), g.random(H)
    k_hat = g.standard_normal((L, d))
    for t in range(L):
        r = orc.index_row(t, q, w, k_hat, None, prm)
        lo, hi = prm.k_sink, t - prm.k_swa
        if lo > hi:
            continue
        elig = list(range(lo, hi + 1))
        sc = {s: float(np.dot(w, np.maximum(q @ k_hat[s], 0))) for s in elig}
        if len(elig) <= prm.k_sparse:
            best = tuple(elig)
        else:
            best = max(itertools.combinations(elig, prm.k_sparse),
                       key=lambda c: (sum(sc[s] for s in c), tuple(-s for s in c)))
        assert tuple(r["sparse"].tolist()) == best, (t, r["sparse"], best)


# ----------------------------------------------------------------------------- Eq. (9)-(12) HI
def pin_sub_block_means(orc):
    """Mean keys: per-dimension mean of each complete sub-block (numpy mean) then one bf16
    rounding (torch's cast, on inputs whose mean is exact in float32)."""
    g = np.random.default_rng(12)
    B, n, d = 8, 43, 6
    k = g.integers(-512, 512, size=(n, d)).astype(np.float64) / 1024.0
    got = orc.sub_block_mean_keys(k, B)
    assert got.shape == (n // B, d)
    exact = np.stack([k[i * B:(i + 1) * B].mean(axis=0) for i in range(n // B)]).astype(np.float32)
    ref = torch.from_numpy(exact).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(got, ref)
    const = np.full((16, 3), 0.375)
    assert np.array_equal(orc.sub_block_mean_keys(const, 4), np.full((4, 3), 0.375))


def pin_page_score_structure(orc):
    """Eq. (9): with one sub-block per page a mean key is scored like a token (Eq. 1); with
    several, a page's score is the sum of its sub-blocks' scores; identical sub-blocks give
    (P/B) times one of them."""
    g = np.random.default_rng(13)
    q, w = g.standard_normal((4, 5)), g.random(4)
    means = g.standard_normal((12, 5))
    one = orc.page_scores(q, w, means, np.arange(12), _prm(orc, page=4, sub_block=4))
    assert np.allclose(one, orc.indexer_scores(q, w, means), rtol=1e-13)
    four = orc.page_scores(q, w, means, np.arange(3), _prm(orc, page=16, sub_block=4))
    sub = orc.indexer_scores(q, w, means)
    assert np.allclose(four, sub.reshape(3, 4).sum(axis=1), rtol=1e-13)
    same = np.repeat(means[:1], 4, axis=0)
    assert np.allclose(orc.page_scores(q, w, same, np.arange(1), _prm(orc, page=16, sub_block=4)),
                       4 * orc.indexer_scores(q, w, means[:1]), rtol=1e-13)


def pin_hi_keep_all_equals_flat(orc):
    """Keeping every eligible page (M >= #pages) reduces Eq. (10)-(12) to Eq. (7)."""
    g = np.random.default_rng(14)
    for P, B in ((8, 8), (8, 2)):
        L = 96
        q, w = g.standard_normal((3, 4)), g.random(3)
        k_hat = g.standard_normal((L, 4))
        k_mean = orc.sub_block_mean_keys(k_hat, B)
        flat = _prm(orc, page=P, sub_block=B, keep_pages=0, k_sparse=6, k_sink=3, k_swa=9)
        keep = _prm(orc, page=P, sub_block=B, keep_pages=L // P + 1, k_sparse=6, k_sink=3, k_swa=9)
        for t in range(L):
            a = orc.index_row(t, q, w, k_hat, k_mean, flat)["S"]
            b = orc.index_row(t, q, w, k_hat, k_mean, keep)["S"]
            assert np.array_equal(a, b), t


def pin_hi_dominant_page(orc):
    """d_I = 1, q = +1: the page whose keys are +1 (others -1) is the only one with a positive
    mean key; with M = 1 it is recalled and the sparse set comes from it alone (earliest first,
    all scores being equal)."""
    P, L = 8, 64
    prm = _prm(orc, page=P, sub_block=P, keep_pages=1, k_sparse=5, k_sink=2, k_swa=8)
    for hot in (0, 2, 5):
        k_hat = -np.ones((L, 1))
        k_hat[hot * P:(hot + 1) * P] = 1.0
        k_mean = orc.sub_block_mean_keys(k_hat, P)
        t = L - 1
        r = orc.index_row(t, np.ones((1, 1)), np.ones(1), k_hat, k_mean, prm)
        assert np.array_equal(r["pages"], [hot])
        cand = [s for s in range(hot * P, hot * P + P) if prm.k_sink <= s <= t - prm.k_swa]
        assert np.array_equal(r["cand"], cand)
        assert np.array_equal(r["sparse"], cand[:prm.k_sparse])


def pin_homogeneity(orc):
    """ReLU(a x) = a ReLU(x) for a > 0: scaling every head weight, or every key (and hence every
    mean key), by a power of two leaves S_t unchanged."""
    g = np.random.default_rng(15)
    prm = _prm(orc, page=8, sub_block=4, keep_pages=3, k_sparse=5, k_sink=2, k_swa=8)
    L = 80
    q, w = g.standard_normal((3, 4)), g.random(3)
    k_hat = g.standard_normal((L, 4))
    km = orc.sub_block_mean_keys(k_hat, prm.sub_block)
    km4 = orc.sub_block_mean_keys(4 * k_hat, prm.sub_block)
    for t in range(0, L, 3):
        base = orc.index_row(t, q, w, k_hat, km, prm)["S"]
        assert np.array_equal(base, orc.index_row(t, q, 8 * w, k_hat, km, prm)["S"])
        assert np.array_equal(base, orc.index_row(t, q, w, 4 * k_hat, km4, prm)["S"])


def pin_minmax_keys(orc):
    """Eq. (13) extrema: on bf16-exact keys every key of a sub-block lies inside [k_min, k_max]
    coordinate-wise, and each bound is attained by one of its keys (brute force over the block)."""
    g = np.random.default_rng(16)
    B, n, d = 4, 22, 5
    k = g.integers(-255, 256, size=(n, d)).astype(np.float64) / 256.0       # bf16-exact
    k_max, k_min = orc.sub_block_minmax_keys(k, B)
    assert k_max.shape == (n // B, d) and k_min.shape == (n // B, d)
    for b in range(n // B):
        blk = k[b * B:(b + 1) * B]
        for c in range(d):
            col = [float(x) for x in blk[:, c]]
            assert k_max[b, c] == max(col) and k_min[b, c] == min(col), (b, c)
    # B = 1: both extrema are the (rounded) key itself
    one_max, one_min = orc.sub_block_minmax_keys(k, 1)
    assert np.array_equal(one_max, k) and np.array_equal(one_min, k)


def pin_minmax_score_is_box_support(orc):
    """Eq. (13) is the largest value of q . x over the box [k_min, k_max]: brute force over the
    2^d corners (d = 4), one head, one sub-block per page, so the page score is ReLU of it times
    the head weight; the box bound is at least every member token's score."""
    g = np.random.default_rng(17)
    prm = _prm(orc, page=4, sub_block=4, pooling="minmax")
    for _ in range(40):
        k = g.integers(-64, 64, size=(4, 4)).astype(np.float64) / 32.0
        k_max, k_min = orc.sub_block_minmax_keys(k, 4)
        q = g.standard_normal((1, 4))
        w = g.random(1) + 0.5
        best = max(float(q[0] @ np.where(np.array(bits) == 1, k_max[0], k_min[0]))
                   for bits in itertools.product((0, 1), repeat=4))
        got = orc.page_scores_minmax(q, w, k_max, k_min, np.arange(1), prm)
        assert np.isclose(got[0], w[0] * max(best, 0.0), rtol=1e-13, atol=1e-15)
        assert best >= float((k @ q[0]).max()) - 1e-12          # upper bound of the block's tokens


def pin_minmax_reduces_to_mean_pooling(orc):
    """With B = 1 the box is a point: Eq. (13) becomes q . k and the min-max page score equals the
    mean-pooled one (Eq. 9), for several heads and sub-blocks per page; and the whole indexer row
    then selects the same set under either pooling."""
    g = np.random.default_rng(18)
    q, w = g.standard_normal((3, 5)), g.random(3)
    k = g.integers(-200, 200, size=(32, 5)).astype(np.float64) / 128.0
    prm_mean = _prm(orc, page=8, sub_block=1)
    prm_mm = _prm(orc, page=8, sub_block=1, pooling="minmax")
    km = orc.sub_block_mean_keys(k, 1)
    kx, kn = orc.sub_block_minmax_keys(k, 1)
    a = orc.page_scores(q, w, km, np.arange(4), prm_mean)
    b = orc.page_scores_minmax(q, w, kx, kn, np.arange(4), prm_mm)
    assert np.allclose(a, b, rtol=1e-13, atol=1e-13)
    hm = _prm(orc, page=8, sub_block=1, keep_pages=2, k_sparse=4, k_sink=2, k_swa=8)
    hx = _prm(orc, page=8, sub_block=1, keep_pages=2, k_sparse=4, k_sink=2, k_swa=8, pooling="minmax")
    for t in range(12, 32):
        assert np.array_equal(orc.index_row(t, q, w, k, km, hm)["S"], orc.index_row(t, q, w, k, (kx, kn), hx)["S"])


# ----------------------------------------------------------------------------- runs
def pin_runs(orc):
    S = [0, 1, 2, 3, 5, 6, 62, 63, 64, 65, 127, 128]
    assert orc.runs_of(S, 64) == [(0, 4), (5, 2), (62, 2), (64, 2), (127, 1), (128, 1)]
    g = np.random.default_rng(16)
    for _ in range(50):
        C = int(g.choice([1, 4, 16, 64]))
        S = np.unique(g.integers(0, 300, size=int(g.integers(1, 120))))
        runs = orc.runs_of(S, C)
        expand = [a + i for a, n in runs for i in range(n)]
        assert expand == S.tolist()
        for a, n in runs:
            assert n >= 1 and (a // C) == ((a + n - 1) // C), "run crosses a multiple of C"
        for (a, n), (b, _) in zip(runs, runs[1:]):
            assert b != a + n or b % C == 0, "runs not maximal"


# ----------------------------------------------------------------------------- Eq. (3)
def _sdpa(q, k, v, scale):
    """torch's scaled_dot_product_attention (float64, CPU) with a causal mask; q [T,H,d]."""
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]            # [1,H,T,d]
    H = q.shape[1]
    kt = torch.from_numpy(k)[None, None].expand(1, H, *k.shape)
    vt = torch.from_numpy(v)[None, None].expand(1, H, *v.shape)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=scale)
    return o[0].permute(1, 0, 2).numpy()


def pin_attention_dense_equals_sdpa(orc):
    """With S_t = [0, t] (K >= t+1) sparse attention is causal softmax attention."""
    g = np.random.default_rng(17)
    T, H, dqk, dv = 13, 4, 8, 6
    q = g.standard_normal((T, H, dqk))
    kv = g.standard_normal((T, dqk))
    vv = g.standard_normal((T, dv))
    scale = 1 / np.sqrt(dqk)
    ref_latent = _sdpa(q, kv, np.ascontiguousarray(kv[:, :dv]), scale)
    ref_sep = _sdpa(q, kv, vv, scale)
    for t in range(T):
        S = np.arange(t + 1)
        o, _ = orc.sparse_attention_row(q[t], kv[S], kv[S, :dv], scale)
        assert np.allclose(o, ref_latent[t], rtol=1e-12, atol=1e-13)
        o, _ = orc.sparse_attention_row(q[t], kv[S], vv[S], scale)
        assert np.allclose(o, ref_sep[t], rtol=1e-12, atol=1e-13)


def pin_attention_closed_forms(orc):
    g = np.random.default_rng(18)
    H, d, dv = 3, 5, 4
    q = g.standard_normal((H, d))
    k = g.standard_normal((6, d))
    v = g.standard_normal((6, dv))
    scale = 0.3
    o, lse = orc.sparse_attention_row(q, k[2:3], v[2:3], scale)       # one token: o = v, lse = z
    assert np.allclose(o, np.repeat(v[2:3], H, 0), rtol=1e-14) and np.allclose(lse, scale * q @ k[2], rtol=1e-14)
    same = np.repeat(k[:1], 6, 0)                                      # identical keys: mean of v
    o, lse = orc.sparse_attention_row(q, same, v, scale)
    assert np.allclose(o, np.repeat(v.mean(0, keepdims=True), H, 0), rtol=1e-13)
    assert np.allclose(lse, scale * q @ k[0] + np.log(6), rtol=1e-13)
    perm = g.permutation(6)                                            # order of the set is irrelevant
    o1, l1 = orc.sparse_attention_row(q, k, v, scale)
    o2, l2 = orc.sparse_attention_row(q, k[perm], v[perm], scale)
    assert np.allclose(o1, o2, rtol=1e-13) and np.allclose(l1, l2, rtol=1e-13)
    oa, la = orc.sparse_attention_row(q, k[:2], v[:2], scale)          # log-sum-exp merge of halves
    ob, lb = orc.sparse_attention_row(q, k[2:], v[2:], scale)
    lse = np.logaddexp(la, lb)
    om = (np.exp(la - lse)[:, None] * oa + np.exp(lb - lse)[:, None] * ob)
    assert np.allclose(om, o1, rtol=1e-12) and np.allclose(lse, l1, rtol=1e-13)


def pin_attention_scale_and_log(orc):
    """lse is a natural log and the scale multiplies q . k: two tokens with z = (0, ln 3)
    give weights (1/4, 3/4) and lse = ln 4."""
    q = np.array([[1.0, 0.0]])
    k = np.array([[0.0, 1.0], [np.log(3.0) / 0.5, 0.0]])
    v = np.array([[4.0], [8.0]])
    o, lse = orc.sparse_attention_row(q, k, v, 0.5)
    assert np.allclose(o, [[7.0]], rtol=1e-14) and np.allclose(lse, [np.log(4.0)], rtol=1e-14)


def pin_attention_for_set_value_columns(orc):
    """One selected row has softmax weight 1, so the output is that row's value vector: with a
    latent cache V is its first d_v columns (MLA absorbed mode), otherwise the separate V row.
    Every other row and column holds distinct values, so a wrong row or column shows."""
    n, d_qk, d_v = 6, 8, 4
    vals = np.arange(n * d_qk, dtype=np.float64).reshape(n, d_qk) / 8.0 - 2.0   # exact in bf16
    kv_bits = orc.f64_to_bf16_bits(vals)
    q_bits = orc.f64_to_bf16_bits(np.full((2, d_qk), 0.25))
    o, lse = orc.attention_for_set(q_bits, kv_bits, None, [3], d_v, 0.5)
    assert np.array_equal(o, np.tile(vals[3, :d_v], (2, 1))), "latent V is not the first d_v columns"
    v_sep = np.arange(n * d_v, dtype=np.float64).reshape(n, d_v) + 100.0
    o2, _ = orc.attention_for_set(q_bits, kv_bits, orc.f64_to_bf16_bits(v_sep), [4], d_v, 0.5)
    assert np.array_equal(o2, np.tile(v_sep[4], (2, 1))), "separate V row not used"
    z = 0.5 * 0.25 * vals[3].sum()
    assert np.allclose(lse, [z, z], rtol=1e-14)


def pin_logical_rows(orc):
    page = 4
    paged = np.arange(6 * page * 2).reshape(6, page, 2)
    table = np.array([3, 0, 5])
    rows = orc.logical_rows(paged, table, 10, page)
    want = np.concatenate([paged[3], paged[0], paged[5]])[:10]
    assert np.array_equal(rows, want)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
