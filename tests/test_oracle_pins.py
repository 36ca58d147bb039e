"""The oracle against its pins, and planted mistakes against the same pins.

A mutant replaces one oracle function with a plausible wrong version (a dropped ReLU, an
off-by-one window, max instead of mean, ...). Each mutant must fail at least one pin, which shows
that the pins would catch that kind of mistake in the oracle itself.
"""
import numpy as np
import pytest

import oracle.lsa_oracle as orc
from tests import oracle_pins as pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(orc)


def _no_relu(q_t, w_t, keys):
    return np.asarray(w_t) @ (np.asarray(q_t) @ np.asarray(keys).T)


def _relu_after_sum(q_t, w_t, keys):
    return np.maximum(np.asarray(w_t) @ (np.asarray(q_t) @ np.asarray(keys).T), 0.0)


def _max_pool(k_hat, sub_block):
    k_hat = np.asarray(k_hat, np.float64)
    n = k_hat.shape[0] // sub_block
    m = k_hat[: n * sub_block].reshape(n, sub_block, -1).max(axis=1)
    return orc.bf16_bits_to_f64(orc.f64_to_bf16_bits(m))


def _window_off_by_one(t, prm):
    sink = np.arange(0, min(prm.k_sink, t + 1))
    swa = np.arange(max(0, t - prm.k_swa), t + 1)
    lo, hi = prm.k_sink, t - prm.k_swa - 1
    return sink, swa, ((lo, hi) if lo <= hi else None)


def _no_sink(t, prm):
    sink = np.arange(0)
    swa = np.arange(max(0, t - prm.k_swa + 1), t + 1)
    lo, hi = prm.k_sink, t - prm.k_swa
    return sink, swa, ((lo, hi) if lo <= hi else None)


def _ties_to_later(scores, ids, k):
    ids = np.asarray(ids, np.int64)
    if len(ids) <= k:
        return np.sort(ids)
    order = np.lexsort((-ids, -np.asarray(scores, np.float64)))
    return np.sort(ids[order[:k]])


def _truncating_bf16(x):
    x = np.asarray(x, np.float64).astype(np.float32)
    return (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _e4m3_bias8(codes):
    c = np.asarray(codes, np.uint8).astype(np.int64)
    e, m = (c >> 3) & 0xF, (c & 7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -10, (1 + m / 8) * np.exp2(e - 8.0))
    mag = np.where((e == 15) & ((c & 7) == 7), np.nan, mag)
    return np.where(c & 0x80, -1.0, 1.0) * mag


def _cand_with_window(pages, lo, hi, prm):
    pages = np.asarray(pages, np.int64)
    pos = (pages[:, None] * prm.page + np.arange(prm.page)[None, :]).reshape(-1)
    return pos[(pos >= lo) & (pos <= hi + 1)]


def _attn_no_scale(q_t, keys, values, scale):
    return orc.__dict__["_orig_attn"](q_t, keys, values, 1.0)


def _attn_log2(q_t, keys, values, scale):
    o, lse = orc.__dict__["_orig_attn"](q_t, keys, values, scale)
    return o, lse / np.log(2.0)


def _page_score_unweighted(q_t, w_t, k_mean, pages, prm):
    return orc.__dict__["_orig_page"](q_t, np.ones_like(np.asarray(w_t)), k_mean, pages, prm)


def _minmax_min_of_products(q_t, w_t, k_max, k_min, pages, prm):
    per_page = prm.page // prm.sub_block
    sub = (np.asarray(pages)[:, None] * per_page + np.arange(per_page)[None, :]).reshape(-1)
    q = np.asarray(q_t, np.float64)
    s = np.minimum(q[:, None, :] * k_max[sub][None], q[:, None, :] * k_min[sub][None]).sum(axis=2)
    relu = np.maximum(s, 0.0).reshape(q.shape[0], len(pages), per_page).sum(axis=2)
    return np.asarray(w_t) @ relu


def _minmax_keys_swapped(k_hat, sub_block):
    k_max, k_min = orc.__dict__["_orig_minmax"](k_hat, sub_block)
    return k_min, k_max


def _pages_shifted(lo, hi, prm):
    return np.arange(lo // prm.page, hi // prm.page)


def _candidates_ignore_pages(pages, lo, hi, prm):
    return np.arange(lo, hi + 1, dtype=np.int64)


def _mean_keys_not_rounded(k_hat, sub_block):
    k_hat = np.asarray(k_hat, np.float64)
    n = k_hat.shape[0] // sub_block
    return k_hat[: n * sub_block].reshape(n, sub_block, -1).mean(axis=1)


def _scores_on_value_columns(q_t_bits, kv_bits, v_bits, S, d_v, scale):
    S = np.asarray(S, np.int64)
    k = orc.bf16_bits_to_f64(kv_bits[S])
    v = k[:, :d_v] if v_bits is None else orc.bf16_bits_to_f64(v_bits[S])
    q = orc.bf16_bits_to_f64(q_t_bits)
    return orc.sparse_attention_row(q[:, :d_v], k[:, :d_v], v, scale)


def _latent_v_last_columns(q_t_bits, kv_bits, v_bits, S, d_v, scale):
    S = np.asarray(S, np.int64)
    k = orc.bf16_bits_to_f64(kv_bits[S])
    v = k[:, -d_v:] if v_bits is None else orc.bf16_bits_to_f64(v_bits[S])
    return orc.sparse_attention_row(orc.bf16_bits_to_f64(q_t_bits), k, v, scale)


def _runs_without_align_cut(S, align):
    runs = []
    for s in np.asarray(S, np.int64).tolist():
        if runs and s == runs[-1][0] + runs[-1][1]:
            runs[-1][1] += 1
        else:
            runs.append([s, 1])
    return [(a, n) for a, n in runs]


def _key_scale_ignored(k, k_scale=None):
    k = np.asarray(k)
    return orc.e4m3fn_to_f64(k) if k.dtype == np.uint8 else orc.bf16_bits_to_f64(k)


MUTANTS = {
    "no_relu": ("indexer_scores", _no_relu),
    "relu_after_head_sum": ("indexer_scores", _relu_after_sum),
    "max_instead_of_mean": ("sub_block_mean_keys", _max_pool),
    "window_off_by_one": ("streaming_sets", _window_off_by_one),
    "sink_excluded": ("streaming_sets", _no_sink),
    "ties_to_later_position": ("arg_top", _ties_to_later),
    "bf16_truncation": ("f64_to_bf16_bits", _truncating_bf16),
    "e4m3_wrong_bias": ("e4m3fn_to_f64", _e4m3_bias8),
    "candidates_leak_into_window": ("candidates_of_pages", _cand_with_window),
    "attention_scale_dropped": ("sparse_attention_row", _attn_no_scale),
    "lse_in_log2": ("sparse_attention_row", _attn_log2),
    "page_score_ignores_w": ("page_scores", _page_score_unweighted),
    "last_eligible_page_dropped": ("eligible_pages", _pages_shifted),
    "minmax_min_of_products": ("page_scores_minmax", _minmax_min_of_products),
    "minmax_extrema_swapped": ("sub_block_minmax_keys", _minmax_keys_swapped),
    "latent_v_from_last_columns": ("attention_for_set", _latent_v_last_columns),
    "runs_not_cut_at_multiples_of_c": ("runs_of", _runs_without_align_cut),
    "key_scale_ignored": ("dequantized_keys", _key_scale_ignored),
    "candidates_ignore_recalled_pages": ("candidates_of_pages", _candidates_ignore_pages),
    "mean_keys_not_rounded_to_bf16": ("sub_block_mean_keys", _mean_keys_not_rounded),
    "attention_scores_on_value_columns_only": ("attention_for_set", _scores_on_value_columns),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    monkeypatch.setitem(orc.__dict__, "_orig_attn", orc.sparse_attention_row)
    monkeypatch.setitem(orc.__dict__, "_orig_page", orc.page_scores)
    monkeypatch.setitem(orc.__dict__, "_orig_minmax", orc.sub_block_minmax_keys)
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(orc, attr, fn)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(orc)
        except Exception:  # an assertion or a crash both count as the pin catching the mutant
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"


def test_worked_example_fixture():
    """The oracle reproduces a worked example derived by hand from Eq. (1), (3), (6)-(7) and
    (9)-(12) (tests/golden/worked_example.json, derivations inside)."""
    import json
    import os
    fx = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")))
    q, w, keys, t = np.array(fx["q"], float), np.array(fx["w"], float), np.array(fx["keys"], float), fx["t"]
    c = fx["cases"]
    assert np.array_equal(orc.indexer_scores(q, w, keys), np.array(c["scores"]["expected"], float))
    for name in ("flat", "flat_tie", "hierarchical"):
        prm = orc.IndexParams(**c[name]["params"])
        k_mean = orc.sub_block_mean_keys(keys, prm.sub_block)
        r = orc.index_row(t, q, w, keys, k_mean, prm)
        assert r["S"].tolist() == c[name]["S"], name
        if "runs" in c[name]:
            assert [list(x) for x in orc.runs_of(r["S"], prm.run_align)] == c[name]["runs"], name
        if "pages" in c[name]:
            assert r["pages"].tolist() == c[name]["pages"]
            assert r["page_ids"].tolist() == c[name]["page_ids"]
            assert np.array_equal(r["page_score"], np.array(c[name]["page_score"], float))
    a = c["attention"]
    o, lse = orc.sparse_attention_row(np.array(a["q"], float), np.array(a["keys"], float), np.array(a["values"], float),
                                      a["scale"])
    assert np.allclose(o, np.array(a["o"]), rtol=1e-14, atol=0) and np.allclose(lse, np.array(a["lse"]), rtol=1e-14)
