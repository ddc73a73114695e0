"""Pins for the CPU oracle against facts fixed outside it.

Each test checks the oracle against something it does not compute itself:
published Philox vectors, hand-computed prologue values from the paper's
equations, library routines (lexsort, argmax, softmax) on cases that reduce
to them, invariants of the truncation rules, and chi-square tests of the
sampling and verification distributions.
"""
import json
import math
import os

import numpy as np
import pytest
from scipy import special, stats

import oracle
from gen import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _num(v):
    if isinstance(v, str):
        return {"-inf": -np.inf, "inf": np.inf, "nan": np.nan, "-0.0": -0.0}[v]
    return v


# --------------------------------------------------------------------------
# Philox4x32-10 and the uniform mapping
# --------------------------------------------------------------------------
def test_philox_published_vectors():
    for v in _load("philox_kat.json")["vectors"]:
        out = oracle.philox4x32_10([int(c, 16) for c in v["ctr"]], [int(k, 16) for k in v["key"]])
        assert out == [int(o, 16) for o in v["out"]]


def test_uniform_layout_uses_counter_request_position():
    # seed 0, request 0, position 0 is the all-zero counter/key vector
    v0 = _load("philox_kat.json")["vectors"][0]
    for word in range(4):
        u = oracle.uniform(0, 0, 0, word)
        assert u == (int(v0["out"][word], 16) + 0.5) / 2.0**32
    us = [oracle.uniform(1234, r, p, w) for r in range(8) for p in range(8) for w in range(2)]
    assert all(0.0 < u < 1.0 for u in us)
    assert len(set(us)) == len(us)


@pytest.mark.parametrize("seed,req,position", [
    (0x0123456789ABCDEF, 5, (1 << 33) + 7),
    (1234, 63, 1),
    (0xFFFFFFFF00000001, 1, 0x7FFFFFFFFFFFFFFF),
])
def test_uniform_counter_words_are_request_then_position(seed, req, position):
    """The uniform of (seed, request, position, word) is word `word` of the
    published Philox4x32-10 block at counter (request, position lo, position
    hi, 0) under key (seed lo, seed hi) (reading R14), mapped as (w + 1/2) 2^-32.
    Non-zero request and a position above 2^32 make every counter word matter,
    so a swapped or shifted word fails here."""
    ctr = [req, position & 0xFFFFFFFF, position >> 32, 0]
    key = [seed & 0xFFFFFFFF, seed >> 32]
    out = oracle.philox4x32_10(ctr, key)
    for word in range(4):
        assert oracle.uniform(seed, req, position, word) == (out[word] + 0.5) / 2.0**32
    swapped = oracle.philox4x32_10([ctr[1], ctr[0], ctr[2], 0], key)
    assert swapped != out


# --------------------------------------------------------------------------
# Prologue: hand-computed values from the paper's equations
# --------------------------------------------------------------------------
@pytest.mark.parametrize("case", _load("prologue_cases.json")["cases"], ids=lambda c: c["name"])
def test_prologue_golden(case):
    if "x_arange" in case:
        x = np.arange(case["x_arange"], dtype=np.float32)
    else:
        x = np.array([_num(v) for v in case["x"]], np.float32)
    y = oracle.process_row(
        x, "f32", case["mode"], rep=case.get("rep", 1.0), freq=case.get("freq", 0.0),
        pres=case.get("pres", 0.0), hist=case.get("hist", []), bias_ids=case.get("bias_ids", []),
        bias_vals=case.get("bias_vals", []),
        mask_row=None if "mask" not in case else np.array(case["mask"], np.uint32))
    if "y_allowed" in case:
        allowed = set(case["y_allowed"])
        for i, v in enumerate(y):
            assert (v == x[i]) if i in allowed else (v == -np.inf)
        return
    want = np.array([_num(v) for v in case["y"]], np.float32)
    assert np.array_equal(y.view(np.uint32), want.view(np.uint32)), (y, want)


def test_prologue_bf16_widening_is_exact():
    rng = np.random.default_rng(0)
    f = rng.normal(0, 3, 4096).astype(np.float32)
    h = W.bf16_bits_from_f32(f)
    y = oracle.process_row(h, "bf16", 0)
    assert np.array_equal(y, W.f32_from_bf16_bits(h))


# --------------------------------------------------------------------------
# Ordering and top-k: brute force against numpy's lexsort
# --------------------------------------------------------------------------
def _lexsort_topk(y, k):
    valid = np.nonzero(y > -np.inf)[0]
    o = valid[np.lexsort((valid, -y[valid].astype(np.float64)))]
    return o[:k]


@pytest.mark.parametrize("kind", ["normal", "ties", "zeros", "bf16_flat", "masked"])
def test_topk_matches_lexsort(kind):
    rng = np.random.default_rng(11)
    B, V, km = 6, 3000, 300
    if kind == "normal":
        x = rng.normal(0, 2, (B, V)).astype(np.float32)
    elif kind == "ties":
        x = rng.integers(-20, 20, (B, V)).astype(np.float32) / 4
    elif kind == "zeros":
        x = np.zeros((B, V), np.float32)
    elif kind == "bf16_flat":
        # U(128.6, 128.7) rounds to 129.0 in bf16: an all-ties row (paper, Section 4.4)
        x = W.f32_from_bf16_bits(W.bf16_bits_from_f32(rng.uniform(128.6, 128.7, (B, V)).astype(np.float32)))
        assert np.all(x == 129.0)
    else:
        x = rng.normal(0, 1, (B, V)).astype(np.float32)
        x[:, ::3] = -np.inf
        x[:, 1::7] = np.nan
    k = np.array([1, 7, 50, 300, 0, 299], np.int32)
    inp = W.custom_rows(x, W.F32, k_max=km, top_k=k)
    val, idx = oracle.topk(inp)
    for b in range(B):
        yb = np.where(np.isnan(x[b]), -np.inf, x[b])
        want = _lexsort_topk(yb, min(int(k[b]), km))
        n = len(want)
        assert np.array_equal(idx[b, :n], want)
        assert np.array_equal(val[b, :n], yb[want])
        assert np.all(idx[b, n:] == -1) and np.all(val[b, n:] == -np.inf)


def test_topk_negative_zero_ties_positive_zero():
    x = np.array([[np.nan, -0.0, 0.0, 1.0]], np.float32)
    val, idx = oracle.topk(W.custom_rows(x, W.F32, k_max=4, top_k=[4]))
    assert list(idx[0]) == [3, 1, 2, -1]
    assert np.array_equal(val[0, :3], np.array([1.0, 0.0, 0.0], np.float32))
    assert not np.signbit(val[0, 1])


# --------------------------------------------------------------------------
# Greedy = first argmax of the processed logits
# --------------------------------------------------------------------------
def test_greedy_is_first_argmax():
    inp = W.config1(B=8)
    inp["mode"][:] = W.MODE_GREEDY | W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
    out = oracle.sample(inp)
    y = oracle.process_logits(inp)["y"]
    for b in range(inp["B"]):
        assert out["token"][b] == int(np.argmax(y[b]))
    # temperature 0 with the TEMP bit also means greedy
    inp2 = W.config0()
    o2 = oracle.sample(inp2)
    assert o2["token"][0] == int(np.argmax(inp2["x"][0]))


def test_greedy_ties_take_lowest_index():
    x = np.zeros((1, 64), np.float32)
    x[0, [5, 9, 40]] = 3.0
    o = oracle.sample(W.custom_rows(x, W.F32, mode=[W.MODE_GREEDY]))
    assert o["token"][0] == 5


def test_empty_row_returns_minus_one():
    x = np.ones((1, 64), np.float32)
    inp = W.custom_rows(x, W.F32, mode=[W.MODE_GRAMMAR | W.MODE_TEMP], bitmask=np.zeros((1, 2), np.uint32))
    o = oracle.sample(inp)
    assert o["token"][0] == -1 and (o["flags"][0] & 1)


# --------------------------------------------------------------------------
# Truncation rules against softmax (scipy) on cases that reduce to it
# --------------------------------------------------------------------------
def _softmax_sorted(y, tau):
    o = np.lexsort((np.arange(y.size), -y.astype(np.float64)))
    p = special.softmax(y[o].astype(np.float64) / tau)
    return o, p


@pytest.mark.parametrize("seed", range(6))
def test_top_p_is_minimal_prefix_with_mass_p(seed):
    rng = np.random.default_rng(100 + seed)
    V = 500
    y = rng.normal(0, 2, V).astype(np.float32)
    tau = float(rng.uniform(0.5, 1.5))
    p = float(rng.uniform(0.3, 0.99))
    d = oracle.row_distribution(y, W.MODE_TEMP | W.MODE_TOPP, temperature=tau, top_p=p, k_cap=V)
    o, sp = _softmax_sorted(y, np.float32(tau))
    assert np.array_equal(d["order"], o)
    cum = np.cumsum(sp)
    n = d["n_p"]
    assert cum[n - 1] >= p - 1e-12          # kept mass reaches p
    assert n == 1 or cum[n - 2] < p + 1e-12  # one fewer does not
    assert np.allclose(d["P"], sp[:n] / sp[:n].sum(), rtol=1e-12, atol=0)


@pytest.mark.parametrize("seed", range(6))
def test_min_p_keeps_tokens_with_p_at_least_theta_pmax(seed):
    rng = np.random.default_rng(200 + seed)
    V = 400
    y = rng.normal(0, 2, V).astype(np.float32)
    tau = float(rng.uniform(0.5, 1.5))
    theta = float(rng.uniform(0.01, 0.5))
    d = oracle.row_distribution(y, W.MODE_TEMP | W.MODE_MINP, temperature=tau, min_p=theta, k_cap=V)
    o, sp = _softmax_sorted(y, np.float32(tau))
    keep = sp >= np.float32(theta) * sp[0]
    assert d["margin_m"] > 1e-9
    assert d["n_m"] == int(keep.sum())
    assert np.all(keep[: d["n_m"]])


def test_top_k_then_top_p_renormalises_within_top_k():
    # three tokens with softmax masses 0.5, 0.3, 0.2 (tau=1); top-k=2 renormalises
    # to 0.625/0.375, so top-p=0.6 keeps one token; without top-k it keeps two.
    y = np.log(np.array([0.5, 0.3, 0.2])).astype(np.float32)
    d1 = oracle.row_distribution(y, W.MODE_TOPK | W.MODE_TOPP, top_k=2, top_p=0.6, k_cap=3)
    d2 = oracle.row_distribution(y, W.MODE_TOPP, top_p=0.6, k_cap=3)
    assert d1["n_s"] == 1 and d2["n_s"] == 2


def test_temperature_two_token_closed_form():
    for a, b, tau in [(1.0, 0.0, 1.0), (2.0, -1.0, 0.5), (0.25, 0.0, 2.0)]:
        y = np.array([a, b], np.float32)
        d = oracle.row_distribution(y, W.MODE_TEMP, temperature=tau, k_cap=2)
        p0 = 1.0 / (1.0 + math.exp(-(a - b) / tau))
        assert abs(d["P"][0] - p0) < 1e-15 and abs(d["P"][1] - (1 - p0)) < 1e-15


def test_probability_ratio_identity():
    rng = np.random.default_rng(5)
    y = rng.normal(0, 1, 64).astype(np.float32)
    d = oracle.row_distribution(y, W.MODE_TEMP, temperature=0.7, k_cap=64)
    ys = y[d["order"]].astype(np.float64)
    r = d["P"][1:] / d["P"][0]
    assert np.allclose(r, np.exp((ys[1:] - ys[0]) / np.float64(np.float32(0.7))), rtol=1e-13)


def test_k_cap_bounds_rows_without_top_k():
    y = np.random.default_rng(3).normal(0, 1, 100).astype(np.float32)
    d = oracle.row_distribution(y, W.MODE_TEMP, k_cap=10)
    assert d["n_k"] == 10 and d["n_s"] == 10 and (d["flags"] & 8)
    d2 = oracle.row_distribution(y, W.MODE_TEMP | W.MODE_TOPK, top_k=5, k_cap=10)
    assert d2["n_k"] == 5 and not (d2["flags"] & 8)


# --------------------------------------------------------------------------
# Draw
# --------------------------------------------------------------------------
@pytest.mark.parametrize("case", _load("draw_cases.json")["cases"])
def test_draw_golden(case):
    assert oracle.draw(case["w"], case["u"]) == case["pick"]


def _chi2_ok(counts, probs, alpha=1e-4):
    n = counts.sum()
    exp = probs * n
    keep = exp > 5
    lump_c = counts[~keep].sum()
    lump_e = exp[~keep].sum()
    c = np.append(counts[keep], lump_c) if lump_e > 0 else counts[keep]
    e = np.append(exp[keep], lump_e) if lump_e > 0 else exp[keep]
    stat, pv = stats.chisquare(c, e * c.sum() / e.sum())
    return pv > alpha, pv


def test_sampling_distribution_chi_square():
    V, B = 12, 40000
    y = np.random.default_rng(7).normal(0, 1, V).astype(np.float32)
    x = np.tile(y, (B, 1))
    inp = W.custom_rows(x, W.F32, k_max=V,
                        mode=np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP),
                        temperature=np.full(B, 0.8), top_k=np.full(B, 9), top_p=np.full(B, 0.95),
                        position=np.arange(B))
    tok = oracle.sample(inp)["token"]
    d = oracle.row_distribution(y, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP, temperature=0.8,
                                top_k=9, top_p=0.95, k_cap=V)
    probs = np.zeros(V)
    probs[d["order"][: d["n_s"]]] = d["P"]
    # kept set equals the softmax top-p rule on the renormalised top-9
    o, sp = _softmax_sorted(y, np.float32(0.8))
    sp9 = sp[:9] / sp[:9].sum()
    n = int(np.searchsorted(np.cumsum(sp9), 0.95) + 1)
    assert d["n_s"] == n
    counts = np.bincount(tok, minlength=V).astype(np.float64)
    assert counts[probs == 0].sum() == 0
    ok, pv = _chi2_ok(counts[probs > 0], probs[probs > 0])
    assert ok, pv


# --------------------------------------------------------------------------
# Full-row truncation for requests without a top-k cut (Appendix C.2)
# --------------------------------------------------------------------------
def _full_rows(y, k_max, mode, **params):
    B = y.shape[0]
    return W.custom_rows(y, W.F32, k_max=k_max, mode=np.full(B, mode), position=np.arange(B) * 3, **params)


@pytest.mark.parametrize("seed", range(4))
def test_full_row_top_p_uses_the_whole_row(seed):
    # a head plus a long tail: the top-p cut over the whole row (scipy softmax
    # over every token) lies inside k_max but differs from the cut over the
    # k_max leading tokens; the kept set and the drawn token's probability
    # follow the whole-row rule
    rng = np.random.default_rng(300 + seed)
    V, k_max, B, p, tau = 600, 64, 16, 0.8, np.float32(0.9)
    y = rng.normal(0, 0.3, (B, V)).astype(np.float32)
    y[:, rng.choice(V, 12, replace=False)] += rng.uniform(5.0, 6.0, 12).astype(np.float32)
    mode = W.MODE_TEMP | W.MODE_TOPP
    inp = _full_rows(y, k_max, mode, temperature=np.full(B, tau), top_p=np.full(B, p))
    o = oracle.sample_full(inp)
    ob = oracle.sample(inp)
    differ = 0
    for b in range(B):
        order, sp = _softmax_sorted(y[b], tau)
        n = int(np.searchsorted(np.cumsum(sp), p) + 1)
        assert n < k_max
        assert o["n_kept"][b] == n
        kept = sp[:n] / sp[:n].sum()
        r = int(np.nonzero(order == o["token"][b])[0][0])
        assert r < n and abs(float(o["logprob"][b]) - math.log(kept[r])) < 1e-6
        assert (o["flags"][b] & 8) == 0  # not bounded
        differ += int(o["n_kept"][b] != ob["n_kept"][b])
    assert differ > 0


def test_full_row_overflow_falls_back_to_the_bounded_result():
    # a flat row keeps ~90 % of 500 tokens under top-p 0.9: more than k_max,
    # so the result is ssref_sample's (top-p over the k_max leading tokens) with
    # the KCAP flag; the same at a kept set of exactly k_max tokens
    V, k_max, B = 500, 64, 6
    y = np.zeros((B, V), np.float32)
    inp = _full_rows(y, k_max, W.MODE_TOPP, top_p=np.full(B, 0.9))
    o, ob = oracle.sample_full(inp), oracle.sample(inp)
    assert np.array_equal(o["token"], ob["token"]) and np.array_equal(o["n_kept"], ob["n_kept"])
    assert np.all(o["flags"] & 8)
    # min-p keeping exactly k_max tokens of a row longer than k_max: overflow
    y2 = np.full((B, V), -10.0, np.float32)
    y2[:, :k_max] = 0.0
    inp2 = _full_rows(y2, k_max, W.MODE_MINP, min_p=np.full(B, 0.5))
    o2 = oracle.sample_full(inp2)
    assert np.all(o2["flags"] & 8) and np.all(o2["n_kept"] == k_max)
    # one token fewer fits: the whole-row result without the flag
    y3 = y2.copy()
    y3[:, k_max - 1] = -10.0
    o3 = oracle.sample_full(_full_rows(y3, k_max, W.MODE_MINP, min_p=np.full(B, 0.5)))
    assert np.all((o3["flags"] & 8) == 0) and np.all(o3["n_kept"] == k_max - 1)
    # a row with fewer valid tokens than k_max always fits; one with exactly
    # k_max keeps them all too, with the flag (its bounded set is the row)
    o4 = oracle.sample_full(_full_rows(np.zeros((B, 50), np.float32), k_max, W.MODE_TEMP))
    assert np.all((o4["flags"] & 8) == 0) and np.all(o4["n_kept"] == 50)
    o5 = oracle.sample_full(_full_rows(np.zeros((B, k_max), np.float32), k_max, W.MODE_TEMP))
    assert np.all(o5["flags"] & 8) and np.all(o5["n_kept"] == k_max)


def test_full_row_leaves_other_requests_alone():
    # top-k requests (k <= k_max and k > k_max) and greedy ones are sampled as by ssref_sample
    rng = np.random.default_rng(12)
    V, B = 300, 12
    y = rng.normal(0, 1, (B, V)).astype(np.float32)
    mode = np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP, np.uint32)
    mode[::4] = W.MODE_GREEDY
    inp = W.custom_rows(y, W.F32, k_max=64, mode=mode, temperature=np.full(B, 0.8),
                        top_k=np.where(np.arange(B) % 3 == 0, 200, 20), top_p=np.full(B, 0.95),
                        position=np.arange(B))
    o, ob = oracle.sample_full(inp), oracle.sample(inp)
    for k in ("token", "logprob", "flags", "n_kept"):
        assert np.array_equal(o[k], ob[k]), k


def test_full_row_draws_follow_the_whole_row_distribution_chi_square():
    V, B, p = 40, 40000, 0.9
    rng = np.random.default_rng(23)
    yv = rng.normal(0, 1.2, V).astype(np.float32)
    inp = W.custom_rows(np.tile(yv, (B, 1)), W.F32, k_max=32, mode=np.full(B, W.MODE_TOPP),
                        top_p=np.full(B, p), position=np.arange(B))
    o = oracle.sample_full(inp)
    order, sp = _softmax_sorted(yv, np.float32(1.0))
    n = int(np.searchsorted(np.cumsum(sp), p) + 1)
    assert n < 32 and np.all(o["n_kept"] == n)
    probs = np.zeros(V)
    probs[order[:n]] = sp[:n] / sp[:n].sum()
    counts = np.bincount(o["token"], minlength=V).astype(np.float64)
    assert counts[probs == 0].sum() == 0
    ok, pv = _chi2_ok(counts[probs > 0], probs[probs > 0])
    assert ok, pv


# --------------------------------------------------------------------------
# Gumbel-max draw (Appendix C.3)
# --------------------------------------------------------------------------
def test_gumbel_draw_follows_truncated_distribution_chi_square():
    # with g = ln z, z ~ Exp(1) fresh per row, the Gumbel-max pick over the kept
    # set is distributed as the truncated distribution P (the reparameterisation)
    V, B = 12, 40000
    rng = np.random.default_rng(17)
    y = rng.normal(0, 1, V).astype(np.float32)
    mode = W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP
    inp = W.custom_rows(np.tile(y, (B, 1)), W.F32, k_max=V, mode=np.full(B, mode), temperature=np.full(B, 0.7),
                        top_k=np.full(B, 9), top_p=np.full(B, 0.95))
    g = np.log(rng.exponential(size=(B, V))).astype(np.float32)
    tok = oracle.sample_gumbel(inp, g)["token"]
    d = oracle.row_distribution(y, mode, temperature=0.7, top_k=9, top_p=0.95, k_cap=V)
    probs = np.zeros(V)
    probs[d["order"][: d["n_s"]]] = d["P"]
    counts = np.bincount(tok, minlength=V).astype(np.float64)
    assert counts[probs == 0].sum() == 0
    ok, pv = _chi2_ok(counts[probs > 0], probs[probs > 0])
    assert ok, pv


def test_gumbel_draw_hand_cases():
    # two tokens y = (1, 0): the pick is token 0 iff (0 - g0) > (-1/tau - g1)
    tau = np.float32(0.5)
    y = np.array([[1.0, 0.0]], np.float32)
    inp = W.custom_rows(y, W.F32, k_max=2, mode=np.array([W.MODE_TEMP]), temperature=np.array([tau]))
    for g0, g1, want in ((0.0, 0.0, 0), (1.9, 0.0, 0), (2.1, 0.0, 1), (0.0, -2.1, 1), (-3.0, -4.9, 0),
                         (-3.0, -5.1, 1)):
        g = np.array([[g0, g1]], np.float32)
        assert int(oracle.sample_gumbel(inp, g)["token"][0]) == want, (g0, g1)
    # equal scores: the lower token id
    y2 = np.array([[0.0, 1.0, 0.0]], np.float32)
    inp2 = W.custom_rows(y2, W.F32, k_max=3, mode=np.array([0]))
    o = oracle.sample_gumbel(inp2, np.array([[0.0, 1.0, 0.0]], np.float32))
    assert int(o["token"][0]) == 0
    # zero noise is the argmax (greedy as z = 1), with its truncated log-probability
    yr = np.random.default_rng(3).normal(0, 1, (4, 50)).astype(np.float32)
    inp3 = W.custom_rows(yr, W.F32, k_max=50, mode=np.full(4, W.MODE_TEMP | W.MODE_TOPK),
                         temperature=np.full(4, 1.3), top_k=np.full(4, 5))
    o = oracle.sample_gumbel(inp3, np.zeros((4, 50), np.float32))
    assert np.array_equal(o["token"], np.argmax(yr, axis=1))
    sp = special.softmax(np.sort(yr.astype(np.float64), axis=1)[:, ::-1][:, :5] / np.float32(1.3), axis=1)
    assert np.allclose(o["logprob"], np.log(sp[:, 0]), rtol=1e-6)


def test_gumbel_draw_never_leaves_the_kept_set():
    # a token outside the top-k with a very large perturbation is still excluded
    V, B = 40, 64
    rng = np.random.default_rng(5)
    y = rng.normal(0, 1, (B, V)).astype(np.float32)
    g = np.log(rng.exponential(size=(B, V))).astype(np.float32)
    order = np.argsort(-y, axis=1, kind="stable")
    for b in range(B):
        g[b, order[b, 6:]] = -1e6  # score +1e6 outside the top 6
    inp = W.custom_rows(y, W.F32, k_max=V, mode=np.full(B, W.MODE_TOPK), top_k=np.full(B, 6))
    tok = oracle.sample_gumbel(inp, g)["token"]
    assert all(tok[b] in order[b, :6] for b in range(B))
    # greedy rows ignore the noise
    inp = W.custom_rows(y, W.F32, k_max=V, mode=np.full(B, W.MODE_GREEDY))
    assert np.array_equal(oracle.sample_gumbel(inp, g)["token"], np.argmax(y, axis=1))


# --------------------------------------------------------------------------
# Speculative verification
# --------------------------------------------------------------------------
def _verify_inputs(x_rows, q, d, mode, L, **params):
    """x_rows [B, L+1, V] float32, q [B, L, V], d [B, L]."""
    B = x_rows.shape[0]
    inp = W.custom_rows(x_rows.reshape(B * (L + 1), -1), W.F32, k_max=x_rows.shape[-1], mode=mode, **params)
    inp["x"] = x_rows
    inp["B"] = B
    for k in ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres", "seed", "position"):
        if inp[k] is not None and inp[k].shape[0] != B:
            inp[k] = inp[k][:B]
    inp["hist_offsets"] = inp["hist_offsets"][: B + 1] if inp["hist_offsets"].shape[0] > B + 1 else inp["hist_offsets"]
    inp["bias_offsets"] = inp["bias_offsets"][: B + 1] if inp["bias_offsets"].shape[0] > B + 1 else inp["bias_offsets"]
    inp["L"] = L
    inp["draft_probs"] = q.astype(np.float32)
    inp["draft_tokens"] = d.astype(np.int32)
    return inp


def test_verify_first_token_follows_target_chi_square():
    V, B, L = 8, 40000, 1
    rng = np.random.default_rng(21)
    t = rng.normal(0, 1, V).astype(np.float32)
    qv = special.softmax(rng.normal(0, 1, V)).astype(np.float32)
    d = rng.choice(V, size=(B, L), p=qv / qv.sum())
    x = np.tile(t, (B, L + 1, 1))
    q = np.tile(qv, (B, L, 1))
    inp = _verify_inputs(x, q, d, np.full(B, W.MODE_TEMP), L, temperature=np.full(B, 0.9),
                         position=np.arange(B) * 7)
    out = oracle.verify(inp)
    first = out["tokens"][:, 0]
    assert np.all(first >= 0)
    p = special.softmax(t.astype(np.float64) / np.float32(0.9))
    ok, pv = _chi2_ok(np.bincount(first, minlength=V).astype(float), p)
    assert ok, pv
    # acceptance rate of one draft equals sum_x min(p(x), q(x)) (Leviathan et al.)
    acc = float(np.mean(out["n_acc"] == 1))
    want = float(np.minimum(p, qv.astype(np.float64)).sum())
    assert abs(acc - want) < 4 * math.sqrt(want * (1 - want) / B)


def test_verify_second_token_uses_accepted_draft_history():
    # With a repetition penalty the target for position 2 depends on token 1;
    # conditioned on token 1, token 2 must follow that penalised target.
    V, B, L = 6, 60000, 2
    rng = np.random.default_rng(33)
    t = rng.normal(0, 0.7, V).astype(np.float32)
    qv = special.softmax(rng.normal(0, 0.5, V)).astype(np.float32)
    d = rng.choice(V, size=(B, L), p=qv / qv.sum())
    x = np.tile(t, (B, L + 1, 1))
    q = np.tile(qv, (B, L, 1))
    mode = W.MODE_TEMP | W.MODE_REP | W.MODE_PRES
    inp = _verify_inputs(x, q, d, np.full(B, mode), L, temperature=np.full(B, 1.0),
                         rep=np.full(B, 3.0), pres=np.full(B, 1.0), position=np.arange(B) * 5,
                         hist_offsets=np.zeros(B + 1, np.int32))
    out = oracle.verify(inp)
    tok = out["tokens"]
    two = tok[:, 1] >= 0
    assert two.sum() > 5000
    for t1 in range(V):
        sel = two & (tok[:, 0] == t1)
        if sel.sum() < 500:
            continue
        ypen = oracle.process_row(t, "f32", mode, rep=3.0, pres=1.0, hist=[t1])
        p2 = special.softmax(ypen.astype(np.float64))
        ok, pv = _chi2_ok(np.bincount(tok[sel, 1], minlength=V).astype(float), p2)
        assert ok, (t1, pv)


def test_verify_special_cases():
    V, L, B = 16, 3, 64
    rng = np.random.default_rng(4)
    t = rng.normal(0, 1, V).astype(np.float32)
    x = np.tile(t, (B, L + 1, 1))
    p = special.softmax(t.astype(np.float64))
    # q equal to the target: every draft is accepted, bonus appended
    d = rng.choice(V, size=(B, L), p=p)
    inp = _verify_inputs(x, np.tile(p.astype(np.float32), (B, L, 1)), d, np.full(B, W.MODE_TEMP), L,
                         position=np.arange(B))
    o = oracle.verify(inp)
    # float32 rounding of q can exceed P by an ulp; acceptance is then u*q <= P almost surely
    assert np.mean(o["n_acc"] == L) > 0.95
    # draft outside the target's top-k: P(d) = 0, always rejected
    order = np.argsort(-t, kind="stable")
    d0 = np.tile(order[-1], (B, L))
    inp = _verify_inputs(x, np.tile(p.astype(np.float32), (B, L, 1)), d0,
                         np.full(B, W.MODE_TEMP | W.MODE_TOPK), L, top_k=np.full(B, 4), position=np.arange(B))
    o = oracle.verify(inp)
    assert np.all(o["n_acc"] == 0) and np.all(np.isin(o["tokens"][:, 0], order[:4]))
    assert np.all(o["tokens"][:, 1:] == -1)
    # greedy: accept iff the draft is the argmax; correction is the argmax
    am = int(np.argmax(t))
    d1 = np.full((B, L), am)
    d1[::2, 1] = order[1]
    inp = _verify_inputs(x, np.tile(p.astype(np.float32), (B, L, 1)), d1, np.full(B, W.MODE_GREEDY), L)
    o = oracle.verify(inp)
    assert np.all(o["n_acc"][1::2] == L) and np.all(o["tokens"][1::2, L] == am)
    assert np.all(o["n_acc"][::2] == 1) and np.all(o["tokens"][::2, :2] == am)
    # a negative draft id ends the draft: that position samples from the target
    d2 = np.full((B, L), -1)
    inp = _verify_inputs(x, np.tile(p.astype(np.float32), (B, L, 1)), d2, np.full(B, W.MODE_GREEDY), L)
    o = oracle.verify(inp)
    assert np.all(o["n_acc"] == 0) and np.all(o["tokens"][:, 0] == am)


def _sparse(inp, idx, qv):
    """Replaces the dense draft distribution of ``inp`` by sparse lists."""
    inp = dict(inp)
    inp.pop("draft_probs")
    inp["draft_idx"] = np.ascontiguousarray(idx, np.int32)
    inp["draft_q"] = np.ascontiguousarray(qv, np.float32)
    return inp


def test_verify_sparse_first_token_follows_target_chi_square():
    # q supported on 4 of 8 ids, listed with a duplicated id (two entries whose
    # sum is its probability), padding and an out-of-range id: the first output
    # token still follows the target exactly (the guarantee of speculative
    # sampling holds for any q the draft was drawn from), and one draft is
    # accepted with probability sum_x min(p(x), q(x)).
    V, B, L = 8, 40000, 1
    rng = np.random.default_rng(27)
    t = rng.normal(0, 1, V).astype(np.float32)
    support = np.array([5, 1, 6, 2])
    qs = np.array([0.4375, 0.25, 0.1875, 0.125])  # exact in float32
    qd = np.zeros(V)
    qd[support] = qs
    d = rng.choice(V, size=(B, L), p=qd)
    idx = np.array([5, 1, -1, 6, 2, 1, V, 9999], np.int32)
    val = np.array([0.4375, 0.125, 0.5, 0.1875, 0.125, 0.125, 0.3, 0.2], np.float32)
    x = np.tile(t, (B, L + 1, 1))
    inp = _verify_inputs(x, np.zeros((B, L, V)), d, np.full(B, W.MODE_TEMP), L, temperature=np.full(B, 0.8),
                         position=np.arange(B) * 3)
    out = oracle.verify(_sparse(inp, np.tile(idx, (B, L, 1)), np.tile(val, (B, L, 1))))
    first = out["tokens"][:, 0]
    assert np.all(first >= 0)
    p = special.softmax(t.astype(np.float64) / np.float32(0.8))
    ok, pv = _chi2_ok(np.bincount(first, minlength=V).astype(float), p)
    assert ok, pv
    acc = float(np.mean(out["n_acc"] == 1))
    want = float(np.minimum(p, qd).sum())
    assert abs(acc - want) < 4 * math.sqrt(want * (1 - want) / B)


def test_verify_sparse_lists_are_per_position():
    # two draft positions with different targets and different sparse lists:
    # conditioned on the first draft being accepted, the second output token
    # follows the second target, which needs the second position's own list
    V, B, L = 6, 60000, 2
    rng = np.random.default_rng(35)
    t = rng.normal(0, 0.8, (L + 1, V)).astype(np.float32)
    lists = [(np.array([0, 3, 4]), np.array([0.5, 0.375, 0.125])),
             (np.array([2, 5, 1]), np.array([0.625, 0.25, 0.125]))]
    idx = np.full((B, L, 3), -1, np.int32)
    val = np.zeros((B, L, 3), np.float32)
    d = np.empty((B, L), np.int64)
    for l, (ii, qq) in enumerate(lists):
        idx[:, l] = ii
        val[:, l] = qq
        d[:, l] = rng.choice(ii, size=B, p=qq)
    x = np.tile(t, (B, 1, 1))
    inp = _verify_inputs(x, np.zeros((B, L, V)), d, np.full(B, W.MODE_TEMP), L, temperature=np.full(B, 1.0),
                         position=np.arange(B) * 5)
    out = oracle.verify(_sparse(inp, idx, val))
    tok = out["tokens"]
    sel = out["n_acc"] >= 1
    assert sel.sum() > 5000
    p2 = special.softmax(t[1].astype(np.float64))
    ok, pv = _chi2_ok(np.bincount(tok[sel, 1], minlength=V).astype(float), p2)
    assert ok, pv


def test_verify_sparse_matches_dense_scatter():
    # lists without repeated ids give the outcome (tokens, accepted counts and
    # admissible sets) of the dense q they scatter to
    V, L, B = 64, 3, 48
    rng = np.random.default_rng(12)
    t = rng.normal(0, 1.5, (B, L + 1, V)).astype(np.float32)
    kq = 12
    idx = np.full((B, L, kq), -1, np.int32)
    val = np.zeros((B, L, kq), np.float32)
    dense = np.zeros((B, L, V), np.float32)
    d = np.empty((B, L), np.int64)
    for b in range(B):
        for l in range(L):
            n = int(rng.integers(1, kq + 1))
            ii = rng.choice(V, size=n, replace=False)
            qq = rng.dirichlet(np.ones(n)).astype(np.float32)
            idx[b, l, :n], val[b, l, :n] = ii, qq
            dense[b, l, ii] = qq
            d[b, l] = ii[0] if b % 3 else int(rng.integers(0, V))  # some drafts outside the list
    mode = np.where(np.arange(B) % 4 == 0, W.MODE_GREEDY, W.MODE_TEMP | W.MODE_TOPP)
    inp = _verify_inputs(t, dense, d, mode, L, temperature=np.full(B, 0.9), top_p=np.full(B, 0.9),
                         position=np.arange(B) * 11)
    a = oracle.verify(inp)
    s_ = oracle.verify(_sparse(inp, idx, val))
    for k in ("tokens", "n_acc", "adm_tokens", "adm_nacc", "n_adm", "flags"):
        assert np.array_equal(a[k], s_[k]), k


def test_verify_sparse_unlisted_draft_is_accepted():
    # an unlisted draft id has q = 0: accepted whenever the target gives it
    # positive probability, rejected (and resampled from p) when it does not
    V, L, B = 16, 2, 256
    rng = np.random.default_rng(8)
    t = rng.normal(0, 1, V).astype(np.float32)
    x = np.tile(t, (B, L + 1, 1))
    order = np.argsort(-t, kind="stable")
    idx = np.tile(np.array([order[0], -1], np.int32), (B, L, 1))
    val = np.tile(np.array([1.0, 0.0], np.float32), (B, L, 1))
    d = np.tile(order[1:1 + L], (B, 1))
    inp = _verify_inputs(x, np.zeros((B, L, V)), d, np.full(B, W.MODE_TEMP), L, position=np.arange(B))
    o = oracle.verify(_sparse(inp, idx, val))
    assert np.all(o["n_acc"] == L) and np.all(o["tokens"][:, :L] == d)
    # top-k 2 excludes order[2]: P(d) = 0, rejected; resampling max(0, P - q)
    # leaves only order[1] (order[0] has q = 1 >= P)
    d2 = np.tile(order[2], (B, L))
    inp = _verify_inputs(x, np.zeros((B, L, V)), d2, np.full(B, W.MODE_TEMP | W.MODE_TOPK), L,
                         top_k=np.full(B, 2), position=np.arange(B))
    o = oracle.verify(_sparse(inp, idx, val))
    assert np.all(o["n_acc"] == 0) and np.all(o["tokens"][:, 0] == order[1])


def _tree_case(seed, B=24, L=3, V=48, kq=10):
    """A path verification input (sparse lists, penalties, grammar rows per
    path position) and the same path hidden in a larger tree of target rows."""
    rng = np.random.default_rng(seed)
    t = rng.normal(0, 1.5, (B, L + 1, V)).astype(np.float32)
    idx = np.full((B, L, kq), -1, np.int32)
    val = np.zeros((B, L, kq), np.float32)
    d = np.empty((B, L), np.int64)
    for b in range(B):
        for l in range(L):
            n = int(rng.integers(1, kq + 1))
            ii = rng.choice(V, size=n, replace=False)
            idx[b, l, :n], val[b, l, :n] = ii, rng.dirichlet(np.ones(n)).astype(np.float32)
            d[b, l] = ii[0]
    mode = np.where(np.arange(B) % 5 == 0, W.MODE_GREEDY | W.MODE_REP | W.MODE_GRAMMAR,
                    W.MODE_TEMP | W.MODE_TOPP | W.MODE_REP | W.MODE_GRAMMAR)
    hist = np.zeros(B + 1, np.int32)
    inp = _verify_inputs(t, np.zeros((B, L, V)), d, mode, L, temperature=np.full(B, 0.9),
                         top_p=np.full(B, 0.9), rep=np.full(B, 1.4), position=np.arange(B) * 7,
                         hist_offsets=hist)
    mask = np.zeros((B * (L + 1), (V + 31) // 32), np.uint32)
    for r in range(B * (L + 1)):
        for i in rng.choice(V, V // 2, replace=False):
            mask[r, i >> 5] |= np.uint32(1 << (int(i) & 31))
        for i in idx.reshape(B, L * kq)[r // (L + 1)]:  # keep most listed drafts allowed
            if i >= 0 and rng.random() < 0.8:
                mask[r, i >> 5] |= np.uint32(1 << (int(i) & 31))
    inp["bitmask"] = mask
    inp["mode"] = mode.astype(np.uint32)
    inp = _sparse(inp, idx, val)
    # the tree: Lt = 2 (L + 1) + 1 rows per request, the path's rows at random
    # places, the others distractors
    Lt = 2 * (L + 1) + 1
    tree = rng.normal(0, 1.5, (B, Lt, V)).astype(np.float32)
    rmap = np.stack([rng.choice(Lt, L + 1, replace=False) for _ in range(B)]).astype(np.int32)
    for b in range(B):
        tree[b, rmap[b]] = t[b]
    tinp = dict(inp, x=tree, row_map=rmap)
    return inp, tinp


def test_verify_tree_rows_are_selected_by_the_map():
    # a path hidden among distractor rows gives the outcomes of the path alone
    for seed in (1, 2):
        inp, tinp = _tree_case(seed)
        a, t_ = oracle.verify(inp), oracle.verify(tinp)
        for k in ("tokens", "n_acc", "adm_tokens", "adm_nacc", "n_adm", "flags"):
            assert np.array_equal(a[k], t_[k]), (seed, k)
        assert a["n_acc"].max() >= 1  # some paths go past the first position


def test_verify_tree_identity_map_is_the_path():
    inp, _ = _tree_case(3)
    L = int(inp["L"])
    a = oracle.verify(inp)
    b = oracle.verify(dict(inp, row_map=np.tile(np.arange(L + 1, dtype=np.int32), (inp["B"], 1))))
    for k in ("tokens", "n_acc", "adm_tokens", "n_adm"):
        assert np.array_equal(a[k], b[k]), k


def test_verify_tree_entry_outside_the_tree_masks_its_row():
    # greedy requests whose first draft is the argmax of their first row: an
    # entry outside [0, Lt) at position 0 rejects at once with no correction;
    # at position 1 it accepts the first draft, then emits nothing
    V, L, B = 16, 2, 4
    rng = np.random.default_rng(9)
    t = rng.normal(0, 1, (B, L + 1, V)).astype(np.float32)
    d = np.stack([[int(np.argmax(t[b, 0])), int(np.argmax(t[b, 1]))] for b in range(B)])
    inp = _verify_inputs(t, np.zeros((B, L, V)), d, np.full(B, W.MODE_GREEDY), L)
    inp = _sparse(inp, np.full((B, L, 1), -1, np.int32), np.zeros((B, L, 1), np.float32))
    rmap = np.tile(np.arange(L + 1, dtype=np.int32), (B, 1))
    rmap[0, 0], rmap[1, 0], rmap[2, 1], rmap[3, 1] = -1, L + 1, L + 1, -5
    o = oracle.verify(dict(inp, row_map=rmap))
    assert list(o["n_acc"]) == [0, 0, 1, 1]
    assert np.all(o["tokens"][:2] == -1)
    assert np.array_equal(o["tokens"][2:, 0], d[2:, 0]) and np.all(o["tokens"][2:, 1:] == -1)
    assert np.all(o["flags"] & 1)  # SS_FLAG_EMPTY


def test_process_logits_distribution_sums_to_one():
    inp = W.config0()
    out = oracle.process_logits(inp)
    P = out["P"]
    assert np.all(np.abs(P.sum(axis=1) - 1.0) < 1e-12)
    assert P[0, np.argmax(inp["x"][0])] == 1.0  # temperature 0: one-hot
    for b in range(1, 4):
        assert np.count_nonzero(P[b]) <= 50


@pytest.mark.parametrize("case", _load("truncation_cases.json")["cases"], ids=lambda c: c["name"])
def test_truncation_golden(case):
    if "y_from_probs" in case:
        y = np.log(np.array(case["y_from_probs"], np.float64)).astype(np.float32)
    else:
        y = np.array(case["y"], np.float32)
    d = oracle.row_distribution(y, case["mode"], temperature=case.get("temperature", 1.0),
                                top_k=case.get("top_k", 0), top_p=case.get("top_p", 1.0),
                                min_p=case.get("min_p", 0.0), k_cap=y.size)
    assert d["n_s"] == case["n_s"]
    if "order" in case:
        assert list(d["order"][: d["n_s"]]) == case["order"]


# --------------------------------------------------------------------------
# Near-boundary band (reading R21): admissible outcomes
# --------------------------------------------------------------------------
BND = _load("boundary_cases.json")


def test_near_band_width():
    assert oracle.near() == BND["near"] == 1e-6


@pytest.mark.parametrize("case", BND["draw"], ids=lambda c: c["why"][:40])
def test_draw_boundary_distance_and_admissible_ranks(case):
    pick, margin, adm = oracle.draw_ex(case["w"], case["u"])
    assert pick == case["pick"]
    assert margin == pytest.approx(case["margin"], rel=1e-6)
    assert adm == case["admissible"]


@pytest.mark.parametrize("case", BND["top_p"], ids=lambda c: "p=%.9f" % c["top_p"])
def test_top_p_boundary_distance_and_admissible_sizes(case):
    d = oracle.row_distribution(np.array(case["y"], np.float32), W.MODE_TOPP, top_p=case["top_p"])
    assert d["margin_p"] == pytest.approx(case["margin"], rel=1e-9)
    assert d["n_s"] == case["n_s"]
    assert [d["ns_lo"], d["ns_hi"]] == case["ns_range"]


@pytest.mark.parametrize("case", BND["min_p"], ids=lambda c: "theta=%.9f" % c["min_p"])
def test_min_p_boundary_distance_and_admissible_sizes(case):
    d = oracle.row_distribution(np.array(case["y"], np.float32), W.MODE_MINP, min_p=case["min_p"])
    assert d["margin_m"] == pytest.approx(case["margin"], rel=1e-9)
    assert d["n_s"] == case["n_s"]
    assert [d["ns_lo"], d["ns_hi"]] == case["ns_range"]


def _two_token_sample(y, mode, **kw):
    x = np.array([y], np.float32)
    return oracle.sample(W.custom_rows(x, W.F32, k_max=2, mode=[mode], **kw))


def test_sample_admits_both_kept_sets_at_a_top_p_boundary():
    """Two equal logits with top-p a hair above 1/2: the kept set is {0, 1}
    or {0} depending on a comparison 1.2e-7 from its boundary, so token 1 (log
    1/2) and token 0 (log 1) are both admissible; far from it, one outcome."""
    near = _two_token_sample([0.0, 0.0], W.MODE_TOPP, top_p=[np.float32(0.5 + 1e-7)], position=[3])
    outs = set(zip(near["adm_token"][0, :near["n_adm"][0]].tolist(),
                   np.round(near["adm_logprob"][0, :near["n_adm"][0]], 6).tolist()))
    assert (0, 0.0) in outs
    assert near["n_adm"][0] >= 2
    assert (near["token"][0], round(float(near["logprob"][0]), 6)) == \
        (near["adm_token"][0, 0], round(float(near["adm_logprob"][0, 0]), 6))
    far = _two_token_sample([0.0, 0.0], W.MODE_TOPP, top_p=[np.float32(0.75)], position=[3])
    assert far["n_adm"][0] == 1


def _accept_case(delta, seed=None):
    """B = 1, L = 1, V = 2, equal target logits (P = 1/2 each), draft token 0
    with q(0) = (1/2)(1 + delta) / a, a the acceptance uniform: a q(0) - P(0)
    is (1/2) delta, a relative distance of delta a / (1 + delta)."""
    for s in range(1, 200):
        a = oracle.uniform(s, 0, 0, 1)
        if a > 0.6:
            break
    q0 = np.float32(0.5 * (1.0 + delta) / a)
    q = np.array([[[q0, np.float32(1.0) - q0]]], np.float32)
    t = np.zeros((1, 2, 2), np.float32)
    inp = W.custom_rows(t.reshape(2, 2), W.F32, k_max=2, mode=[0, 0], position=[0, 0])
    for k in ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres", "seed", "position"):
        inp[k] = inp[k][:1]
    inp["seed"] = np.array([s], np.uint64)
    inp.update(x=t, B=1, L=1, draft_probs=q, draft_tokens=np.array([[0]], np.int32))
    return oracle.verify(inp), a


def test_verify_admits_accept_and_reject_at_the_acceptance_boundary():
    out, a = _accept_case(3e-7)
    seqs = {(tuple(out["adm_tokens"][0, e]), int(out["adm_nacc"][0, e])) for e in range(out["n_adm"][0])}
    # u q(0) exceeds P(0) by a relative 1.8e-7: rejected, the residual puts all
    # its mass on token 1; accepted is admissible too (then a bonus token)
    assert out["n_acc"][0] == 0 and out["tokens"][0].tolist() == [1, -1]
    assert ((1, -1), 0) in seqs
    assert any(n == 1 and t[0] == 0 for t, n in seqs)
    assert out["n_adm"][0] >= 2
    far, _ = _accept_case(1e-4)
    assert far["n_adm"][0] == 1 and far["tokens"][0].tolist() == [1, -1]


# --------------------------------------------------------------------------
# Top-k log-probabilities (indicator bit 0x400)
# --------------------------------------------------------------------------
def _lp_rows(rng, B, V, tau, mask=False):
    x = rng.normal(0.0, 2.0, (B, V)).astype(np.float32)
    x[:, : V // 8] = np.round(x[:, : V // 8])  # exact ties among the leaders
    mode = np.full(B, W.MODE_LOGPROBS | W.MODE_TEMP | W.MODE_REP | W.MODE_BIAS, np.uint32)
    hist = [rng.integers(0, V, 12).astype(np.int32) for _ in range(B)]
    bids = [rng.choice(V, 3, replace=False).astype(np.int32) for _ in range(B)]
    extra = {}
    if mask:
        m = np.full((B, (V + 31) // 32), 0xFFFFFFFF, np.uint32)
        m[:, 0] = 0x0000FFFF  # ids 16..31 denied
        extra = dict(bitmask=m)
        mode |= np.uint32(W.MODE_GRAMMAR)
    return W.custom_rows(x, W.F32, k_max=V, mode=mode, temperature=np.asarray(tau, np.float32),
                         rep=np.full(B, 1.3, np.float32),
                         hist_offsets=np.arange(0, 12 * B + 1, 12, dtype=np.int32), hist_ids=np.concatenate(hist),
                         bias_offsets=np.arange(0, 3 * B + 1, 3, dtype=np.int32), bias_ids=np.concatenate(bids),
                         bias_vals=rng.uniform(-3, 3, 3 * B).astype(np.float32), **extra)


def test_logprobs_two_token_closed_form():
    """Two logits 0 and ln 3: probabilities 1/4 and 3/4."""
    y1 = np.float32(np.log(3.0))
    inp = W.custom_rows(np.array([[0.0, y1]], np.float32), W.F32, k_max=2, mode=np.array([W.MODE_LOGPROBS]))
    idx, lp = oracle.logprobs(inp, 2)
    assert idx.tolist() == [[1, 0]]
    z = 1.0 + math.exp(float(y1))
    assert lp[0, 0] == pytest.approx(float(y1) - math.log(z), abs=1e-7)
    assert lp[0, 1] == pytest.approx(-math.log(z), abs=1e-7)


@pytest.mark.parametrize("mask", [False, True])
def test_logprobs_match_scipy_log_softmax(mask):
    """The leading n_lp tokens and their log-probabilities equal scipy's
    log_softmax of the processed logits at the row's temperature, the
    normaliser running over every valid token (masked ids excluded)."""
    rng = np.random.default_rng(77)
    B, V, n = 6, 200, 17
    tau = rng.uniform(0.4, 2.0, B)
    inp = _lp_rows(rng, B, V, tau, mask)
    idx, lp = oracle.logprobs(inp, n)
    y = oracle.process_logits(inp)["y"].astype(np.float64)
    for b in range(B):
        valid = np.isfinite(y[b])
        ls = np.full(V, -np.inf)
        ls[valid] = special.log_softmax(y[b][valid] / float(np.float32(tau[b])))
        order = np.lexsort((np.arange(V), -y[b]))
        order = order[valid[order]]
        assert idx[b].tolist() == order[:n].tolist()
        np.testing.assert_allclose(lp[b], ls[order[:n]], rtol=1e-6, atol=1e-6)


def test_logprobs_full_list_sums_to_one():
    rng = np.random.default_rng(78)
    B, V = 4, 96
    inp = _lp_rows(rng, B, V, rng.uniform(0.5, 1.5, B), mask=True)
    idx, lp = oracle.logprobs(inp, V)
    for b in range(B):
        k = idx[b] >= 0
        assert np.exp(lp[b][k].astype(np.float64)).sum() == pytest.approx(1.0, abs=1e-5)
        assert (~k).sum() == 16  # the denied ids pad the tail


def test_logprobs_temperature_scales_differences():
    """lp_i - lp_j = (y_i - y_j) / tau for any two listed tokens."""
    rng = np.random.default_rng(79)
    B, V, n = 3, 128, 10
    tau = np.array([0.5, 1.0, 1.7])
    inp = _lp_rows(rng, B, V, tau)
    idx, lp = oracle.logprobs(inp, n)
    y = oracle.process_logits(inp)["y"].astype(np.float64)
    for b in range(B):
        t = float(np.float32(tau[b]))
        d_lp = lp[b, 0] - lp[b, 1:]
        d_y = (y[b, idx[b, 0]] - y[b, idx[b, 1:]]) / t
        np.testing.assert_allclose(d_lp, d_y, atol=2e-6)


def test_logprobs_rows_without_the_bit_greedy_and_empty():
    """Rows without bit 0x400 and fully masked rows are padded; a greedy row
    (or one with the temperature bit off) reports tau = 1 log-probabilities."""
    rng = np.random.default_rng(80)
    V = 64
    x = rng.normal(0, 1, (4, V)).astype(np.float32)
    mask = np.full((4, 2), 0xFFFFFFFF, np.uint32)
    mask[3] = 0
    mode = np.array([0, W.MODE_LOGPROBS | W.MODE_GREEDY | W.MODE_TEMP, W.MODE_LOGPROBS,
                     W.MODE_LOGPROBS | W.MODE_GRAMMAR], np.uint32)
    inp = W.custom_rows(x, W.F32, k_max=V, mode=mode, temperature=np.array([1.0, 0.3, 0.3, 1.0], np.float32),
                        bitmask=mask)
    idx, lp = oracle.logprobs(inp, 5)
    assert (idx[0] == -1).all() and np.isneginf(lp[0]).all()
    assert (idx[3] == -1).all() and np.isneginf(lp[3]).all()
    for b in (1, 2):
        ls = special.log_softmax(x[b].astype(np.float64))
        order = np.lexsort((np.arange(V), -x[b]))[:5]
        assert idx[b].tolist() == order.tolist()
        np.testing.assert_allclose(lp[b], ls[order], atol=1e-6)
