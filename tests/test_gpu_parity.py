"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: top-k values/indices, greedy ids, processed logits and verification ids
are bit-exact; probabilities and log-probabilities agree to 1e-5 relative.
Where a data-dependent comparison (top-p, min-p, the draw, the acceptance
test) lies within 1e-6 of its boundary the oracle lists every outcome the row
admits (each such comparison taken both ways); the GPU's outcome must be one
of them, and those rows are counted.  Counts are printed at the end of the run.
"""
import sys

import numpy as np
import pytest
import torch

import oracle
from gen import workloads as W

pytestmark = pytest.mark.gpu

EMPTY, FALLBACK, OUT_TRUNC, KCAP = 1, 2, 4, 8


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _counts(parity_counts):
    global COUNTS
    COUNTS = parity_counts
    yield


COUNTS = None


@pytest.fixture(scope="module")
def ssb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_20475_amd import binding
    binding.lib()
    return binding


def _np(t):
    return t.detach().cpu().numpy()


def run_sample(ssb, inp, k_out=0):
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    out = ssb.sample(x, prm, inp["k_max"], k_out=k_out)
    torch.cuda.synchronize()
    return [_np(o) for o in out]


def _admissible(ref, tok, lp):
    """Per row: the GPU's (token, log-prob) is one of the oracle's admissible outcomes."""
    A = ref["adm_token"].shape[1]
    valid = np.arange(A)[None, :] < ref["n_adm"][:, None]
    al = ref["adm_logprob"].astype(np.float64)
    lp_ok = np.abs(lp.astype(np.float64)[:, None] - al) <= 1e-5 * np.abs(al) + 1e-6
    return (valid & (ref["adm_token"] == tok[:, None]) & lp_ok).any(axis=1)


def check_sample(inp, tok, lp, fl, label, counts=None):
    ref = oracle.sample(inp)
    ok = _admissible(ref, tok, lp)
    bad = np.nonzero(~ok)[0]
    assert bad.size == 0, (label, bad[:10], tok[bad[:10]], lp[bad[:10]], ref["token"][bad[:10]],
                           ref["logprob"][bad[:10]], ref["n_adm"][bad[:10]])
    assert np.array_equal(fl & (EMPTY | KCAP), ref["flags"] & (EMPTY | KCAP)), label
    near = int((ref["n_adm"] > 1).sum())
    alt = int((tok != ref["token"]).sum())
    fb = int(((fl & FALLBACK) > 0).sum())
    counts = counts or COUNTS
    if counts is not None:
        counts.add(label, tok.size, near, alt, fb)
    say(f"[{label}] rows={tok.size} near-boundary rows={near} (outcome other than the oracle's own: {alt}) "
        f"fallback={fb}")
    return ref


# --------------------------------------------------------------------------
# Standalone top-k
# --------------------------------------------------------------------------
def check_topk(ssb, inp, label):
    x = ssb.logits_tensor(inp)
    k = torch.from_numpy(inp["top_k"].astype(np.int32)).cuda() if inp.get("top_k") is not None else None
    fl = torch.zeros(inp["B"], dtype=torch.int32, device="cuda")
    say(f"[{label}] topk B={inp['B']} V={inp['V']} k_max={inp['k_max']} dtype={inp['dtype']}")
    val, idx = ssb.topk(x, k, inp["k_max"], flags=fl)
    torch.cuda.synchronize()
    rv, ri = oracle.topk(inp)
    gv, gi = _np(val), _np(idx)
    bad = np.nonzero(~(gi == ri).all(axis=1))[0]
    assert bad.size == 0, (label, bad[:5])
    assert np.array_equal(gv.view(np.uint32), rv.view(np.uint32)), label
    say(f"[{label}] ok, fallback rows={int((_np(fl) & FALLBACK > 0).sum())}")


def test_topk_config2_full(ssb):
    check_topk(ssb, W.config2(), "cfg2")


@pytest.mark.parametrize("kind", ["zeros", "bf16_flat", "ties", "nan_inf", "sorted", "small_v", "odd_v"])
def test_topk_edge_cases(ssb, kind):
    rng = np.random.default_rng(5)
    B, V, km, dt = 8, 40000, 600, W.F32
    if kind == "zeros":
        x = np.zeros((B, V), np.float32)
    elif kind == "bf16_flat":
        x = W.bf16_bits_from_f32(rng.uniform(128.6, 128.7, (B, V)).astype(np.float32))
        dt = W.BF16
    elif kind == "ties":
        x = (rng.integers(-8, 8, (B, V)) / 4).astype(np.float32)
    elif kind == "nan_inf":
        x = rng.normal(0, 1, (B, V)).astype(np.float32)
        x[:, ::5] = np.nan
        x[:, 1::7] = -np.inf
        x[:, 2::11] = -0.0
        x[1] = -np.inf
        x[2, :] = np.nan
        x[2, 17] = 3.0
    elif kind == "sorted":
        x = np.sort(rng.normal(0, 1, (B, V)).astype(np.float32), axis=1)[:, ::-1].copy()
    elif kind == "small_v":
        V = 100
        x = rng.normal(0, 1, (B, V)).astype(np.float32)
        km = 64
    else:
        V = 40001
        x = W.bf16_bits_from_f32(rng.normal(0, 2, (B, V)).astype(np.float32))
        dt = W.BF16
    k = np.array([1, 2, 50, km, 0, km - 1, 600, 7][:B], np.int32)
    k = np.minimum(k, km)
    inp = W.custom_rows(x, dt, k_max=km, top_k=k)
    check_topk(ssb, inp, f"topk-{kind}")


def test_topk_large_k_small_vocab(ssb):
    rng = np.random.default_rng(9)
    x = rng.normal(0, 1, (3, 20000)).astype(np.float32)
    inp = W.custom_rows(x, W.F32, k_max=4096, top_k=np.array([4096, 4095, 3000], np.int32))
    check_topk(ssb, inp, "topk-k4096-V20000")


# --------------------------------------------------------------------------
# Fused sampling
# --------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["cfg0", "cfg1", "cfg3"])
def test_sample_configs(ssb, name):
    inp = W.make_config(name)
    say(f"[{name}] sample B={inp['B']} V={inp['V']} dtype={inp['dtype']}")
    tok, lp, fl = run_sample(ssb, inp)
    check_sample(inp, tok, lp, fl, name)


def test_sample_penalised_heads(ssb):
    """bf16 rows whose head tokens are penalised and biased, so their final
    values leave the bf16 grid and sit next to the top-k, top-p, min-p and
    draw boundaries; several Philox positions per row."""
    rng = np.random.default_rng(97)
    B, V = 48, 1 << 15
    xf = rng.normal(0.0, 2.0, (B, V))
    hist, bids, bvals = [], [], []
    for r in range(B):
        heads = rng.choice(V, 24, replace=False)
        xf[r, heads] += rng.uniform(4.0, 10.0, 24)
        hist.append(np.concatenate([np.repeat(heads, rng.integers(1, 4, 24)), rng.integers(0, V, 100)]).astype(np.int32))
        bids.append(rng.choice(heads, 8, replace=False).astype(np.int32))
        bvals.append(rng.uniform(-2.0, 2.0, 8).astype(np.float32))
    x = W.bf16_bits_from_f32(xf.astype(np.float32))
    pen = W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
    hoff = np.concatenate([[0], np.cumsum([len(h) for h in hist])]).astype(np.int32)
    boff = np.concatenate([[0], np.cumsum([len(v) for v in bids])]).astype(np.int32)
    min_p = np.where(np.arange(B) % 2 == 0, 0.0, rng.uniform(0.01, 0.3, B)).astype(np.float32)
    inp = W.custom_rows(x, dtype=W.BF16, k_max=512,
                        mode=np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_MINP | pen, np.uint32),
                        temperature=rng.uniform(0.5, 1.5, B).astype(np.float32),
                        top_k=rng.integers(2, 301, B).astype(np.int32),
                        top_p=rng.uniform(0.3, 0.99, B).astype(np.float32), min_p=min_p,
                        rep=rng.uniform(1.05, 1.5, B).astype(np.float32),
                        freq=rng.uniform(0.0, 0.7, B).astype(np.float32),
                        pres=rng.uniform(0.0, 0.7, B).astype(np.float32),
                        hist_offsets=hoff, hist_ids=np.concatenate(hist),
                        bias_offsets=boff, bias_ids=np.concatenate(bids), bias_vals=np.concatenate(bvals))
    for pos in range(3):
        inp["position"] = np.full(B, pos, np.int64)
        say(f"[penalised-heads] sample B={B} V={V} position={pos}")
        tok, lp, fl = run_sample(ssb, inp)
        check_sample(inp, tok, lp, fl, f"penalised-heads-{pos}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_greedy_patched_maxima(ssb, dtype):
    """Greedy rows whose largest raw logits are penalised below other values:
    the units holding them are re-read (the other units' candidates bound the
    maximum).  Rows mix one penalised head, many penalised heads spread over
    the units, a grammar mask, rows with no lists (tied maxima, so the units
    overflow their candidate regions) and rows where every head is penalised."""
    rng = np.random.default_rng(4242 if dtype == "bf16" else 4243)
    B, V = 32, 1 << 17
    xf = rng.normal(0.0, 1.0, (B, V))
    hist, mask = [], np.full((B, (V + 31) // 32), 0xFFFFFFFF, np.uint32)
    mode = np.full(B, W.MODE_GREEDY | W.MODE_REP | W.MODE_FREQ, np.uint32)
    for r in range(B):
        kind = r % 4
        nheads = (1, 40, 6, 0)[kind]
        heads = rng.choice(V, max(nheads, 1), replace=False)
        if kind == 3:  # no lists: tied maxima in every unit
            xf[r, rng.choice(V, 8000, replace=False)] = 6.0
            mode[r] = W.MODE_GREEDY
            hist.append(np.zeros(0, np.int32))
            continue
        xf[r, heads] += rng.uniform(6.0, 9.0, heads.size)
        h = np.repeat(heads, 2)
        if r % 8 == 2:  # one penalised head stays above the rest
            h = h[2:]
        hist.append(np.concatenate([h, rng.integers(0, V, 64)]).astype(np.int32))
        if kind == 2:  # grammar: deny a third of the words
            mask[r, rng.choice(mask.shape[1], mask.shape[1] // 3, replace=False)] = 0
            mode[r] |= W.MODE_GRAMMAR
    x = xf.astype(np.float32)
    if dtype == "bf16":
        x = W.bf16_bits_from_f32(x)
    hoff = np.concatenate([[0], np.cumsum([len(h) for h in hist])]).astype(np.int32)
    inp = W.custom_rows(x, dtype=W.BF16 if dtype == "bf16" else W.F32, k_max=64, mode=mode,
                        rep=np.full(B, 4.0, np.float32), freq=np.full(B, 0.5, np.float32),
                        hist_offsets=hoff, hist_ids=np.concatenate(hist), bitmask=mask)
    say(f"[greedy-patched-{dtype}] sample B={B} V={V}")
    tok, lp, fl = run_sample(ssb, inp)
    ref = check_sample(inp, tok, lp, fl, f"greedy-patched-{dtype}")
    assert np.array_equal(tok, ref["token"]), f"greedy-patched-{dtype}"


def test_sample_large_vocab_patched(ssb):
    """V = 2^18 bf16 with penalties and bias: the patched-id bitmap is hashed
    above 2^17 ids, so pooled raw copies are checked against the hash table."""
    rng = np.random.default_rng(2718)
    B, V = 8, 1 << 18
    xf = rng.normal(0.0, 2.0, (B, V))
    hist, bids, bvals = [], [], []
    for r in range(B):
        heads = rng.choice(V, 16, replace=False)
        xf[r, heads] += rng.uniform(6.0, 12.0, 16)
        hist.append(np.concatenate([heads[:8], rng.integers(0, V, 600)]).astype(np.int32))
        bids.append(rng.choice(V, 12, replace=False).astype(np.int32))
        bvals.append(rng.uniform(-3.0, 3.0, 12).astype(np.float32))
    x = W.bf16_bits_from_f32(xf.astype(np.float32))
    pen = W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
    mode = np.array([W.MODE_GREEDY | pen if r % 4 == 0 else W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | pen
                     for r in range(B)], np.uint32)
    inp = W.custom_rows(x, dtype=W.BF16, k_max=256, mode=mode,
                        temperature=rng.uniform(0.6, 1.4, B).astype(np.float32),
                        top_k=rng.integers(2, 257, B).astype(np.int32),
                        top_p=rng.uniform(0.5, 0.95, B).astype(np.float32),
                        rep=rng.uniform(1.1, 1.4, B).astype(np.float32),
                        freq=rng.uniform(0.0, 0.5, B).astype(np.float32),
                        pres=rng.uniform(0.0, 0.5, B).astype(np.float32),
                        hist_offsets=np.concatenate([[0], np.cumsum([len(h) for h in hist])]).astype(np.int32),
                        hist_ids=np.concatenate(hist),
                        bias_offsets=np.concatenate([[0], np.cumsum([len(v) for v in bids])]).astype(np.int32),
                        bias_ids=np.concatenate(bids), bias_vals=np.concatenate(bvals))
    say(f"[large-vocab-patched] sample B={B} V={V}")
    tok, lp, fl = run_sample(ssb, inp)
    check_sample(inp, tok, lp, fl, "large-vocab-patched")


def test_sample_kept_distribution_outputs(ssb):
    inp = W.config1(B=16)
    say("[cfg1-B16] sample with k_out=64")
    tok, lp, fl, idx, prob = run_sample(ssb, inp, k_out=64)
    check_sample(inp, tok, lp, fl, "cfg1-kout")
    ref = oracle.process_logits(inp)
    for b in range(inp["B"]):
        P = ref["P"][b]
        n = int(np.count_nonzero(P))
        o = np.lexsort((np.arange(P.size), -P))[:n]
        m = min(n, 64)
        if (inp["mode"][b] & W.MODE_GREEDY) == 0:
            assert np.array_equal(np.sort(idx[b, :m]), np.sort(o[:m])), b
        np.testing.assert_allclose(prob[b, :m], P[idx[b, :m]], rtol=1e-5, atol=1e-30)
        assert np.all(idx[b, m:] == -1)


def check_sample_full(ssb, inp, label, k_out=0):
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    r = ssb.sample_full(x, prm, inp["k_max"], k_out=k_out)
    torch.cuda.synchronize()
    tok, lp, fl = _np(r[0]), _np(r[1]), _np(r[2])
    ref = oracle.sample_full(inp)
    ok = _admissible(ref, tok, lp)
    bad = np.nonzero(~ok)[0]
    assert bad.size == 0, (label, bad[:10], tok[bad[:10]], lp[bad[:10]], ref["token"][bad[:10]],
                           ref["logprob"][bad[:10]], ref["n_adm"][bad[:10]])
    # the fit test may go either way only where a kept-set boundary is near
    sure = ref["n_adm"] == 1
    assert np.array_equal((fl & (EMPTY | KCAP))[sure], (ref["flags"] & (EMPTY | KCAP))[sure]), label
    near = int((ref["n_adm"] > 1).sum())
    alt = int((tok != ref["token"]).sum())
    fb = int(((fl & FALLBACK) > 0).sum())
    over = int(((ref["flags"] & KCAP) > 0).sum())
    if COUNTS is not None:
        COUNTS.add(label, tok.size, near, alt, fb)
    say(f"[{label}] rows={tok.size} near-boundary rows={near} (outcome other than the oracle's own: {alt}) "
        f"fallback={fb} bounded (KCAP)={over}")
    return ref


def nucleus_rows(inp):
    """The input with the top-k bit cleared on every stochastic request."""
    inp = dict(inp)
    greedy = (inp["mode"] & W.MODE_GREEDY) != 0
    inp["mode"] = np.where(greedy, inp["mode"], inp["mode"] & ~np.uint32(W.MODE_TOPK)).astype(np.uint32)
    return inp


@pytest.mark.parametrize("name", ["cfg0", "cfg1", "cfg3"])
def test_sample_full_configs(ssb, name):
    inp = nucleus_rows(W.make_config(name))
    say(f"[{name}-full] sample B={inp['B']} V={inp['V']} dtype={inp['dtype']}")
    ref = check_sample_full(ssb, inp, f"{name}-full")
    stoch = (inp["mode"] & W.MODE_GREEDY) == 0
    assert ((ref["flags"][stoch] & KCAP) == 0).any()  # some requests take the full-row result


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_sample_full_edge_cases(ssb, dtype):
    # long tails (the whole-row cut differs from the bounded one), flat rows
    # (overflow), min-p keeping exactly k_max and one fewer, short valid sets,
    # masked and NaN entries, penalised and biased heads, a long history that
    # overflows the LDS patch table, and top-k requests beside
    rng = np.random.default_rng(123)
    B, V, k_max = 16, 20000, 128
    x = rng.normal(0, 0.3, (B, V)).astype(np.float32)
    for b in range(B):
        x[b, rng.choice(V, 10, replace=False)] += rng.uniform(5.0, 6.5, 10).astype(np.float32)
    x[2] = 0.0                                        # flat: overflow
    x[3] = -20.0
    x[3, :k_max] = 0.0                                # min-p keeps exactly k_max: overflow
    x[4] = -20.0
    x[4, : k_max - 1] = 0.0                           # ... k_max - 1: fits
    x[5, 40:] = -np.inf                               # 40 valid tokens
    x[6, ::3] = np.nan
    mode = np.full(B, W.MODE_TEMP | W.MODE_TOPP | W.MODE_MINP | W.MODE_REP | W.MODE_BIAS, np.uint32)
    mode[3] = mode[4] = W.MODE_MINP
    mode[7] = W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP
    mode[8] = W.MODE_GREEDY
    top_p = np.full(B, 0.9, np.float32)
    top_p[9] = 0.999
    min_p = np.full(B, 0.001, np.float32)
    min_p[3] = min_p[4] = 0.5
    hist = [rng.integers(0, V, 64).astype(np.int32) for _ in range(B)]
    hist[10] = rng.choice(V, 3000, replace=False).astype(np.int32)  # beyond the LDS table
    off = np.zeros(B + 1, np.int32)
    off[1:] = np.cumsum([len(h) for h in hist])
    bids = [rng.choice(V, 8, replace=False).astype(np.int32) for _ in range(B)]
    boff = np.arange(B + 1, dtype=np.int32) * 8
    xx = x if dtype == W.F32 else W.bf16_bits_from_f32(x)
    inp = W.custom_rows(xx, dtype, k_max=k_max, mode=mode, temperature=np.full(B, 0.8), top_k=np.full(B, 50),
                        top_p=top_p, min_p=min_p, rep=np.full(B, 1.3), position=np.arange(B) * 5)
    inp["hist_offsets"], inp["hist_ids"] = off, np.concatenate(hist)
    inp["bias_offsets"], inp["bias_ids"] = boff, np.concatenate(bids)
    inp["bias_vals"] = rng.uniform(-3, 3, B * 8).astype(np.float32)
    label = f"full-edge-{dtype}"
    say(f"[{label}] B={B} V={V} k_max={k_max}")
    x_t = ssb.logits_tensor(inp)
    r = ssb.sample_full(x_t, ssb.Params.from_arrays(inp), k_max, k_out=16)
    torch.cuda.synchronize()
    gidx, gprob = _np(r[3]), _np(r[4])
    ref = check_sample_full(ssb, inp, label, k_out=16)
    assert ref["flags"][2] & KCAP and ref["flags"][3] & KCAP and not ref["flags"][4] & KCAP
    # the kept list of rows that fit: the n_kept leading tokens of the processed
    # row (canonical order) with their probabilities over the kept set
    y = oracle.process_logits(inp)["y"]
    tau = np.float32(0.8)
    for b in range(B):
        stoch = (mode[b] & W.MODE_GREEDY) == 0
        if not stoch or ref["n_adm"][b] != 1 or (ref["flags"][b] & KCAP) or (mode[b] & W.MODE_TOPK):
            continue
        yb = y[b].astype(np.float64)
        order = np.lexsort((np.arange(V), -yb))
        n = int(ref["n_kept"][b])
        t_b = float(tau) if mode[b] & W.MODE_TEMP else 1.0
        w = np.exp((yb[order[:n]] - yb[order[0]]) / t_b)
        P = w / w.sum()
        m = min(n, 16)
        assert np.array_equal(gidx[b, :m], order[:m]), b
        np.testing.assert_allclose(gprob[b, :m], P[:m], rtol=1e-5, atol=1e-30)
        assert np.all(gidx[b, m:] == -1)


def check_sample_gumbel(ssb, inp, noise, label, k_out=0):
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    g = torch.from_numpy(np.ascontiguousarray(noise, np.float32)).cuda()
    r = ssb.sample_gumbel(x, prm, inp["k_max"], g, k_out=k_out)
    torch.cuda.synchronize()
    tok, lp, fl = _np(r[0]), _np(r[1]), _np(r[2])
    ref = oracle.sample_gumbel(inp, noise)
    ok = _admissible(ref, tok, lp)
    bad = np.nonzero(~ok)[0]
    assert bad.size == 0, (label, bad[:10], tok[bad[:10]], lp[bad[:10]], ref["token"][bad[:10]],
                           ref["logprob"][bad[:10]], ref["n_adm"][bad[:10]])
    assert np.array_equal(fl & (EMPTY | KCAP), ref["flags"] & (EMPTY | KCAP)), label
    near = int((ref["n_adm"] > 1).sum())
    alt = int((tok != ref["token"]).sum())
    fb = int(((fl & FALLBACK) > 0).sum())
    if COUNTS is not None:
        COUNTS.add(label, tok.size, near, alt, fb)
    say(f"[{label}] rows={tok.size} near-boundary rows={near} (outcome other than the oracle's own: {alt}) "
        f"fallback={fb}")
    return r


@pytest.mark.parametrize("name", ["cfg0", "cfg1", "cfg3"])
def test_sample_gumbel_configs(ssb, name):
    inp = W.make_config(name)
    say(f"[{name}-gumbel] sample B={inp['B']} V={inp['V']} dtype={inp['dtype']}")
    check_sample_gumbel(ssb, inp, W.gumbel_noise(inp["B"], inp["V"], 500 + len(name)), f"{name}-gumbel")


def test_sample_gumbel_edge_cases(ssb):
    # zero noise (the argmax of the kept set), equal scores (lower id), heavy
    # noise outside the kept set, tied and masked rows, a k_out list beside
    rng = np.random.default_rng(88)
    B, V = 12, 3000
    x = rng.normal(0, 1, (B, V)).astype(np.float32)
    x[3] = 0.0                               # every logit tied
    x[4, ::2] = -np.inf                      # half masked
    x[5, 7] = np.nan
    noise = np.log(rng.exponential(size=(B, V))).astype(np.float32)
    noise[0] = 0.0                           # zero noise: the argmax
    order = np.argsort(-x[1], kind="stable")
    noise[1, order[20:]] = -1e30             # huge scores outside the kept set
    noise[2] = 0.0
    x[2, :4] = np.array([1.0, 2.0, 1.0, 2.0], np.float32)
    x[2, 4:] = -5.0
    # tau 0.5: scores (1 - 2)/0.5 + 1 = -1 (id 0) and 0 - 1 = -1 (id 1) tie: the lower id
    noise[2, :4] = np.array([-1.0, 1.0, 5.0, 5.0], np.float32)
    mode = np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_MINP, np.uint32)
    mode[6] = W.MODE_GREEDY
    mode[7] = W.MODE_TEMP                    # no truncation: the k_max bound
    inp = W.custom_rows(x, W.F32, k_max=256, mode=mode, temperature=np.full(B, 0.5), top_k=np.full(B, 20),
                        top_p=np.full(B, 0.97), min_p=np.full(B, 0.001), position=np.arange(B))
    r = check_sample_gumbel(ssb, inp, noise, "gumbel-edge", k_out=32)
    assert int(_np(r[0])[2]) == 0


def _edge_inputs(kind):
    rng = np.random.default_rng(77)
    B = 8
    stoch = W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_MINP
    if kind == "zeros":
        V = 30000
        x = np.zeros((B, V), np.float32)
        return W.custom_rows(x, W.F32, k_max=256, mode=np.full(B, stoch), top_k=np.full(B, 200),
                             top_p=np.full(B, 0.9), min_p=np.full(B, 0.0), position=np.arange(B))
    if kind == "bf16_flat":
        V = 65536
        x = W.bf16_bits_from_f32(rng.uniform(128.6, 128.7, (B, V)).astype(np.float32))
        return W.custom_rows(x, W.BF16, k_max=128, mode=np.full(B, stoch), top_k=np.full(B, 128),
                             top_p=np.full(B, 0.5), position=np.arange(B))
    if kind == "ragged_odd":
        V = 50001
        x = W.bf16_bits_from_f32(rng.normal(0, 2, (B, V)).astype(np.float32))
        return W.custom_rows(x, W.BF16, k_max=300, mode=np.full(B, stoch), top_k=np.arange(1, B + 1) * 37,
                             top_p=np.full(B, 0.97), min_p=np.full(B, 0.001), temperature=np.full(B, 1.1),
                             position=np.arange(B) + 5)
    if kind == "small_v":
        V = 70
        x = rng.normal(0, 1, (B, V)).astype(np.float32)
        return W.custom_rows(x, W.F32, k_max=64, mode=np.full(B, stoch), top_k=np.array([1, 5, 64, 0, 70, 3, 2, 9]),
                             top_p=np.full(B, 0.99), position=np.arange(B))
    if kind == "nan_empty":
        V = 20000
        x = rng.normal(0, 1, (B, V)).astype(np.float32)
        x[0] = np.nan
        x[1] = -np.inf
        x[2, ::2] = np.nan
        x[3, 1::3] = -np.inf
        x[4, :] = -0.0
        return W.custom_rows(x, W.F32, k_max=64, mode=np.full(B, stoch), top_k=np.full(B, 40),
                             position=np.arange(B))
    if kind == "no_topk":
        V = 40000
        x = rng.normal(0, 3, (B, V)).astype(np.float32)
        return W.custom_rows(x, W.F32, k_max=512, mode=np.full(B, W.MODE_TEMP | W.MODE_TOPP),
                             temperature=np.full(B, 0.8), top_p=np.full(B, 0.999), position=np.arange(B))
    if kind == "grammar_few":
        V = 65536
        x = rng.normal(0, 2, (B, V)).astype(np.float32)
        mask = np.zeros((B, V // 32), np.uint32)
        for b in range(B):
            ids = rng.choice(V, 10 + b, replace=False)
            for i in ids:
                mask[b, i >> 5] |= np.uint32(1 << (int(i) & 31))
        mask[7] = 0
        return W.custom_rows(x, W.F32, k_max=256, mode=np.full(B, stoch | W.MODE_GRAMMAR), top_k=np.full(B, 100),
                             bitmask=mask, position=np.arange(B))
    if kind == "long_history":
        V = 65536
        x = W.bf16_bits_from_f32(rng.normal(0, 2, (B, V)).astype(np.float32))
        hist = [np.concatenate([rng.integers(0, 5000, 3000), rng.integers(0, V, 500)]).astype(np.int32) for _ in range(B)]
        off = np.zeros(B + 1, np.int32)
        off[1:] = np.cumsum([len(h) for h in hist])
        bias_ids = [np.array([3, 3, 9, 70000, -1, 3], np.int32) for _ in range(B)]
        bias_vals = [np.array([0.5, 0.25, -1.0, 9.0, 9.0, 0.125], np.float32) for _ in range(B)]
        boff = np.zeros(B + 1, np.int32)
        boff[1:] = np.cumsum([len(h) for h in bias_ids])
        m = stoch | W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
        mode = np.full(B, m)
        mode[::2] = W.MODE_GREEDY | W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
        return W.custom_rows(x, W.BF16, k_max=256, mode=mode, top_k=np.full(B, 200), top_p=np.full(B, 0.95),
                             rep=np.full(B, 1.2), freq=np.full(B, 0.1), pres=np.full(B, 0.3),
                             hist_offsets=off, hist_ids=np.concatenate(hist), bias_offsets=boff,
                             bias_ids=np.concatenate(bias_ids), bias_vals=np.concatenate(bias_vals),
                             position=np.arange(B))
    if kind == "dense_patch":
        # consecutive penalised / biased ids: one thread holds several patched slots
        V = 40000
        x = W.bf16_bits_from_f32(rng.normal(0, 2, (B, V)).astype(np.float32))
        hist = [np.concatenate([np.arange(96, 112), np.arange(9000, 9040), rng.integers(0, V, 64)]).astype(np.int32)
                for _ in range(B)]
        off = np.zeros(B + 1, np.int32)
        off[1:] = np.cumsum([len(h) for h in hist])
        bids = [np.arange(200, 216, dtype=np.int32) for _ in range(B)]
        bvals = [np.full(16, 3.0, np.float32) for _ in range(B)]
        boff = np.zeros(B + 1, np.int32)
        boff[1:] = np.cumsum([len(h) for h in bids])
        m = stoch | W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
        mode = np.full(B, m)
        mode[::2] = W.MODE_GREEDY | W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
        return W.custom_rows(x, W.BF16, k_max=128, mode=mode, top_k=np.full(B, 100), top_p=np.full(B, 0.99),
                             rep=np.full(B, 1.2), freq=np.full(B, 0.1), pres=np.full(B, 0.3),
                             hist_offsets=off, hist_ids=np.concatenate(hist), bias_offsets=boff,
                             bias_ids=np.concatenate(bids), bias_vals=np.concatenate(bvals),
                             position=np.arange(B))
    if kind == "greedy_ties":
        V = 30000
        x = np.zeros((B, V), np.float32)
        for b in range(B):
            x[b, rng.choice(V, 5, replace=False)] = 4.0
        return W.custom_rows(x, W.F32, k_max=64, mode=np.full(B, W.MODE_GREEDY))
    raise KeyError(kind)


@pytest.mark.parametrize("kind", ["zeros", "bf16_flat", "ragged_odd", "small_v", "nan_empty", "no_topk",
                                  "grammar_few", "long_history", "dense_patch", "greedy_ties"])
def test_sample_edge_cases(ssb, kind):
    inp = _edge_inputs(kind)
    say(f"[{kind}] sample B={inp['B']} V={inp['V']}")
    tok, lp, fl = run_sample(ssb, inp)
    check_sample(inp, tok, lp, fl, kind)


def _patched_rows(V, n_distinct, B=4, seed=31, dtype=None):
    """Rows whose penalty history holds n_distinct[b] distinct ids (including
    the row's boosted heads, so penalties move the top tokens)."""
    rng = np.random.default_rng(seed)
    xf = rng.normal(0.0, 2.0, (B, V))
    hist, bids, bvals = [], [], []
    for r in range(B):
        heads = rng.choice(V, 16, replace=False)
        xf[r, heads] += rng.uniform(6.0, 12.0, 16)
        ids = np.unique(np.concatenate([heads, rng.choice(V, n_distinct[r], replace=False)]))[:n_distinct[r]]
        ids = np.concatenate([ids, heads[:8], ids[:100]])  # some ids repeat
        hist.append(rng.permutation(ids).astype(np.int32))
        bids.append(np.concatenate([heads[8:12], heads[8:10], rng.choice(V, 10, replace=False)]).astype(np.int32))
        bvals.append(rng.uniform(-3.0, 3.0, 16).astype(np.float32))
    x = W.bf16_bits_from_f32(xf.astype(np.float32))
    pen = W.MODE_REP | W.MODE_FREQ | W.MODE_PRES | W.MODE_BIAS
    mode = np.array([W.MODE_GREEDY | pen if r == 0 else W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_MINP | pen
                     for r in range(B)], np.uint32)
    return W.custom_rows(x, dtype=W.BF16, k_max=256, mode=mode,
                         temperature=rng.uniform(0.6, 1.4, B).astype(np.float32),
                         top_k=rng.integers(20, 257, B).astype(np.int32),
                         top_p=rng.uniform(0.5, 0.95, B).astype(np.float32),
                         min_p=rng.uniform(0.0, 0.05, B).astype(np.float32),
                         rep=rng.uniform(1.1, 1.4, B).astype(np.float32),
                         freq=rng.uniform(0.0, 0.5, B).astype(np.float32),
                         pres=rng.uniform(0.0, 0.5, B).astype(np.float32),
                         hist_offsets=np.concatenate([[0], np.cumsum([len(h) for h in hist])]).astype(np.int32),
                         hist_ids=np.concatenate(hist),
                         bias_offsets=np.concatenate([[0], np.cumsum([len(v) for v in bids])]).astype(np.int32),
                         bias_ids=np.concatenate(bids), bias_vals=np.concatenate(bvals),
                         position=np.arange(B))


def test_sample_patch_table_modes(ssb):
    """Histories of 20 000 distinct ids overflow both patch tables (the merge
    then looks every id up in the lists); 5 000 overflow only the LDS table
    (the row's table in the workspace); 1 000 fit the LDS table."""
    inp = _patched_rows(1 << 17, [20000, 20000, 5000, 1000])
    say("[patch-modes] sample B=4 V=131072 distinct history ids 20000/20000/5000/1000")
    tok, lp, fl = run_sample(ssb, inp)
    check_sample(inp, tok, lp, fl, "patch-modes")


def test_workspace_contents_do_not_matter(ssb):
    """A workspace sized for a larger call and filled with arbitrary bytes
    serves the global-patch-table case: nothing is read before it is written."""
    inp = _edge_inputs("long_history")
    n = ssb.workspace_bytes(ssb.OP_SAMPLE, 64, 1 << 17, 0, 1024, ssb.BF16)
    assert n >= ssb.workspace_bytes(ssb.OP_SAMPLE, inp["B"], inp["V"], 0, inp["k_max"], ssb.BF16)
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    ws = torch.randint(0, 256, (n,), dtype=torch.uint8, device="cuda", generator=g)
    big = W.config1()
    say("[ws-reuse] cfg1 then long_history on one workspace of random bytes")
    ssb.sample(ssb.logits_tensor(big), ssb.Params.from_arrays(big), big["k_max"], ws=ws)
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    for rep in range(2):
        tok, lp, fl = [_np(t) for t in ssb.sample(x, prm, inp["k_max"], ws=ws)]
        torch.cuda.synchronize()
        check_sample(inp, tok, lp, fl, f"ws-reuse-{rep}")
        ws.random_(0, 256, generator=g)


@pytest.mark.parametrize("kind", ["f32_zeros_2e18", "bf16_ties_2e17"])
def test_flat_rows_full_size(ssb, kind):
    """The paper's correctness inputs (all zero; U(128.6, 128.7), all 129.0
    in bf16) at full vocabulary size: every unit's ties overflow its candidate
    region, so each keeps its lowest-index tie groups.  Sampling (k_max 1024)
    finds its top-k in the first unit's groups without the slow path; top-k
    rows beyond one unit's capacity take the exact slow path."""
    rng = np.random.default_rng(13)
    B = 4
    if kind == "f32_zeros_2e18":
        V, dt = 1 << 18, W.F32
        x = np.zeros((B, V), np.float32)
    else:
        V, dt = 1 << 17, W.BF16
        x = W.bf16_bits_from_f32(rng.uniform(128.6, 128.7, (B, V)).astype(np.float32))
    k = np.array([4096, 1024, 1, 3000], np.int32)
    inp = W.custom_rows(x, dt, k_max=4096, top_k=k)
    check_topk(ssb, inp, f"topk-flat-{kind}")
    stoch = W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP
    smp = W.custom_rows(x, dt, k_max=1024, mode=np.full(B, stoch), top_k=np.array([1024, 1000, 64, 1024]),
                        top_p=np.array([0.9, 1.0, 0.5, 0.999]), temperature=np.full(B, 0.8), position=np.arange(B))
    say(f"[flat-{kind}] sample B={B} V={V}")
    tok, lp, fl = run_sample(ssb, smp)
    ref = check_sample(smp, tok, lp, fl, f"flat-{kind}")
    assert not (fl & FALLBACK).any(), fl


def test_tied_rows_headline_params(ssb):
    """B=64 rows of one tied bf16 value (V=2^17) with the headline workload's
    per-request parameters (mixed greedy and stochastic, k up to 900,
    penalties over a 512-id history, bias): the tie cut keeps every row off
    the slow path and the results match the oracle."""
    inp = W.config1()
    inp["x"] = np.full_like(inp["x"], W.bf16_bits_from_f32(np.array([0.5], np.float32))[0])
    # k <= 900: the first unit's 1024 tie elements, less the listed ids among
    # them (a few), cover every row's top-k
    inp["top_k"] = np.minimum(inp["top_k"], 900).astype(np.int32)
    say("[tied-headline] sample B=64 V=131072 bf16, one tied value")
    tok, lp, fl = run_sample(ssb, inp)
    check_sample(inp, tok, lp, fl, "tied-headline")
    assert not (fl & FALLBACK).any(), np.nonzero(fl & FALLBACK)[0]


# --------------------------------------------------------------------------
# Top-k log-probabilities
# --------------------------------------------------------------------------
def check_logprobs(ssb, inp, n_lp, label):
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    fl = torch.zeros(inp["B"], dtype=torch.int32, device="cuda")
    say(f"[{label}] logprobs B={inp['B']} V={inp['V']} n_lp={n_lp} dtype={inp['dtype']}")
    idx, lp = ssb.logprobs(x, prm, n_lp, flags=fl)
    torch.cuda.synchronize()
    ri, rl = oracle.logprobs(inp, n_lp)
    gi, gl = _np(idx), _np(lp)
    bad = np.nonzero(~(gi == ri).all(axis=1))[0]
    assert bad.size == 0, (label, bad[:5], gi[bad[:1]], ri[bad[:1]])
    fin = ri >= 0
    assert np.isneginf(gl[~fin]).all(), label
    # float32 exponentials summed in double: the normaliser's relative error is
    # a few 1e-7, so each log-probability is within 1e-5 (absolute, or
    # relative for magnitudes above 1)
    err = np.abs(gl[fin].astype(np.float64) - rl[fin]) / np.maximum(1.0, np.abs(rl[fin]))
    assert err.max(initial=0.0) <= 1e-5, (label, float(err.max()))
    fb = int(((_np(fl) & FALLBACK) > 0).sum())
    say(f"[{label}] ok, max error {err.max(initial=0.0):.2e}, fallback rows={fb}")


@pytest.mark.parametrize("name", ["cfg1", "cfg3", "cfg0"])
def test_logprobs_configs(ssb, name):
    """The workloads' rows (penalties, bias, grammar, temperatures, greedy
    rows) with the log-probability bit on every other row."""
    inp = W.make_config(name)
    inp["mode"] = inp["mode"] | np.where(np.arange(inp["B"]) % 2 == 1, W.MODE_LOGPROBS, 0).astype(np.uint32)
    inp["mode"][0] |= np.uint32(W.MODE_LOGPROBS)  # a greedy row too (cfg1/cfg3)
    for n in (1, 20, 700):
        check_logprobs(ssb, inp, n, f"logprobs-{name}-{n}")


def test_logprobs_edge_cases(ssb):
    """Tied rows, a fully masked row, NaN and -inf, long histories (the
    merge's global patch table), and a vocabulary that is not a multiple of a
    unit."""
    rng = np.random.default_rng(91)
    B, V = 6, 40000
    x = rng.normal(0, 3, (B, V)).astype(np.float32)
    x[0] = 1.5
    x[2, ::7] = np.nan
    x[3, :100] = -np.inf
    mask = np.full((B, (V + 31) // 32), 0xFFFFFFFF, np.uint32)
    mask[1] = 0
    hist = [rng.integers(0, V, 20).astype(np.int32) for _ in range(B)]
    hist[4] = rng.integers(0, V, 5000).astype(np.int32)  # more distinct ids than the LDS table
    pen = W.MODE_LOGPROBS | W.MODE_REP | W.MODE_FREQ | W.MODE_TEMP | W.MODE_GRAMMAR
    inp = W.custom_rows(x, W.F32, k_max=64, mode=np.full(B, pen, np.uint32),
                        temperature=rng.uniform(0.5, 2.0, B).astype(np.float32), rep=np.full(B, 1.2, np.float32),
                        freq=np.full(B, 0.3, np.float32), bitmask=mask,
                        hist_offsets=np.concatenate([[0], np.cumsum([len(h) for h in hist])]).astype(np.int32),
                        hist_ids=np.concatenate(hist))
    check_logprobs(ssb, inp, 50, "logprobs-edges-f32")
    inp_b = dict(inp)
    inp_b["x"] = W.bf16_bits_from_f32(x)
    inp_b["dtype"] = W.BF16
    check_logprobs(ssb, inp_b, 50, "logprobs-edges-bf16")


# --------------------------------------------------------------------------
# Materialised pipeline
# --------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["cfg0", "cfg1", "long_history", "dense_patch", "nan_empty", "grammar_few"])
def test_process_logits(ssb, name):
    inp = W.make_config(name) if name.startswith("cfg") else _edge_inputs(name)
    if name == "cfg1":
        inp = W.config1(B=16)
    say(f"[{name}] process B={inp['B']} V={inp['V']}")
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    y, P, fl = ssb.process_logits(x, prm, inp["k_max"])
    torch.cuda.synchronize()
    y, P = _np(y), _np(P)
    ref = oracle.process_logits(inp)
    assert np.array_equal(y.view(np.uint32), ref["y"].view(np.uint32)), name
    lo, hi = ref["ns_range"][:, 0], ref["ns_range"][:, 1]

    def close(Pr):
        err = np.abs(P.astype(np.float64) - Pr)
        return np.all(err <= 1e-5 * Pr + 1e-38, axis=1)

    ok = close(ref["P"])
    # rows whose kept-set size depends on a comparison within 1e-6 of its
    # boundary: the GPU's P must equal the oracle's for one admissible size
    for j in range(int((hi - lo).max()) + 1 if hi.size else 0):
        alt = oracle.process_logits(inp, force_ns=np.minimum(lo + j, hi))
        ok |= close(alt["P"])
    bad = np.nonzero(~ok)[0]
    assert bad.size == 0, (name, bad[:5])
    near = int((hi > lo).sum())
    if COUNTS is not None:
        COUNTS.add(f"process-{name}", inp["B"], near, 0, int(((_np(fl) & FALLBACK) > 0).sum()))
    say(f"[{name}] ok, rows with several admissible kept sets: {near}")


# --------------------------------------------------------------------------
# Verification
# --------------------------------------------------------------------------
def run_verify(ssb, inp):
    x = ssb.logits_tensor(inp)
    q = torch.from_numpy(np.ascontiguousarray(inp["draft_probs"], np.float32)).cuda()
    d = torch.from_numpy(np.ascontiguousarray(inp["draft_tokens"], np.int32)).cuda()
    prm = ssb.Params.from_arrays(inp)
    out, nacc, fl = ssb.verify(x, q, d, prm, inp["k_max"])
    torch.cuda.synchronize()
    return _np(out), _np(nacc), _np(fl)


def check_verify(inp, out, nacc, fl, label):
    ref = oracle.verify(inp)
    A = ref["adm_nacc"].shape[1]
    valid = np.arange(A)[None, :] < ref["n_adm"][:, None]
    same = (ref["adm_tokens"] == out[:, None, :]).all(axis=2) & (ref["adm_nacc"] == nacc[:, None]) & valid
    ok = same.any(axis=1)
    bad = np.nonzero(~ok)[0]
    assert bad.size == 0, (label, bad[:5], out[bad[:5]], nacc[bad[:5]], ref["tokens"][bad[:5]], ref["n_adm"][bad[:5]])
    assert np.array_equal(fl & (EMPTY | KCAP), ref["flags"] & (EMPTY | KCAP)), label
    near = int((ref["n_adm"] > 1).sum())
    alt = int((~((out == ref["tokens"]).all(axis=1) & (nacc == ref["n_acc"]))).sum())
    if COUNTS is not None:
        COUNTS.add(label, nacc.size, near, alt, int(((fl & FALLBACK) > 0).sum()))
    say(f"[{label}] requests={nacc.size} mean accepted={nacc.mean():.2f} near-boundary requests={near} "
        f"(outcome other than the oracle's own: {alt})")


def test_verify_config4(ssb):
    inp = W.config4()
    say("[cfg4] verify B=64 L=4 V=131072")
    out, nacc, fl = run_verify(ssb, inp)
    check_verify(inp, out, nacc, fl, "cfg4")


def test_verify_edge_cases(ssb):
    rng = np.random.default_rng(41)
    B, L, V = 12, 3, 5000
    t = rng.normal(0, 1.5, (B, L + 1, V)).astype(np.float32)
    q = rng.dirichlet(np.ones(V) * 0.3, size=(B, L)).astype(np.float32)
    d = np.stack([[rng.choice(V, p=q[b, l] / q[b, l].sum()) for l in range(L)] for b in range(B)]).astype(np.int32)
    d[1, 1] = -1          # end of draft
    d[2, 0] = V + 5       # out-of-range draft
    mode = np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_REP | W.MODE_PRES)
    mode[3] = W.MODE_GREEDY
    mode[4] = W.MODE_GREEDY | W.MODE_REP
    d[3, :] = np.argmax(t[3, 0])
    hist = [rng.integers(0, V, 50).astype(np.int32) for _ in range(B)]
    off = np.zeros(B + 1, np.int32)
    off[1:] = np.cumsum([len(h) for h in hist])
    inp = W.custom_rows(t.reshape(B * (L + 1), V), W.F32, k_max=256, mode=mode,
                        temperature=np.full(B * (L + 1), 0.9), top_k=np.full(B * (L + 1), 100),
                        top_p=np.full(B * (L + 1), 0.95), rep=np.full(B * (L + 1), 1.5),
                        pres=np.full(B * (L + 1), 0.5), position=np.arange(B * (L + 1)) * 3)
    for k in ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres", "seed", "position"):
        inp[k] = inp[k][:B]
    inp["mode"] = mode.astype(np.uint32)
    inp["hist_offsets"], inp["hist_ids"] = off, np.concatenate(hist)
    inp["bias_offsets"] = np.zeros(B + 1, np.int32)
    inp.update(x=t, B=B, L=L, draft_probs=q, draft_tokens=d)
    say("[verify-edge] B=12 L=3 V=5000")
    out, nacc, fl = run_verify(ssb, inp)
    check_verify(inp, out, nacc, fl, "verify-edge")


def test_verify_grammar(ssb):
    """Verification with an allow bitmask per target row (B (L+1) rows): draft
    tokens outside a row's allowed set have P(d) = 0 and are always rejected."""
    rng = np.random.default_rng(57)
    B, L, V = 8, 3, 1 << 15
    t = rng.normal(0.0, 2.0, (B, L + 1, V))
    for b in range(B):
        for l in range(L + 1):
            t[b, l, rng.choice(V, 12, replace=False)] += rng.uniform(6.0, 12.0, 12)
    z = t[:, :L] + rng.normal(0.0, 1.0, (B, L, V))
    q64 = np.exp(z - z.max(axis=2, keepdims=True))
    q64 /= q64.sum(axis=2, keepdims=True)
    q = q64.astype(np.float32)
    d = np.stack([[rng.choice(V, p=q64[b, l]) for l in range(L)] for b in range(B)]).astype(np.int32)
    mask = np.zeros((B * (L + 1), V // 32), np.uint32)
    for r in range(B * (L + 1)):
        allow = rng.choice(V, V // 4, replace=False)
        b, l = divmod(r, L + 1)
        allow = np.concatenate([allow, [int(np.argmax(t[b, l]))]]) if (b + l) % 2 == 0 else allow
        if l < L and b % 3 == 0:
            allow = np.concatenate([allow, [d[b, l]]])
        for i in allow:
            mask[r, i >> 5] |= np.uint32(1 << (int(i) & 31))
    mode = np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_GRAMMAR | W.MODE_REP)
    mode[1] = W.MODE_GREEDY | W.MODE_GRAMMAR
    hist = [rng.integers(0, V, 64).astype(np.int32) for _ in range(B)]
    off = np.zeros(B + 1, np.int32)
    off[1:] = np.cumsum([len(h) for h in hist])
    xb = W.bf16_bits_from_f32(t.astype(np.float32))
    inp = W.custom_rows(xb.reshape(B * (L + 1), V), W.BF16, k_max=256, mode=np.zeros(B * (L + 1)))
    for k in ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres", "seed", "position"):
        inp[k] = inp[k][:B]
    inp["mode"] = mode.astype(np.uint32)
    inp["temperature"] = np.full(B, 0.9, np.float32)
    inp["top_k"] = np.full(B, 200, np.int32)
    inp["top_p"] = np.full(B, 0.95, np.float32)
    inp["rep"] = np.full(B, 1.3, np.float32)
    inp["position"] = np.arange(B, dtype=np.int64) * 7
    inp["hist_offsets"], inp["hist_ids"] = off, np.concatenate(hist)
    inp["bias_offsets"] = np.zeros(B + 1, np.int32)
    inp["bitmask"] = mask
    inp.update(x=xb, B=B, L=L, draft_probs=q, draft_tokens=d)
    say(f"[verify-grammar] B={B} L={L} V={V}")
    out, nacc, fl = run_verify(ssb, inp)
    check_verify(inp, out, nacc, fl, "verify-grammar")


def run_verify_sparse(ssb, inp):
    x = ssb.logits_tensor(inp)
    qi = torch.from_numpy(np.ascontiguousarray(inp["draft_idx"], np.int32)).cuda()
    qv = torch.from_numpy(np.ascontiguousarray(inp["draft_q"], np.float32)).cuda()
    d = torch.from_numpy(np.ascontiguousarray(inp["draft_tokens"], np.int32)).cuda()
    prm = ssb.Params.from_arrays(inp)
    out, nacc, fl = ssb.verify_sparse(x, qi, qv, d, prm, inp["k_max"])
    torch.cuda.synchronize()
    return _np(out), _np(nacc), _np(fl)


def test_verify_sparse_config4(ssb):
    inp = W.config4_sparse()
    say("[cfg4_sparse] verify B=64 L=4 V=131072 kq=64")
    out, nacc, fl = run_verify_sparse(ssb, inp)
    check_verify(inp, out, nacc, fl, "cfg4_sparse")


def _sparse_edge_input(rng, B, L, V, kq, dtype, k_max):
    """Target rows with a few heads, sparse lists holding duplicates, padding
    (-1), out-of-range ids and unlisted drafts; greedy, end-of-draft and
    penalised requests mixed in."""
    t = rng.normal(0.0, 1.5, (B, L + 1, V))
    for b in range(B):
        for l in range(L + 1):
            t[b, l, rng.choice(V, 24, replace=False)] += rng.uniform(3.0, 8.0, 24)
    idx = np.full((B, L, kq), -1, np.int32)
    val = np.zeros((B, L, kq), np.float32)
    d = np.empty((B, L), np.int32)
    for b in range(B):
        for l in range(L):
            n = int(rng.integers(1, kq + 1))
            heads = np.argsort(-t[b, l], kind="stable")[: min(n, 32)]
            ids = np.concatenate([heads, rng.choice(V, n - heads.size)]) if n > heads.size else heads
            q = rng.dirichlet(np.ones(n)).astype(np.float32)
            idx[b, l, :n], val[b, l, :n] = ids, q
            if n >= 4:
                idx[b, l, n - 1] = ids[0]          # a repeated id: its entries add up
                idx[b, l, n - 2] = V + 3           # out of range: ignored
            d[b, l] = ids[int(rng.integers(0, n))] if b % 4 else int(rng.integers(0, V))  # some unlisted drafts
    d[1, -1] = -1                                   # end of draft
    mode = np.full(B, W.MODE_TEMP | W.MODE_TOPK | W.MODE_TOPP | W.MODE_REP)
    mode[2] = W.MODE_GREEDY
    mode[5 % B] = W.MODE_TEMP | W.MODE_MINP
    tt = t.astype(np.float32)
    x = tt if dtype == W.F32 else W.bf16_bits_from_f32(tt)
    inp = W.custom_rows(x.reshape(B * (L + 1), V), dtype, k_max=k_max, mode=np.zeros(B * (L + 1)))
    for k in ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres", "seed", "position"):
        inp[k] = inp[k][:B]
    inp["mode"] = mode.astype(np.uint32)
    inp["temperature"] = np.full(B, 0.9, np.float32)
    inp["top_k"] = np.full(B, k_max, np.int32)
    inp["top_p"] = np.full(B, 0.97, np.float32)
    inp["min_p"] = np.full(B, 0.01, np.float32)
    inp["rep"] = np.full(B, 1.2, np.float32)
    inp["position"] = np.arange(B, dtype=np.int64) * 13
    hist = [rng.integers(0, V, 40).astype(np.int32) for _ in range(B)]
    off = np.zeros(B + 1, np.int32)
    off[1:] = np.cumsum([len(h) for h in hist])
    inp["hist_offsets"], inp["hist_ids"] = off, np.concatenate(hist)
    inp["bias_offsets"] = np.zeros(B + 1, np.int32)
    inp.update(x=x, B=B, L=L, draft_idx=idx, draft_q=val, draft_tokens=d)
    return inp


@pytest.mark.parametrize("dtype,kq,V,k_max", [(W.F32, 1, 3000, 64), (W.F32, 40, 5000, 256),
                                             (W.BF16, 700, 1 << 15, 1024), (W.BF16, 4096, 1 << 16, 2048)],
                         ids=["f32-kq1", "f32-kq40", "bf16-kq700", "bf16-kq4096"])
def test_verify_sparse_edge_cases(ssb, dtype, kq, V, k_max):
    rng = np.random.default_rng(60 + kq)
    B, L = 10, 3
    inp = _sparse_edge_input(rng, B, L, V, kq, dtype, k_max)
    label = f"verify-sparse-{dtype}-kq{kq}"
    say(f"[{label}] B={B} L={L} V={V} k_max={k_max}")
    out, nacc, fl = run_verify_sparse(ssb, inp)
    check_verify(inp, out, nacc, fl, label)


def test_verify_sparse_equals_dense_scatter(ssb):
    # repeat-free lists: the sparse call gives the dense call's outputs for
    # the q they scatter to (same kernels, only the q lookup differs)
    inp = W.config4_sparse(B=16)
    V = inp["V"]
    dense = np.zeros(inp["draft_idx"].shape[:2] + (V,), np.float32)
    for b in range(dense.shape[0]):
        for l in range(dense.shape[1]):
            m = inp["draft_idx"][b, l] >= 0
            dense[b, l, inp["draft_idx"][b, l, m]] = inp["draft_q"][b, l, m]
    sp = run_verify_sparse(ssb, inp)
    dn = run_verify(ssb, dict(inp, draft_probs=dense))
    for a_, b_ in zip(sp, dn):
        assert np.array_equal(a_, b_)


def run_verify_tree(ssb, inp):
    x = ssb.logits_tensor(inp)
    rm = torch.from_numpy(np.ascontiguousarray(inp["row_map"], np.int32)).cuda()
    qi = torch.from_numpy(np.ascontiguousarray(inp["draft_idx"], np.int32)).cuda()
    qv = torch.from_numpy(np.ascontiguousarray(inp["draft_q"], np.float32)).cuda()
    d = torch.from_numpy(np.ascontiguousarray(inp["draft_tokens"], np.int32)).cuda()
    prm = ssb.Params.from_arrays(inp)
    out, nacc, fl = ssb.verify_tree(x, rm, qi, qv, d, prm, inp["k_max"])
    torch.cuda.synchronize()
    return _np(out), _np(nacc), _np(fl)


def test_verify_tree_config4(ssb):
    # the sparse-list verification workload's paths hidden in trees of 9 rows
    inp = W.tree_from_path(W.config4_sparse(), 9, 4242)
    say("[cfg4_tree] verify B=64 L=4 Lt=9 V=131072 kq=64")
    out, nacc, fl = run_verify_tree(ssb, inp)
    check_verify(inp, out, nacc, fl, "cfg4_tree")


@pytest.mark.parametrize("dtype", [W.F32, W.BF16])
def test_verify_tree_edge_cases(ssb, dtype):
    # penalties, grammar rows along the path, greedy rows, map entries outside
    # the tree at the first and at later positions, repeated rows in one map
    rng = np.random.default_rng(71)
    B, L, V, kq = 10, 3, 1 << 14, 48
    path = _sparse_edge_input(rng, B, L, V, kq, dtype, 512)
    mask = np.zeros((B * (L + 1), V // 32), np.uint32)
    for r in range(B * (L + 1)):
        b, l = divmod(r, L + 1)
        allow = rng.choice(V, V // 3, replace=False)
        if l < L:
            allow = np.concatenate([allow, path["draft_idx"][b, l][path["draft_idx"][b, l] >= 0]])
        ok = allow[(allow >= 0) & (allow < V)]
        np.bitwise_or.at(mask[r], ok >> 5, (np.uint32(1) << (ok & 31).astype(np.uint32)))
    path["bitmask"] = mask
    path["mode"] = path["mode"] | np.uint32(W.MODE_GRAMMAR)
    inp = W.tree_from_path(path, 2 * (L + 1), 99)
    rm = inp["row_map"]
    rm[0, 0] = -1                # outside the tree at the first position
    rm[1, 2] = 2 * (L + 1)       # ... at a later one
    rm[4, 1] = rm[4, 0]          # the same row twice
    label = f"verify-tree-{dtype}"
    say(f"[{label}] B={B} L={L} Lt={2 * (L + 1)} V={V}")
    out, nacc, fl = run_verify_tree(ssb, inp)
    check_verify(inp, out, nacc, fl, label)
    assert nacc[0] == 0 and np.all(out[0] == -1) and (fl[0] & EMPTY)


# --------------------------------------------------------------------------
# Graph capture and determinism
# --------------------------------------------------------------------------
def test_graph_replay_matches_eager(ssb):
    inp = W.config1()
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    ws = ssb.workspace(ssb.OP_SAMPLE, inp["B"], inp["V"], 0, inp["k_max"], ssb.BF16)
    tok = torch.empty(inp["B"], dtype=torch.int32, device="cuda")
    lp = torch.empty(inp["B"], dtype=torch.float32, device="cuda")
    fl = torch.empty(inp["B"], dtype=torch.int32, device="cuda")
    say("[graph] eager reference")
    ssb.sample(x, prm, inp["k_max"], out_token=tok, out_logprob=lp, flags=fl, ws=ws)
    torch.cuda.synchronize()
    ref = (_np(tok).copy(), _np(lp).copy())
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ssb.sample(x, prm, inp["k_max"], out_token=tok, out_logprob=lp, flags=fl, ws=ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say("[graph] capture")
    with torch.cuda.graph(g):
        ssb.sample(x, prm, inp["k_max"], out_token=tok, out_logprob=lp, flags=fl, ws=ws)
    for rep in range(3):
        tok.fill_(-7)
        say(f"[graph] replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(_np(tok), ref[0]) and np.array_equal(_np(lp), ref[1]), rep
        # eager work between replays
        ssb.sample(x, prm, inp["k_max"], ws=ws)
        torch.cuda.synchronize()
    # new step: the graph reads positions from device memory
    prm.position.add_(1)
    g.replay()
    torch.cuda.synchronize()
    inp2 = dict(inp)
    inp2["position"] = inp["position"] + 1
    check_sample(inp2, _np(tok), _np(lp), _np(fl), "graph-pos+1")


@pytest.mark.parametrize("entry", ["sample_full", "sample_gumbel", "verify_sparse", "verify_tree"])
def test_graph_replay_of_the_extended_entry_points(ssb, entry):
    """Each extended entry point captured in a HIP graph: every replay (with
    eager calls between replays) gives the eager result."""
    if entry.startswith("sample"):
        inp = nucleus_rows(W.config1(B=16)) if entry == "sample_full" else W.config1(B=16)
        x = ssb.logits_tensor(inp)
        prm = ssb.Params.from_arrays(inp)
        ws = ssb.workspace(ssb.OP_SAMPLE, inp["B"], inp["V"], 0, inp["k_max"], ssb.BF16)
        outs = [torch.empty(inp["B"], dtype=dt, device="cuda") for dt in (torch.int32, torch.float32, torch.int32)]
        g_noise = torch.from_numpy(W.gumbel_noise(inp["B"], inp["V"], 77)).cuda()

        def call(o):
            if entry == "sample_full":
                ssb.sample_full(x, prm, inp["k_max"], out_token=o[0], out_logprob=o[1], flags=o[2], ws=ws)
            else:
                ssb.sample_gumbel(x, prm, inp["k_max"], g_noise, out_token=o[0], out_logprob=o[1], flags=o[2], ws=ws)
    else:
        inp = W.config4_sparse(B=8)
        if entry == "verify_tree":
            inp = W.tree_from_path(inp, 7, 5)
        x = ssb.logits_tensor(inp)
        qi = torch.from_numpy(np.ascontiguousarray(inp["draft_idx"], np.int32)).cuda()
        qv = torch.from_numpy(np.ascontiguousarray(inp["draft_q"], np.float32)).cuda()
        d = torch.from_numpy(np.ascontiguousarray(inp["draft_tokens"], np.int32)).cuda()
        prm = ssb.Params.from_arrays(inp)
        L = inp["L"]
        ws = ssb.workspace(ssb.OP_VERIFY, inp["B"], inp["V"], L, inp["k_max"], ssb.BF16)
        outs = [torch.empty(inp["B"], L + 1, dtype=torch.int32, device="cuda"),
                torch.empty(inp["B"], dtype=torch.int32, device="cuda"),
                torch.empty(inp["B"], dtype=torch.int32, device="cuda")]
        rm = torch.from_numpy(np.ascontiguousarray(inp.get("row_map", np.zeros((1, 1))), np.int32)).cuda()

        def call(o):
            if entry == "verify_tree":
                ssb.verify_tree(x, rm, qi, qv, d, prm, inp["k_max"], out_tokens=o[0], out_nacc=o[1], flags=o[2], ws=ws)
            else:
                ssb.verify_sparse(x, qi, qv, d, prm, inp["k_max"], out_tokens=o[0], out_nacc=o[1], flags=o[2], ws=ws)
    say(f"[graph-{entry}] eager reference")
    call(outs)
    torch.cuda.synchronize()
    ref = [_np(o).copy() for o in outs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call(outs)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    say(f"[graph-{entry}] capture")
    with torch.cuda.graph(g):
        call(outs)
    scratch = [torch.empty_like(o) for o in outs]
    for rep in range(3):
        for o in outs:
            o.fill_(-7)
        say(f"[graph-{entry}] replay {rep}")
        g.replay()
        torch.cuda.synchronize()
        for a_, r_ in zip(outs, ref):
            assert np.array_equal(_np(a_), r_), (entry, rep)
        call(scratch)  # eager work between replays
        torch.cuda.synchronize()


def test_repeat_calls_are_bitwise_identical(ssb):
    inp = W.config3(B=32)
    say("[determinism] cfg3 B=32 x3")
    outs = [run_sample(ssb, inp) for _ in range(3)]
    for o in outs[1:]:
        assert all(np.array_equal(a, b) for a, b in zip(outs[0], o))
