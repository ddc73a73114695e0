"""Seeded synthetic workloads (numpy only, no sampling arithmetic).

Every generator returns a plain ``dict`` of numpy arrays that both the CPU
oracle and the HIP binding accept:

  x              logits, float32 ``[R, V]`` or raw bfloat16 bits (uint16) ``[R, V]``;
                 for verification ``[B, L+1, V]``
  dtype          ``F32`` or ``BF16``
  B, V, L        requests, vocabulary, draft length (0 outside verification)
  mode           uint32 ``[B]`` per-request bit indicators (paper, Section 3.5 table)
  temperature, top_p, min_p, rep, freq, pres   float32 ``[B]``
  top_k          int32 ``[B]``
  hist_offsets, hist_ids                 CSR of previously decoded token ids
  bias_offsets, bias_ids, bias_vals      CSR of sparse logit-bias entries
  bitmask        uint32 ``[R, ceil(V/32)]`` grammar allow bits (or None)
  seed           uint64 ``[B]``;  position  int64 ``[B]``
  k_max          candidate bound (int)
  draft_probs    float32 ``[B, L, V]`` and draft_tokens int32 ``[B, L]`` (verification)
  draft_idx, draft_q  int32 / float32 ``[B, L, kq]``: sparse draft distributions
                 (the (id, probability) list a draft step emits over its kept
                 set, padded with (-1, 0)); they replace ``draft_probs``

Logits follow the paper's evaluation regime (concentrated next-token
distributions, Section 3.3) with the shapes of the five evaluated
workloads; the recipes are listed in the design notes.  The draft
distribution ``q`` is part of the *input* (a stand-in for a draft model), so
its softmax is computed here in float64 as input preparation.
"""
from __future__ import annotations

import numpy as np

# Per-request indicator bits, as enumerated in the paper's bit-level encoding
# table (Section 3.5).  These are data-format constants only.
MODE_GRAMMAR = 0x001
MODE_REP = 0x002
MODE_FREQ = 0x004
MODE_PRES = 0x008
MODE_BIAS = 0x010
MODE_TEMP = 0x020
MODE_GREEDY = 0x040
MODE_TOPK = 0x080
MODE_TOPP = 0x100
MODE_MINP = 0x200
MODE_LOGPROBS = 0x400

F32 = "f32"
BF16 = "bf16"

CONFIG_NAMES = ("cfg0", "cfg1", "cfg2", "cfg3", "cfg4")


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even), return raw uint16 bits."""
    a = np.asarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r[nan] = np.uint16(0x7FC0)
    return r


def f32_from_bf16_bits(h: np.ndarray) -> np.ndarray:
    """Exact widening of raw bfloat16 bits to float32."""
    h = np.asarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


def empty_params(B: int) -> dict:
    """Neutral per-request parameters (no bits set, empty sparse lists)."""
    return dict(
        mode=np.zeros(B, np.uint32),
        temperature=np.ones(B, np.float32),
        top_k=np.zeros(B, np.int32),
        top_p=np.ones(B, np.float32),
        min_p=np.zeros(B, np.float32),
        rep=np.ones(B, np.float32),
        freq=np.zeros(B, np.float32),
        pres=np.zeros(B, np.float32),
        hist_offsets=np.zeros(B + 1, np.int32),
        hist_ids=np.zeros(0, np.int32),
        bias_offsets=np.zeros(B + 1, np.int32),
        bias_ids=np.zeros(0, np.int32),
        bias_vals=np.zeros(0, np.float32),
        bitmask=None,
        seed=np.full(B, 1234, np.uint64),
        position=np.zeros(B, np.int64),
    )


def _head_logits(rng, rows: int, V: int, heads: int, std: float = 2.0) -> np.ndarray:
    """N(0, std) background plus `heads` distinct ids per row boosted by U(8, 16)."""
    x = rng.normal(0.0, std, size=(rows, V))
    for r in range(rows):
        ids = rng.choice(V, size=heads, replace=False)
        x[r, ids] += rng.uniform(8.0, 16.0, size=heads)
    return x.astype(np.float32)


def _csr(lists) -> tuple[np.ndarray, np.ndarray]:
    off = np.zeros(len(lists) + 1, np.int32)
    off[1:] = np.cumsum([len(a) for a in lists])
    flat = np.concatenate([np.asarray(a) for a in lists]) if lists else np.zeros(0)
    return off, flat


def _hetero_params(rng, B: int, V: int, greedy_even: bool = True) -> dict:
    """Mixed greedy / stochastic requests with penalties, history and sparse bias."""
    p = empty_params(B)
    pen = MODE_REP | MODE_FREQ | MODE_PRES | MODE_BIAS
    for b in range(B):
        if greedy_even and b % 2 == 0:
            p["mode"][b] = MODE_GREEDY | pen
        else:
            p["mode"][b] = MODE_TEMP | MODE_TOPK | MODE_TOPP | MODE_MINP | pen
    p["temperature"][:] = rng.uniform(0.3, 1.5, B)
    p["top_k"][:] = rng.integers(1, 1025, B)
    p["top_p"][:] = rng.uniform(0.5, 1.0, B)
    p["min_p"][:] = rng.uniform(0.0, 0.1, B)
    p["rep"][:] = rng.uniform(1.0, 1.3, B)
    p["freq"][:] = rng.uniform(0.0, 0.5, B)
    p["pres"][:] = rng.uniform(0.0, 0.5, B)
    hist = [rng.integers(0, V, 512).astype(np.int32) for _ in range(B)]
    p["hist_offsets"], p["hist_ids"] = _csr(hist)
    p["hist_ids"] = p["hist_ids"].astype(np.int32)
    bids = [rng.choice(V, 16, replace=False).astype(np.int32) for _ in range(B)]
    bvals = [rng.uniform(-5.0, 5.0, 16).astype(np.float32) for _ in range(B)]
    p["bias_offsets"], p["bias_ids"] = _csr(bids)
    p["bias_ids"] = p["bias_ids"].astype(np.int32)
    p["bias_vals"] = np.concatenate(bvals).astype(np.float32)
    return p


def config0(B: int = 4) -> dict:
    """Singular fused sampling, tiny case: V=32768 fp32, 8 heads, mixed temperature."""
    rng = np.random.default_rng(1000 * 0 + 7)
    V = 32768
    x = _head_logits(rng, B, V, heads=8)
    p = empty_params(B)
    temps = np.array([0.0, 0.7, 1.0, 1.3], np.float32)
    p["temperature"][:] = temps[np.arange(B) % 4]
    p["mode"][:] = MODE_TEMP | MODE_TOPK | MODE_TOPP | MODE_MINP
    p["top_k"][:] = 50
    p["top_p"][:] = 0.9
    p["min_p"][:] = 0.0
    return dict(name="cfg0", x=x, dtype=F32, B=B, V=V, L=0, k_max=64, **p)


def config1(B: int = 64) -> dict:
    """Heterogeneous singular batch: V=2^17 bf16, 16 heads, penalties, bias."""
    rng = np.random.default_rng(1000 * 1 + 7)
    V = 1 << 17
    x = bf16_bits_from_f32(_head_logits(rng, B, V, heads=16))
    p = _hetero_params(rng, B, V)
    return dict(name="cfg1", x=x, dtype=BF16, B=B, V=V, L=0, k_max=1024, **p)


def config2(B: int = 256) -> dict:
    """Standalone top-k stress: V=2^18 fp32, low-entropy and flat rows, k in {1,50,1024,4096}."""
    rng = np.random.default_rng(1000 * 2 + 7)
    V = 1 << 18
    x = np.empty((B, V), np.float32)
    for b in range(B):
        if b % 2 == 0:
            x[b] = _head_logits(rng, 1, V, heads=32)[0]
        else:
            # U(-1, 1) on a 2^-23 grid: exactly representable, many exact ties
            x[b] = (rng.integers(-(1 << 23), 1 << 23, V) / float(1 << 23)).astype(np.float32)
    p = empty_params(B)
    p["mode"][:] = MODE_TOPK
    p["top_k"][:] = rng.choice(np.array([1, 50, 1024, 4096], np.int32), B)
    return dict(name="cfg2", x=x, dtype=F32, B=B, V=V, L=0, k_max=4096, **p)


def config3(B: int = 128) -> dict:
    """Grammar-constrained fused sampling: config-1 generator plus a 5% allow bitmask."""
    rng = np.random.default_rng(1000 * 3 + 7)
    V = 1 << 17
    x = bf16_bits_from_f32(_head_logits(rng, B, V, heads=16))
    p = _hetero_params(rng, B, V)
    W = (V + 31) // 32
    n_allow = int(round(0.05 * V))
    mask = np.zeros((B, W), np.uint32)
    xf = f32_from_bf16_bits(x)
    for b in range(B):
        am = int(np.argmax(xf[b]))
        pool = np.delete(np.arange(V), am)
        allow = rng.choice(pool, n_allow, replace=False)
        if ((b >> 1) & 1) == 0:
            allow[rng.integers(0, n_allow)] = am  # force-allow the raw argmax
        for i in allow:
            mask[b, i >> 5] |= np.uint32(1 << (int(i) & 31))
    p["bitmask"] = mask
    p["mode"] |= np.uint32(MODE_GRAMMAR)
    return dict(name="cfg3", x=x, dtype=BF16, B=B, V=V, L=0, k_max=1024, **p)


def config4(B: int = 64, L: int = 4) -> dict:
    """Multistep speculative verification: target [B, L+1, 2^17] bf16, draft q [B, L, V] fp32."""
    rng = np.random.default_rng(1000 * 4 + 7)
    V = 1 << 17
    xf = _head_logits(rng, B * (L + 1), V, heads=16)
    x = bf16_bits_from_f32(xf).reshape(B, L + 1, V)
    p = _hetero_params(rng, B, V)
    # draft distribution: softmax(target + N(0,1)) at temperature 1 (input preparation)
    tgt = f32_from_bf16_bits(x[:, :L, :]).astype(np.float64)
    noisy = tgt + rng.normal(0.0, 1.0, size=tgt.shape)
    noisy -= noisy.max(axis=-1, keepdims=True)
    e = np.exp(noisy)
    q64 = e / e.sum(axis=-1, keepdims=True)
    q = q64.astype(np.float32)
    rng_d = np.random.default_rng(1000 * 4 + 8)
    d = np.empty((B, L), np.int32)
    for b in range(B):
        for l in range(L):
            c = np.cumsum(q64[b, l])
            d[b, l] = min(int(np.searchsorted(c, rng_d.random() * c[-1], side="right")), V - 1)
    return dict(name="cfg4", x=x, dtype=BF16, B=B, V=V, L=L, k_max=1024,
                draft_probs=q, draft_tokens=d, **p)


def sparse_drafts(noisy: np.ndarray, kq: int, top_p: float, rng_d) -> tuple:
    """Sparse draft lists from draft logits ``noisy`` [B, L, V] (float64): per
    position the kq leading ids (value descending, lower index first), cut to
    the shortest prefix whose softmax mass reaches top_p, renormalised, as
    float32 (id, q) pairs padded with (-1, 0); and one draft token drawn from
    each list.  Input preparation standing in for a draft model's sampler."""
    B, L, V = noisy.shape
    idx = np.full((B, L, kq), -1, np.int32)
    qv = np.zeros((B, L, kq), np.float32)
    d = np.empty((B, L), np.int32)
    for b in range(B):
        for l in range(L):
            row = noisy[b, l]
            top = np.argpartition(-row, kq - 1)[:kq]
            top = top[np.lexsort((top, -row[top]))]
            w = np.exp(row[top] - row[top[0]])
            c = np.cumsum(w)
            n = min(int(np.searchsorted(c, top_p * c[-1], side="left")) + 1, kq)
            q = w[:n] / c[n - 1]
            idx[b, l, :n] = top[:n]
            qv[b, l, :n] = q.astype(np.float32)
            cq = np.cumsum(q)
            d[b, l] = int(top[min(int(np.searchsorted(cq, rng_d.random() * cq[-1], side="right")), n - 1)])
    return idx, qv, d


def config4_sparse(B: int = 64, L: int = 4, kq: int = 64) -> dict:
    """Verification against sparse draft lists: the target and parameters of
    config4, each draft position carrying at most kq (id, q) pairs (the draft
    distribution of config4 cut to its kq leading ids and top-p 0.95)."""
    rng = np.random.default_rng(1000 * 4 + 7)
    V = 1 << 17
    xf = _head_logits(rng, B * (L + 1), V, heads=16)
    x = bf16_bits_from_f32(xf).reshape(B, L + 1, V)
    p = _hetero_params(rng, B, V)
    tgt = f32_from_bf16_bits(x[:, :L, :]).astype(np.float64)
    noisy = tgt + rng.normal(0.0, 1.0, size=tgt.shape)
    idx, qv, d = sparse_drafts(noisy, kq, 0.95, np.random.default_rng(1000 * 4 + 9))
    return dict(name="cfg4_sparse", x=x, dtype=BF16, B=B, V=V, L=L, k_max=1024,
                draft_idx=idx, draft_q=qv, draft_tokens=d, **p)


def tree_from_path(inp: dict, Lt: int, seed: int) -> dict:
    """A draft tree holding a verification input's path: ``x`` becomes
    ``[B, Lt, V]`` with the path's L+1 target rows at distinct random rows of
    each request and N(0, 2) distractor rows elsewhere; ``row_map`` [B, L+1]
    names the path's rows.  Everything else is the path input's."""
    x = np.asarray(inp["x"])
    B, L1, V = x.shape
    assert Lt >= L1
    rng = np.random.default_rng(seed)
    noise = rng.normal(0.0, 2.0, size=(B, Lt, V)).astype(np.float32)
    tree = bf16_bits_from_f32(noise) if inp["dtype"] == BF16 else noise
    rmap = np.stack([rng.choice(Lt, L1, replace=False) for _ in range(B)]).astype(np.int32)
    for b in range(B):
        tree[b, rmap[b]] = x[b]
    out = dict(inp, x=tree, row_map=rmap)
    out["name"] = str(inp.get("name", "custom")) + "_tree"
    return out


def gumbel_noise(B: int, V: int, seed: int) -> np.ndarray:
    """Pre-drawn noise for the Gumbel-max draw: g = ln z, z ~ Exp(1), float32
    ``[B, V]`` (one value per token; the draw subtracts it at the kept ids)."""
    rng = np.random.default_rng(seed)
    return np.log(rng.standard_exponential(size=(B, V))).astype(np.float32)


def make_config(name: str, **kw) -> dict:
    return {"cfg0": config0, "cfg1": config1, "cfg2": config2,
            "cfg3": config3, "cfg4": config4, "cfg4_sparse": config4_sparse}[name](**kw)


def custom_rows(x, dtype: str = F32, k_max: int = 64, L: int = 0, **params) -> dict:
    """Wrap explicit logits (and optional per-request params) into an input dict."""
    x = np.asarray(x)
    if dtype == F32:
        x = x.astype(np.float32)
    else:
        x = x.astype(np.uint16)
    B = x.shape[0]
    V = x.shape[-1]
    p = empty_params(B)
    for k, v in params.items():
        if k not in p:
            raise KeyError(k)
        p[k] = v if v is None else np.asarray(v, dtype=(p[k].dtype if p[k] is not None else np.uint32))
    d = dict(name="custom", x=x, dtype=dtype, B=B, V=V, L=L, k_max=k_max, **p)
    return d
