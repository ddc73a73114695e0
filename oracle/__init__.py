"""CPU oracle for the fused sampler -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It wraps ``ssref.c`` (plain C, float32
prologue without contraction, double-precision probabilities) through ctypes
and shares nothing with the HIP implementation.

Functions take the input dicts produced by ``gen.workloads``.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from .build import build as _build, LIB_PATH

_lib = None


class _Params(C.Structure):
    _fields_ = [
        ("B", C.c_int), ("V", C.c_int),
        ("mode", C.c_void_p),
        ("temperature", C.c_void_p), ("top_p", C.c_void_p), ("min_p", C.c_void_p),
        ("rep", C.c_void_p), ("freq", C.c_void_p), ("pres", C.c_void_p),
        ("top_k", C.c_void_p),
        ("hist_off", C.c_void_p), ("hist_ids", C.c_void_p),
        ("bias_off", C.c_void_p), ("bias_ids", C.c_void_p),
        ("bias_vals", C.c_void_p),
        ("bitmask", C.c_void_p),
        ("mask_ld", C.c_int64),
        ("seed", C.c_void_p),
        ("position", C.c_void_p),
        ("k_cap", C.c_int),
    ]


def lib():
    global _lib
    if _lib is None:
        # SSREF_LIB: a library built from a modified copy of ssref.c (the
        # planted-mistake tests load one to check that the pins catch it)
        path = os.environ.get("SSREF_LIB")
        if not path:
            if not os.path.exists(LIB_PATH):
                _build()
            path = LIB_PATH
        _lib = C.CDLL(path)
        _lib.ssref_uniform.restype = C.c_double
        _lib.ssref_uniform.argtypes = [C.c_uint64, C.c_uint32, C.c_int64, C.c_int]
        _lib.ssref_near.restype = C.c_double
    return _lib


def near():
    """Width of the near-boundary band inside which a comparison may go either way."""
    return float(lib().ssref_near())


def adm_max():
    return int(lib().ssref_adm_max())


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dt):
    return None if a is None else np.ascontiguousarray(a, dtype=dt)


def _dtype_code(inp):
    return 1 if inp["dtype"] == "bf16" else 0


class _Bundle:
    """Keeps the contiguous arrays alive while the C call runs."""

    def __init__(self, inp, B=None):
        self.arrs = dict(
            mode=_c(inp.get("mode"), np.uint32),
            temperature=_c(inp.get("temperature"), np.float32),
            top_p=_c(inp.get("top_p"), np.float32),
            min_p=_c(inp.get("min_p"), np.float32),
            rep=_c(inp.get("rep"), np.float32),
            freq=_c(inp.get("freq"), np.float32),
            pres=_c(inp.get("pres"), np.float32),
            top_k=_c(inp.get("top_k"), np.int32),
            hist_off=_c(inp.get("hist_offsets"), np.int32),
            hist_ids=_c(inp.get("hist_ids"), np.int32),
            bias_off=_c(inp.get("bias_offsets"), np.int32),
            bias_ids=_c(inp.get("bias_ids"), np.int32),
            bias_vals=_c(inp.get("bias_vals"), np.float32),
            bitmask=_c(inp.get("bitmask"), np.uint32),
            seed=_c(inp.get("seed"), np.uint64),
            position=_c(inp.get("position"), np.int64),
        )
        a = self.arrs
        # zero-length CSR payloads still need a valid pointer
        for k in ("hist_ids", "bias_ids", "bias_vals"):
            if a[k] is not None and a[k].size == 0:
                a[k] = np.zeros(1, a[k].dtype)
        bm = a["bitmask"]
        self.p = _Params(
            B=int(inp["B"] if B is None else B), V=int(inp["V"]),
            mode=_ptr(a["mode"]), temperature=_ptr(a["temperature"]), top_p=_ptr(a["top_p"]),
            min_p=_ptr(a["min_p"]), rep=_ptr(a["rep"]), freq=_ptr(a["freq"]), pres=_ptr(a["pres"]),
            top_k=_ptr(a["top_k"]), hist_off=_ptr(a["hist_off"]), hist_ids=_ptr(a["hist_ids"]),
            bias_off=_ptr(a["bias_off"]), bias_ids=_ptr(a["bias_ids"]),
            bias_vals=_ptr(a["bias_vals"]), bitmask=_ptr(bm),
            mask_ld=0 if bm is None else int(bm.shape[-1]),
            seed=_ptr(a["seed"]), position=_ptr(a["position"]),
            k_cap=int(inp["k_max"]),
        )


def _x(inp):
    x = inp["x"]
    return np.ascontiguousarray(x, dtype=np.uint16 if inp["dtype"] == "bf16" else np.float32)


def philox4x32_10(ctr, key):
    c = (C.c_uint32 * 4)(*[int(v) & 0xFFFFFFFF for v in ctr])
    k = (C.c_uint32 * 2)(*[int(v) & 0xFFFFFFFF for v in key])
    o = (C.c_uint32 * 4)()
    lib().ssref_philox4x32_10(c, k, o)
    return [int(v) for v in o]


def uniform(seed, request, position, word):
    return float(lib().ssref_uniform(int(seed), int(request), int(position), int(word)))


def sample(inp, nthreads=0):
    """Singular-mode sampling.

    Returns dict(token, logprob, flags, margin, n_kept, adm_token [B, A],
    adm_logprob [B, A], n_adm): the oracle's own outcome and every admissible
    (token, log-probability) outcome when comparisons within ``near()`` of
    their boundary may go either way (entry 0 is the oracle's own, -1 pads).
    """
    B, V = int(inp["B"]), int(inp["V"])
    A = adm_max()
    x = _x(inp)
    bd = _Bundle(inp)
    tok = np.empty(B, np.int32)
    lp = np.empty(B, np.float32)
    fl = np.empty(B, np.int32)
    mg = np.empty(B, np.float64)
    nk = np.empty(B, np.int32)
    at = np.empty((B, A), np.int32)
    al = np.empty((B, A), np.float32)
    na = np.empty(B, np.int32)
    lib().ssref_sample(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), C.byref(bd.p),
                       _ptr(tok), _ptr(lp), _ptr(fl), _ptr(mg), _ptr(nk), _ptr(at), _ptr(al), _ptr(na),
                       C.c_int(nthreads))
    return dict(token=tok, logprob=lp, flags=fl, margin=mg, n_kept=nk, adm_token=at, adm_logprob=al, n_adm=na)


def sample_full(inp, nthreads=0):
    """Sampling with full-row truncation for requests without a top-k cut
    (top-p / min-p over the whole row when the kept set fits ``k_max``, else
    the bounded result flagged KCAP).  Returns the keys of ``sample`` except
    ``margin``."""
    B, V = int(inp["B"]), int(inp["V"])
    A = adm_max()
    x = _x(inp)
    bd = _Bundle(inp)
    tok = np.empty(B, np.int32)
    lp = np.empty(B, np.float32)
    fl = np.empty(B, np.int32)
    nk = np.empty(B, np.int32)
    at = np.empty((B, A), np.int32)
    al = np.empty((B, A), np.float32)
    na = np.empty(B, np.int32)
    lib().ssref_sample_full(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), C.byref(bd.p), _ptr(tok), _ptr(lp),
                            _ptr(fl), _ptr(nk), _ptr(at), _ptr(al), _ptr(na), C.c_int(nthreads))
    return dict(token=tok, logprob=lp, flags=fl, n_kept=nk, adm_token=at, adm_logprob=al, n_adm=na)


def sample_gumbel(inp, noise, nthreads=0):
    """Singular-mode sampling with the Gumbel-max draw: ``noise`` float32
    [B, V] holds g = ln z (z ~ Exp(1)) per token.  Returns the keys of
    ``sample`` except ``margin`` (the pick has no tolerance band of its own;
    the admissible outcomes cover the kept-set boundaries)."""
    B, V = int(inp["B"]), int(inp["V"])
    A = adm_max()
    x = _x(inp)
    g = np.ascontiguousarray(noise, dtype=np.float32)
    assert g.shape == (B, V)
    bd = _Bundle(inp)
    tok = np.empty(B, np.int32)
    lp = np.empty(B, np.float32)
    fl = np.empty(B, np.int32)
    nk = np.empty(B, np.int32)
    at = np.empty((B, A), np.int32)
    al = np.empty((B, A), np.float32)
    na = np.empty(B, np.int32)
    lib().ssref_sample_gumbel(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), C.byref(bd.p), _ptr(g),
                              C.c_int64(V), _ptr(tok), _ptr(lp), _ptr(fl), _ptr(nk), _ptr(at), _ptr(al),
                              _ptr(na), C.c_int(nthreads))
    return dict(token=tok, logprob=lp, flags=fl, n_kept=nk, adm_token=at, adm_logprob=al, n_adm=na)


def process_logits(inp, nthreads=0, force_ns=None):
    """Processed logits y [B,V] (float32) and final probabilities P [B,V] (float64).

    Also returns ns_range [B, 2], the admissible kept-set sizes.  ``force_ns``
    ([B] int) replaces a row's kept-set size by another admissible one."""
    B, V = int(inp["B"]), int(inp["V"])
    x = _x(inp)
    bd = _Bundle(inp)
    y = np.empty((B, V), np.float32)
    P = np.empty((B, V), np.float64)
    fl = np.empty(B, np.int32)
    rng = np.empty((B, 2), np.int32)
    fns = None if force_ns is None else np.ascontiguousarray(force_ns, dtype=np.int32)
    lib().ssref_process_logits(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), C.byref(bd.p),
                               _ptr(y), _ptr(P), _ptr(fl), _ptr(rng), _ptr(fns), C.c_int(nthreads))
    return dict(y=y, P=P, flags=fl, ns_range=rng)


def topk(inp, nthreads=0):
    """Standalone top-k on raw values: (values [B,k_max] float32, indices [B,k_max] int32)."""
    B, V, km = int(inp["B"]), int(inp["V"]), int(inp["k_max"])
    x = _x(inp)
    k = _c(inp.get("top_k"), np.int32)
    val = np.empty((B, km), np.float32)
    idx = np.empty((B, km), np.int32)
    lib().ssref_topk(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int(B), C.c_int(V), C.c_int64(V),
                     _ptr(k), C.c_int(km), _ptr(val), _ptr(idx), C.c_int(nthreads))
    return val, idx


def logprobs(inp, n_lp, nthreads=0):
    """Top-k log-probabilities of the rows with indicator bit 0x400: indices
    [B, n_lp] int32 (canonical order of the processed logits, -1 padded) and
    log-probabilities [B, n_lp] float32 under the untruncated softmax(y / tau)
    of the row (-inf padded)."""
    B, V = int(inp["B"]), int(inp["V"])
    x = _x(inp)
    bd = _Bundle(inp)
    idx = np.empty((B, n_lp), np.int32)
    lp = np.empty((B, n_lp), np.float32)
    lib().ssref_logprobs(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), C.byref(bd.p), C.c_int(n_lp),
                         _ptr(idx), _ptr(lp), C.c_int(nthreads))
    return idx, lp


def verify(inp, nthreads=0):
    """Multistep verification, against dense ``draft_probs`` [B, L, V] or, when
    the input holds ``draft_idx`` / ``draft_q`` [B, L, kq], sparse draft lists;
    with ``row_map`` [B, L+1] the logits ``x`` are [B, Lt, V] target rows of a
    draft tree and path position l reads row ``row_map[b, l]``.

    Returns dict(tokens [B,L+1], n_acc [B], flags, margin, adm_tokens [B,A,L+1],
    adm_nacc [B,A], n_adm): the oracle's own outcome and every admissible
    outcome when comparisons within ``near()`` of their boundary may go either
    way (entry 0 is the oracle's own)."""
    B, V, L = int(inp["B"]), int(inp["V"]), int(inp["L"])
    A = adm_max()
    x = _x(inp)
    sparse = inp.get("draft_idx") is not None
    if sparse:
        qi = np.ascontiguousarray(inp["draft_idx"], dtype=np.int32)
        qv = np.ascontiguousarray(inp["draft_q"], dtype=np.float32)
        assert qi.shape == qv.shape and qi.shape[:2] == (B, L)
    else:
        q = np.ascontiguousarray(inp["draft_probs"], dtype=np.float32)
    d = np.ascontiguousarray(inp["draft_tokens"], dtype=np.int32)
    bd = _Bundle(inp)
    tok = np.empty((B, L + 1), np.int32)
    na = np.empty(B, np.int32)
    fl = np.empty(B, np.int32)
    mg = np.empty(B, np.float64)
    aseq = np.empty((B, A, L + 1), np.int32)
    anacc = np.empty((B, A), np.int32)
    nadm = np.empty(B, np.int32)
    outs = (_ptr(tok), _ptr(na), _ptr(fl), _ptr(mg), _ptr(aseq), _ptr(anacc), _ptr(nadm), C.c_int(nthreads))
    if inp.get("row_map") is not None:
        assert sparse, "tree paths take sparse draft lists"
        rm = np.ascontiguousarray(inp["row_map"], dtype=np.int32)
        Lt = int(np.asarray(inp["x"]).shape[1])
        assert rm.shape == (B, L + 1)
        rc = lib().ssref_verify_tree(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), C.c_int(Lt), _ptr(rm),
                                     _ptr(qi), _ptr(qv), C.c_int(qi.shape[2]), _ptr(d), C.c_int(L),
                                     C.byref(bd.p), *outs)
        assert rc == 0
    elif sparse:
        rc = lib().ssref_verify_sparse(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), _ptr(qi), _ptr(qv),
                                       C.c_int(qi.shape[2]), _ptr(d), C.c_int(L), C.byref(bd.p), *outs)
        assert rc == 0
    else:
        lib().ssref_verify(_ptr(x), C.c_int(_dtype_code(inp)), C.c_int64(V), _ptr(q), C.c_int64(V),
                           _ptr(d), C.c_int(L), C.byref(bd.p), *outs)
    return dict(tokens=tok, n_acc=na, flags=fl, margin=mg, adm_tokens=aseq, adm_nacc=anacc, n_adm=nadm)


def row_distribution(y, mode, temperature=1.0, top_k=0, top_p=1.0, min_p=0.0, k_cap=None):
    """Truncated distribution of one processed row ``y`` (float32).

    Returns dict(order, P (canonical order, length n_s), n_valid, n_k, n_p, n_m,
    n_s, greedy, flags, ns_lo, ns_hi (admissible kept-set sizes), M, tau, Z_k,
    Z_s, margin_p, margin_m).
    """
    y = np.ascontiguousarray(y, dtype=np.float32)
    V = y.size
    if k_cap is None:
        k_cap = max(V, 1)
    order = np.empty(max(V, 1), np.int32)
    P = np.empty(max(k_cap, 1), np.float64)
    cnt = np.empty(9, np.int32)
    sums = np.empty(6, np.float64)
    nv = lib().ssref_row_distribution(
        _ptr(y), C.c_int(V), C.c_uint32(mode), C.c_float(temperature), C.c_int32(top_k),
        C.c_float(top_p), C.c_float(min_p), C.c_int(k_cap), _ptr(order), _ptr(P), _ptr(cnt), _ptr(sums))
    ns = int(cnt[4])
    return dict(order=order[:nv].copy(), P=P[:ns].copy(), n_valid=int(cnt[0]), n_k=int(cnt[1]),
                n_p=int(cnt[2]), n_m=int(cnt[3]), n_s=ns, greedy=int(cnt[5]), flags=int(cnt[6]),
                ns_lo=int(cnt[7]), ns_hi=int(cnt[8]),
                M=float(sums[0]), tau=float(sums[1]), Z_k=float(sums[2]), Z_s=float(sums[3]),
                margin_p=float(sums[4]), margin_m=float(sums[5]))


def process_row(x, dtype="f32", mode=0, rep=1.0, freq=0.0, pres=0.0, hist=(), extra=(),
                bias_ids=(), bias_vals=(), mask_row=None):
    """Prologue of one row; returns processed float32 logits."""
    if dtype == "bf16":
        xa = np.ascontiguousarray(x, dtype=np.uint16)
    else:
        xa = np.ascontiguousarray(x, dtype=np.float32)
    V = xa.size
    h = np.ascontiguousarray(np.asarray(hist, np.int32).reshape(-1)) if len(hist) else np.zeros(1, np.int32)
    e = np.ascontiguousarray(np.asarray(extra, np.int32).reshape(-1)) if len(extra) else np.zeros(1, np.int32)
    bi = np.ascontiguousarray(np.asarray(bias_ids, np.int32)) if len(bias_ids) else np.zeros(1, np.int32)
    bv = np.ascontiguousarray(np.asarray(bias_vals, np.float32)) if len(bias_vals) else np.zeros(1, np.float32)
    m = None if mask_row is None else np.ascontiguousarray(mask_row, dtype=np.uint32)
    y = np.empty(V, np.float32)
    lib().ssref_process_row(_ptr(xa), C.c_int(1 if dtype == "bf16" else 0), C.c_int(V), C.c_uint32(mode),
                            C.c_float(rep), C.c_float(freq), C.c_float(pres),
                            _ptr(h), C.c_int(len(hist)), _ptr(e), C.c_int(len(extra)),
                            _ptr(bi), _ptr(bv), C.c_int(len(bias_ids)), _ptr(m), _ptr(y))
    return y


def draw(w, u):
    """Inverse-CDF pick over weights ``w`` for uniform ``u``."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    return int(lib().ssref_draw(_ptr(w), C.c_int(w.size), C.c_double(u)))


def draw_ex(w, u):
    """Inverse-CDF pick with its boundary distance and admissible ranks.

    Returns (pick, margin relative to sum(w), admissible ranks, own pick first)."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    A = adm_max()
    mg = C.c_double()
    adm = np.empty(A, np.int32)
    na = C.c_int32()
    pick = lib().ssref_draw_ex(_ptr(w), C.c_int(w.size), C.c_double(u), C.byref(mg), _ptr(adm), C.c_int(A),
                               C.byref(na))
    return int(pick), float(mg.value), [int(v) for v in adm[:na.value]]
