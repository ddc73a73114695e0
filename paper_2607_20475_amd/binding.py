"""Thin ctypes binding of libss.so (argument marshalling only).

Every function takes torch tensors that already live on the GPU, passes their
device pointers and torch's current HIP stream to the C ABI declared in
``include/ss.h``, and raises on a non-zero status.  All computation runs in the
library's HIP kernels; there is no CPU or PyTorch fallback -- if ``libss.so`` is
missing the import fails.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libss.so")

# indicator bits (paper, Section 3.5 table) and flags, as declared in ss.h
GRAMMAR, REP, FREQ, PRES, BIAS, TEMP = 0x001, 0x002, 0x004, 0x008, 0x010, 0x020
GREEDY, TOPK, TOPP, MINP, LOGPROBS = 0x040, 0x080, 0x100, 0x200, 0x400
FLAG_EMPTY, FLAG_FALLBACK, FLAG_OUT_TRUNC, FLAG_KCAP = 1, 2, 4, 8
OP_TOPK, OP_SAMPLE, OP_VERIFY, OP_PROCESS, OP_LOGPROBS = 0, 1, 2, 3, 4
F32, BF16 = 0, 1

_lib = None


class SSError(RuntimeError):
    pass


class _Params(C.Structure):
    _fields_ = [
        ("B", C.c_int32), ("V", C.c_int32),
        ("mode", C.c_void_p), ("temperature", C.c_void_p), ("top_k", C.c_void_p),
        ("top_p", C.c_void_p), ("min_p", C.c_void_p),
        ("rep_penalty", C.c_void_p), ("freq_penalty", C.c_void_p), ("pres_penalty", C.c_void_p),
        ("hist_offsets", C.c_void_p), ("hist_ids", C.c_void_p),
        ("bias_offsets", C.c_void_p), ("bias_ids", C.c_void_p), ("bias_vals", C.c_void_p),
        ("bitmask", C.c_void_p), ("bitmask_ld", C.c_int64),
        ("seed", C.c_void_p), ("position", C.c_void_p),
    ]


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
        L.ss_workspace_bytes.restype = sz
        L.ss_workspace_bytes.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int]
        L.ss_workspace_init.restype = i32
        L.ss_workspace_init.argtypes = [vp, sz, vp]
        L.ss_topk.restype = i32
        L.ss_topk.argtypes = [vp, C.c_int, C.c_int, C.c_int, i64, vp, C.c_int, vp, vp, vp, vp, sz, vp]
        L.ss_sample.restype = i32
        L.ss_sample.argtypes = [vp, C.c_int, i64, C.POINTER(_Params), C.c_int, vp, vp, vp, vp, C.c_int, vp,
                                vp, sz, vp]
        if hasattr(L, "ss_sample_full"):
            L.ss_sample_full.restype = i32
            L.ss_sample_full.argtypes = [vp, C.c_int, i64, C.POINTER(_Params), C.c_int, vp, vp, vp, vp, C.c_int,
                                         vp, vp, sz, vp]
        if hasattr(L, "ss_sample_gumbel"):
            L.ss_sample_gumbel.restype = i32
            L.ss_sample_gumbel.argtypes = [vp, C.c_int, i64, C.POINTER(_Params), C.c_int, vp, i64, vp, vp, vp, vp,
                                           C.c_int, vp, vp, sz, vp]
        if hasattr(L, "ss_sample_noalloc"):
            L.ss_sample_noalloc.restype = i32
            L.ss_sample_noalloc.argtypes = [vp, C.c_int, i64, C.POINTER(_Params), C.c_int, vp, vp, vp, vp, C.c_int,
                                            vp, vp]
        L.ss_verify.restype = i32
        L.ss_verify.argtypes = [vp, C.c_int, i64, vp, i64, vp, C.c_int, C.POINTER(_Params), C.c_int, vp, vp,
                                vp, vp, sz, vp]
        if hasattr(L, "ss_verify_tree"):
            L.ss_verify_tree.restype = i32
            L.ss_verify_tree.argtypes = [vp, C.c_int, i64, C.c_int, vp, vp, vp, C.c_int, vp, C.c_int,
                                         C.POINTER(_Params), C.c_int, vp, vp, vp, vp, sz, vp]
        if hasattr(L, "ss_verify_sparse"):
            L.ss_verify_sparse.restype = i32
            L.ss_verify_sparse.argtypes = [vp, C.c_int, i64, vp, vp, C.c_int, vp, C.c_int, C.POINTER(_Params),
                                           C.c_int, vp, vp, vp, vp, sz, vp]
        if hasattr(L, "ss_logprobs"):
            L.ss_logprobs.restype = i32
            L.ss_logprobs.argtypes = [vp, C.c_int, i64, C.POINTER(_Params), C.c_int, vp, vp, vp, vp, sz, vp]
        L.ss_process_logits.restype = i32
        L.ss_process_logits.argtypes = [vp, C.c_int, i64, C.POINTER(_Params), C.c_int, vp, vp, vp, vp, sz, vp]
        L.ss_status_string.restype = C.c_char_p
        L.ss_status_string.argtypes = [i32]
        _lib = L
    return _lib


def _check(st):
    if st != 0:
        raise SSError(f"libss: {lib().ss_status_string(st).decode()} ({st})")


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise SSError(f"unsupported logits dtype {t.dtype}")


def workspace_bytes(op, B, V, L, k_max, dtype):
    return int(lib().ss_workspace_bytes(op, B, V, L, k_max, dtype))


def workspace(op, B, V, L, k_max, dtype, device="cuda"):
    """A zero-filled workspace for `op` (caller keeps it across calls)."""
    n = workspace_bytes(op, B, V, L, k_max, dtype)
    if n == 0:
        raise SSError("invalid sizes for workspace")
    return torch.zeros(n, dtype=torch.uint8, device=device)


class Params:
    """Per-request parameters as device tensors (see ss_params in ss.h)."""

    FIELDS = ("mode", "temperature", "top_k", "top_p", "min_p", "rep", "freq", "pres",
              "hist_offsets", "hist_ids", "bias_offsets", "bias_ids", "bias_vals",
              "bitmask", "seed", "position")
    DTYPES = dict(mode=torch.int32, temperature=torch.float32, top_k=torch.int32, top_p=torch.float32,
                  min_p=torch.float32, rep=torch.float32, freq=torch.float32, pres=torch.float32,
                  hist_offsets=torch.int32, hist_ids=torch.int32, bias_offsets=torch.int32,
                  bias_ids=torch.int32, bias_vals=torch.float32, bitmask=torch.int32,
                  seed=torch.int64, position=torch.int64)

    def __init__(self, B, V, **tensors):
        self.B, self.V = int(B), int(V)
        for f in self.FIELDS:
            setattr(self, f, tensors.get(f))

    @classmethod
    def from_arrays(cls, d, device="cuda"):
        """Build from a dict of numpy arrays (the gen.workloads layout)."""
        t = {}
        for f in cls.FIELDS:
            a = d.get(f)
            if a is None:
                continue
            a = np.ascontiguousarray(a)
            if a.size == 0:
                a = np.zeros(1, a.dtype)  # CSR payloads need a valid pointer
            if a.dtype == np.uint32:
                a = a.view(np.int32)
            elif a.dtype == np.uint64:
                a = a.view(np.int64)
            t[f] = torch.from_numpy(a).to(device=device, dtype=cls.DTYPES[f])
        return cls(d["B"], d["V"], **t)

    def struct(self):
        bm = self.bitmask
        return _Params(
            B=self.B, V=self.V, mode=_ptr(self.mode), temperature=_ptr(self.temperature),
            top_k=_ptr(self.top_k), top_p=_ptr(self.top_p), min_p=_ptr(self.min_p),
            rep_penalty=_ptr(self.rep), freq_penalty=_ptr(self.freq), pres_penalty=_ptr(self.pres),
            hist_offsets=_ptr(self.hist_offsets), hist_ids=_ptr(self.hist_ids),
            bias_offsets=_ptr(self.bias_offsets), bias_ids=_ptr(self.bias_ids), bias_vals=_ptr(self.bias_vals),
            bitmask=_ptr(bm), bitmask_ld=0 if bm is None else int(bm.shape[-1]),
            seed=_ptr(self.seed), position=_ptr(self.position))


def _ws(ws, op, B, V, L, k_max, dtype, device):
    if ws is None:
        ws = workspace(op, B, V, L, k_max, dtype, device)
    return ws


def topk(x, k, k_max, out_val=None, out_idx=None, flags=None, ws=None):
    """Exact top-k per row of x [B, V] (row stride x.stride(0)).  k: int32 [B] or None."""
    B, V = x.shape
    dt = _dtype_code(x)
    ws = _ws(ws, OP_TOPK, B, V, 0, k_max, dt, x.device)
    if out_val is None:
        out_val = torch.empty(B, k_max, dtype=torch.float32, device=x.device)
    if out_idx is None:
        out_idx = torch.empty(B, k_max, dtype=torch.int32, device=x.device)
    _check(lib().ss_topk(_ptr(x), dt, B, V, x.stride(0), _ptr(k), k_max, _ptr(out_val), _ptr(out_idx),
                         _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    return out_val, out_idx


def logprobs(logits, params, n_lp, out_idx=None, out_lp=None, flags=None, ws=None):
    """Top-k log-probabilities (rows whose mode has bit 0x400): indices and
    log-probabilities [B, n_lp] under the full-row distribution."""
    B, V = logits.shape
    dt = _dtype_code(logits)
    ws = _ws(ws, OP_LOGPROBS, B, V, 0, n_lp, dt, logits.device)
    if out_idx is None:
        out_idx = torch.empty(B, n_lp, dtype=torch.int32, device=logits.device)
    if out_lp is None:
        out_lp = torch.empty(B, n_lp, dtype=torch.float32, device=logits.device)
    p = params.struct()
    _check(lib().ss_logprobs(_ptr(logits), dt, logits.stride(0), C.byref(p), n_lp, _ptr(out_idx), _ptr(out_lp),
                             _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    return out_idx, out_lp


def sample(logits, params, k_max, k_out=0, out_token=None, out_logprob=None, out_idx=None, out_prob=None,
           flags=None, ws=None):
    """Singular-mode sampling of logits [B, V]; returns (token, logprob, flags[, idx, prob])."""
    B, V = logits.shape
    dt = _dtype_code(logits)
    dev = logits.device
    ws = _ws(ws, OP_SAMPLE, B, V, 0, k_max, dt, dev)
    if out_token is None:
        out_token = torch.empty(B, dtype=torch.int32, device=dev)
    if out_logprob is None:
        out_logprob = torch.empty(B, dtype=torch.float32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    if k_out > 0:
        if out_idx is None:
            out_idx = torch.empty(B, k_out, dtype=torch.int32, device=dev)
        if out_prob is None:
            out_prob = torch.empty(B, k_out, dtype=torch.float32, device=dev)
    p = params.struct()
    _check(lib().ss_sample(_ptr(logits), dt, logits.stride(0), C.byref(p), k_max, _ptr(out_token),
                           _ptr(out_logprob), _ptr(out_idx), _ptr(out_prob), k_out, _ptr(flags), _ptr(ws),
                           ws.numel(), _stream()))
    if k_out > 0:
        return out_token, out_logprob, flags, out_idx, out_prob
    return out_token, out_logprob, flags


def sample_full(logits, params, k_max, k_out=0, out_token=None, out_logprob=None, out_idx=None, out_prob=None,
                flags=None, ws=None):
    """ss_sample_full: sampling with full-row top-p / min-p for requests
    without a top-k cut.  Returns as ``sample``."""
    B, V = logits.shape
    dt = _dtype_code(logits)
    dev = logits.device
    ws = _ws(ws, OP_SAMPLE, B, V, 0, k_max, dt, dev)
    if out_token is None:
        out_token = torch.empty(B, dtype=torch.int32, device=dev)
    if out_logprob is None:
        out_logprob = torch.empty(B, dtype=torch.float32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    if k_out > 0:
        if out_idx is None:
            out_idx = torch.empty(B, k_out, dtype=torch.int32, device=dev)
        if out_prob is None:
            out_prob = torch.empty(B, k_out, dtype=torch.float32, device=dev)
    p = params.struct()
    _check(lib().ss_sample_full(_ptr(logits), dt, logits.stride(0), C.byref(p), k_max, _ptr(out_token),
                                _ptr(out_logprob), _ptr(out_idx), _ptr(out_prob), k_out, _ptr(flags), _ptr(ws),
                                ws.numel(), _stream()))
    if k_out > 0:
        return out_token, out_logprob, flags, out_idx, out_prob
    return out_token, out_logprob, flags


def sample_gumbel(logits, params, k_max, noise, k_out=0, out_token=None, out_logprob=None, out_idx=None,
                  out_prob=None, flags=None, ws=None):
    """ss_sample_gumbel: sampling with the Gumbel-max draw; noise float32 [B, >= V]
    holds g = ln z (z ~ Exp(1)) per token.  Returns as ``sample``."""
    B, V = logits.shape
    dt = _dtype_code(logits)
    dev = logits.device
    if noise.dtype != torch.float32 or noise.dim() != 2 or noise.shape[0] != B or noise.shape[1] < V \
            or noise.stride(1) != 1:
        raise SSError("noise must be float32 [B, >= V] with unit column stride")
    ws = _ws(ws, OP_SAMPLE, B, V, 0, k_max, dt, dev)
    if out_token is None:
        out_token = torch.empty(B, dtype=torch.int32, device=dev)
    if out_logprob is None:
        out_logprob = torch.empty(B, dtype=torch.float32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    if k_out > 0:
        if out_idx is None:
            out_idx = torch.empty(B, k_out, dtype=torch.int32, device=dev)
        if out_prob is None:
            out_prob = torch.empty(B, k_out, dtype=torch.float32, device=dev)
    p = params.struct()
    _check(lib().ss_sample_gumbel(_ptr(logits), dt, logits.stride(0), C.byref(p), k_max, _ptr(noise), noise.stride(0),
                                  _ptr(out_token), _ptr(out_logprob), _ptr(out_idx), _ptr(out_prob), k_out,
                                  _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    if k_out > 0:
        return out_token, out_logprob, flags, out_idx, out_prob
    return out_token, out_logprob, flags


def sample_noalloc(logits, params, k_max, out_token, out_logprob, flags, k_out=0, out_idx=None, out_prob=None):
    """ss_sample_noalloc: sampling into caller-provided outputs with the
    library's own per-GPU workspace (nothing is allocated by this call)."""
    B, V = logits.shape
    p = params.struct()
    _check(lib().ss_sample_noalloc(_ptr(logits), _dtype_code(logits), logits.stride(0), C.byref(p), k_max,
                                   _ptr(out_token), _ptr(out_logprob), _ptr(out_idx), _ptr(out_prob), k_out,
                                   _ptr(flags), _stream()))
    return out_token, out_logprob, flags


def verify(target_logits, draft_probs, draft_tokens, params, k_max, out_tokens=None, out_nacc=None, flags=None,
           ws=None):
    """target_logits [B, L+1, V], draft_probs [B, L, V] float32, draft_tokens [B, L] int32."""
    B, L1, V = target_logits.shape
    L = L1 - 1
    dt = _dtype_code(target_logits)
    dev = target_logits.device
    ws = _ws(ws, OP_VERIFY, B, V, L, k_max, dt, dev)
    if out_tokens is None:
        out_tokens = torch.empty(B, L + 1, dtype=torch.int32, device=dev)
    if out_nacc is None:
        out_nacc = torch.empty(B, dtype=torch.int32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    if target_logits.stride(0) != L1 * target_logits.stride(1) or draft_probs.stride(0) != L * draft_probs.stride(1):
        raise SSError("target rows and draft rows must be evenly strided")
    p = params.struct()
    _check(lib().ss_verify(_ptr(target_logits), dt, target_logits.stride(1), _ptr(draft_probs),
                           draft_probs.stride(1), _ptr(draft_tokens), L, C.byref(p), k_max, _ptr(out_tokens),
                           _ptr(out_nacc), _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    return out_tokens, out_nacc, flags


def verify_sparse(target_logits, draft_idx, draft_q, draft_tokens, params, k_max, out_tokens=None, out_nacc=None,
                  flags=None, ws=None):
    """target_logits [B, L+1, V]; draft_idx int32 / draft_q float32 [B, L, kq]
    (sparse draft lists); draft_tokens [B, L] int32."""
    B, L1, V = target_logits.shape
    L = L1 - 1
    kq = draft_idx.shape[-1]
    dt = _dtype_code(target_logits)
    dev = target_logits.device
    ws = _ws(ws, OP_VERIFY, B, V, L, k_max, dt, dev)
    if out_tokens is None:
        out_tokens = torch.empty(B, L + 1, dtype=torch.int32, device=dev)
    if out_nacc is None:
        out_nacc = torch.empty(B, dtype=torch.int32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    if target_logits.stride(0) != L1 * target_logits.stride(1):
        raise SSError("target rows must be evenly strided")
    for t, dtype in ((draft_idx, torch.int32), (draft_q, torch.float32)):
        if t.shape != (B, L, kq) or t.dtype != dtype or not t.is_contiguous():
            raise SSError("draft lists must be contiguous [B, L, kq] int32 ids and float32 probabilities")
    p = params.struct()
    _check(lib().ss_verify_sparse(_ptr(target_logits), dt, target_logits.stride(1), _ptr(draft_idx), _ptr(draft_q),
                                  kq, _ptr(draft_tokens), L, C.byref(p), k_max, _ptr(out_tokens), _ptr(out_nacc),
                                  _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    return out_tokens, out_nacc, flags


def verify_tree(target_logits, row_map, draft_idx, draft_q, draft_tokens, params, k_max, out_tokens=None,
                out_nacc=None, flags=None, ws=None):
    """target_logits [B, Lt, V] (a draft tree's target rows); row_map int32
    [B, L+1] (path position -> row); draft_idx int32 / draft_q float32
    [B, L, kq]; draft_tokens [B, L] int32."""
    B, Lt, V = target_logits.shape
    L = row_map.shape[1] - 1
    kq = draft_idx.shape[-1]
    dt = _dtype_code(target_logits)
    dev = target_logits.device
    ws = _ws(ws, OP_VERIFY, B, V, L, k_max, dt, dev)
    if out_tokens is None:
        out_tokens = torch.empty(B, L + 1, dtype=torch.int32, device=dev)
    if out_nacc is None:
        out_nacc = torch.empty(B, dtype=torch.int32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    if target_logits.stride(0) != Lt * target_logits.stride(1):
        raise SSError("target rows must be evenly strided")
    if row_map.shape != (B, L + 1) or row_map.dtype != torch.int32 or not row_map.is_contiguous():
        raise SSError("row_map must be contiguous int32 [B, L+1]")
    for t, dtype in ((draft_idx, torch.int32), (draft_q, torch.float32)):
        if t.shape != (B, L, kq) or t.dtype != dtype or not t.is_contiguous():
            raise SSError("draft lists must be contiguous [B, L, kq] int32 ids and float32 probabilities")
    p = params.struct()
    _check(lib().ss_verify_tree(_ptr(target_logits), dt, target_logits.stride(1), Lt, _ptr(row_map), _ptr(draft_idx),
                                _ptr(draft_q), kq, _ptr(draft_tokens), L, C.byref(p), k_max, _ptr(out_tokens),
                                _ptr(out_nacc), _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    return out_tokens, out_nacc, flags


def process_logits(logits, params, k_max, out_logits=None, out_probs=None, flags=None, ws=None):
    """Materialised processed logits and final probabilities, both float32 [B, V]."""
    B, V = logits.shape
    dt = _dtype_code(logits)
    dev = logits.device
    ws = _ws(ws, OP_PROCESS, B, V, 0, k_max, dt, dev)
    if out_logits is None:
        out_logits = torch.empty(B, V, dtype=torch.float32, device=dev)
    if out_probs is None:
        out_probs = torch.empty(B, V, dtype=torch.float32, device=dev)
    if flags is None:
        flags = torch.empty(B, dtype=torch.int32, device=dev)
    p = params.struct()
    _check(lib().ss_process_logits(_ptr(logits), dt, logits.stride(0), C.byref(p), k_max, _ptr(out_logits),
                                   _ptr(out_probs), _ptr(flags), _ptr(ws), ws.numel(), _stream()))
    return out_logits, out_probs, flags


def logits_tensor(d, device="cuda"):
    """Device logits tensor from a gen.workloads dict (bf16 from raw bits)."""
    x = np.ascontiguousarray(d["x"])
    if d["dtype"] == "bf16":
        return torch.from_numpy(x.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(x.astype(np.float32)).to(device)
