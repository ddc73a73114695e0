"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function declared in include/ss.h, size
workspaces, and reject invalid arguments before launching anything.
"""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_20475_amd import build as b
    if b.is_stale():
        b.build()
    from paper_2607_20475_amd import binding
    binding._lib = None
    return binding.lib()


def _declared():
    src = open(os.path.join(ROOT, "include", "ss.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ss_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) >= {"ss_topk", "ss_sample", "ss_verify", "ss_process_logits", "ss_workspace_bytes",
                          "ss_workspace_init", "ss_status_string"}
    for n in names:
        assert hasattr(lib, n), n


def test_workspace_sizes(lib):
    from paper_2607_20475_amd import binding as b
    n1 = b.workspace_bytes(b.OP_SAMPLE, 64, 1 << 17, 0, 1024, b.BF16)
    n2 = b.workspace_bytes(b.OP_SAMPLE, 128, 1 << 17, 0, 1024, b.BF16)
    assert 0 < n1 < n2
    assert b.workspace_bytes(b.OP_VERIFY, 64, 1 << 17, 4, 1024, b.BF16) > n1
    # invalid sizes
    assert b.workspace_bytes(b.OP_SAMPLE, 0, 100, 0, 10, b.F32) == 0
    assert b.workspace_bytes(b.OP_SAMPLE, 4, (1 << 20) + 1, 0, 10, b.F32) == 0
    assert b.workspace_bytes(b.OP_SAMPLE, 4, 100, 0, 4097, b.F32) == 0
    assert b.workspace_bytes(b.OP_VERIFY, 4, 100, 0, 10, b.F32) == 0
    assert b.workspace_bytes(b.OP_VERIFY, 4, 100, 17, 10, b.F32) == 0
    assert b.workspace_bytes(b.OP_TOPK, 4, 100, 0, 10, 7) == 0
    # workspace for the largest top-k stress case stays modest (no vocab-scale buffer)
    assert b.workspace_bytes(b.OP_TOPK, 256, 1 << 18, 0, 4096, b.F32) < 256 * (1 << 18) * 4 // 2


def test_logprobs_arguments_are_checked_before_launch(lib):
    from paper_2607_20475_amd import binding as b
    fake = C.c_void_p(0x10000)  # never dereferenced: validation fails first
    p = b._Params(B=4, V=100)
    mode = (C.c_uint32 * 4)()
    p.mode = C.cast(mode, C.c_void_p)
    bad = -1  # SS_ERR_INVALID_ARG
    assert lib.ss_logprobs(None, 0, 100, C.byref(p), 10, fake, fake, None, fake, 1 << 20, None) == bad
    assert lib.ss_logprobs(fake, 0, 100, C.byref(p), 0, fake, fake, None, fake, 1 << 20, None) == bad
    assert lib.ss_logprobs(fake, 0, 100, C.byref(p), 4097, fake, fake, None, fake, 1 << 20, None) == bad
    assert lib.ss_logprobs(fake, 0, 99, C.byref(p), 10, fake, fake, None, fake, 1 << 20, None) == bad
    assert lib.ss_logprobs(fake, 0, 100, C.byref(p), 10, None, fake, None, fake, 1 << 20, None) == bad
    n = b.workspace_bytes(b.OP_LOGPROBS, 4, 100, 0, 10, b.F32)
    assert n >= b.workspace_bytes(b.OP_TOPK, 4, 100, 0, 10, b.F32)
    assert lib.ss_logprobs(fake, 0, 100, C.byref(p), 10, fake, fake, None, fake, n - 256, None) == -3  # SS_ERR_WORKSPACE


def test_verify_sparse_arguments_are_checked_before_launch(lib):
    from paper_2607_20475_amd import binding as b
    fake = C.c_void_p(0x10000)  # never dereferenced: validation fails first
    p = b._Params(B=4, V=100)
    mode = (C.c_uint32 * 4)()
    p.mode = C.cast(mode, C.c_void_p)
    p.seed = fake
    p.position = fake
    bad = -1  # SS_ERR_INVALID_ARG

    def call(x=fake, idx=fake, q=fake, kq=8, L=2, ws_bytes=1 << 24):
        return lib.ss_verify_sparse(x, 0, 100, idx, q, kq, fake, L, C.byref(p), 16, fake, fake, None, fake,
                                    ws_bytes, None)
    assert call(kq=0) == bad
    assert call(kq=4097) == bad
    assert call(idx=None) == bad
    assert call(q=None) == bad
    assert call(x=None) == bad
    assert call(L=0) == bad
    n = b.workspace_bytes(b.OP_VERIFY, 4, 100, 2, 16, b.F32)
    assert call(ws_bytes=n - 256) == -3  # SS_ERR_WORKSPACE: every argument passed its check


def test_sample_gumbel_arguments_are_checked_before_launch(lib):
    from paper_2607_20475_amd import binding as b
    fake = C.c_void_p(0x10000)  # never dereferenced: validation fails first
    p = b._Params(B=4, V=100)
    mode = (C.c_uint32 * 4)()
    p.mode = C.cast(mode, C.c_void_p)

    def call(noise=fake, ld_noise=100, ws_bytes=1 << 24, k_max=10):
        return lib.ss_sample_gumbel(fake, 0, 100, C.byref(p), k_max, noise, ld_noise, fake, None, None, None, 0,
                                    None, fake, ws_bytes, None)
    assert call(noise=None) == -1
    assert call(ld_noise=99) == -1
    assert call(k_max=0) == -1
    n = b.workspace_bytes(b.OP_SAMPLE, 4, 100, 0, 10, b.F32)
    assert call(ws_bytes=n - 256) == -3  # SS_ERR_WORKSPACE: every argument passed its check


def test_verify_tree_arguments_are_checked_before_launch(lib):
    from paper_2607_20475_amd import binding as b
    fake = C.c_void_p(0x10000)  # never dereferenced: validation fails first
    p = b._Params(B=4, V=100)
    mode = (C.c_uint32 * 4)()
    p.mode = C.cast(mode, C.c_void_p)
    p.seed = fake
    p.position = fake

    def call(Lt=7, rmap=fake, kq=8, ws_bytes=1 << 24):
        return lib.ss_verify_tree(fake, 0, 100, Lt, rmap, fake, fake, kq, fake, 2, C.byref(p), 16, fake, fake,
                                  None, fake, ws_bytes, None)
    assert call(Lt=0) == -1
    assert call(rmap=None) == -1
    assert call(kq=0) == -1
    n = b.workspace_bytes(b.OP_VERIFY, 4, 100, 2, 16, b.F32)
    assert call(ws_bytes=n - 256) == -3


def test_invalid_arguments_are_rejected_before_launch(lib):
    from paper_2607_20475_amd import binding as b
    fake = C.c_void_p(0x10000)  # never dereferenced: validation fails first
    p = b._Params(B=4, V=100)
    st = lib.ss_sample(None, 0, 100, C.byref(p), 10, fake, None, None, None, 0, None, fake, 1 << 20, None)
    assert st == -1
    p.mode = fake
    st = lib.ss_sample(fake, 0, 99, C.byref(p), 10, fake, None, None, None, 0, None, fake, 1 << 20, None)
    assert st == -1  # ld < V
    st = lib.ss_sample(fake, 0, 100, C.byref(p), 10, fake, None, None, None, 0, None, fake, 16, None)
    assert st == -3  # workspace too small
    st = lib.ss_sample(fake, 0, 100, C.byref(p), 0, fake, None, None, None, 0, None, fake, 1 << 20, None)
    assert st == -1  # k_max out of range
    st = lib.ss_sample(fake, 0, 100, C.byref(p), 10, fake, None, None, None, 5, None, fake, 1 << 20, None)
    assert st == -1  # k_out without buffers
    st = lib.ss_topk(fake, 3, 4, 100, 100, None, 10, fake, fake, None, fake, 1 << 20, None)
    assert st == -1  # dtype
    st = lib.ss_verify(fake, 0, 100, fake, 100, fake, 0, C.byref(p), 10, fake, fake, None, fake, 1 << 20, None)
    assert st == -1  # L = 0
    p.bitmask = fake
    p.bitmask_ld = 3  # < ceil(100 / 32)
    st = lib.ss_process_logits(fake, 0, 100, C.byref(p), 10, fake, fake, None, fake, 1 << 20, None)
    assert st == -1
    assert lib.ss_status_string(-3) == b"workspace too small or misaligned"
    assert lib.ss_workspace_init(C.c_void_p(0x10001), 64, None) == -1  # misaligned


def test_product_path_does_not_touch_the_oracle():
    pkg = os.path.join(ROOT, "paper_2607_20475_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                txt = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in txt, f
                assert "ssref" not in txt, f
