"""ss_sample_noalloc (no workspace argument, library-owned per-GPU scratch)
against ss_sample with a caller workspace: identical outputs on two calls in
a row, the second with a smaller batch and vocabulary, and the size limit."""
import numpy as np
import pytest
import torch

from gen import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ssb():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_20475_amd import binding
    binding.lib()
    assert hasattr(binding.lib(), "ss_sample_noalloc")
    return binding


def _both(ssb, inp, k_out=0):
    x = ssb.logits_tensor(inp)
    prm = ssb.Params.from_arrays(inp)
    B = inp["B"]
    ref = ssb.sample(x, prm, inp["k_max"], k_out=k_out)
    outs = [torch.full((B,), -7, dtype=torch.int32, device="cuda"), torch.full((B,), 9.0, device="cuda"),
            torch.full((B,), -7, dtype=torch.int32, device="cuda")]
    extra = {}
    if k_out:
        extra = dict(k_out=k_out, out_idx=torch.full((B, k_out), -7, dtype=torch.int32, device="cuda"),
                     out_prob=torch.full((B, k_out), 9.0, device="cuda"))
    ssb.sample_noalloc(x, prm, inp["k_max"], *outs, **extra)
    torch.cuda.synchronize()
    got = outs + ([extra["out_idx"], extra["out_prob"]] if k_out else [])
    for r, g in zip(ref, got):
        assert np.array_equal(r.cpu().numpy(), g.cpu().numpy())


def test_noalloc_matches_workspace_entry_point(ssb):
    print("[noalloc] cfg1 B=64 V=131072 bf16, then cfg0 B=4 V=32768 f32", flush=True)
    _both(ssb, W.config1())
    _both(ssb, W.config0(), k_out=16)
    # history long enough for the row tables in the scratch array
    rng = np.random.default_rng(8)
    B, V = 6, 1 << 16
    x = W.bf16_bits_from_f32(rng.normal(0, 2, (B, V)).astype(np.float32))
    hist = [rng.integers(0, V, 6000).astype(np.int32) for _ in range(B)]
    off = np.concatenate([[0], np.cumsum([len(h) for h in hist])]).astype(np.int32)
    pen = W.MODE_REP | W.MODE_FREQ | W.MODE_PRES
    inp = W.custom_rows(x, W.BF16, k_max=256, mode=np.full(B, W.MODE_TEMP | W.MODE_TOPK | pen),
                        top_k=np.full(B, 100), rep=np.full(B, 1.2), freq=np.full(B, 0.1), pres=np.full(B, 0.2),
                        hist_offsets=off, hist_ids=np.concatenate(hist), position=np.arange(B))
    print("[noalloc] long histories B=6 V=65536", flush=True)
    _both(ssb, inp)


def test_noalloc_rejects_sizes_beyond_its_array(ssb):
    inp = W.config1(B=8)
    n = ssb.workspace_bytes(ssb.OP_SAMPLE, 4096, 1 << 17, 0, 1024, ssb.BF16)
    assert n > (48 << 20)
    x = torch.zeros(4096, 1 << 17, dtype=torch.bfloat16, device="cuda")
    prm = ssb.Params(4096, 1 << 17, mode=torch.zeros(4096, dtype=torch.int32, device="cuda"))
    o = [torch.empty(4096, dtype=torch.int32, device="cuda"), torch.empty(4096, device="cuda"),
         torch.empty(4096, dtype=torch.int32, device="cuda")]
    with pytest.raises(ssb.SSError, match="workspace"):
        ssb.sample_noalloc(x, prm, 1024, *o)
