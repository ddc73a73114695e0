"""Host-side checks of the seeded input generators (CPU only): the sparse
draft lists, the draft trees and the Gumbel noise have the layout the entry
points and the oracle expect."""
import numpy as np

from gen import workloads as W


def test_sparse_drafts_are_padded_distributions_holding_their_draft():
    rng = np.random.default_rng(3)
    noisy = rng.normal(0, 2, (3, 2, 500))
    idx, q, d = W.sparse_drafts(noisy, 16, 0.9, np.random.default_rng(4))
    assert idx.shape == q.shape == (3, 2, 16) and idx.dtype == np.int32 and q.dtype == np.float32
    for b in range(3):
        for l in range(2):
            n = int((idx[b, l] >= 0).sum())
            assert n >= 1 and np.all(idx[b, l, :n] >= 0) and np.all(idx[b, l, n:] == -1)
            assert np.all(q[b, l, n:] == 0) and abs(float(q[b, l, :n].astype(np.float64).sum()) - 1) < 1e-6
            assert len(set(idx[b, l, :n].tolist())) == n          # no repeated ids
            assert np.all(np.diff(q[b, l, :n]) <= 0)              # leading ids first
            assert d[b, l] in idx[b, l, :n]
            # the listed ids are the n largest draft logits
            top = np.argsort(-noisy[b, l], kind="stable")[:n]
            assert set(top.tolist()) == set(idx[b, l, :n].tolist())


def test_tree_from_path_places_every_path_row():
    rng = np.random.default_rng(5)
    x = rng.normal(0, 1, (4, 3, 64)).astype(np.float32)
    inp = dict(x=x, dtype=W.F32, B=4, V=64, L=2, name="t")
    t = W.tree_from_path(inp, 7, 11)
    assert t["x"].shape == (4, 7, 64) and t["row_map"].shape == (4, 3)
    for b in range(4):
        assert len(set(t["row_map"][b].tolist())) == 3
        assert np.array_equal(t["x"][b, t["row_map"][b]], x[b])
    xb = W.bf16_bits_from_f32(x)
    tb = W.tree_from_path(dict(inp, x=xb, dtype=W.BF16), 5, 2)
    assert tb["x"].dtype == np.uint16
    for b in range(4):
        assert np.array_equal(tb["x"][b, tb["row_map"][b]], xb[b])


def test_gumbel_noise_is_log_of_unit_exponentials():
    g = W.gumbel_noise(4, 50000, 9)
    assert g.shape == (4, 50000) and g.dtype == np.float32 and np.all(np.isfinite(g))
    z = np.exp(g.astype(np.float64))
    # Exp(1): mean 1, P(z > 1) = e^-1
    assert abs(z.mean() - 1) < 0.01 and abs((z > 1).mean() - np.exp(-1)) < 0.005
    assert np.array_equal(g, W.gumbel_noise(4, 50000, 9))  # seeded
