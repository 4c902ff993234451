"""Seeded input generator: determinism, column access and distribution shape (CPU only)."""
import numpy as np
import torch

import synth


def test_columns_match_full_matrix_and_are_deterministic():
    s = synth.small_spec(64, 256, 1000)
    X = synth.gen_matrix(s.x)
    cols = [0, 7, 100, 255]
    assert torch.equal(synth.gen_columns(s.x, cols), X[:, cols])
    assert torch.equal(synth.gen_matrix(s.x, rows=(300, 700)), X[300:700])
    assert torch.equal(synth.gen_matrix(s.x, chunk_elems=1000), X)


def test_heavy_tail_and_scales():
    s = synth.workload(2, n_tokens=4096)
    X = synth.gen_matrix(s.x).float()
    sel = s.x.dist_idx.astype(bool)
    assert sel.sum() == 41  # 1% of 4096 channels are Student-t(3)
    kurt_t = (X[:, sel] ** 4).mean() / (X[:, sel] ** 2).mean() ** 2
    kurt_n = (X[:, ~sel] ** 4).mean() / (X[:, ~sel] ** 2).mean() ** 2
    assert kurt_t > 6.0 and abs(kurt_n - 3.0) < 0.1
    G = synth.gen_matrix(s.g).float()
    ratio = G.std(0) / torch.from_numpy(s.g.col_scale)
    assert torch.allclose(ratio, torch.ones_like(ratio), rtol=0.1)


def test_rotation_params_shapes():
    r = synth.rotation_params(28 * 512, 2, "t")
    assert r.sign.dtype == np.int8 and set(np.unique(r.sign)) == {-1, 1}
    assert r.q28.dtype == np.float32 and r.q28.shape == (28, 28)
    assert synth.rotation_params(4096, 1, "t").q28 is None
