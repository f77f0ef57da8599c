"""Checks of the seeded input generators and the host mask selection."""
import numpy as np
import pytest
import torch

import workloads as w


def test_bf16_rounding_matches_torch_rne():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-6, 6, 20000),
        # exact ties between two bf16 neighbours, both parities of the kept bit
        (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        -(np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0], np.float32)])
    ours = w.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(w.bf16_bits_to_f32(ours),
                                  torch.from_numpy(ours.view(np.int16).copy()).view(torch.bfloat16).float().numpy())


def test_chunks_are_reproducible_and_thread_independent():
    cfg = w.Q_PROJ.with_tokens(3 * 2048 + 100)
    a = w.x_all(cfg, threads=1)
    b = w.x_all(cfg, threads=4)
    np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(a[2048:4096], w.x_chunk(cfg, 1))
    assert a.shape == (3 * 2048 + 100, 4096) and a.dtype == np.uint16
    assert w.x_chunk(cfg, 3).shape == (100, 4096)


def test_recipes_have_the_stated_structure():
    tiny = w.x_chunk(w.TINY, 0).astype(np.float64)
    c = np.cov(tiny.T)
    assert abs(c[10, 10] - 1.0) < 0.15 and abs(c[10, 11] - 0.5) < 0.12 and abs(c[10, 12] - 0.25) < 0.12
    q = w.x_to_f64(w.x_chunk(w.Q_PROJ, 0))
    out = w.outlier_channels(w.Q_PROJ)
    rest = np.setdiff1d(np.arange(4096), out)
    ratio = np.median(np.abs(q[:, out])) / np.median(np.abs(q[:, rest]))
    assert 40 < ratio < 60
    assert w.round_to_bf16(w.w0(w.Q_PROJ)[:4]).tobytes() == w.w0(w.Q_PROJ)[:4].tobytes()
    down = w.x_to_f64(w.x_chunk(w.DOWN_PROJ.with_tokens(256), 0))
    assert 0.3 < down.var() < 0.42


def test_unstructured_mask_counts_and_ties():
    rng = np.random.default_rng(1)
    W0 = rng.standard_normal((50, 37)).astype(np.float32)
    cs = rng.uniform(0.5, 2, 37)
    for s in (0.0, 0.5, 0.6, 1.0):
        m = w.wanda_unstructured(W0, cs, s)
        assert np.all(m.sum(1) == 37 - int(np.floor(s * 37)))
    # kept entries dominate pruned ones in score
    m = w.wanda_unstructured(W0, cs, 0.6)
    sc = np.abs(W0.astype(np.float64)) * np.sqrt(cs)
    for j in range(50):
        assert sc[j][m[j] == 1].min() >= sc[j][m[j] == 0].max()
    # ties: lower index kept first
    m = w.wanda_unstructured(np.ones((1, 6), np.float32), np.ones(6), 0.5)
    np.testing.assert_array_equal(m[0], [1, 1, 1, 0, 0, 0])


def test_2to4_mask_validity_and_ties():
    rng = np.random.default_rng(2)
    W0 = rng.standard_normal((30, 64)).astype(np.float32)
    cs = rng.uniform(0.5, 2, 64)
    m = w.wanda_2to4(W0, cs)
    assert np.all(m.reshape(30, 16, 4).sum(2) == 2)
    m = w.wanda_2to4(np.ones((1, 8), np.float32), np.ones(8))
    np.testing.assert_array_equal(m[0], [1, 1, 0, 0, 1, 1, 0, 0])
    with pytest.raises(ValueError):
        w.wanda_2to4(np.ones((1, 6), np.float32), np.ones(6))


def test_config_shapes():
    assert (w.TINY.d, w.TINY.n_cols, w.TINY.n_tok) == (128, 64, 512)
    assert (w.GPT2_FC.d, w.GPT2_FC.n_cols, w.GPT2_FC.n_tok) == (768, 3072, 262144)
    assert (w.Q_PROJ.d, w.Q_PROJ.n_cols, w.Q_PROJ.mask_kind) == (4096, 4096, "2:4")
    assert (w.DOWN_PROJ.d, w.DOWN_PROJ.n_cols, w.DOWN_PROJ.sparsity) == (14336, 4096, 0.6)
