"""GPU parity of the Wanda mask selection (optima_wanda_mask) with the oracle.

Masks are integer results: the device must reproduce the oracle's mask bit for
bit on the same inputs, including every tie (lower index first), NaN scores
(ranked last) and -0 (equal to +0).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, to_dev, to_dev_x, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def gpu_mask(L, W0, col_sq, pattern, sparsity=0.5, stride=1):
    Wd = W0 if isinstance(W0, torch.Tensor) else to_dev(W0)
    cd = col_sq if isinstance(col_sq, torch.Tensor) else torch.from_numpy(col_sq).to(dev())
    m = torch.full(tuple(Wd.shape), 7, dtype=torch.uint8, device=dev())
    L.optima_wanda_mask(Wd, cd, m, pattern, sparsity, col_sq_stride=stride)
    return m.cpu().numpy()


def tied_inputs(n, d, seed):
    rng = np.random.default_rng(seed)
    W = (rng.integers(-4, 5, (n, d)) * 0.125).astype(np.float32)
    c = rng.choice([0.5, 2.0, 8.0], d)
    return W, c


@pytest.mark.parametrize("d", [3, 77, 1000, 4096])
@pytest.mark.parametrize("sparsity", [0.0, 0.3, 0.5, 0.6, 1.0])
def test_unstructured_bit_exact_with_ties(L, d, sparsity):
    W, c = tied_inputs(9, d, d)
    for cs in (c.astype(np.float64), c.astype(np.float32)):
        g = gpu_mask(L, W, cs, L.MASK_UNSTRUCTURED, sparsity)
        ref = oracle.wanda_mask(W, cs, "unstructured", sparsity)
        np.testing.assert_array_equal(g, ref)


@pytest.mark.parametrize("d", [4, 12, 1000, 4096])
def test_2to4_bit_exact_with_ties(L, d):
    W, c = tied_inputs(7, d, 100 + d)
    g = gpu_mask(L, W, c, L.MASK_2TO4)
    np.testing.assert_array_equal(g, oracle.wanda_mask(W, c, "2:4"))


def test_special_values(L):
    W = np.array([[np.nan, 0.0, -0.0, 2.0, -3.0, np.nan, 1.0, 0.5,
                   np.inf, -np.inf, 1.0, np.nan, 0.0, -0.0, 0.0, 0.0]], dtype=np.float32)
    c = np.ones(16)
    c[14] = -0.0
    for pat, name in ((L.MASK_2TO4, "2:4"), (L.MASK_UNSTRUCTURED, "unstructured")):
        g = gpu_mask(L, W, c, pat, 0.5)
        np.testing.assert_array_equal(g, oracle.wanda_mask(W, c, name, 0.5))


def test_layers_match_the_host_generator(L):
    # The benchmark layer (q_proj, 2:4) and the GPT-2 layer (50 % unstructured)
    # with their fp64 column norms: the device reproduces the generator's mask.
    for cfg in (workloads.Q_PROJ.with_tokens(8192), workloads.GPT2_FC.with_tokens(8192)):
        log(f"mask {cfg.name}")
        X = workloads.x_all(cfg)
        W0 = workloads.w0(cfg)
        cs = workloads.col_sq_norms(cfg, X)
        ref = workloads.layer_mask(cfg, W0, cs)
        pat = L.MASK_2TO4 if cfg.mask_kind == "2:4" else L.MASK_UNSTRUCTURED
        g = gpu_mask(L, W0, cs, pat, cfg.sparsity)
        np.testing.assert_array_equal(g, ref)
        assert np.array_equal(g, oracle.wanda_mask(W0, cs, cfg.mask_kind, cfg.sparsity))


def test_from_the_device_hessian_diagonal(L):
    # col_sq read in place from the undamped device Hessian (stride d + 1).
    cfg = workloads.GPT2_FC.with_tokens(4096).with_cols(256)
    X = workloads.x_all(cfg)
    W0 = workloads.w0(cfg)
    H = torch.empty((cfg.d, cfg.d), dtype=torch.float32, device=dev())
    L.optima_hessian_accumulate(to_dev_x(X), H)
    diag = np.diag(H.cpu().numpy()).astype(np.float64)
    for pat, name in ((L.MASK_UNSTRUCTURED, "unstructured"), (L.MASK_2TO4, "2:4")):
        g = gpu_mask(L, W0, H, pat, 0.5, stride=cfg.d + 1)
        np.testing.assert_array_equal(g, oracle.wanda_mask(W0, diag, name, 0.5))


def test_mask_error_paths(L):
    W = to_dev(np.ones((2, 6), dtype=np.float32))
    c = torch.ones(6, dtype=torch.float64, device=dev())
    m = torch.empty((2, 6), dtype=torch.uint8, device=dev())
    for kw in ({"pattern": L.MASK_2TO4}, {"pattern": 5}, {"sparsity": 1.5},
               {"sparsity": -0.1}):
        with pytest.raises(L.OptimaError) as e:
            L.optima_wanda_mask(W, c, m, **{"pattern": L.MASK_UNSTRUCTURED, **kw})
        assert e.value.status == -1
    with pytest.raises(ValueError):
        L.optima_wanda_mask(W, c.to(torch.float16), m)
    # n_cols = 0 is a no-op.
    L.optima_wanda_mask(W[:0], c, m[:0])
