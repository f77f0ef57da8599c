"""The cooperative few-column launch (opts.cooperative): with at most 8 active
columns and d <= 4096, the iterations between two checks run as one launch
that keeps H's split planes in registers. It forms the same products, in the
same summation order, as one few-column launch per iteration, so both must
give the same bits: W, every per-column statistic, and the iteration counts.
"""
import numpy as np
import pytest

from gpu_util import gpu_solve, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib
    return lib


def _spd(rng, d):
    """A damped Gram matrix with a spread spectrum (condition number ~1e3)."""
    A = rng.standard_normal((d + 16, d)).astype(np.float64)
    A *= np.exp(rng.normal(0.0, 1.0, d))[None, :]
    H = A.T @ A
    H += 0.01 * np.trace(H) / d * np.eye(d)
    return H.astype(np.float32)


def _mask_2to4(rng, n, d):
    keep = np.zeros((n, d), np.uint8)
    for j in range(n):
        for g in range(d // 4):
            keep[j, 4 * g + rng.choice(4, 2, replace=False)] = 1
    return keep


def _both(L, H, lm, W0, M, **kw):
    out = {}
    for coop in (0, 1):
        o = L.SolverOpts.default(cooperative=coop, **kw)
        W, st, info = gpu_solve(L, H, lm, W0, M, o)
        out[coop] = (W.cpu().numpy(), st, info)
    return out


def _assert_same_bits(out):
    W0_, st0, _ = out[0]
    W1_, st1, _ = out[1]
    assert np.array_equal(W0_.view(np.uint32), W1_.view(np.uint32))
    for k in st0:
        assert np.array_equal(st0[k], st1[k]), k


def _lambda_max(L, H):
    import torch
    lm = torch.empty(1, dtype=torch.float32, device="cuda:0")
    V0 = np.random.default_rng(7).standard_normal((16, H.shape[0])).astype(np.float32)
    L.optima_spectral_norm(to_dev(H), to_dev(V0), lm)
    return lm


@pytest.mark.parametrize("d,n", [(128, 1), (128, 8), (1024, 5), (4096, 5)])
def test_sparse_cooperative_matches_per_iteration_launches(L, d, n):
    rng = np.random.default_rng(1000 + d + n)
    H = _spd(rng, d)
    W0 = (0.015 * rng.standard_normal((n, d))).astype(np.float32)
    M = _mask_2to4(rng, n, d)
    Hd, lm = to_dev(H), _lambda_max(L, H)
    out = _both(L, Hd, lm, W0, M, max_iters=200, fixed_iters=1)
    _assert_same_bits(out)
    i0, i1 = out[0][2], out[1][2]
    assert i0["sparse_products"] == 1 and i1["sparse_products"] == 1
    assert i0["persistent_launches"] == 0
    assert i1["persistent_launches"] == 4            # blocks of 64, 64, 64 and 8 iterations
    assert i0["few_launches"] == i1["few_launches"] == 200


@pytest.mark.parametrize("d,n", [(256, 3), (4096, 7)])
def test_dense_cooperative_matches_per_iteration_launches(L, d, n):
    # 50 % unstructured masks: dense bf16x3 products
    rng = np.random.default_rng(2000 + d + n)
    H = _spd(rng, d)
    W0 = (0.02 * rng.standard_normal((n, d))).astype(np.float32)
    M = (rng.random((n, d)) < 0.5).astype(np.uint8)
    Hd, lm = to_dev(H), _lambda_max(L, H)
    out = _both(L, Hd, lm, W0, M, max_iters=130, fixed_iters=1)
    _assert_same_bits(out)
    assert out[0][2]["sparse_products"] == 0
    assert out[1][2]["persistent_launches"] == 3      # 64, 64 and 2 iterations
    assert out[0][2]["few_launches"] == out[1][2]["few_launches"] == 130


def test_paper_mode_tail_is_cooperative_and_identical(L):
    # A paper-mode solve whose last columns run past the first check: the tail
    # runs cooperatively and every column stops where it did before.
    rng = np.random.default_rng(3)
    d, n = 512, 64
    H = _spd(rng, d)
    W0 = (0.015 * rng.standard_normal((n, d))).astype(np.float32)
    M = _mask_2to4(rng, n, d)
    Hd, lm = to_dev(H), _lambda_max(L, H)
    out = _both(L, Hd, lm, W0, M, eps_rel=1e-4, eps_abs=0.0)
    _assert_same_bits(out)
    assert out[0][2]["iterations"] == out[1][2]["iterations"]
    if out[1][2]["few_launches"]:
        assert out[1][2]["persistent_launches"] >= 1


def test_no_cooperative_launch_beyond_4096(L):
    rng = np.random.default_rng(4)
    d, n = 4096 + 128, 2
    H = _spd(rng, d)
    W0 = (0.015 * rng.standard_normal((n, d))).astype(np.float32)
    M = _mask_2to4(rng, n, d)
    Hd, lm = to_dev(H), _lambda_max(L, H)
    _, _, info = gpu_solve(L, Hd, lm, W0, M, L.SolverOpts.default(max_iters=64, fixed_iters=1))
    assert info["persistent_launches"] == 0 and info["few_launches"] == 64


def test_cooperative_option_validation(L):
    rng = np.random.default_rng(5)
    H = _spd(rng, 128)
    W0 = (0.015 * rng.standard_normal((2, 128))).astype(np.float32)
    M = _mask_2to4(rng, 2, 128)
    with pytest.raises(L.OptimaError) as e:
        gpu_solve(L, to_dev(H), _lambda_max(L, H), W0, M, L.SolverOpts.default(cooperative=2))
    assert e.value.status == -1
