"""GPU parity of the 2:4-sparse iteration products (opts.sparse).

A mask that keeps at most 2 of every group of 4 consecutive columns (the 2:4
pattern of Section 4, or one pruned further) lets the bf16x3 rAPDHG products
store x compressed and run on the sparse MFMA. The same products are formed
(the skipped ones are exact zeros), summed in another order, so the bar is the
bf16x3 one: W within 1e-4 relative Frobenius of the oracle, objectives within
1e-5, pruned entries +0.0. Each case also checks which path ran.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads
from gpu_util import dev, to_dev, gpu_solve, rel_fro, f32_exact, log
from test_gpu_solver import _assert_w_and_f, _assert_zero_pattern, _oracle_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _tiny_2to4():
    cfg = workloads.TINY
    H, W0, _, lam = _oracle_layer(cfg)
    M = oracle.wanda_mask(W0, workloads.col_sq_norms(cfg), "2:4")
    return H, W0, M, lam


def _opts(L, **kw):
    return L.SolverOpts.default(**kw)


def test_sparse_fixed_1000_matches_oracle_and_dense(L):
    H, W0, M, lam = _tiny_2to4()
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    o = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions(max_iters=1000, fixed_iters=True))
    ref = oracle.closed_form(H, W0, M)
    Ws, st, info = gpu_solve(L, Hd, lmd, W0, M, _opts(L, max_iters=1000, fixed_iters=1))
    assert info["sparse_products"] == 1
    Wd, _, info_d = gpu_solve(L, Hd, lmd, W0, M, _opts(L, max_iters=1000, fixed_iters=1,
                                                        sparse=0))
    assert info_d["sparse_products"] == 0
    Ws, Wd = Ws.cpu().numpy(), Wd.cpu().numpy()
    _assert_w_and_f(H, W0, M, Ws, o.W, label="sparse vs oracle rapdhg")
    _assert_w_and_f(H, W0, M, Ws, ref, label="sparse vs closed form")
    assert rel_fro(Ws, Wd) <= 1e-4
    assert np.all(st["iters"] == 1000)
    assert np.all(st["restarts"] > 0)


@pytest.mark.parametrize("T", [1, 2, 7, 63])
def test_sparse_trajectory_before_first_check(L, T):
    H, W0, M, lam = _tiny_2to4()
    o = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions(max_iters=T, fixed_iters=True))
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                             _opts(L, max_iters=T, fixed_iters=1))
    assert info["sparse_products"] == 1
    Wg = Wg.cpu().numpy()
    _assert_zero_pattern(Wg, M)
    per_col = np.linalg.norm(Wg - o.W, axis=1) / np.linalg.norm(o.W, axis=1)
    log(f"  T={T} worst column rel={per_col.max():.3e}")
    assert per_col.max() <= 1e-4


def test_sparse_paper_mode_tiny(L):
    H, W0, M, lam = _tiny_2to4()
    o = oracle.rapdhg(H, W0, M, lam, oracle.SolverOptions())
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M, _opts(L))
    assert info["sparse_products"] == 1
    Wg = Wg.cpu().numpy()
    same = st["iters"] == o.iters
    log(f"  same stopping check on {same.mean():.2%} of columns")
    assert same.mean() >= 0.95 and st["converged"].all()
    _assert_w_and_f(H, W0[same], M[same], Wg[same], o.W[same], label="sparse paper mode")


def _thinned_2to4(rng, n, d, extra=0.3):
    """2:4 rows with a further share of the kept entries pruned, some groups
    and some whole rows pruned: every group keeps 0, 1 or 2."""
    M = np.zeros((n, d), dtype=np.uint8)
    for j in range(n):
        for g in range(0, d - d % 4, 4):
            M[j, g + rng.choice(4, 2, replace=False)] = 1
        if d % 4:
            tail = np.arange(d - d % 4, d)
            M[j, rng.choice(tail, min(2, tail.size), replace=False)] = 1
    M[rng.random((n, d)) < extra] = 0
    M[:, 8:12] = 0
    M[n // 2] = 0
    return M


@pytest.mark.parametrize("d,n", [(100, 3), (200, 130), (300, 257), (512, 200)])
def test_sparse_ragged_and_thinned_masks(L, d, n):
    # d not a multiple of 64 or 128 (stored groups in the padding), columns
    # over several row tiles with a ragged tail, groups keeping 0, 1 or 2.
    rng = np.random.default_rng(11 + d)
    X = rng.standard_normal((4 * d, d)).astype(np.float32)
    X[:, :3] *= 10
    H, _ = oracle.damp(oracle.hessian([X]), 0.01)
    H = f32_exact(H)
    W0 = (rng.standard_normal((n, d)) * 0.02).astype(np.float32)
    M = _thinned_2to4(rng, n, d)
    lam = float(np.float32(np.linalg.eigvalsh(H)[-1]))
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                             _opts(L, max_iters=3000, fixed_iters=1))
    assert info["sparse_products"] == 1
    log(f"  d={d} n={n}: kept {M.mean():.3f}")
    _assert_w_and_f(H, W0, M, Wg.cpu().numpy(), oracle.closed_form(H, W0, M),
                    label=f"sparse d={d} n={n}")


def test_mask_with_three_kept_falls_back_to_dense(L):
    H, W0, M, lam = _tiny_2to4()
    M = M.copy()
    M[5, 40:44] = 1  # one group of one row keeps 4
    Wg, st, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                             _opts(L, max_iters=1000, fixed_iters=1))
    assert info["sparse_products"] == 0
    _assert_w_and_f(H, W0, M, Wg.cpu().numpy(), oracle.closed_form(H, W0, M), label="fallback")


def test_sparse_columns_are_independent(L):
    H, W0, M, lam = _tiny_2to4()
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    opts = _opts(L, max_iters=2000, fixed_iters=1)
    full, _, _ = gpu_solve(L, Hd, lmd, W0, M, opts)
    again, _, _ = gpu_solve(L, Hd, lmd, W0, M, opts)
    assert torch.equal(full, again)
    full = full.cpu().numpy()
    for sl in (slice(5, 6), slice(10, 30), slice(0, 64, 7)):
        part, _, info = gpu_solve(L, Hd, lmd, W0[sl], M[sl], opts)
        assert info["sparse_products"] == 1
        assert rel_fro(part.cpu().numpy(), full[sl]) <= 1e-5


def test_sparse_option_validation(L):
    H, W0, M, lam = _tiny_2to4()
    W0d, Md = to_dev(W0), to_dev(M, torch.uint8)
    out = torch.empty_like(W0d)
    with pytest.raises(L.OptimaError) as e:
        L.optima_qp_solve_batched(to_dev(H), to_dev(np.array([lam])), W0d, Md, out,
                                  opts=_opts(L, sparse=2))
    assert e.value.status == -1
    # fp32 products and CG never take the sparse path.
    for kw in (dict(precision=L.PREC_FP32), dict(method=L.METHOD_CG)):
        _, _, info = gpu_solve(L, to_dev(H), to_dev(np.array([lam])), W0, M,
                               _opts(L, max_iters=64, fixed_iters=1, **kw))
        assert info["sparse_products"] == 0


@pytest.mark.parametrize("n", [1, 5, 8, 9])
def test_sparse_few_columns_match_closed_form(L, n):
    # 1 to 8 active columns of a 2:4 solve run the few-column sparse kernel
    # (H streamed once per iteration, x compressed); 9 take the tiles. Both
    # reach the closed form, and the columns agree with the same columns of a
    # full batch.
    H, W0, M, lam = _tiny_2to4()
    Hd, lmd = to_dev(H), to_dev(np.array([lam]))
    opts = _opts(L, max_iters=1000, fixed_iters=1)
    Wg, st, info = gpu_solve(L, Hd, lmd, W0[:n], M[:n], opts)
    assert info["sparse_products"] == 1
    assert info["few_launches"] == (1000 if n <= 8 else 0)
    Wg = Wg.cpu().numpy()
    _assert_w_and_f(H, W0[:n], M[:n], Wg, oracle.closed_form(H, W0[:n], M[:n]),
                    label=f"sparse {n} columns")
    full, _, _ = gpu_solve(L, Hd, lmd, W0, M, opts)
    assert rel_fro(Wg, full.cpu().numpy()[:n]) <= 1e-5
