"""GPU parity of the layer forward pass and of the layer loop of Algorithm 1.

optima_linear_forward against the oracle's fp64 forward (bf16 weights, exact
products): fp32 outputs within the fp32 summation error, bf16 outputs within
one bf16 step of the rounded oracle value, the squared output error within
1e-6 relative. The chain of three layers is then checked layer by layer: each
layer's inputs as the device produced them go to the oracle. The oracle then
gives that layer's mask, the closed form of its damped QPs, its two output
errors and the next layer's inputs.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline_oracle as po
import workloads
from gpu_util import dev, to_dev, rel_fro, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _bf16_dev(x64: np.ndarray) -> torch.Tensor:
    """Device bfloat16 tensor of values that are exact in bf16."""
    return torch.from_numpy(np.ascontiguousarray(x64, dtype=np.float32)).to(dev()).to(torch.bfloat16)


def _sum_abs_bound(X, W):
    return np.abs(X) @ np.abs(po.bf16_round(W)).T


@pytest.mark.parametrize("n_tok,d_in,d_out", [(300, 128, 100), (1000, 256, 260), (129, 64, 4),
                                              (2048, 512, 384)])
@pytest.mark.parametrize("act", ["none", "silu"])
def test_forward_matches_oracle(L, n_tok, d_in, d_out, act):
    rng = np.random.default_rng(n_tok + d_in)
    X = po.bf16_round(rng.standard_normal((n_tok, d_in)) * 2)
    W = (rng.standard_normal((d_out, d_in)) * 0.05).astype(np.float32)
    Xd, Wd = _bf16_dev(X), to_dev(W)
    a = L.ACT_SILU if act == "silu" else L.ACT_NONE
    Y32 = torch.empty((n_tok, d_out), dtype=torch.float32, device=dev())
    L.optima_linear_forward(Xd, Wd, Y=Y32, act=a)
    Y16 = torch.empty((n_tok, d_out), dtype=torch.bfloat16, device=dev())
    L.optima_linear_forward(Xd, Wd, Y=Y16, act=a)
    ref = po.linear_forward(X, W, act)
    y32 = Y32.cpu().numpy().astype(np.float64)
    bound = 2.0 ** -18 * _sum_abs_bound(X, W) + 1e-30
    err = np.abs(y32 - ref)
    log(f"  n={n_tok} d_in={d_in} d_out={d_out} {act}: max |y - ref| / bound = "
        f"{float(np.max(err / bound)):.3f}")
    assert np.all(err <= bound)
    # bf16 outputs: the rounding of the device's fp32 value, so within the
    # fp32 bound plus one bf16 step of the rounded oracle value (near zero
    # the fp32 bound, relative to the summed magnitudes, dominates), and
    # equal to it almost always
    y16 = Y16.float().cpu().numpy().astype(np.float64)
    r16 = po.bf16_round(ref.astype(np.float32))
    step = np.maximum(np.abs(r16), np.abs(y16)) * 2.0 ** -7 + 2 * bound
    assert np.all(np.abs(y16 - r16) <= step)
    assert np.mean(y16 != r16) < 1e-3
    np.testing.assert_array_equal(y16, po.bf16_round(Y32.cpu().numpy()))


def test_forward_squared_error(L):
    rng = np.random.default_rng(7)
    n_tok, d_in, d_out = 777, 192, 136
    X = po.bf16_round(rng.standard_normal((n_tok, d_in)))
    W = (rng.standard_normal((d_out, d_in)) * 0.05).astype(np.float32)
    Wr = W + (rng.standard_normal(W.shape) * 0.01).astype(np.float32)
    Xd = _bf16_dev(X)
    Yref = torch.empty((n_tok, d_out), dtype=torch.float32, device=dev())
    L.optima_linear_forward(Xd, to_dev(Wr), Y=Yref)
    err = torch.zeros(1, dtype=torch.float64, device=dev())
    L.optima_linear_forward(Xd, to_dev(W), Y_ref=Yref, err_out=err)
    # oracle: the same sum against the device reference values
    Z = po.linear_forward(X, W)
    want = float(np.sum((Z - Yref.cpu().numpy().astype(np.float64)) ** 2))
    assert err.item() == pytest.approx(want, rel=1e-6)
    assert err.item() == pytest.approx(po.output_sq_error(X, W, Wr), rel=1e-4)
    # the same weights against their own outputs: exactly zero
    L.optima_linear_forward(Xd, to_dev(Wr), Y_ref=Yref, err_out=err)
    assert err.item() == 0.0
    # no tokens: zero error, nothing written
    L.optima_linear_forward(Xd[:0], to_dev(W), Y_ref=Yref[:0], err_out=err)
    assert err.item() == 0.0


def test_forward_error_paths(L):
    X = _bf16_dev(np.ones((16, 64)))
    W = torch.ones((8, 64), dtype=torch.float32, device=dev())
    W[3, 5] = float("nan")
    Y = torch.empty((16, 8), dtype=torch.float32, device=dev())
    with pytest.raises(L.OptimaError) as e:
        L.optima_linear_forward(X, W, Y=Y)
    assert e.value.status == -3
    with pytest.raises(ValueError):
        L.optima_linear_forward(X, W[:, :32], Y=Y)


def _chain(n_tok=1024, d=128, layers=3, seed=11):
    rng = np.random.default_rng(seed)
    mix = np.eye(d) + 0.5 * rng.standard_normal((d, d)) / np.sqrt(d) * 4
    X0 = po.bf16_round((rng.standard_normal((n_tok, d)) @ mix) * np.exp(0.5 * rng.standard_normal(d)))
    Ws = [(rng.standard_normal((d, d)) / np.sqrt(d)).astype(np.float32) for _ in range(layers)]
    return X0, Ws


def _run_chain(L, X0, Ws, opts):
    from paper_2512_13886_amd.pipeline import prune_chain
    start = lambda d: to_dev(workloads.power_start_block(d, 16))  # noqa: E731
    return prune_chain(_bf16_dev(X0), [to_dev(W) for W in Ws], start, sparsity=0.5,
                       rel_damp=0.01, opts=opts)


def test_chain_layer_by_layer(L):
    X0, Ws = _chain()
    opts = L.SolverOpts.default(max_iters=3000, fixed_iters=1)
    kept, masks, reps, _ = _run_chain(L, X0, Ws, opts)
    # Re-run the forward passes to collect each layer's device inputs.
    X = X0
    for l, (W0, Wk, Mk, rep) in enumerate(zip(Ws, kept, masks, reps)):
        Wk, Mk = Wk.cpu().numpy(), Mk.cpu().numpy()
        r = po.prune_layer(X, W0, 0.5, 0.01, act="silu")
        np.testing.assert_array_equal(Mk, r.mask)
        assert not rep.skipped
        assert np.all(Wk[Mk == 0].view(np.uint32) == 0)
        assert rel_fro(Wk, r.W) <= 1e-4
        e_kept = po.output_sq_error(X, Wk, W0)
        e_wanda = po.output_sq_error(X, np.where(Mk != 0, W0, 0).astype(np.float32), W0)
        log(f"  layer {l}: W rel={rel_fro(Wk, r.W):.2e} ratio gpu {rep.error_ratio:.4f} "
            f"oracle {r.ratio:.4f}")
        assert rep.err_kept == pytest.approx(e_kept, rel=1e-4)
        assert rep.err_wanda == pytest.approx(e_wanda, rel=1e-4)
        assert rep.error_ratio < 1.0
        # the next inputs: bf16(silu(X bf16(W_kept)^T)) from the device's weights
        Xn = torch.empty((X.shape[0], Wk.shape[0]), dtype=torch.bfloat16, device=dev())
        L.optima_linear_forward(_bf16_dev(X), to_dev(Wk), Y=Xn, act=L.ACT_SILU)
        xn = Xn.float().cpu().numpy().astype(np.float64)
        want = po.bf16_round(po.linear_forward(X, Wk, "silu").astype(np.float32))
        tol = (np.maximum(np.abs(want), np.abs(xn)) * 2.0 ** -7
               + 2.0 ** -17 * _sum_abs_bound(X, Wk))
        assert np.all(np.abs(xn - want) <= tol)
        X = xn


def test_chain_skip_rule(L):
    # One iteration at a tolerance no column meets: every layer is skipped,
    # keeps the mask-only weights and has an error ratio of exactly 1.
    X0, Ws = _chain(layers=2, seed=12)
    opts = L.SolverOpts.default(max_iters=1, eps_rel=1e-9, eps_abs=0.0)
    kept, masks, reps, _ = _run_chain(L, X0, Ws, opts)
    for W0, Wk, Mk, rep in zip(Ws, kept, masks, reps):
        assert rep.skipped and rep.converged == 0
        np.testing.assert_array_equal(Wk.cpu().numpy(),
                                      np.where(Mk.cpu().numpy() != 0, W0, 0).astype(np.float32))
        assert rep.error_ratio == 1.0
