"""Pins of the layer-loop oracle (Algorithm 1): bf16 rounding, SiLU, the
layer forward pass, the squared output error, the skip rule and one layer of
the chain."""
import numpy as np
import pytest
import torch

import oracle
from oracle import pipeline_oracle as po


def test_bf16_round_matches_torch_and_ties():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(4000) * 10.0 ** rng.integers(-6, 6, 4000),
                        [0.0, -0.0, 1.0, -1.0, 65504.0, 1e-30]]).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(po.bf16_round(x), ref)
    # ties go to the even mantissa: 1 + 2^-8 lies halfway between 1 and
    # 1 + 2^-7 (even: 1); 1 + 3 * 2^-8 halfway between 1 + 2^-7 and 1 + 2^-6
    assert po.bf16_round(np.float32(1 + 2.0 ** -8)) == 1.0
    assert po.bf16_round(np.float32(1 + 3 * 2.0 ** -8)) == 1 + 2.0 ** -6
    assert po.bf16_round(np.float32(1 + 2.0 ** -8 + 2.0 ** -20)) == 1 + 2.0 ** -7


def test_silu_values():
    assert po.silu(0.0) == 0.0
    assert po.silu(1.0) == pytest.approx(0.7310585786300049, rel=1e-15)
    assert po.silu(-1.0) == pytest.approx(-0.2689414213699951, rel=1e-15)
    z = np.linspace(-30, 30, 601)
    np.testing.assert_allclose(po.silu(z) - po.silu(-z), z, rtol=0, atol=1e-12)
    assert po.silu(-1000.0) == 0.0 and po.silu(1000.0) == 1000.0


def test_linear_forward_brute_force():
    rng = np.random.default_rng(1)
    X = rng.integers(-8, 9, (7, 5)).astype(np.float64)   # exact in bf16
    W = rng.integers(-8, 9, (3, 5)).astype(np.float32)
    Z = np.zeros((7, 3))
    for t in range(7):
        for j in range(3):
            for k in range(5):
                Z[t, j] += X[t, k] * W[j, k]
    np.testing.assert_array_equal(po.linear_forward(X, W), Z)
    np.testing.assert_array_equal(po.linear_forward(X, W, "silu"), po.silu(Z))
    # the weights are rounded to bf16 first: 1 + 2^-9 becomes 1
    W1 = np.full((1, 5), 1 + 2.0 ** -9, dtype=np.float32)
    np.testing.assert_array_equal(po.linear_forward(X, W1)[:, 0], X.sum(axis=1))


def test_output_sq_error_identity():
    rng = np.random.default_rng(2)
    X = po.bf16_round(rng.standard_normal((64, 24)))
    Wa = rng.standard_normal((10, 24)).astype(np.float32)
    Wb = rng.standard_normal((10, 24)).astype(np.float32)
    H = oracle.hessian([X])
    D = po.bf16_round(Wa) - po.bf16_round(Wb)
    via_h = sum(D[j] @ H @ D[j] for j in range(10))
    assert po.output_sq_error(X, Wa, Wb) == pytest.approx(via_h, rel=1e-12)
    assert po.output_sq_error(X, Wa, Wb) == pytest.approx(po.output_sq_error(X, Wb, Wa),
                                                          rel=1e-15)
    assert po.output_sq_error(X, Wa, Wa) == 0.0


def test_skip_rule_cases():
    ok = np.ones(10, dtype=bool)
    assert not po.skip_layer(ok, np.ones(10), np.full(10, 0.5))
    half = ok.copy()
    half[:5] = False
    assert not po.skip_layer(half, np.ones(10), np.full(10, 0.5))   # exactly half: not most
    half[5] = False
    assert po.skip_layer(half, np.ones(10), np.full(10, 0.5))       # 6 of 10 unconverged
    f_fin = np.full(10, 0.5)
    f_fin[0] = 6.0                                                  # sum 10.5 > 10
    assert po.skip_layer(ok, np.ones(10), f_fin)
    assert not po.skip_layer(np.zeros(0, dtype=bool), [], [])


def _chain_inputs(n_tok=600, d=24, seed=3):
    # correlated features (a random mixing of independent ones), so that the
    # weight update has something to compensate
    rng = np.random.default_rng(seed)
    mix = np.eye(d) + 0.5 * rng.standard_normal((d, d))
    X0 = po.bf16_round((rng.standard_normal((n_tok, d)) @ mix) * np.exp(rng.standard_normal(d)))
    Ws = [(rng.standard_normal((d, d)) * 0.2).astype(np.float32) for _ in range(3)]
    return X0, Ws


def test_chain_layers_are_their_closed_forms():
    X0, Ws = _chain_inputs()
    res = po.prune_chain(X0, Ws, 0.5, 0.01)
    X = X0
    for W0, r in zip(Ws, res):
        H, _ = oracle.damp(oracle.hessian([X]), 0.01)
        H = H.astype(np.float32).astype(np.float64)
        np.testing.assert_array_equal(r.mask, oracle.wanda_mask(W0, np.diag(oracle.hessian([X])),
                                                                "unstructured", 0.5))
        np.testing.assert_allclose(r.W, oracle.closed_form(H, W0, r.mask), rtol=1e-6,
                                   atol=1e-9)
        assert np.all(r.W[r.mask == 0] == 0)
        np.testing.assert_array_equal(
            r.X_next, po.bf16_round(po.silu(X @ po.bf16_round(r.W).T).astype(np.float32)))
        X = r.X_next


def test_closed_form_lowers_the_output_error_without_damping():
    # With the damping going to zero the closed form minimises exactly the
    # output error X (w - w0) over the kept entries, so it cannot do worse
    # than Wanda's zeroing on the same mask (the bf16 rounding of the weights
    # aside, which is far below the gap here).
    X0, Ws = _chain_inputs(seed=4)
    for rel in (1e-6, 1e-8):
        r = po.prune_layer(X0, Ws[0], 0.5, rel)
        assert r.err_optima <= r.err_wanda
        assert r.ratio < 0.8


def test_skipped_layer_keeps_wanda_weights():
    X0, Ws = _chain_inputs(seed=5)
    Hd, _ = oracle.damp(oracle.hessian([X0]), 0.01)
    lam = float(np.linalg.eigvalsh(Hd)[-1])
    # one iteration cannot converge at these tolerances: the layer is skipped
    r = po.prune_layer(X0, Ws[0], 0.5, 0.01, solver="rapdhg", lambda_max=lam,
                       opts=oracle.SolverOptions(max_iters=1, eps_rel=1e-9, eps_abs=0.0))
    assert r.skipped
    np.testing.assert_array_equal(r.W, np.where(r.mask != 0, Ws[0], 0).astype(np.float32))
    assert r.ratio == 1.0
