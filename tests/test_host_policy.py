"""Host logic of the package, on the CPU: the step-size policy, the skip rule
and the binding's argument checks (no kernel runs here)."""
import numpy as np
import pytest
import torch


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


@pytest.fixture(scope="module")
def pipeline(L):
    from paper_2512_13886_amd import pipeline as mod
    return mod


class _FakeSpectral:
    """Stands in for the two spectral entry points and records the calls."""

    def __init__(self, block_passes_run):
        self.block_passes_run = block_passes_run
        self.calls = []

    def norm(self, H, V0, lam, max_iters, tol, iters):
        self.calls.append(("block", max_iters, tol, V0.shape))
        iters.fill_(min(self.block_passes_run, max_iters))
        lam.fill_(1.0)

    def lanczos(self, H, v0, lam, tol, steps):
        self.calls.append(("lanczos", tol, v0.shape, v0.data_ptr()))
        steps.fill_(42)
        lam.fill_(2.0)


@pytest.mark.parametrize("passes,method", [(4, "subspace"), (7, "subspace"), (8, "lanczos")])
def test_step_size_falls_back_to_lanczos(monkeypatch, pipeline, passes, method):
    fake = _FakeSpectral(passes)
    monkeypatch.setattr(pipeline.L, "optima_spectral_norm", fake.norm)
    monkeypatch.setattr(pipeline.L, "optima_spectral_lanczos", fake.lanczos)
    H = torch.zeros(8, 8)
    V0 = torch.randn(16, 8)
    lam = torch.zeros(1)
    rep = pipeline.spectral_step_size(H, V0, lam)
    assert rep["method"] == method
    assert fake.calls[0] == ("block", pipeline.BLOCK_PASSES, 1e-6, (16, 8))
    if method == "lanczos":
        # Lanczos starts from the block's first vector, at tol 1e-7.
        assert len(fake.calls) == 2 and fake.calls[1][:3] == ("lanczos", 1e-7, (8,))
        assert fake.calls[1][3] == V0[0].data_ptr()
        assert rep["lanczos_steps"] == 42 and float(lam) == 2.0
    else:
        assert len(fake.calls) == 1 and rep["lanczos_steps"] == 0 and float(lam) == 1.0
    assert rep["block_passes"] == min(passes, pipeline.BLOCK_PASSES)


def test_skip_rule(pipeline):
    ones = torch.ones(10, dtype=torch.uint8)
    f0 = torch.ones(10)
    assert not pipeline.skip_layer(ones, f0, f0 * 0.5)
    half = ones.clone()
    half[:5] = 0
    assert not pipeline.skip_layer(half, f0, f0 * 0.5)     # exactly half unconverged: not most
    half[5] = 0
    assert pipeline.skip_layer(half, f0, f0 * 0.5)         # 6 of 10 unconverged
    worse = f0 * 0.5
    worse[0] = 10.0                                        # sum f_final above sum f_initial
    assert pipeline.skip_layer(ones, f0, worse)
    assert not pipeline.skip_layer(torch.zeros(0, dtype=torch.uint8), torch.zeros(0),
                                   torch.zeros(0))


def test_binding_rejects_host_tensors_before_any_call(L):
    H = torch.zeros(8, 8)
    lam = torch.zeros(1)
    with pytest.raises(ValueError, match="device tensor"):
        L.optima_spectral_lanczos(H, torch.ones(8), lam)
    with pytest.raises(ValueError, match="device tensor"):
        L.optima_spectral_norm(H, torch.ones(8), lam)
    with pytest.raises(ValueError):
        L.optima_hessian_damp(H, 0.01, lam)
    assert np.isfinite(L.optima_spectral_lanczos_workspace_bytes(4096, 64))
