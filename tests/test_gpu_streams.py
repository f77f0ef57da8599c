"""The library on a side stream and from a second host thread.

Every host wait of the library (the solve's read-backs, the spectral
iterations' convergence polls) copies into a pinned buffer held per host
thread and device, and polls an event recorded on the caller's stream. The
other GPU tests run on torch's default stream from the main thread. Here the
same spectral norm, Lanczos step size and solve run on a created stream, then
from another host thread on a stream of its own, and must match the
default-stream run. The kernels and their reduction orders are the same, so
the results agree to rounding.
"""
import threading

import numpy as np
import pytest
import torch

from gpu_util import dev, to_dev, rel_fro, f32_exact, log

pytestmark = pytest.mark.gpu

D, N_COLS, RANK = 512, 300, 64


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


@pytest.fixture(scope="module")
def problem():
    rng = np.random.default_rng(97)
    B = rng.standard_normal((D, RANK))
    H = f32_exact(B @ B.T / RANK + 0.5 * np.eye(D))
    W0 = (rng.standard_normal((N_COLS, D)) * 0.02).astype(np.float32)
    keep = np.argsort(-np.abs(W0), axis=1, kind="stable")[:, :D // 2]
    M = np.zeros((N_COLS, D), dtype=np.uint8)
    np.put_along_axis(M, keep, 1, axis=1)
    V0 = rng.standard_normal((16, D)).astype(np.float32)
    return to_dev(H), to_dev(W0), to_dev(M, torch.uint8), to_dev(V0)


def run_all(L, Hd, W0d, Md, V0d, stream):
    lm = torch.zeros(1, dtype=torch.float32, device=dev())
    it = torch.zeros(1, dtype=torch.int32, device=dev())
    L.optima_spectral_norm(Hd, V0d, lm, max_iters=200, tol=1e-6, iters=it, stream=stream)
    lz = torch.zeros(1, dtype=torch.float32, device=dev())
    st = torch.zeros(1, dtype=torch.int32, device=dev())
    L.optima_spectral_lanczos(Hd, V0d[0].contiguous(), lz, steps=st, stream=stream)
    W = torch.empty_like(W0d)
    conv = torch.zeros(N_COLS, dtype=torch.uint8, device=dev())
    info = L.optima_qp_solve_batched(Hd, lm, W0d, Md, W, stats={"converged": conv},
                                     stream=stream)
    if stream is None:
        torch.cuda.synchronize()
    else:
        stream.synchronize()
    return (float(lm.item()), int(it.item()), float(lz.item()), int(st.item()),
            W.cpu().numpy(), conv.cpu().numpy(), info)


def check_same(ref, got, label):
    lam_r, it_r, lz_r, st_r, W_r, c_r, inf_r = ref
    lam, it, lz, st, W, c, inf = got
    log(f"{label}: lambda {lam:.7e} vs {lam_r:.7e}, {it} vs {it_r} passes, Lanczos {lz:.7e} "
        f"({st} steps), W rel_fro {rel_fro(W, W_r):.2e}, {inf['iterations']} iterations")
    assert lam == pytest.approx(lam_r, rel=1e-6) and lz == pytest.approx(lz_r, rel=1e-6)
    assert it == it_r and st == st_r
    assert c.all() and np.array_equal(c, c_r)
    assert inf["iterations"] == inf_r["iterations"] and inf["checks"] == inf_r["checks"]
    assert rel_fro(W, W_r) <= 1e-6


def test_side_stream_and_second_thread_match_default_stream(L, problem):
    Hd, W0d, Md, V0d = problem
    torch.cuda.synchronize()
    ref = run_all(L, Hd, W0d, Md, V0d, None)

    side = torch.cuda.Stream()
    check_same(ref, run_all(L, Hd, W0d, Md, V0d, side), "side stream")

    out, err = {}, []

    def worker():
        try:
            torch.cuda.set_device(dev())
            out["r"] = run_all(L, Hd, W0d, Md, V0d, torch.cuda.Stream())
        except Exception as e:  # reported in the main thread
            err.append(e)

    t = threading.Thread(target=worker)
    t.start()
    t.join(timeout=120)
    assert not t.is_alive(), "the second host thread did not finish"
    assert not err, err
    check_same(ref, out["r"], "second host thread")
