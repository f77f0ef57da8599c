"""The library on a side stream and from a second host thread.

Every host wait of the library (the solve's read-backs, the spectral
iterations' convergence polls) copies into a pinned buffer held per host
thread and device, and polls an event recorded on the caller's stream. The
other GPU tests run on torch's default stream from the main thread. Here the
Hessian accumulation, the layer forward pass (both asynchronous, with the
workspace the binding allocates on the call's stream), the spectral norm, the
Lanczos step size and the solve run on a created stream, then from another
host thread on a stream of its own, and must match the default-stream run.
The kernels and their reduction orders are the same, so the results agree
bit for bit (the Hessian and the forward pass) or to rounding.
"""
import threading

import numpy as np
import pytest
import torch

from gpu_util import dev, to_dev, rel_fro, f32_exact, log

pytestmark = pytest.mark.gpu

D, N_COLS, RANK = 512, 300, 64
N_TOK, D_OUT = 3000, 256


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
    X = to_dev(rng.standard_normal((N_TOK, D)).astype(np.float32)).to(torch.bfloat16)
    Wf = to_dev((rng.standard_normal((D_OUT, D)) * 0.05).astype(np.float32))
    Yref = to_dev(rng.standard_normal((N_TOK, D_OUT)).astype(np.float32))
    torch.cuda.synchronize()
    return to_dev(H), to_dev(W0), to_dev(M, torch.uint8), to_dev(V0), X, Wf, Yref


def run_all(L, prob, stream):
    Hd, W0d, Md, V0d, X, Wf, Yref = prob
    # Outputs are allocated (and zero-filled) on the stream the library runs
    # on, so the fills are ordered before its kernels.
    with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
        Hx = torch.empty((D, D), dtype=torch.float32, device=dev())
        Y = torch.empty((N_TOK, D_OUT), dtype=torch.bfloat16, device=dev())
        err = torch.zeros(1, dtype=torch.float64, device=dev())
        lm = torch.zeros(1, dtype=torch.float32, device=dev())
        it = torch.zeros(1, dtype=torch.int32, device=dev())
        lz = torch.zeros(1, dtype=torch.float32, device=dev())
        st = torch.zeros(1, dtype=torch.int32, device=dev())
        W = torch.empty_like(W0d)
        conv = torch.zeros(N_COLS, dtype=torch.uint8, device=dev())
        v0 = V0d[0].contiguous()
    L.optima_hessian_accumulate(X, Hx, stream=stream)
    L.optima_linear_forward(X, Wf, Y, L.ACT_SILU, Y_ref=Yref, err_out=err, stream=stream)
    L.optima_spectral_norm(Hd, V0d, lm, max_iters=200, tol=1e-6, iters=it, stream=stream)
    L.optima_spectral_lanczos(Hd, v0, lz, steps=st, stream=stream)
    info = L.optima_qp_solve_batched(Hd, lm, W0d, Md, W, stats={"converged": conv},
                                     stream=stream)
    if stream is None:
        torch.cuda.synchronize()
    else:
        stream.synchronize()
    return (float(lm.item()), int(it.item()), float(lz.item()), int(st.item()),
            W.cpu().numpy(), conv.cpu().numpy(), info, Hx.cpu(), Y.cpu(), float(err.item()))


def check_same(ref, got, label):
    lam_r, it_r, lz_r, st_r, W_r, c_r, inf_r, H_r, Y_r, e_r = ref
    lam, it, lz, st, W, c, inf, Hx, Y, e = got
    log(f"{label}: Hessian identical {torch.equal(Hx, H_r)}, forward identical "
        f"{torch.equal(Y, Y_r)}, error sum {e:.9e} vs {e_r:.9e}")
    assert torch.equal(Hx, H_r) and torch.equal(Y, Y_r) and e == e_r
    log(f"{label}: lambda {lam:.7e} vs {lam_r:.7e}, {it} vs {it_r} passes, Lanczos {lz:.7e} "
        f"({st} steps), W rel_fro {rel_fro(W, W_r):.2e}, {inf['iterations']} iterations")
    assert lam == pytest.approx(lam_r, rel=1e-6) and lz == pytest.approx(lz_r, rel=1e-6)
    assert it == it_r and st == st_r
    assert c.all() and np.array_equal(c, c_r)
    assert inf["iterations"] == inf_r["iterations"] and inf["checks"] == inf_r["checks"]
    assert rel_fro(W, W_r) <= 1e-6


def test_side_stream_and_second_thread_match_default_stream(L, problem):
    torch.cuda.synchronize()
    ref = run_all(L, problem, None)

    side = torch.cuda.Stream()
    check_same(ref, run_all(L, problem, side), "side stream")

    out, err = {}, []

    def worker():
        try:
            torch.cuda.set_device(dev())
            out["r"] = run_all(L, problem, torch.cuda.Stream())
        except Exception as e:  # reported in the main thread
            err.append(e)

    t = threading.Thread(target=worker)
    t.start()
    t.join(timeout=120)
    assert not t.is_alive(), "the second host thread did not finish"
    assert not err, err
    check_same(ref, out["r"], "second host thread")
