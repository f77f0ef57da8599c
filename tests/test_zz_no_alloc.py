"""optima_spectral_norm_noalloc against optima_spectral_norm.

The entry point for callers that cannot allocate runs the same iterations
on the library's fixed per-device work array. Through the C ABI (ctypes
binding) it must return the same lambda_max and pass count as the
workspace entry point, bit for bit, on two calls in a row (the second on a
smaller matrix, over the contents the first call left in the array), for the
block iteration and the power iteration, and reject a matrix wider than its
limit before any launch.
"""
import ctypes

import numpy as np
import pytest
import torch

from gpu_util import dev, to_dev, f32_exact, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    import paper_2512_13886_amd as lib_mod  # fails loudly when the library is missing
    return lib_mod


def _spd(d, rank, seed):
    rng = np.random.default_rng(seed)
    B = rng.standard_normal((d, rank))
    s = np.ones(rank)
    s[:8] = 10.0 + np.arange(8)  # a cluster of large eigenvalues, as outlier channels give
    H = f32_exact((B * s) @ B.T / rank + 0.25 * np.eye(d))
    return to_dev(H), to_dev(rng.standard_normal((16, d)).astype(np.float32))


def _pair(L, H, V0, max_iters=1000, tol=1e-6):
    ref_l = torch.zeros(1, dtype=torch.float32, device=dev())
    ref_i = torch.zeros(1, dtype=torch.int32, device=dev())
    L.optima_spectral_norm(H, V0, ref_l, max_iters=max_iters, tol=tol, iters=ref_i)
    got_l = torch.full((1,), -1.0, dtype=torch.float32, device=dev())
    got_i = torch.full((1,), -1, dtype=torch.int32, device=dev())
    L.optima_spectral_norm_noalloc(H, V0, got_l, max_iters=max_iters, tol=tol, iters=got_i)
    torch.cuda.synchronize()
    return (float(ref_l.item()), int(ref_i.item())), (float(got_l.item()), int(got_i.item()))


@pytest.mark.parametrize("block", [16, 1])
def test_noalloc_matches_workspace_entry_point_twice(L, block):
    # First call on a 4096-wide matrix, then a smaller, odd-sized one (no
    # vector loads) over whatever the first call left in the array.
    for d, seed in ((4096, 11), (1000, 12)):
        H, V0 = _spd(d, 256, seed)
        V = V0 if block == 16 else V0[0].contiguous()
        ref, got = _pair(L, H, V, max_iters=300 if block == 16 else 2000)
        log(f"d={d} block={block}: lambda {got[0]:.9e} ({got[1]} passes) vs workspace entry "
            f"{ref[0]:.9e} ({ref[1]} passes)")
        assert got[0] == ref[0] and got[1] == ref[1]
        assert np.float32(got[0]) == np.float32(ref[0])
        lam = float(np.linalg.eigvalsh(H.double().cpu().numpy())[-1])
        assert got[0] <= lam * (1 + 1e-5) and got[0] >= lam * (1 - 1e-3)


def test_noalloc_rejects_a_matrix_beyond_its_array(L):
    lib = ctypes.CDLL(L.library_path())
    f = lib.optima_spectral_norm_noalloc
    f.restype = ctypes.c_int
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    f.argtypes = [vp, i64, vp, ctypes.c_int, ctypes.c_int, ctypes.c_float, vp, vp, vp]
    H = torch.zeros(16, dtype=torch.float32, device=dev())
    out = torch.zeros(1, dtype=torch.float32, device=dev())
    # Validation returns before any launch: d beyond the limit is a workspace
    # error; a bad block or iteration count is an invalid argument.
    st = f(vp(H.data_ptr()), L.SPECTRAL_NOALLOC_MAX_DIM + 1, vp(H.data_ptr()), 16, 10, 1e-6,
           vp(out.data_ptr()), None, None)
    assert st == -4, st
    assert f(vp(H.data_ptr()), 4, vp(H.data_ptr()), 17, 10, 1e-6, vp(out.data_ptr()), None,
             None) == -1
    assert f(vp(H.data_ptr()), 4, vp(H.data_ptr()), 1, 0, 1e-6, vp(out.data_ptr()), None,
             None) == -1
