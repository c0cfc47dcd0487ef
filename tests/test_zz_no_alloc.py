"""GPU check of the allocation-free wide ridge solve (cb_ridge_solve_noalloc).

It factors in the library's fixed device scratch array instead of a caller
workspace, so its results must equal those of cb_ridge_solve_ws (same kernel,
same fp64 arithmetic per system) on the same fp32 moments: two calls in a row,
the second on a smaller input, each compared element by element with the
workspace solve, plus a system with G = 0 whose info and zero maps must match.
"""
import sys

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def cb():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2609_00891_amd as cbmod
    return cbmod


def moments(n, P, d_t, rows, seed):
    """Augmented moments of random data: G = X~^T X~ (last column 1), C = X~^T Y, fp32 on the device."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    X = torch.randn((n, rows, P), generator=g)
    X[:, :, P - 1] = 1.0
    X *= torch.exp(0.5 * torch.randn((n, 1, P), generator=g))
    Y = torch.randn((n, rows, d_t), generator=g)
    X, Y = X.to("cuda"), Y.to("cuda")
    Xt = X.transpose(1, 2).contiguous()
    G = torch.bmm(Xt, X)
    C = torch.bmm(Xt, Y)
    G = 0.5 * (G + G.transpose(1, 2).contiguous())     # exactly symmetric
    torch.cuda.synchronize()
    return G.contiguous(), C.contiguous()


def solve_both(cb, G, C, flags):
    n, P, _ = G.shape
    d_t = C.shape[2]
    per = cb.cb_ridge_solve_workspace_bytes(P, d_t, 1)
    assert per <= cb.cb_ridge_solve_noalloc_max_bytes()
    ws = torch.empty((per * n,), dtype=torch.uint8, device="cuda")
    m_ws = torch.full_like(C, 7.0)
    i_ws = torch.full((n,), -5, dtype=torch.int32, device="cuda")
    cb.cb_ridge_solve_ws(G, C, 1e-2, flags, m_ws, i_ws, ws)
    torch.cuda.synchronize()
    del ws
    m_na = torch.full_like(C, -3.0)
    i_na = torch.full((n,), -9, dtype=torch.int32, device="cuda")
    cb.cb_ridge_solve_noalloc(G, C, 1e-2, flags, m_na, i_na)
    torch.cuda.synchronize()
    return m_ws, i_ws, m_na, i_na


def compare(m_ws, i_ws, m_na, i_na, label):
    a, b = m_na.double().cpu().numpy(), m_ws.double().cpu().numpy()
    rel = max(float(np.linalg.norm(a[i] - b[i]) / max(np.linalg.norm(b[i]), 1e-300)) for i in range(a.shape[0]))
    same = bool(torch.equal(m_na, m_ws))
    say(f"  {label}: worst per-map relF vs cb_ridge_solve_ws {rel:.3e}, bitwise equal {same}, "
        f"info {i_na.cpu().tolist()}")
    assert torch.equal(i_na, i_ws)
    assert rel <= 1e-6
    assert same


def test_noalloc_solve_matches_workspace_solve_two_calls(cb):
    flags = cb.CB_LAMBDA_RELATIVE | cb.CB_RIDGE_BIAS_UNPENALIZED
    # first call: the k = 8 width (P = 1025), 30 systems, several scratch batches
    n, P, d_t = 30, 1025, 128
    per = cb.cb_ridge_solve_workspace_bytes(P, d_t, 1)
    say(f"noalloc solve call 1: {n} systems, P={P}, d_t={d_t}, {cb.cb_ridge_solve_noalloc_max_bytes() // per} "
        f"systems per scratch batch")
    G, C = moments(n, P, d_t, 2 * P, seed=11)
    G[4].zero_()                                        # a system with no data: info = 1, zero maps
    C[4].zero_()
    m_ws, i_ws, m_na, i_na = solve_both(cb, G, C, flags)
    assert int(i_ws[4]) == 1 and int((i_ws != 0).sum()) == 1
    assert not m_na[4].any()
    compare(m_ws, i_ws, m_na, i_na, f"P={P}")
    del G, C, m_ws, m_na
    torch.cuda.empty_cache()
    # second call: smaller systems and fewer of them, default ridge flags
    n, P, d_t = 7, 513, 64
    say(f"noalloc solve call 2: {n} systems, P={P}, d_t={d_t}")
    G, C = moments(n, P, d_t, 3 * P, seed=12)
    m_ws, i_ws, m_na, i_na = solve_both(cb, G, C, cb.CB_LAMBDA_RELATIVE)
    assert int((i_ws != 0).sum()) == 0
    compare(m_ws, i_ws, m_na, i_na, f"P={P}")


def test_noalloc_solve_narrow_systems_use_the_register_solver(cb):
    # P <= 129 needs no scratch: the call is cb_ridge_solve
    n, P, d_t = 9, 129, 128
    G, C = moments(n, P, d_t, 4 * P, seed=13)
    m_ref = torch.empty_like(C)
    i_ref = torch.empty((n,), dtype=torch.int32, device="cuda")
    cb.cb_ridge_solve(G, C, 1e-2, cb.CB_LAMBDA_RELATIVE, m_ref, i_ref)
    m_na = torch.empty_like(C)
    i_na = torch.empty((n,), dtype=torch.int32, device="cuda")
    cb.cb_ridge_solve_noalloc(G, C, 1e-2, cb.CB_LAMBDA_RELATIVE, m_na, i_na)
    torch.cuda.synchronize()
    assert torch.equal(m_na, m_ref) and torch.equal(i_na, i_ref)
