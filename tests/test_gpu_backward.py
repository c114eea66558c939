"""GPU parity of the contraction backward (tri_mul_contract_backward) against
the fp64 oracle (oracle.contract_backward): dA_c = dC_c B_c, dB_c = dC_c^T A_c.

Tolerances: exact on small-integer data (every product and partial sum is an
integer below 2^24, so fp32 accumulation and the bf16 rounding of dC are
exact).  On Gaussian data the fp32 path is held to relative Frobenius error
<= 1e-5; the bf16 path rounds dC to bf16 once (relative error <= 2^-9 per
element, about 1e-3 RMS over independent terms), so it is held to relative
Frobenius error <= 3e-3 and max-abs error <= 1e-2 * max |reference|."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import synth
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import errors, host, make_layer, say

pytestmark = pytest.mark.gpu

TOL = {"f32": (1e-5, None), "bf16": (3e-3, 1e-2)}


def check(got, ref, dtype, what):
    mx, rel = errors(got, ref)
    rel_tol, max_rel = TOL[dtype]
    say(f"  {what}: max_abs={mx:.3e} rel_fro={rel:.3e} max|ref|={np.abs(ref).max():.3e}")
    assert np.all(np.isfinite(got)), what
    assert rel <= rel_tol, f"{what}: relative Frobenius error {rel:.3e} > {rel_tol}"
    if max_rel is not None:
        assert mx <= max_rel * np.abs(ref).max(), f"{what}: max-abs error {mx:.3e}"


def run(layer, A, B, dC_dense, N):
    """A, B dense [c][N][N] (device), dC dense [c][N][N] fp32 (device)."""
    dA, dB = layer.contract_backward(T.dense_to_result(dC_dense), T.dense_to_panel(A), T.dense_to_panel(B), N)
    torch.cuda.synchronize()
    return T.result_to_dense(dA, N), T.result_to_dense(dB, N)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("N", [1, 33, 64, 100, 300])
def test_contract_backward_exact_on_integers(dtype, N):
    say(f"contract backward exact dtype={dtype} N={N}")
    layer, _ = make_layer(dtype)
    g = torch.Generator().manual_seed(100 + N)
    A = torch.randint(-4, 5, (128, N, N), generator=g).to(synth.DTYPES[dtype])
    B = torch.randint(-4, 5, (128, N, N), generator=g).to(synth.DTYPES[dtype])
    dC = torch.randint(-4, 5, (128, N, N), generator=g).float()
    dA, dB = run(layer, A.cuda(), B.cuda(), dC.cuda(), N)
    rA, rB = oracle.contract_backward(host(A), host(B), host(dC))
    np.testing.assert_array_equal(host(dA), rA)
    np.testing.assert_array_equal(host(dB), rB)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("N", [96, 257])
def test_contract_backward_gaussian(dtype, N):
    say(f"contract backward gaussian dtype={dtype} N={N}")
    layer, _ = make_layer(dtype)
    g = torch.Generator().manual_seed(200 + N)
    A = torch.randn((128, N, N), generator=g).to(synth.DTYPES[dtype])
    B = torch.randn((128, N, N), generator=g).to(synth.DTYPES[dtype])
    dC = torch.randn((128, N, N), generator=g)
    dA, dB = run(layer, A.cuda(), B.cuda(), dC.cuda(), N)
    rA, rB = oracle.contract_backward(host(A), host(B), host(dC))
    check(host(dA), rA, dtype, "dA")
    check(host(dB), rB, dtype, "dB")


def poisoned_panel(X):
    """dense_to_panel with NaN in every padding element."""
    c, N = X.shape[0], X.shape[1]
    _, tr, S = T._panel_dims(N, c)
    Y = torch.full((c, tr * 256, S * 32), float("nan"), dtype=X.dtype, device=X.device)
    Y[:, :N, :N] = X
    return Y.reshape(c, tr, 256, S, 32).permute(0, 1, 3, 2, 4).contiguous().reshape(-1)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("N", [100, 300])
def test_contract_backward_ignores_padding(dtype, N):
    """NaN in the padding rows and columns of the A and B panels, in the
    padding columns of dC's result layout and in the whole workspace: the
    products reach no padding element (k past N is zeroed in LDS, output
    rows and columns past N are not stored), so integer data stay exact."""
    say(f"contract backward poisoned padding dtype={dtype} N={N}")
    layer, _ = make_layer(dtype)
    g = torch.Generator().manual_seed(300 + N)
    A = torch.randint(-4, 5, (128, N, N), generator=g).to(synth.DTYPES[dtype]).cuda()
    B = torch.randint(-4, 5, (128, N, N), generator=g).to(synth.DTYPES[dtype]).cuda()
    dC = torch.randint(-4, 5, (128, N, N), generator=g).float().cuda()
    J = -(-N // 32)
    dCr = torch.full((128, N, J * 32), float("nan"), device="cuda")
    dCr[:, :, :N] = dC
    dCr = dCr.reshape(128, N, J, 32).permute(1, 2, 0, 3).contiguous().reshape(-1)
    n = N * J * 32 * 128
    dA = torch.empty(n, device="cuda")
    dB = torch.empty(n, device="cuda")
    wsb = T.tri_mul_contract_backward_workspace_size(layer.h, N)
    ws = torch.full((wsb,), 0xff, dtype=torch.uint8, device="cuda")       # NaN in both dtypes
    T.tri_mul_contract_backward(layer.h, dCr, poisoned_panel(A), poisoned_panel(B), N, dA, dB, ws, wsb)
    torch.cuda.synchronize()
    rA, rB = oracle.contract_backward(host(A), host(B), host(dC))
    np.testing.assert_array_equal(host(T.result_to_dense(dA, N)), rA)
    np.testing.assert_array_equal(host(T.result_to_dense(dB, N)), rB)


def test_contract_backward_n4096_sampled():
    """The benchmark size (N = 4096, bf16) in the launch configuration the
    benchmark times; sampled rows of dA and dB against the oracle, one channel
    at a time on the host."""
    N = 4096
    say(f"contract backward N={N} sampled")
    layer, _ = make_layer("bf16")
    g = torch.Generator(device="cuda").manual_seed(4096)
    A = torch.randn((128, N, N), generator=g, device="cuda").to(torch.bfloat16)
    B = torch.randn((128, N, N), generator=g, device="cuda").to(torch.bfloat16)
    dCr = torch.randn(N * N * 128, generator=g, device="cuda")          # result layout, N % 32 == 0
    dA, dB = layer.contract_backward(dCr, T.dense_to_panel(A), T.dense_to_panel(B), N)
    torch.cuda.synchronize()
    dC = T.result_to_dense(dCr, N)
    rows = [0, 1, 1234, 2049, 4095]
    gA = host(T.result_to_dense(dA, N)[:, rows])
    gB = host(T.result_to_dense(dB, N)[:, rows])
    del dA, dB
    rA = np.empty_like(gA)
    rB = np.empty_like(gB)
    for c in range(128):
        rA[c] = host(dC[c, rows]) @ host(B[c])
        rB[c] = host(dC[c][:, rows]).T @ host(A[c])
    check(gA, rA, "bf16", "dA rows")
    check(gB, rB, "bf16", "dB rows")


def test_contract_backward_errors():
    layer, _ = make_layer("bf16")
    N = 64
    need = T.tri_mul_contract_backward_workspace_size(layer.h, N)
    n = N * N * 128
    dC = torch.zeros(n, device="cuda")
    P = torch.zeros(n, dtype=torch.bfloat16, device="cuda")
    dA, dB = torch.empty(n, device="cuda"), torch.empty(n, device="cuda")
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_contract_backward(layer.h, dC, P, P, N, dA, dB, ws, need - 1)
    assert e.value.code == -3
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_contract_backward(layer.h, None, P, P, N, dA, dB, ws, need)
    assert e.value.code == -1
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_contract_backward(layer.h, dC, P, P, 0, dA, dB, ws, need)
    assert e.value.code == -1
