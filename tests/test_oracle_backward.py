"""Pins of the oracle's backward pass (gradients of the update) against things
other than itself: automatic differentiation of an independent torch forward,
central finite differences of the oracle's own forward, brute-force loops for
the contraction backward, the bilinear identity, and exact zeros on masked
pairs.  CPU only, fp64."""
import numpy as np
import pytest
import torch

import oracle
from oracle import f64
from paper_2603_14806_amd import synth

DIRS = ("outgoing", "incoming")


def rand_weights(c_z, c, seed):
    W = synth.weights(c_z, c, dtype="f32", seed=seed, affine=True)
    return {k: f64(v) for k, v in W.items()}


def torch_forward(z, mask, W, direction, eps=1e-5):
    """The layer written with torch ops (independent of the oracle's code),
    differentiable in z and every weight."""
    ln = torch.nn.functional.layer_norm
    cz = z.shape[-1]
    m = (mask != 0).double()
    mp = (m[:, None] * m[None, :])[..., None]
    x = ln(z, (cz,), W["ln_in_w"], W["ln_in_b"], eps=eps)
    a = mp * torch.sigmoid(x @ W["w_ga"].T) * (x @ W["w_a"].T)
    b = mp * torch.sigmoid(x @ W["w_gb"].T) * (x @ W["w_b"].T)
    if direction == "outgoing":
        C = torch.einsum("ikc,jkc->ijc", a, b)
    else:
        C = torch.einsum("kic,kjc->ijc", a, b)
    c = C.shape[-1]
    y = ln(C, (c,), W["ln_out_w"], W["ln_out_b"], eps=eps) @ W["w_o"].T
    return mp * torch.sigmoid(x @ W["w_g"].T) * y


def setup(N, c_z, c, seed, masked=True):
    rng = np.random.default_rng(seed)
    z = rng.standard_normal((N, N, c_z))
    mask = np.ones(N)
    if masked and N > 3:
        mask[rng.choice(N, size=2, replace=False)] = 0
    W = rand_weights(c_z, c, seed + 1)
    dout = rng.standard_normal((N, N, c_z))
    return z, mask, W, dout


@pytest.mark.parametrize("direction", DIRS)
@pytest.mark.parametrize("N,c_z,c", [(1, 4, 4), (5, 8, 4), (6, 4, 8)])
def test_backward_matches_autograd(direction, N, c_z, c):
    z, mask, W, dout = setup(N, c_z, c, seed=10 * N + c)
    zt = torch.tensor(z, requires_grad=True)
    Wt = {k: torch.tensor(v, requires_grad=True) for k, v in W.items()}
    out = torch_forward(zt, torch.tensor(mask), Wt, direction)
    # the torch forward is the oracle's function
    np.testing.assert_allclose(out.detach().numpy(), oracle.tri_mul(z, mask, W, direction), rtol=1e-12, atol=1e-12)
    (out * torch.tensor(dout)).sum().backward()
    g = oracle.tri_mul_backward(z, mask, W, direction, dout)
    np.testing.assert_allclose(g["dz"], zt.grad.numpy(), rtol=1e-10, atol=1e-11)
    for k in oracle.WEIGHT_NAMES:
        np.testing.assert_allclose(g[k], Wt[k].grad.numpy(), rtol=1e-10, atol=1e-11, err_msg=k)


@pytest.mark.parametrize("direction", DIRS)
def test_backward_finite_differences(direction):
    N, c_z, c = 5, 6, 4
    z, mask, W, dout = setup(N, c_z, c, seed=3)
    g = oracle.tri_mul_backward(z, mask, W, direction, dout)
    rng = np.random.default_rng(4)

    def L(zz, WW):
        return float((oracle.tri_mul(zz, mask, WW, direction) * dout).sum())

    eps = 1e-5
    V = rng.standard_normal(z.shape)
    fd = (L(z + eps * V, W) - L(z - eps * V, W)) / (2 * eps)
    assert abs(fd - (g["dz"] * V).sum()) <= 1e-7 * max(1.0, abs(fd))
    for k in ("w_a", "w_gb", "w_g", "w_o", "ln_out_w", "ln_in_b"):
        V = rng.standard_normal(W[k].shape)
        Wp = dict(W, **{k: W[k] + eps * V})
        Wm = dict(W, **{k: W[k] - eps * V})
        fd = (L(z, Wp) - L(z, Wm)) / (2 * eps)
        assert abs(fd - (g[k] * V).sum()) <= 1e-7 * max(1.0, abs(fd)), k


def test_contract_backward_brute_force():
    rng = np.random.default_rng(5)
    c, n, m, K = 3, 4, 5, 6
    A, B, dC = rng.standard_normal((c, n, K)), rng.standard_normal((c, m, K)), rng.standard_normal((c, n, m))
    dA, dB = oracle.contract_backward(A, B, dC)
    for ch in range(c):
        for i in range(n):
            for k in range(K):
                s = 0.0
                for j in range(m):
                    s += dC[ch, i, j] * B[ch, j, k]
                assert abs(dA[ch, i, k] - s) < 1e-12
        for j in range(m):
            for k in range(K):
                s = 0.0
                for i in range(n):
                    s += dC[ch, i, j] * A[ch, i, k]
                assert abs(dB[ch, j, k] - s) < 1e-12


def test_contract_backward_bilinear_identity():
    # C is bilinear in (A, B), so <dA, A> = <dB, B> = <dC, C>.
    rng = np.random.default_rng(6)
    A, B, dC = rng.standard_normal((4, 7, 9)), rng.standard_normal((4, 8, 9)), rng.standard_normal((4, 7, 8))
    dA, dB = oracle.contract_backward(A, B, dC)
    ref = (dC * (A @ B.transpose(0, 2, 1))).sum()
    assert abs((dA * A).sum() - ref) < 1e-10 * abs(ref)
    assert abs((dB * B).sum() - ref) < 1e-10 * abs(ref)


def test_layer_norm_backward_matches_torch():
    rng = np.random.default_rng(7)
    v = rng.standard_normal((20, 33)) * 3 + 1
    gamma, beta, dy = rng.standard_normal(33), rng.standard_normal(33), rng.standard_normal((20, 33))
    vt = torch.tensor(v, requires_grad=True)
    gt, bt = torch.tensor(gamma, requires_grad=True), torch.tensor(beta, requires_grad=True)
    (torch.nn.functional.layer_norm(vt, (33,), gt, bt, eps=1e-5) * torch.tensor(dy)).sum().backward()
    dv, dg, db = oracle.layer_norm_backward(dy, v, gamma)
    np.testing.assert_allclose(dv, vt.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("direction", DIRS)
def test_masked_pairs_get_exactly_zero_gradient(direction):
    z, mask, W, dout = setup(7, 4, 4, seed=8)
    g = oracle.tri_mul_backward(z, mask, W, direction, dout)
    dead = (mask[:, None] == 0) | (mask[None, :] == 0)
    assert dead.any()
    assert np.all(g["dz"][dead] == 0.0)
    assert np.abs(g["dz"][~dead]).max() > 0
