"""Pins of the fp64 oracle against things other than itself: brute force on
tiny inputs, library routines for single stages, closed forms, and the
invariants the definition (Section 3.3, Eq. 2/3) implies.  CPU only."""
import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle import f64
from paper_2603_14806_amd import synth
from tests.brute_force import brute_tri_mul

DIRS = ("outgoing", "incoming")


def rand_weights(c_z, c, seed, affine=True):
    W = synth.weights(c_z, c, dtype="f32", seed=seed, affine=affine)
    return {k: f64(v) for k, v in W.items()}


def rand_z(N, c_z, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal((N, N, c_z)) * scale


def as_lists(W):
    return {k: v.tolist() for k, v in W.items()}


# ---------------------------------------------------------------- stage pins

def test_layer_norm_matches_torch():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((50, 37)) * rng.uniform(1e-4, 10, size=(50, 1)) + rng.standard_normal((50, 1))
    v[0] = 3.0                      # zero variance: eps decides the result
    v[1] = 1e-3 * rng.standard_normal(37)  # variance ~ eps
    gamma, beta = rng.standard_normal(37), rng.standard_normal(37)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(v), (37,), torch.from_numpy(gamma),
                                         torch.from_numpy(beta), eps=1e-5).numpy()
    np.testing.assert_allclose(oracle.layer_norm(v, gamma, beta), ref, rtol=1e-12, atol=1e-12)


def test_sigmoid_matches_expit():
    t = np.concatenate([np.linspace(-800, 800, 2001), np.random.default_rng(2).standard_normal(1000) * 5])
    np.testing.assert_allclose(oracle.sigmoid(t), scipy.special.expit(t), rtol=1e-14, atol=1e-300)


def test_layer_norm_hand_value():
    # (1,2,3,4): mean 2.5, biased variance 1.25.
    out = oracle.layer_norm(np.array([1.0, 2.0, 3.0, 4.0]), np.ones(4), np.zeros(4))
    s = np.sqrt(1.25 + 1e-5)
    np.testing.assert_allclose(out, np.array([-1.5, -0.5, 0.5, 1.5]) / s, rtol=1e-15)


def test_project_identity_weights_hand_value():
    # W_a = I, W_ga = 0 -> a = 0.5 * m * LN(z); W_b = -I, W_gb = 0 -> b = -a.
    c = 4
    W = {"ln_in_w": np.ones(c), "ln_in_b": np.zeros(c), "w_a": np.eye(c),
         "w_ga": np.zeros((c, c)), "w_b": -np.eye(c), "w_gb": np.zeros((c, c)),
         "w_g": np.zeros((c, c))}
    z = np.array([[1.0, 2.0, 3.0, 4.0]])
    a, b, g = oracle.project(z, np.array([1.0]), W)
    ln = np.array([-1.5, -0.5, 0.5, 1.5]) / np.sqrt(1.25 + 1e-5)
    np.testing.assert_allclose(a[0], 0.5 * ln, rtol=1e-15)
    np.testing.assert_allclose(b[0], -0.5 * ln, rtol=1e-15)
    np.testing.assert_allclose(g[0], 0.5 * np.ones(c), rtol=0)
    a0, _, _ = oracle.project(z, np.array([0.0]), W)
    assert np.all(a0 == 0)


# ------------------------------------------------------------- brute force

@pytest.mark.parametrize("N,c_z,c", [(1, 4, 4), (2, 4, 4), (3, 4, 8), (5, 8, 4), (4, 8, 8)])
@pytest.mark.parametrize("direction", DIRS)
def test_brute_force_tiny(N, c_z, c, direction):
    W = rand_weights(c_z, c, seed=10 + N + c_z + c)
    z = rand_z(N, c_z, seed=N * 7 + c)
    mask = np.ones(N)
    if N >= 3:
        mask[N - 1] = 0
    ref = np.array(brute_tri_mul(z.tolist(), mask.tolist(), as_lists(W), direction))
    got = oracle.tri_mul(z, mask, W, direction)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)


def test_brute_force_c128_n2():
    W = rand_weights(128, 128, seed=3)
    z = rand_z(2, 128, seed=4)
    mask = np.ones(2)
    for d in DIRS:
        ref = np.array(brute_tri_mul(z.tolist(), mask.tolist(), as_lists(W), d))
        np.testing.assert_allclose(oracle.tri_mul(z, mask, W, d), ref, rtol=1e-10, atol=1e-12)


def test_sampled_rows_cols_equal_full():
    N, W = 9, rand_weights(8, 8, seed=5)
    z = rand_z(N, 8, seed=6)
    mask = np.ones(N)
    mask[7] = 0
    rows, cols = np.array([0, 3, 7, 8]), np.array([8, 1, 2])
    for d in DIRS:
        full = oracle.tri_mul(z, mask, W, d)
        np.testing.assert_allclose(oracle.tri_mul(z, mask, W, d, rows, cols),
                                   full[np.ix_(rows, cols)], rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------- closed forms

def test_n1_outgoing_equals_incoming():
    W = rand_weights(8, 8, seed=7)
    z = rand_z(1, 8, seed=8)
    a, b, g = oracle.project(z, np.ones((1, 1)), W)
    C = oracle.contract_outgoing(a, b)
    np.testing.assert_array_equal(C, a * b)
    np.testing.assert_array_equal(oracle.tri_mul(z, np.ones(1), W, "outgoing"),
                                  oracle.tri_mul(z, np.ones(1), W, "incoming"))


@pytest.mark.parametrize("n_valid", [1, 3, 6])
def test_constant_z(n_valid):
    """z_ij = v for all pairs: C_ij = n * (a* . b*) on valid pairs, so the
    output is g* . W_o LN_out(n a* . b*) there and 0 elsewhere; both
    directions agree exactly."""
    N, cz = 6, 8
    W = rand_weights(cz, cz, seed=9)
    v = np.random.default_rng(10).standard_normal(cz)
    z = np.broadcast_to(v, (N, N, cz)).copy()
    mask = np.zeros(N)
    mask[:n_valid] = 1
    a1, b1, g1 = oracle.project(v[None], np.ones(1), W)
    m = oracle.pair_mask(mask)
    a, b, _ = oracle.project(z, m, W)
    for d, contract in (("outgoing", oracle.contract_outgoing),
                        ("incoming", lambda x, y: oracle.contract_incoming(x, y))):
        C = contract(a, b)
        expect_C = m[..., None] * (n_valid * a1[0] * b1[0])
        np.testing.assert_allclose(C, expect_C, rtol=1e-13, atol=1e-15)
    y = oracle.linear(oracle.layer_norm(n_valid * a1[0] * b1[0], W["ln_out_w"], W["ln_out_b"]), W["w_o"])
    expect = m[..., None] * (g1[0] * y)
    for d in DIRS:
        np.testing.assert_allclose(oracle.tri_mul(z, mask, W, d), expect, rtol=1e-12, atol=1e-14)


def test_row_constant_z_separates_directions():
    """z_ij = u_i: outgoing C_ij = N a(u_i) . b(u_j) (rank-one per channel),
    incoming C_ij = sum_k a(u_k) . b(u_k), the same for every pair."""
    N, cz = 5, 8
    W = rand_weights(cz, cz, seed=11)
    u = np.random.default_rng(12).standard_normal((N, cz))
    z = np.repeat(u[:, None, :], N, axis=1)
    au, bu, _ = oracle.project(u, np.ones(N), W)
    a, b, _ = oracle.project(z, np.ones((N, N)), W)
    C_out = oracle.contract_outgoing(a, b)
    np.testing.assert_allclose(C_out, N * au[:, None, :] * bu[None, :, :], rtol=1e-12, atol=1e-14)
    C_in = oracle.contract_incoming(a, b)
    np.testing.assert_allclose(C_in, np.broadcast_to((au * bu).sum(0), C_in.shape), rtol=1e-12, atol=1e-14)


def test_zero_cases():
    N, cz = 6, 8
    W = rand_weights(cz, cz, seed=13, affine=False)
    z = rand_z(N, cz, seed=14)
    for d in DIRS:
        assert np.all(oracle.tri_mul(z, np.zeros(N), W, d) == 0)
    W0 = dict(W, w_a=np.zeros_like(W["w_a"]))
    for d in DIRS:
        assert np.all(oracle.tri_mul(z, np.ones(N), W0, d) == 0)


# --------------------------------------------------------------- invariants

def swapped(W):
    return dict(W, w_a=W["w_b"], w_ga=W["w_gb"], w_b=W["w_a"], w_gb=W["w_ga"])


def test_incoming_is_transposed_outgoing_with_swapped_weights():
    N, cz = 7, 8
    W = rand_weights(cz, cz, seed=15)
    z = rand_z(N, cz, seed=16)
    mask = np.ones(N)
    mask[2] = 0
    zt = z.transpose(1, 0, 2)
    inc = oracle.tri_mul(z, mask, W, "incoming")
    out_t = oracle.tri_mul(zt, mask, swapped(W), "outgoing").transpose(1, 0, 2)
    np.testing.assert_allclose(inc, out_t, rtol=1e-12, atol=1e-14)
    # The contraction alone needs no weight swap: C_in(z) = C_out(z^T).
    m = oracle.pair_mask(mask)
    a, b, _ = oracle.project(z, m, W)
    at, bt, _ = oracle.project(zt, m, W)
    np.testing.assert_allclose(oracle.contract_incoming(a, b), oracle.contract_outgoing(at, bt),
                               rtol=1e-12, atol=1e-14)


def test_same_weight_form_fails_in_general():
    """incoming(z) == outgoing(z^T) with unchanged weights does not hold for a
    full layer: the output gate reads z_ij, not z_ji."""
    N, cz = 6, 8
    W = rand_weights(cz, cz, seed=17)
    z = rand_z(N, cz, seed=18)
    inc = oracle.tri_mul(z, np.ones(N), W, "incoming")
    out = oracle.tri_mul(z.transpose(1, 0, 2), np.ones(N), W, "outgoing")
    assert np.max(np.abs(inc - out)) > 1e-3


@pytest.mark.parametrize("direction", DIRS)
def test_token_permutation_equivariance(direction):
    N, cz = 8, 8
    W = rand_weights(cz, cz, seed=19)
    z = rand_z(N, cz, seed=20)
    mask = np.ones(N)
    mask[[1, 5]] = 0
    P = np.random.default_rng(21).permutation(N)
    out = oracle.tri_mul(z, mask, W, direction)
    outp = oracle.tri_mul(z[np.ix_(P, P)], mask[P], W, direction)
    np.testing.assert_allclose(outp, out[np.ix_(P, P)], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("direction", DIRS)
def test_padding_invariance_bitwise(direction):
    N, cz = 9, 8
    W = rand_weights(cz, cz, seed=22)
    z = rand_z(N, cz, seed=23)
    mask = np.ones(N)
    mask[6:] = 0
    z2 = z.copy()
    z2[6:, :, :] = 100 * rand_z(N, cz, seed=24)[6:]
    z2[:, 6:, :] = -50 * rand_z(N, cz, seed=25)[:, 6:]
    o1 = oracle.tri_mul(z, mask, W, direction)
    o2 = oracle.tri_mul(z2, mask, W, direction)
    np.testing.assert_array_equal(o1[:6, :6], o2[:6, :6])
    assert np.all(o2[6:] == 0) and np.all(o2[:, 6:] == 0)


@pytest.mark.parametrize("direction", DIRS)
def test_hidden_channel_permutation_invariance(direction):
    N, cz, c = 6, 8, 8
    W = rand_weights(cz, c, seed=26)
    z = rand_z(N, cz, seed=27)
    P = np.random.default_rng(28).permutation(c)
    Wp = dict(W, w_a=W["w_a"][P], w_ga=W["w_ga"][P], w_b=W["w_b"][P], w_gb=W["w_gb"][P],
              ln_out_w=W["ln_out_w"][P], ln_out_b=W["ln_out_b"][P], w_o=W["w_o"][:, P])
    np.testing.assert_allclose(oracle.tri_mul(z, np.ones(N), Wp, direction),
                               oracle.tri_mul(z, np.ones(N), W, direction), rtol=1e-11, atol=1e-13)


def test_symmetric_z_equal_weights():
    N, cz = 7, 8
    W = rand_weights(cz, cz, seed=29)
    W = dict(W, w_b=W["w_a"], w_gb=W["w_ga"])
    z = rand_z(N, cz, seed=30)
    z = z + z.transpose(1, 0, 2)
    out = oracle.tri_mul(z, np.ones(N), W, "outgoing")
    inc = oracle.tri_mul(z, np.ones(N), W, "incoming")
    np.testing.assert_allclose(out, out.transpose(1, 0, 2), rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out, inc, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("direction", DIRS)
@pytest.mark.parametrize("N,g", [(12, 3), (10, 2)])
def test_block_decomposition_matches_full(direction, N, g):
    """Each tile (r, c) of a g x g grid, accumulated over g k-panels and
    finished by the tile epilogue, reproduces the full update on that tile."""
    cz = 8
    W = rand_weights(cz, cz, seed=31)
    z = rand_z(N, cz, seed=32)
    mask = np.ones(N)
    mask[-2:] = 0
    full = oracle.tri_mul(z, mask, W, direction)
    A, B = oracle.projected_panels(z, mask, W, direction)       # [c][N][N]
    b = N // g
    edges = [(t * b, (t + 1) * b) for t in range(g)]
    for r0, r1 in edges:
        for c0, c1 in edges:
            ap = [A[:, r0:r1, k0:k1] for k0, k1 in edges]
            bp = [B[:, c0:c1, k0:k1] for k0, k1 in edges]
            km = [np.ones(k1 - k0) for k0, k1 in edges]
            C = oracle.block_contract(ap, bp, km)
            out = oracle.block_epilogue(C, z[r0:r1, c0:c1], mask[r0:r1], mask[c0:c1], W)
            np.testing.assert_allclose(out, full[r0:r1, c0:c1], rtol=1e-12, atol=1e-14)


def test_block_kmask_drops_masked_k():
    rng = np.random.default_rng(33)
    ap = [rng.standard_normal((3, 4, 5)), rng.standard_normal((3, 4, 6))]
    bp = [rng.standard_normal((3, 2, 5)), rng.standard_normal((3, 2, 6))]
    km = [np.array([1, 0, 1, 1, 0]), np.array([0, 0, 0, 0, 0, 1])]
    C = oracle.block_contract(ap, bp, km)
    for i in range(4):
        for j in range(2):
            for c in range(3):
                s = sum(ap[0][c, i, k] * bp[0][c, j, k] for k in (0, 2, 3)) + ap[1][c, i, 5] * bp[1][c, j, 5]
                assert abs(C[i, j, c] - s) < 1e-12


def test_sampling_from_torch_input_matches_numpy():
    N = 10
    W = rand_weights(8, 8, seed=34)
    z = rand_z(N, 8, seed=35)
    rows, cols = np.array([9, 0, 4]), np.array([2, 7])
    for d in DIRS:
        np.testing.assert_array_equal(oracle.tri_mul(torch.from_numpy(z), np.ones(N), W, d, rows, cols),
                                      oracle.tri_mul(z, np.ones(N), W, d, rows, cols))
