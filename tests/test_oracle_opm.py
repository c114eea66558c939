"""Pins of the outer-product-mean oracle (oracle/opm.py, Section 3.5) against
things other than itself: brute-force Python loops, the closed form for one
sequence, the mean of identical sequences, exact results for masked inputs,
token-permutation equivariance, the channel-permutation and a/b-swap
identities, the split of the sequence sum into panels, and the tile view.
CPU only, fp64."""
import numpy as np
import pytest

import oracle


def rand_case(S, N, D, cz, seed, masked=False):
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((S, N, D))
    b = rng.standard_normal((S, N, D))
    w = rng.standard_normal((cz, D * D)) / D
    bo = rng.standard_normal(cz)
    mask = None
    if masked:
        mask = (rng.random((S, N)) > 0.3).astype(np.uint8)
    return a, b, mask, w, bo


def test_brute_force_loops():
    S, N, D, cz = 3, 4, 3, 5
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=1, masked=True)
    mask[:, 2] = 0                                  # token 2 absent everywhere: n = 0 rows
    out = oracle.outer_product_mean(a, b, mask, w, bo)
    for i in range(N):
        for j in range(N):
            n = 0
            for s in range(S):
                n += int(mask[s, i]) * int(mask[s, j])
            for e in range(cz):
                acc = 0.0
                for c in range(D):
                    for d in range(D):
                        t = 0.0
                        for s in range(S):
                            if mask[s, i] and mask[s, j]:
                                t += a[s, i, c] * b[s, j, d]
                        if n:
                            acc += w[e, c * D + d] * (t / n)
                ref = acc + bo[e]
                assert abs(out[i, j, e] - ref) < 1e-12 * max(1.0, abs(ref)), (i, j, e)


def test_one_sequence_is_the_outer_product():
    S, N, D, cz = 1, 5, 4, 6
    a, b, _, w, bo = rand_case(S, N, D, cz, seed=2)
    out = oracle.outer_product_mean(a, b, None, w, bo)
    for i in range(N):
        for j in range(N):
            ref = w @ np.outer(a[0, i], b[0, j]).reshape(-1) + bo
            np.testing.assert_allclose(out[i, j], ref, rtol=1e-13, atol=1e-13)


def test_identical_sequences_average_to_one():
    N, D, cz = 4, 3, 5
    a1, b1, _, w, bo = rand_case(1, N, D, cz, seed=3)
    a = np.repeat(a1, 7, axis=0)
    b = np.repeat(b1, 7, axis=0)
    np.testing.assert_allclose(oracle.outer_product_mean(a, b, None, w, bo),
                               oracle.outer_product_mean(a1, b1, None, w, bo), rtol=1e-13, atol=1e-13)


def test_all_masked_gives_the_bias_and_masked_entries_do_not_matter():
    S, N, D, cz = 5, 6, 4, 7
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=4, masked=True)
    out0 = oracle.outer_product_mean(a, b, np.zeros((S, N), np.uint8), w, bo)
    assert np.array_equal(out0, np.broadcast_to(bo, out0.shape))
    rng = np.random.default_rng(5)
    a2, b2 = a.copy(), b.copy()
    a2[mask == 0] = rng.standard_normal(a2[mask == 0].shape) * 100
    b2[mask == 0] = rng.standard_normal(b2[mask == 0].shape) * 100
    np.testing.assert_array_equal(oracle.outer_product_mean(a, b, mask, w, bo),
                                  oracle.outer_product_mean(a2, b2, mask, w, bo))


def test_all_present_mean_divides_by_the_sequence_count():
    S, N, D, cz = 6, 3, 2, 4
    a, b, _, w, bo = rand_case(S, N, D, cz, seed=6)
    total = np.einsum("sic,sjd->ijcd", a, b)        # independent of the oracle's matmul path
    ref = (total / S).reshape(N, N, D * D) @ w.T + bo
    np.testing.assert_allclose(oracle.outer_product_mean(a, b, None, w, bo), ref, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(oracle.pair_counts(None, S, N), np.full((N, N), float(S)))


def test_token_permutation_equivariance():
    S, N, D, cz = 4, 7, 3, 5
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=7, masked=True)
    p = np.random.default_rng(8).permutation(N)
    out = oracle.outer_product_mean(a, b, mask, w, bo)
    outp = oracle.outer_product_mean(a[:, p], b[:, p], mask[:, p], w, bo)
    np.testing.assert_allclose(outp, out[p][:, p], rtol=1e-13, atol=1e-13)


def test_channel_permutation_moves_into_the_projection():
    # permuting a's channels c and b's channels d is undone by permuting W_o's columns
    S, N, D, cz = 3, 4, 5, 6
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=9, masked=True)
    rng = np.random.default_rng(10)
    pc, pd = rng.permutation(D), rng.permutation(D)
    w3 = w.reshape(cz, D, D)
    wp = w3[:, pc][:, :, pd].reshape(cz, D * D)
    np.testing.assert_allclose(oracle.outer_product_mean(a[..., pc], b[..., pd], mask, wp, bo),
                               oracle.outer_product_mean(a, b, mask, w, bo), rtol=1e-12, atol=1e-12)


def test_swapping_a_and_b_transposes_pairs_and_the_flatten():
    S, N, D, cz = 3, 5, 3, 4
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=11, masked=True)
    wt = w.reshape(cz, D, D).transpose(0, 2, 1).reshape(cz, D * D)
    out = oracle.outer_product_mean(a, b, mask, w, bo)
    outs = oracle.outer_product_mean(b, a, mask, wt, bo)
    np.testing.assert_allclose(outs, out.transpose(1, 0, 2), rtol=1e-12, atol=1e-12)


def test_sequence_panels_combine_by_their_counts():
    # the ring accumulates sums and counts per panel; the mean is their ratio
    S, N, D, cz = 11, 4, 3, 5
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=12, masked=True)
    cuts = [0, 4, 5, 11]
    tot = np.zeros((N, N, D, D))
    cnt = np.zeros((N, N))
    for s0, s1 in zip(cuts[:-1], cuts[1:]):
        tot += oracle.outer_sum(a[s0:s1], b[s0:s1], (mask[s0:s1], mask[s0:s1]))
        cnt += oracle.pair_counts(mask[s0:s1], s1 - s0, N)
    inv = np.divide(1.0, cnt, out=np.zeros_like(cnt), where=cnt > 0)
    ref = (tot * inv[..., None, None]).reshape(N, N, D * D) @ w.T + bo
    np.testing.assert_allclose(oracle.outer_product_mean(a, b, mask, w, bo), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("row0,rows,col0,cols", [(0, 3, 2, 4), (5, 2, 0, 7), (1, 6, 1, 6)])
def test_tile_view_is_the_restriction(row0, rows, col0, cols):
    S, N, D, cz = 5, 7, 3, 4
    a, b, mask, w, bo = rand_case(S, N, D, cz, seed=13, masked=True)
    full = oracle.outer_product_mean(a, b, mask, w, bo)
    tile = oracle.outer_product_mean_tile(a, b, mask, w, bo, row0, rows, col0, cols)
    np.testing.assert_allclose(tile, full[row0:row0 + rows, col0:col0 + cols], rtol=1e-13, atol=1e-13)
