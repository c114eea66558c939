"""Pins of the triangle-attention oracle (oracle/triattn.py, Section 3.2,
Eq. 1) against things other than itself: brute-force Python loops, torch's
scaled_dot_product_attention (a different library routine) in fp64, closed
forms (uniform scores, one present key, a dominant bias), the softmax's
invariance to per-query shifts, key and query permutations, and the chunked
log-sum-exp merge against the plain softmax.  CPU only, fp64."""
import math

import numpy as np
import pytest
import torch

import oracle


def rand_case(rows, N, H, d, seed, masked=False):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((rows, N, H, d))
    k = rng.standard_normal((rows, N, H, d))
    v = rng.standard_normal((rows, N, H, d))
    b = rng.standard_normal((H, N, N))
    mask = None
    if masked:
        mask = (rng.random(N) > 0.3).astype(np.uint8)
        mask[0] = 1
    return q, k, v, b, mask


def test_brute_force_loops():
    rows, N, H, d = 2, 4, 2, 3
    q, k, v, b, mask = rand_case(rows, N, H, d, seed=1, masked=True)
    mask[2] = 0
    out = oracle.triangle_attention(q, k, v, b, mask)
    for i in range(rows):
        for h in range(H):
            for j in range(N):
                s = []
                for kk in range(N):
                    if mask[kk]:
                        dot = 0.0
                        for c in range(d):
                            dot += q[i, j, h, c] * k[i, kk, h, c]
                        s.append((kk, dot / math.sqrt(d) + b[h, j, kk]))
                top = max(x for _, x in s)
                den = sum(math.exp(x - top) for _, x in s)
                for c in range(d):
                    ref = sum(math.exp(x - top) / den * v[i, kk, h, c] for kk, x in s)
                    assert abs(out[i, j, h, c] - ref) < 1e-12, (i, j, h, c)


def test_matches_torch_sdpa_in_fp64():
    rows, N, H, d = 3, 9, 2, 8
    q, k, v, b, mask = rand_case(rows, N, H, d, seed=2, masked=True)
    bias = torch.tensor(b)[None].expand(rows, H, N, N).clone()
    bias[..., torch.tensor(mask) == 0] = -math.inf
    out = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).transpose(1, 2), torch.tensor(k).transpose(1, 2), torch.tensor(v).transpose(1, 2),
        attn_mask=bias).transpose(1, 2).numpy()
    np.testing.assert_allclose(oracle.triangle_attention(q, k, v, b, mask), out, rtol=1e-12, atol=1e-12)


def test_uniform_scores_average_the_present_values():
    rows, N, H, d = 2, 6, 2, 4
    _, k, v, _, mask = rand_case(rows, N, H, d, seed=3, masked=True)
    q = np.zeros((rows, N, H, d))
    b = np.zeros((H, N, N))
    out = oracle.triangle_attention(q, k, v, b, mask)
    ref = v[:, mask != 0].mean(axis=1)                      # [rows][H][d]
    np.testing.assert_allclose(out, np.broadcast_to(ref[:, None], out.shape), rtol=1e-13, atol=1e-13)


def test_one_present_key_and_no_key():
    rows, N, H, d = 2, 5, 3, 4
    q, k, v, b, _ = rand_case(rows, N, H, d, seed=4)
    mask = np.zeros(N, np.uint8)
    mask[3] = 1
    out = oracle.triangle_attention(q, k, v, b, mask)
    np.testing.assert_allclose(out, np.broadcast_to(v[:, 3:4], out.shape), rtol=1e-14, atol=1e-14)
    none = oracle.triangle_attention(q, k, v, b, np.zeros(N, np.uint8))
    assert np.array_equal(none, np.zeros_like(none))


def test_dominant_bias_selects_its_key():
    rows, N, H, d = 2, 6, 2, 3
    q, k, v, b, _ = rand_case(rows, N, H, d, seed=5)
    b = b * 0.1
    b[:, :, 4] += 200.0
    out = oracle.triangle_attention(q, k, v, b, None)
    np.testing.assert_allclose(out, np.broadcast_to(v[:, 4:5], out.shape), rtol=1e-12, atol=1e-12)


def test_per_query_bias_shift_changes_nothing():
    rows, N, H, d = 2, 7, 2, 4
    q, k, v, b, mask = rand_case(rows, N, H, d, seed=6, masked=True)
    shift = np.random.default_rng(7).standard_normal((H, N, 1)) * 5
    np.testing.assert_allclose(oracle.triangle_attention(q, k, v, b + shift, mask),
                               oracle.triangle_attention(q, k, v, b, mask), rtol=1e-11, atol=1e-12)


def test_key_and_query_permutations():
    rows, N, H, d = 2, 8, 2, 3
    q, k, v, b, mask = rand_case(rows, N, H, d, seed=8, masked=True)
    rng = np.random.default_rng(9)
    pk, pq = rng.permutation(N), rng.permutation(N)
    out = oracle.triangle_attention(q, k, v, b, mask)
    outk = oracle.triangle_attention(q, k[:, pk], v[:, pk], b[:, :, pk], mask[pk])
    np.testing.assert_allclose(outk, out, rtol=1e-12, atol=1e-12)
    outq = oracle.triangle_attention(q[:, pq], k, v, b[:, pq], mask)
    np.testing.assert_allclose(outq, out[:, pq], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("cuts", [[0, 10], [0, 1, 10], [0, 3, 4, 9, 10], [0, 5, 10]])
def test_chunked_merge_equals_the_plain_softmax(cuts):
    rows, N, H, d = 2, 10, 2, 4
    q, k, v, b, mask = rand_case(rows, N, H, d, seed=10, masked=True)
    mask[5:9] = 0                                           # a chunk with no present key
    np.testing.assert_allclose(oracle.chunked_attention(q, k, v, b, mask, cuts),
                               oracle.triangle_attention(q, k, v, b, mask), rtol=1e-12, atol=1e-13)
