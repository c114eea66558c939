"""The panel layout conversion helpers of the binding follow the layout the
header documents (element (c, i, k) at ((c*T + i/256)*S + k/32)*8192 +
(i%256)*32 + k%32).  CPU only."""
import pytest
import torch

from paper_2603_14806_amd import trimul as T


@pytest.mark.parametrize("N", [1, 31, 33, 256, 300, 520])
def test_panel_index_formula(N):
    X = torch.arange(3 * N * N, dtype=torch.float64).reshape(3, N, N)
    P = T.dense_to_panel(X)
    Tn, S = -(-N // 256), -(-N // 32)
    assert P.numel() == 3 * Tn * 256 * S * 32
    for c in range(3):
        for i in {0, N // 2, N - 1, min(N - 1, 255)}:
            for k in {0, N // 3, N - 1, min(N - 1, 31)}:
                idx = ((c * Tn + i // 256) * S + k // 32) * 8192 + (i % 256) * 32 + k % 32
                assert P[idx] == X[c, i, k]
    assert torch.equal(T.panel_to_dense(P, N, 3), X)


@pytest.mark.parametrize("N", [1, 31, 33, 100])
def test_result_index_formula(N):
    c = 5
    X = torch.arange(c * N * N, dtype=torch.float64).reshape(c, N, N)
    R = T.dense_to_result(X)
    J = -(-N // 32)
    assert R.numel() == N * J * 32 * c
    for ch in range(c):
        for i in {0, N // 2, N - 1}:
            for j in {0, N // 3, N - 1}:
                assert R[((i * J + j // 32) * c + ch) * 32 + j % 32] == X[ch, i, j]
    assert torch.equal(T.result_to_dense(R, N, c), X)
