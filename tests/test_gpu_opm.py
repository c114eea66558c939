"""GPU parity of the outer product mean (include/opm.h) against the fp64
oracle (oracle.outer_product_mean / outer_product_mean_tile).

Tolerance (fp32 output): relative Frobenius error <= 1e-4 and max-abs error
<= 1e-4 * max|reference|.  Derivation: the products a_sic b_sjd of bf16
inputs are exact in fp32 and their sums over s carry fp32 rounding only
(relative ~1e-7 sqrt(S)); the epilogue feeds each mean into the projection
as bf16 hi + lo (relative truncation <= 2^-17 ~ 7.6e-6 per value) against
bf16 weights (exact), with fp32 accumulation.  With bf16 output one more
rounding (<= 2^-9 relative) is added: relative Frobenius <= 3e-3.  Pairs
whose tokens share no sequence get exactly the bias."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import errors, host, say

pytestmark = pytest.mark.gpu
D, CZ = 32, 128


def inputs(S, N, seed, masked):
    g = torch.Generator().manual_seed(seed)
    a = torch.randn((S, N, D), generator=g).to(torch.bfloat16)
    b = torch.randn((S, N, D), generator=g).to(torch.bfloat16)
    w = (torch.randn((CZ, D * D), generator=g) / D).to(torch.bfloat16)
    bo = torch.randn(CZ, generator=g).to(torch.bfloat16)
    mask = None
    if masked:
        mask = (torch.rand((S, N), generator=g) > 0.25).to(torch.uint8)
        if N > 3:
            mask[:, 3] = 0                      # token 3 absent everywhere: its pairs get the bias
    return a, b, mask, w, bo


def check(got, ref, what, rel_tol=1e-4, max_rel=1e-4):
    mx, rel = errors(got, ref)
    say(f"  {what}: rel_fro={rel:.3e} max_abs={mx:.3e} max|ref|={np.abs(ref).max():.3e}")
    assert np.all(np.isfinite(got)), what
    assert rel <= rel_tol, f"{what}: relative Frobenius error {rel:.3e} > {rel_tol}"
    if max_rel is not None:
        assert mx <= max_rel * np.abs(ref).max(), f"{what}: max-abs error {mx:.3e}"


@pytest.mark.parametrize("S,N,masked", [(1, 8, False), (37, 100, True), (300, 64, False), (64, 257, True)])
def test_opm_forward_matches_oracle(S, N, masked):
    say(f"opm forward S={S} N={N} masked={masked}")
    a, b, mask, w, bo = inputs(S, N, seed=S * 1000 + N, masked=masked)
    op = T.OuterProductMean(w, bo, out_dtype="f32")
    out = op.forward(a.cuda(), b.cuda(), None if mask is None else mask.cuda())
    torch.cuda.synchronize()
    ref = oracle.outer_product_mean(host(a), host(b), None if mask is None else mask.numpy(), host(w), host(bo))
    got = host(out)
    check(got, ref, "out")
    if masked and N > 3:
        assert np.array_equal(got[3], np.broadcast_to(host(bo), got[3].shape))
        assert np.array_equal(got[:, 3], np.broadcast_to(host(bo), got[:, 3].shape))


def test_opm_forward_bf16_output():
    S, N = 50, 96
    a, b, mask, w, bo = inputs(S, N, seed=7, masked=True)
    op = T.OuterProductMean(w, bo, out_dtype="bf16")
    out = op.forward(a.cuda(), b.cuda(), mask.cuda())
    torch.cuda.synchronize()
    ref = oracle.outer_product_mean(host(a), host(b), mask.numpy(), host(w), host(bo))
    check(host(out), ref, "out bf16", rel_tol=3e-3, max_rel=1e-2)


def test_opm_block_steps_reproduce_the_full_op():
    """2 x 2 pair tiles (ragged) and three sequence panels (ragged), each tile
    accumulating over the panels as the ring would."""
    S, N = 101, 150
    a, b, mask, w, bo = inputs(S, N, seed=11, masked=True)
    ad, bd, md = a.cuda(), b.cuda(), mask.cuda()
    op = T.OuterProductMean(w, bo, out_dtype="f32")
    ref = oracle.outer_product_mean(host(a), host(b), mask.numpy(), host(w), host(bo))
    cuts = [0, 40, 41, 101]
    for (r0, r1) in ((0, 77), (77, 150)):
        for (c0, c1) in ((0, 64), (64, 150)):
            acc = op.accumulator(r1 - r0, c1 - c0)
            out = torch.full((r1 - r0, c1 - c0, CZ), float("nan"), device="cuda")
            for k, (s0, s1) in enumerate(zip(cuts[:-1], cuts[1:])):
                v = T.OpmBlockView(N, S, r0, r1 - r0, c0, c1 - c0, s0, s1 - s0, k, len(cuts) - 1)
                op.block_accumulate(v, ad, bd, md, acc, out if k == len(cuts) - 2 else None)
            torch.cuda.synchronize()
            check(host(out), ref[r0:r1, c0:c1], f"tile rows {r0}:{r1} cols {c0}:{c1}")


def test_opm_one_panel_of_sequences_is_the_tile_oracle():
    S, N = 90, 70
    a, b, mask, w, bo = inputs(S, N, seed=13, masked=True)
    op = T.OuterProductMean(w, bo, out_dtype="f32")
    acc = op.accumulator(30, 45)
    out = torch.empty((30, 45, CZ), device="cuda")
    v = T.OpmBlockView(N, S, 20, 30, 10, 45, 33, 40, 0, 1)
    op.block_accumulate(v, a.cuda(), b.cuda(), mask.cuda(), acc, out)
    torch.cuda.synchronize()
    ref = oracle.outer_product_mean_tile(host(a), host(b), mask.numpy(), host(w), host(bo), 20, 30, 10, 45, 33, 40)
    check(host(out), ref, "tile with sequences 33:73")


def test_opm_n1024_s4096_sampled():
    """The benchmark size (N = 1024 tokens, S = 4096 sequences) in the launch
    configuration the benchmark times; blocks of pairs against the oracle's
    tile function."""
    S, N = 4096, 1024
    say(f"opm forward S={S} N={N} sampled")
    g = torch.Generator(device="cuda").manual_seed(4096)
    a = torch.randn((S, N, D), generator=g, device="cuda").to(torch.bfloat16)
    b = torch.randn((S, N, D), generator=g, device="cuda").to(torch.bfloat16)
    w = (torch.randn((CZ, D * D), generator=g, device="cuda") / D).to(torch.bfloat16)
    bo = torch.randn(CZ, generator=g, device="cuda").to(torch.bfloat16)
    op = T.OuterProductMean(w, bo, out_dtype="f32")
    out = op.forward(a, b, None)
    torch.cuda.synchronize()
    ah, bh, wh, boh = host(a), host(b), host(w), host(bo)
    for (r0, c0) in ((0, 0), (1020, 1016), (517, 3)):
        ref = oracle.outer_product_mean_tile(ah, bh, None, wh, boh, r0, 4, c0, 8)
        check(host(out[r0:r0 + 4, c0:c0 + 8]), ref, f"pairs {r0}:{r0 + 4} x {c0}:{c0 + 8}")


def test_opm_errors():
    a, b, mask, w, bo = inputs(4, 16, seed=1, masked=False)
    op = T.OuterProductMean(w, bo)
    acc = op.accumulator(8, 8)
    ad, bd = a.cuda(), b.cuda()
    n = T.opm_workspace_size(op.h, 8, 8, 4)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    out = torch.empty((8, 8, CZ), device="cuda")
    with pytest.raises(T.TriMulError) as e:         # tile past the tokens
        T.opm_block_accumulate(op.h, T.OpmBlockView(16, 4, 10, 8, 0, 8, 0, 4, 0, 1), ad, bd, None, acc, out, ws, n)
    assert e.value.code == T.TRI_MUL_EINVAL
    with pytest.raises(T.TriMulError) as e:         # workspace too small
        T.opm_block_accumulate(op.h, T.OpmBlockView(16, 4, 0, 8, 0, 8, 0, 4, 0, 1), ad, bd, None, acc, out, ws, n - 1)
    assert e.value.code == T.TRI_MUL_ENOMEM
    with pytest.raises(T.TriMulError) as e:         # step index out of range
        T.opm_block_accumulate(op.h, T.OpmBlockView(16, 4, 0, 8, 0, 8, 0, 4, 2, 2), ad, bd, None, acc, out, ws, n)
    assert e.value.code == T.TRI_MUL_EINVAL
    with pytest.raises(T.TriMulError) as e:         # last step without an output tile
        T.opm_block_accumulate(op.h, T.OpmBlockView(16, 4, 0, 8, 0, 8, 0, 4, 0, 1), ad, bd, None, acc, None, ws, n)
    assert e.value.code == T.TRI_MUL_EINVAL
