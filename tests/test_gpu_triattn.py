"""GPU parity of the triangle attention core (include/triattn.h) against the
fp64 oracle (oracle.triangle_attention / chunked_attention).

Tolerance (fp32 output): relative Frobenius error <= 1e-4 and max-abs error
<= 1e-4 * max|reference|.  Derivation: q . k of bf16 inputs is exact per
product in fp32 (sums of 32 terms carry ~1e-7 relative rounding); scale and
bias are added in fp32; exp is v_exp_f32 (about 1 ulp) of an fp32 argument,
so each weight carries ~|s| 2^-24 relative error; the weights enter the
P V product as bf16 hi + lo (relative truncation <= 2^-17 ~ 7.6e-6) against
bf16 values (exact), fp32 accumulation and normalisation.  With bf16 output
the weights enter the product as bf16 alone (<= 2^-9 relative each; since
the output is itself a weighted mean, these roundings are of the same
relative size in it as in the weights, ~1.1e-3 RMS) and the output is
rounded once more (<= 2^-9): ~1.6e-3 in quadrature, measured 2.0e-3 (1.7e-3
with hi + lo weights); relative Frobenius <= 3e-3."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import errors, host, say

pytestmark = pytest.mark.gpu


def inputs(rows, n, H, seed, masked, ld=None):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((rows, n, H, 32), generator=g).to(torch.bfloat16)
    k = torch.randn((rows, n, H, 32), generator=g).to(torch.bfloat16)
    v = torch.randn((rows, n, H, 32), generator=g).to(torch.bfloat16)
    ld = ld or (n + 7) // 8 * 8
    bfull = torch.zeros((H, n, ld), dtype=torch.bfloat16)
    bfull[:, :, :n] = torch.randn((H, n, n), generator=g).to(torch.bfloat16)
    mask = None
    if masked:
        mask = (torch.rand(n, generator=g) > 0.3).to(torch.uint8)
        mask[0] = 1
    return q, k, v, bfull, mask


def check(got, ref, what, rel_tol=1e-4, max_rel=1e-4):
    mx, rel = errors(got, ref)
    say(f"  {what}: rel_fro={rel:.3e} max_abs={mx:.3e} max|ref|={np.abs(ref).max():.3e}")
    assert np.all(np.isfinite(got)), what
    assert rel <= rel_tol, f"{what}: relative Frobenius error {rel:.3e} > {rel_tol}"
    if max_rel is not None:
        assert mx <= max_rel * np.abs(ref).max(), f"{what}: max-abs error {mx:.3e}"


def dev(*ts):
    return [None if t is None else t.cuda() for t in ts]


# n = 129 and 257 end with a one-key chunk on a tile's last bias row: a bias
# range ending inside a dword once dropped that key (regression case)
@pytest.mark.parametrize("rows,n,H,masked", [(2, 64, 4, False), (3, 100, 4, True), (1, 257, 2, True),
                                             (2, 130, 1, False), (1, 129, 1, False)])
def test_triangle_attention_matches_oracle(rows, n, H, masked):
    say(f"triangle attention rows={rows} n={n} H={H} masked={masked}")
    q, k, v, bfull, mask = inputs(rows, n, H, seed=rows * 1000 + n, masked=masked)
    qd, kd, vd, bd, md = dev(q, k, v, bfull, mask)
    out = T.triangle_attention(qd, kd, vd, bd[:, :, :n], md)
    torch.cuda.synchronize()
    ref = oracle.triangle_attention(host(q), host(k), host(v), host(bfull[:, :, :n]),
                                    None if mask is None else mask.numpy())
    check(host(out), ref, "out")


def test_triangle_attention_bf16_output_and_no_keys():
    rows, n, H = 2, 96, 4
    q, k, v, bfull, mask = inputs(rows, n, H, seed=5, masked=True)
    qd, kd, vd, bd, md = dev(q, k, v, bfull, mask)
    out = T.triangle_attention(qd, kd, vd, bd, md, out_dtype="bf16")
    torch.cuda.synchronize()
    ref = oracle.triangle_attention(host(q), host(k), host(v), host(bfull), mask.numpy())
    check(host(out), ref, "out bf16", rel_tol=3e-3, max_rel=1e-2)
    none = T.triangle_attention(qd, kd, vd, bd, torch.zeros(n, dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    assert torch.count_nonzero(none).item() == 0


@pytest.mark.parametrize("cuts", [[0, 64, 128, 200], [0, 40, 104, 200], [0, 200], [0, 8, 200]])
def test_chunked_steps_merge_exactly(cuts):
    rows, n, H = 2, 200, 4
    q, k, v, bfull, mask = inputs(rows, n, H, seed=9, masked=True)
    mask[130:180] = 0                                  # a chunk of [104, 200) partly empty
    qd, kd, vd, bd, md = dev(q, k, v, bfull, mask)
    view = T.TriAttnView(rows, n, H, T.TRI_MUL_F32, bfull.shape[2], 0, n, 0, 1)
    state = torch.full((T.tri_attn_state_size(view) // 4,), float("nan"), device="cuda")
    out = torch.empty((rows, n, H, 32), device="cuda")
    for t, (k0, k1) in enumerate(zip(cuts[:-1], cuts[1:])):
        v_t = T.TriAttnView(rows, n, H, T.TRI_MUL_F32, bfull.shape[2], k0, k1 - k0, t, len(cuts) - 1)
        T.tri_attn_chunk(v_t, qd, kd, vd, bd, md, state, out)
    torch.cuda.synchronize()
    ref = oracle.triangle_attention(host(q), host(k), host(v), host(bfull[:, :, :n]), mask.numpy())
    check(host(out), ref, f"chunks {cuts}")


def test_triangle_attention_n2048_sampled_rows():
    """The benchmark size (rows = n = 2048, 4 heads) in the launch
    configuration the benchmark times; two sampled rows against the oracle."""
    rows, n, H = 2048, 2048, 4
    say(f"triangle attention rows={rows} n={n} H={H} sampled")
    g = torch.Generator(device="cuda").manual_seed(2048)
    q = torch.randn((rows, n, H, 32), generator=g, device="cuda").to(torch.bfloat16)
    k = torch.randn((rows, n, H, 32), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((rows, n, H, 32), generator=g, device="cuda").to(torch.bfloat16)
    b = torch.randn((H, n, n), generator=g, device="cuda").to(torch.bfloat16)
    out = T.triangle_attention(q, k, v, b, None)
    torch.cuda.synchronize()
    for i in (0, 1537):
        ref = oracle.triangle_attention(host(q[i:i + 1]), host(k[i:i + 1]), host(v[i:i + 1]), host(b), None)
        check(host(out[i:i + 1]), ref, f"row {i}")


def test_triangle_attention_errors():
    rows, n, H = 1, 64, 4
    q, k, v, bfull, _ = inputs(rows, n, H, seed=1, masked=False)
    qd, kd, vd, bd = dev(q, k, v, bfull)
    out = torch.empty((rows, n, H, 32), device="cuda")
    with pytest.raises(T.TriMulError) as e:          # bias row stride not a multiple of 8
        T.tri_attn_forward(qd, kd, vd, bd, None, rows, n, H, 60, "f32", out)
    assert e.value.code == T.TRI_MUL_EINVAL
    with pytest.raises(T.TriMulError) as e:          # k0 not a multiple of 8
        T.tri_attn_chunk(T.TriAttnView(rows, n, H, T.TRI_MUL_F32, n, 4, 60, 1, 2), qd, kd, vd, bd, None,
                         torch.empty(1 << 16, device="cuda"), out)
    assert e.value.code == T.TRI_MUL_EINVAL
    with pytest.raises(T.TriMulError) as e:          # a chunked attention without a state
        T.tri_attn_chunk(T.TriAttnView(rows, n, H, T.TRI_MUL_F32, n, 0, 32, 0, 2), qd, kd, vd, bd, None, None, out)
    assert e.value.code == T.TRI_MUL_EINVAL


@pytest.mark.parametrize("cuts", [[0, 64, 128, 200], [0, 8, 200]])
def test_chunked_steps_bf16_output(cuts):
    """The ring's chunk merge with bf16 output (the weights enter the PV
    product as bf16 alone in every chunk; the merge state stays fp32): the
    bf16 bar of a single call."""
    rows, n, H = 2, 200, 4
    q, k, v, bfull, mask = inputs(rows, n, H, seed=13, masked=True)
    mask[130:180] = 0
    qd, kd, vd, bd, md = dev(q, k, v, bfull, mask)
    view = T.TriAttnView(rows, n, H, T.TRI_MUL_BF16, bfull.shape[2], 0, n, 0, 1)
    state = torch.full((T.tri_attn_state_size(view) // 4,), float("nan"), device="cuda")
    out = torch.empty((rows, n, H, 32), dtype=torch.bfloat16, device="cuda")
    for t, (k0, k1) in enumerate(zip(cuts[:-1], cuts[1:])):
        v_t = T.TriAttnView(rows, n, H, T.TRI_MUL_BF16, bfull.shape[2], k0, k1 - k0, t, len(cuts) - 1)
        T.tri_attn_chunk(v_t, qd, kd, vd, bd, md, state, out)
    torch.cuda.synchronize()
    ref = oracle.triangle_attention(host(q), host(k), host(v), host(bfull[:, :, :n]), mask.numpy())
    check(host(out), ref, f"bf16 chunks {cuts}", rel_tol=3e-3, max_rel=1e-2)
