"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Sizes here let the oracle compute every output; they span several tiles of
every kernel and ragged tails (N not a multiple of 8, 64 or 256)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import synth
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import TOL, assert_close, errors, host, make_layer, needs_gpu, say

pytestmark = [pytest.mark.gpu, needs_gpu]
DIRS = ("outgoing", "incoming")


# ------------------------------------------------------------ contraction

@pytest.mark.parametrize("dtype,N", [("bf16", 64), ("bf16", 264), ("bf16", 300), ("bf16", 520), ("f32", 65), ("f32", 130)])
def test_contract_exact_on_integers(dtype, N):
    """Small-integer operands make every product and partial sum exact in
    fp32, so the kernel must match the fp64 contraction bit for bit (this also
    pins the matrix-core operand and accumulator layouts)."""
    say(f"contract exact dtype={dtype} N={N}")
    layer, _ = make_layer(dtype)
    g = torch.Generator().manual_seed(N)
    A = torch.randint(-4, 5, (128, N, N), generator=g).to(synth.DTYPES[dtype])
    B = torch.randint(-4, 5, (128, N, N), generator=g).to(synth.DTYPES[dtype])
    C = layer.contract(T.dense_to_panel(A).cuda(), T.dense_to_panel(B).cuda(), N)
    torch.cuda.synchronize()
    ref = oracle.block_contract([host(A)], [host(B)], [np.ones(N)])    # [i][j][c]
    np.testing.assert_array_equal(host(T.result_to_dense(C, N)).transpose(1, 2, 0), ref)


@pytest.mark.parametrize("N", [64, 300, 520])
def test_contract_transposed_exact_on_integers(N):
    """tri_mul_contract_transposed takes the operands transposed (A_c^T,
    B_c^T in the panel layout): on small integers it must give the fp64
    contraction of A and B bit for bit."""
    say(f"contract transposed exact N={N}")
    layer, _ = make_layer("bf16")
    g = torch.Generator().manual_seed(N + 1)
    A = torch.randint(-4, 5, (128, N, N), generator=g).to(torch.bfloat16)
    B = torch.randint(-4, 5, (128, N, N), generator=g).to(torch.bfloat16)
    AT = T.dense_to_panel(A.transpose(1, 2).contiguous()).cuda()
    BT = T.dense_to_panel(B.transpose(1, 2).contiguous()).cuda()
    C = layer.contract_transposed(AT, BT, N)
    torch.cuda.synchronize()
    ref = oracle.block_contract([host(A)], [host(B)], [np.ones(N)])    # [i][j][c]
    np.testing.assert_array_equal(host(T.result_to_dense(C, N)).transpose(1, 2, 0), ref)


@pytest.mark.parametrize("N", [65, 300, 1000])
@pytest.mark.parametrize("direction", DIRS)
def test_contract_transposed_from_opposite_projection_is_bitwise_plain(N, direction):
    """The projection with the opposite direction writes the direction's
    operands transposed; contracting those with tri_mul_contract_transposed
    (the full calls' order) equals tri_mul_contract of the direction's own
    panels bit for bit, and the full call's output equals the stage calls'."""
    say(f"contract transposed == plain N={N} {direction}")
    layer, _ = make_layer("bf16", affine=True, seed=5)
    z = synth.pair_tensor(N, dtype="bf16", seed=5, device="cuda")
    mask = synth.random_mask(N, 0.9, sub=2).cuda()
    other = "incoming" if direction == "outgoing" else "outgoing"
    A, B = layer.project(z, mask, direction)
    AT, BT = layer.project(z, mask, other)
    C = layer.contract(A, B, N)
    CT = layer.contract_transposed(AT, BT, N)
    out_stage = layer.epilogue(CT, z, mask)
    out_full = layer(z, mask, direction)
    torch.cuda.synchronize()
    assert torch.equal(T.result_to_dense(C, N), T.result_to_dense(CT, N))
    assert torch.equal(T.panel_to_dense(AT, N), T.panel_to_dense(A, N).transpose(1, 2))
    assert torch.equal(out_stage, out_full)


def test_contract_transposed_errors():
    layer, _ = make_layer("bf16")
    N = 64
    buf = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    L = T.lib()
    s = torch.cuda.current_stream().cuda_stream
    assert L.tri_mul_contract_transposed(layer.h, None, buf.data_ptr(), N, buf.data_ptr(), s) == T.TRI_MUL_EINVAL
    assert L.tri_mul_contract_transposed(layer.h, buf.data_ptr() + 4, buf.data_ptr(), N, buf.data_ptr(), s) == T.TRI_MUL_EINVAL
    assert L.tri_mul_contract_transposed(layer.h, buf.data_ptr(), buf.data_ptr(), 0, buf.data_ptr(), s) == T.TRI_MUL_EINVAL
    f32, _ = make_layer("f32")
    assert L.tri_mul_contract_transposed(f32.h, buf.data_ptr(), buf.data_ptr(), N, buf.data_ptr(), s) == T.TRI_MUL_EUNSUPPORTED
    assert "bf16" in T.last_error()
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype,use_ws", [("bf16", False), ("bf16", True), ("f32", False), ("f32", True)])
def test_block_accumulate_kmask_exact(dtype, use_ws):
    """Two k-panels with a token mask over k, ragged tile (300 x 200) and
    panel lengths (130, 77) with padded row strides: overwrite on the first
    panel, accumulate on the second, exact on integer data; both entry
    points (with use_ws the panels are repacked into the workspace)."""
    say(f"block accumulate exact dtype={dtype} ws={use_ws}")
    layer, W = make_layer(dtype)
    rows, cols, n_total = 300, 200, 1000
    g = torch.Generator().manual_seed(7)
    mask = (torch.rand(n_total, generator=g) < 0.8).to(torch.uint8)
    mask_d = mask.cuda()
    acc = torch.full((128, rows, cols), float("nan"), device="cuda")
    ks = [(100, 130), (500, 77)]
    aps, bps = [], []
    for idx, (k0, klen) in enumerate(ks):
        ld = (klen + 7) // 8 * 8 + 8
        ap = torch.randint(-4, 5, (128, rows, ld), generator=g).to(synth.DTYPES[dtype])
        bp = torch.randint(-4, 5, (128, cols, ld), generator=g).to(synth.DTYPES[dtype])
        # padding columns hold garbage the kernel must ignore
        ap[:, :, klen:] = 1e4
        bp[:, :, klen:] = float("nan")
        aps.append(ap[:, :, :klen])
        bps.append(bp[:, :, :klen])
        v = T.BlockView(n_total, 700, 10, rows, cols, k0, klen, ld, ld, idx, 3)
        ws = None
        if use_ws:   # a fresh workspace full of garbage for every panel
            ws = torch.full((max(layer.block_workspace_size(v), 1),), 0xff, dtype=torch.uint8, device="cuda")
        layer.block_accumulate(v, ap.cuda(), bp.cuda(), acc, mask_d, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.block_contract([host(a) for a in aps], [host(b) for b in bps],
                                [host(mask[k0:k0 + kl]) for k0, kl in ks])
    np.testing.assert_array_equal(host(acc).transpose(1, 2, 0), ref)


def test_block_accumulate_ws_errors():
    """The workspace entry points reject a short or misaligned workspace (and
    a bad CU reserve) before launching anything."""
    layer, _ = make_layer("bf16")
    rows, cols, klen, ld = 64, 40, 50, 56
    ap = torch.zeros((128, rows, ld), dtype=torch.bfloat16, device="cuda")
    bp = torch.zeros((128, cols, ld), dtype=torch.bfloat16, device="cuda")
    acc = torch.zeros((128, rows, cols), device="cuda")
    v = T.BlockView(200, 0, 0, rows, cols, 0, klen, ld, ld, 0, 2)
    need = layer.block_workspace_size(v)
    # one 256-row tile and two k-steps per operand, then the staged k-mask (64 bytes, 256-byte aligned)
    assert need == 128 * 1 * 2 * 16384 * 2 + 256
    ws = torch.empty(need + 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_block_accumulate_ws(layer.h, v, ap, bp, acc, None, None, None, ws, need - 1)
    assert e.value.code == T.TRI_MUL_ENOMEM
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_block_accumulate_ws(layer.h, v, ap, bp, acc, None, None, None, ws[16:], need)
    assert e.value.code == T.TRI_MUL_EINVAL
    # the split form: the same workspace checks, a packed accumulator of
    # rows * ceil(cols / 32) * 32 * 128 floats, and the CU reserve's range
    assert layer.block_accumulator_size(v) == rows * 64 * 128 * 4
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_block_repack(layer.h, v, ap, bp, None, ws, need - 1)
    assert e.value.code == T.TRI_MUL_ENOMEM
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_block_accumulate_packed(layer.h, v, ws, need, acc, None, None, None, reserve_cus=-1)
    assert e.value.code == T.TRI_MUL_EINVAL
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_block_accumulate_packed(layer.h, v, ws[16:], need, acc, None, None, None)
    assert e.value.code == T.TRI_MUL_EINVAL


@pytest.mark.parametrize("use_ws", [False, True])
def test_block_accumulate_no_mask_ignores_padding(use_ws):
    """Without a token mask the contraction must still ignore the padding
    columns past klen of row-major panels (NaN and huge values here), in the
    last, ragged k-step that loads them; three panels, one shorter than a
    k-step, exact on integer data (bf16)."""
    say("block accumulate without mask, garbage padding")
    layer, _ = make_layer("bf16")
    rows, cols, n_total = 260, 33, 600
    g = torch.Generator().manual_seed(11)
    acc = torch.full((128, rows, cols), float("nan"), device="cuda")
    ks = [(0, 61), (61, 20), (81, 100)]
    aps, bps = [], []
    for idx, (k0, klen) in enumerate(ks):
        ld = (klen + 7) // 8 * 8 + 16
        ap = torch.randint(-4, 5, (128, rows, ld), generator=g).to(torch.bfloat16)
        bp = torch.randint(-4, 5, (128, cols, ld), generator=g).to(torch.bfloat16)
        ap[:, :, klen:] = float("nan")
        bp[:, :, klen:] = -3e38
        aps.append(ap[:, :, :klen])
        bps.append(bp[:, :, :klen])
        v = T.BlockView(n_total, 100, 300, rows, cols, k0, klen, ld, ld, idx, len(ks) + 1)   # no epilogue
        ws = None
        if use_ws:
            ws = torch.full((layer.block_workspace_size(v),), 0xff, dtype=torch.uint8, device="cuda")
        layer.block_accumulate(v, ap.cuda(), bp.cuda(), acc, None, ws=ws)
    torch.cuda.synchronize()
    ref = oracle.block_contract([host(a) for a in aps], [host(b) for b in bps], [np.ones(kl) for _, kl in ks])
    np.testing.assert_array_equal(host(acc).transpose(1, 2, 0), ref)


# ------------------------------------------------------------- projection

@pytest.mark.parametrize("dtype,N", [("bf16", 72), ("bf16", 300), ("f32", 65)])
@pytest.mark.parametrize("direction", DIRS)
def test_project_matches_oracle(dtype, N, direction):
    say(f"project dtype={dtype} N={N} {direction}")
    layer, W = make_layer(dtype, affine=True)
    z = synth.pair_tensor(N, dtype=dtype)
    mask = synth.random_mask(N, 0.85)
    A, B = layer.project(z.cuda(), mask.cuda(), direction)
    torch.cuda.synchronize()
    rA, rB = oracle.projected_panels(z, mask, W, direction)
    # Per-element error terms of the bf16 path, from the oracle's pieces: the
    # values W x and the gates run on x rounded once to fp16 (the kernel
    # scales x and W by powers of two so that neither overflows nor falls
    # into fp16's subnormals: |x - fl(x)| <= 2^-11 |x|, weights exact), the
    # logistic is 1/4-Lipschitz, then one bf16 rounding of the product
    # (<= 2^-8 relative).
    x = oracle.layer_norm(oracle.f64(z), W["ln_in_w"], W["ln_in_b"])
    ax = np.abs(x)
    m = oracle.pair_mask(mask)[..., None]
    lay = (2, 0, 1) if direction == "outgoing" else (2, 1, 0)
    extra = {}
    for name, wv, wg in (("A", "w_a", "w_ga"), ("B", "w_b", "w_gb")):
        p = np.abs(oracle.linear(x, W[wv]))
        gate = 2.0 ** -13 * (ax @ np.abs(oracle.f64(W[wg])).T)
        vals = 2.0 ** -11 * (ax @ np.abs(oracle.f64(W[wv])).T)
        extra[name] = (m * (gate * p + vals)).transpose(lay)
    for got, ref, name in ((A, rA, "A"), (B, rB, "B")):
        got = host(T.panel_to_dense(got, N))
        if dtype == "f32":
            mx, rel = errors(got, ref)
            say(f"  {name}: max_abs={mx:.2e} rel_fro={rel:.2e}")
            assert rel <= 1e-6
        else:
            bound = 2.0 ** -8 * np.abs(ref) + (1 + 2.0 ** -8) * extra[name] + 1e-5
            bad = np.abs(got - ref) > bound
            mx, rel = errors(got, ref)
            say(f"  {name}: max_abs={mx:.2e} rel_fro={rel:.2e}")
            assert not bad.any(), f"{name}: {bad.sum()} elements beyond the bound"
        # masked pairs are exact zeros
        m = oracle.pair_mask(mask)
        mm = m if direction == "outgoing" else m.T
        assert np.all(got[:, mm == 0] == 0)


# --------------------------------------------------------------- epilogue

@pytest.mark.parametrize("dtype,out_dtype,N", [("bf16", "f32", 100), ("bf16", "bf16", 64), ("f32", "f32", 65)])
def test_epilogue_matches_oracle(dtype, out_dtype, N):
    say(f"epilogue dtype={dtype} out={out_dtype} N={N}")
    layer, W = make_layer(dtype, out_dtype, affine=True)
    z = synth.pair_tensor(N, dtype=dtype)
    mask = synth.random_mask(N, 0.85, sub=3)
    # contraction-like input: sums of ~N unit products have scale sqrt(N)
    C = (torch.randn((128, N, N), generator=torch.Generator().manual_seed(5)) * np.sqrt(N)).float()
    out = layer.epilogue(T.dense_to_result(C).cuda(), z.cuda(), mask.cuda())
    torch.cuda.synchronize()
    m = oracle.pair_mask(mask)
    _, _, gate = oracle.project(z, m, W)
    ref = oracle.epilogue(host(C).transpose(1, 2, 0), gate, m, W)
    tol_dtype = "f32" if (dtype == "f32" and out_dtype == "f32") else "bf16"
    assert_close(host(out), ref, tol_dtype, "epilogue")
    assert np.all(host(out)[m == 0] == 0)


# ------------------------------------------------------- whole update, full

def run_full(dtype, N, mask, direction, out_dtype="f32", affine=False, scale=None):
    layer, W = make_layer(dtype, out_dtype, affine=affine)
    z = synth.pair_tensor(N, dtype=dtype, scale=scale)
    out = layer(z.cuda(), None if mask is None else mask.cuda(), direction)
    torch.cuda.synchronize()
    ref = oracle.tri_mul(z, np.ones(N) if mask is None else mask, W, direction)
    return host(out), ref, layer, W, z


@pytest.mark.parametrize("direction", DIRS)
def test_config1_fp32_n64(direction):
    say(f"config 1: fp32 N=64 {direction}")
    got, ref, *_ = run_full("f32", 64, None, direction)
    assert_close(got, ref, "f32", "c1")


@pytest.mark.parametrize("direction", DIRS)
def test_config2_bf16_n512_pad51(direction):
    say(f"config 2: bf16 N=512, last 51 tokens padded, {direction}")
    mask = synth.token_mask(512, 51)
    got, ref, *_ = run_full("bf16", 512, mask, direction)
    assert_close(got[:461, :461], ref[:461, :461], "bf16", "c2 unmasked block")
    assert np.all(got[461:] == 0) and np.all(got[:, 461:] == 0)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("N", [1, 2, 17, 63, 65, 257, 300])
def test_ragged_sizes(dtype, N):
    for direction in DIRS:
        say(f"ragged dtype={dtype} N={N} {direction}")
        mask = synth.random_mask(N, 0.8, sub=N)
        if N > 1:
            mask[0] = 1
        got, ref, *_ = run_full(dtype, N, mask, direction, affine=True)
        if not np.any(ref):
            assert not np.any(got)
        else:
            assert_close(got, ref, dtype, f"N={N}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_all_masked_gives_zero(dtype):
    N = 40
    got, ref, *_ = run_full(dtype, N, torch.zeros(N, dtype=torch.uint8), "outgoing")
    assert not np.any(got)


def test_bf16_output_dtype():
    say("bf16 output N=256")
    got, ref, *_ = run_full("bf16", 256, None, "incoming", out_dtype="bf16")
    assert_close(got, ref, "bf16", "bf16 out")


# ------------------------------------------------------------ invariants

@pytest.mark.parametrize("direction", DIRS)
def test_padding_invariance_bitwise(direction):
    N, n_real = 200, 170
    layer, W = make_layer("bf16")
    mask = synth.token_mask(N, N - n_real).cuda()
    z = synth.pair_tensor(N, dtype="bf16").cuda()
    z2 = z.clone()
    z2[n_real:] = 100 * synth.pair_tensor(N, dtype="bf16", seed=5)[n_real:].cuda()
    z2[:, n_real:] = -30 * synth.pair_tensor(N, dtype="bf16", seed=6)[:, n_real:].cuda()
    o1 = layer(z, mask, direction).clone()
    o2 = layer(z2, mask, direction)
    torch.cuda.synchronize()
    assert torch.equal(o1[:n_real, :n_real], o2[:n_real, :n_real])
    assert not o2[n_real:].any() and not o2[:, n_real:].any()


def test_deterministic_bitwise():
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(320, dtype="bf16").cuda()
    o1 = layer(z, None, "outgoing").clone()
    o2 = layer(z, None, "outgoing")
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def test_incoming_equals_transposed_outgoing_with_swapped_weights():
    N = 192
    Wt = synth.weights(128, 128, dtype="bf16")
    Ws = dict(Wt, w_a=Wt["w_b"], w_ga=Wt["w_gb"], w_b=Wt["w_a"], w_gb=Wt["w_ga"])
    la = T.TriMul(Wt, "bf16", "f32")
    lb = T.TriMul(Ws, "bf16", "f32")
    z = synth.pair_tensor(N, dtype="bf16").cuda()
    inc = la.incoming(z)
    out_t = lb.outgoing(z.transpose(0, 1).contiguous()).transpose(0, 1)
    torch.cuda.synchronize()
    mx, rel = errors(host(inc), host(out_t))
    say(f"  swap relation: max_abs={mx:.2e} rel={rel:.2e}")
    assert rel <= 1e-6


# ------------------------------------------------------------- ABI errors

def test_abi_errors_on_device():
    layer, _ = make_layer("bf16")
    N = 64
    z = torch.zeros((N, N, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((N, N, 128), dtype=torch.float32, device="cuda")
    need = T.tri_mul_workspace_size(layer.h, N)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    L = T.lib()
    s = torch.cuda.current_stream().cuda_stream
    assert L.tri_mul_outgoing(layer.h, z.data_ptr(), None, N, out.data_ptr(), ws.data_ptr(), need - 1, s) == T.TRI_MUL_ENOMEM
    assert L.tri_mul_outgoing(layer.h, z.data_ptr() + 2, None, N, out.data_ptr(), ws.data_ptr(), need, s) == T.TRI_MUL_EINVAL
    assert L.tri_mul_outgoing(layer.h, z.data_ptr(), None, 0, out.data_ptr(), ws.data_ptr(), need, s) == T.TRI_MUL_EINVAL
    assert L.tri_mul_outgoing(layer.h, z.data_ptr(), None, -5, out.data_ptr(), ws.data_ptr(), need, s) == T.TRI_MUL_EINVAL
    assert L.tri_mul_project(layer.h, z.data_ptr(), None, N, 7, ws.data_ptr(), ws.data_ptr(), s) == T.TRI_MUL_EINVAL
    v = T.BlockView(100, 90, 0, 20, 10, 0, 10, 16, 16, 0, 1)      # rows exceed n_total
    assert L.tri_mul_block_accumulate(layer.h, v, ws.data_ptr(), ws.data_ptr(), ws.data_ptr(), None,
                                      z.data_ptr(), out.data_ptr(), s) == T.TRI_MUL_EINVAL
    v = T.BlockView(100, 0, 0, 20, 10, 0, 10, 12, 16, 0, 1)       # ld_a not a multiple of 8
    assert L.tri_mul_block_accumulate(layer.h, v, ws.data_ptr(), ws.data_ptr(), ws.data_ptr(), None,
                                      z.data_ptr(), out.data_ptr(), s) == T.TRI_MUL_EINVAL
    v = T.BlockView(100, 0, 0, 20, 10, 0, 10, 16, 16, 0, 1)       # last panel without z_tile
    assert L.tri_mul_block_accumulate(layer.h, v, ws.data_ptr(), ws.data_ptr(), ws.data_ptr(), None,
                                      None, out.data_ptr(), s) == T.TRI_MUL_EINVAL
    assert "z_tile" in T.last_error()
    torch.cuda.synchronize()
    layer.close()
    layer.close()


def test_init_range_of_projection_operands():
    """The bf16 path's projection runs on fp16 operands scaled by powers of
    two chosen at init: weights and LayerNorm parameters far apart in
    magnitude still give the oracle's projections (to the projection's
    per-element bound, through the whole update), and values beyond what
    the largest scale can bring into fp16 range are refused."""
    W = synth.weights(128, 128, dtype="bf16", affine=True)
    for name, f in (("w_a", 2.0 ** -30), ("w_gb", 2.0 ** 20), ("ln_in_w", 2.0 ** -25), ("ln_in_b", 2.0 ** -25)):
        W[name] = (W[name].double() * f).to(torch.bfloat16)
    layer = T.TriMul(W, dtype="bf16", out_dtype="f32")
    Wd = {k: oracle.f64(v) for k, v in W.items()}
    N = 40
    z = synth.pair_tensor(N, dtype="bf16")
    mask = synth.random_mask(N, 0.9)
    for direction in DIRS:
        A, B = layer.project(z.cuda(), mask.cuda(), direction)
        torch.cuda.synchronize()
        rA, rB = oracle.projected_panels(z, mask, Wd, direction)
        for got, ref in ((A, rA), (B, rB)):
            mx, rel = errors(host(T.panel_to_dense(got, N)), ref)
            say(f"  scaled weights {direction}: rel_fro={rel:.2e}")
            assert rel <= 4e-3
    layer.close()
    for name in ("w_ga", "ln_in_w"):
        Wb = dict(W)
        Wb[name] = torch.full_like(W[name], 1e30)
        with pytest.raises(T.TriMulError) as e:
            T.TriMul(Wb, dtype="bf16", out_dtype="f32")
        assert "supported range" in str(e.value)
