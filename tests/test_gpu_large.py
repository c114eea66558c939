"""GPU parity at the benchmark table's full sizes (N = 2048, N = 4096, and one
3750 x 3750 tile of an 8 x 8 grid at N = 30000), checked on sampled outputs
the oracle computes one by one and on four full output rows (at N = 4096 the
oracle projects all 16.7M pairs for them, in column chunks on worker
processes), plus the block decomposition of the full update (each tile
accumulated over k-panels equals the full result)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import synth
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import assert_close, errors, host, make_layer, needs_gpu, say

pytestmark = [pytest.mark.gpu, needs_gpu]
DIRS = ("outgoing", "incoming")


def sample_index(N, n_rand, seed, extra=()):
    """Sorted unique indices: n_rand random ones plus edges and tile seams."""
    rng = np.random.default_rng(seed)
    fixed = [0, 1, 31, 32, 63, 64, 255, 256, N // 2, N - 2, N - 1] + list(extra)
    idx = set(int(i) for i in fixed if 0 <= i < N)
    idx |= set(rng.choice(N, size=n_rand, replace=False).tolist())
    return np.array(sorted(idx))


def ring_packed(layer, views, aps, bps, mask, z_tile, out, pacc, wss, reserve_cus=0):
    """The ring steps of one tile through tri_mul_block_repack +
    tri_mul_block_accumulate_packed: panel p + 1 is repacked on a second
    stream while panel p is contracted on the current one, alternating
    between two workspaces (ordered by events)."""
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    n = len(views)
    packed = [torch.cuda.Event() for _ in range(n)]
    done = [torch.cuda.Event() for _ in range(n)]
    layer.block_repack(views[0], aps[0], bps[0], mask, wss[0], main)
    packed[0].record(main)
    side.wait_stream(main)
    for p in range(n):
        if p + 1 < n:
            if p >= 1:
                side.wait_event(done[p - 1])   # that step read the workspace this repack overwrites
            layer.block_repack(views[p + 1], aps[p + 1], bps[p + 1], mask, wss[(p + 1) % 2], side)
            packed[p + 1].record(side)
        main.wait_event(packed[p])
        layer.block_accumulate_packed(views[p], wss[p % 2], pacc, mask, z_tile, out,
                                      reserve_cus=reserve_cus if p + 1 < n else 0, stream=main)
        done[p].record(main)
    main.wait_stream(side)


@pytest.mark.parametrize("direction", DIRS)
def test_config3_bf16_n2048_channel_scaled(direction):
    N = 2048
    say(f"config 3: bf16 N={N}, per-channel scale U(0.5,2), {direction}")
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", scale=synth.channel_scale(), device="cuda")
    out = layer(z, None, direction)
    torch.cuda.synchronize()
    I, J = sample_index(N, 110, 1), sample_index(N, 110, 2)
    ref = oracle.tri_mul(z, np.ones(N), W, direction, I, J)
    got = host(out[torch.as_tensor(I, device="cuda")][:, torch.as_tensor(J, device="cuda")])
    assert_close(got, ref, "bf16", f"c3 {len(I)}x{len(J)} sampled pairs")
    # four full output rows
    R = np.array([0, 777, 1500, N - 1])
    ref_r = oracle.tri_mul(z, np.ones(N), W, direction, R, None)
    assert_close(host(out[torch.as_tensor(R, device="cuda")]), ref_r, "bf16", "c3 full rows")


@pytest.mark.parametrize("direction", DIRS)
def test_config4_bf16_n4096(direction):
    N = 4096
    say(f"config 4: bf16 N={N}, {direction}")
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", device="cuda")
    out = layer(z, None, direction)
    torch.cuda.synchronize()
    I, J = sample_index(N, 117, 3), sample_index(N, 117, 4)
    ref = oracle.tri_mul(z, np.ones(N), W, direction, I, J)
    got = host(out[torch.as_tensor(I, device="cuda")][:, torch.as_tensor(J, device="cuda")])
    assert_close(got, ref, "bf16", f"c4 {len(I)}x{len(J)} sampled pairs")
    del out, z
    layer.close()
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_config4_full_rows_n4096():
    """Four full output rows of each direction at N = 4096 (all 4096 columns,
    all 128 channels), against oracle.tri_mul over 64-column chunks."""
    from tests.oracle_pool import tri_mul_rows
    N = 4096
    say(f"config 4: bf16 N={N}, four full output rows per direction")
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", device="cuda")
    R = np.array([0, 1537, 2890, N - 1])
    Rt = torch.as_tensor(R, device="cuda")
    got = {}
    for direction in DIRS:
        got[direction] = host(layer(z, None, direction)[Rt])
    torch.cuda.synchronize()
    say("  device runs done")
    pieces = ((r0, z[r0:r0 + 256].float().cpu().numpy()) for r0 in range(0, N, 256))
    ref = tri_mul_rows(pieces, N, np.ones(N), W, DIRS, R, say=say)
    for direction in DIRS:
        assert_close(got[direction], ref[direction], "bf16", f"c4 {direction} rows {R.tolist()}")
    layer.close()
    del z
    torch.cuda.empty_cache()


def test_config5_tile_of_8x8_grid_n30000():
    """Tile (7, 7) of an 8 x 8 grid at N = 30000: 3750 x 3750 outputs, 8
    k-panels of 3750 tokens, the last 300 tokens padded (rows, columns and the
    last k-panel).  Panels ~ N(0,1) bf16 generated on the device.  Three
    ways run on the same panels: tri_mul_block_accumulate (row-major panels
    read in place), tri_mul_block_accumulate_ws (panels repacked through the
    workspace), and tri_mul_block_repack + tri_mul_block_accumulate_packed
    with the next panel's repack on a second stream and a packed
    accumulator (the one the benchmark times)."""
    n_total, g = 30000, 8
    b = n_total // g
    row0 = col0 = 7 * b
    ld = (b + 7) // 8 * 8
    say(f"config 5: tile ({row0},{col0}) {b}x{b}, 8 k-panels, ld={ld}")
    layer, W = make_layer("bf16")
    mask = synth.token_mask(n_total, 300, device="cuda")
    aps, bps = [], []
    for p in range(g):
        aps.append(synth.pair_tensor(0, dtype="bf16", device="cuda", name="a_panel", seed=synth.SEED + p,
                                     shape=(128, b, ld)))
        bps.append(synth.pair_tensor(0, dtype="bf16", device="cuda", name="b_panel", seed=synth.SEED + p,
                                     shape=(128, b, ld)))
    z_tile = synth.pair_tensor(0, dtype="bf16", device="cuda", name="z_tile", shape=(b, b, 128))
    acc = torch.empty((128, b, b), dtype=torch.float32, device="cuda")
    out = torch.empty((b, b, 128), dtype=torch.float32, device="cuda")
    I = sample_index(b, 114, 5, extra=(3449, 3450, 3451, 3700, 3748))
    J = sample_index(b, 114, 6, extra=(3449, 3450, 3451, 3700, 3748))
    It, Jt = torch.as_tensor(I, device="cuda"), torch.as_tensor(J, device="cuda")
    mask_h = host(mask)
    ref_C = oracle.block_contract([host(a[:, It, :b]) for a in aps], [host(bb[:, Jt, :b]) for bb in bps],
                                  [mask_h[p * b:(p + 1) * b] for p in range(g)])
    ref = oracle.block_epilogue(ref_C, oracle.take_pairs(z_tile, I, J), mask_h[row0 + I], mask_h[col0 + J], W)
    valid = (mask_h[row0 + I] != 0)[:, None] & (mask_h[col0 + J] != 0)[None, :]
    v0 = T.BlockView(n_total, row0, col0, b, b, 0, b, ld, ld, 0, g)
    ws = torch.empty(layer.block_workspace_size(v0), dtype=torch.uint8, device="cuda")
    outs = {}
    for mode in ("plain", "ws", "packed", "blocked"):
        acc.fill_(float("nan"))   # the first ring step must overwrite every element
        out.fill_(float("nan"))
        if mode == "blocked":
            # the panels in the contraction's blocked layout (here made by the
            # repack, as tri_mul_block_project would send them) contracted by
            # tri_mul_block_accumulate_blocked
            pacc = torch.full((layer.block_accumulator_size(v0) // 4,), float("nan"), device="cuda")
            ob = -(-layer.block_panel_size(b, b) // 256) * 256
            for p in range(g):
                v = T.BlockView(n_total, row0, col0, b, b, p * b, b, ld, ld, p, g)
                layer.block_repack(v, aps[p], bps[p], mask, ws)
                layer.block_accumulate_blocked(v, ws, ws[ob:], pacc, mask, z_tile, out)
            torch.cuda.synchronize()
            acc.copy_(T.result_to_dense(pacc, b, cols=b))
        elif mode == "packed":
            # the next panel's repack on a second stream while the current one
            # is contracted on 16 fewer compute units; two workspaces
            pacc = torch.full((layer.block_accumulator_size(v0) // 4,), float("nan"), device="cuda")
            ring_packed(layer, [T.BlockView(n_total, row0, col0, b, b, p * b, b, ld, ld, p, g) for p in range(g)],
                        aps, bps, mask, z_tile, out, pacc, [ws, torch.empty_like(ws)], reserve_cus=16)
            torch.cuda.synchronize()
            acc.copy_(T.result_to_dense(pacc, b, cols=b))
        else:
            for p in range(g):
                v = T.BlockView(n_total, row0, col0, b, b, p * b, b, ld, ld, p, g)
                layer.block_accumulate(v, aps[p], bps[p], acc, mask, z_tile, out, ws=ws if mode == "ws" else None)
        torch.cuda.synchronize()
        say(f"  device run done ({mode})")
        got_C = host(acc[:, It][:, :, Jt]).transpose(1, 2, 0)
        mx, rel = errors(got_C, ref_C)
        say(f"  accumulator: max_abs={mx:.3e} rel_fro={rel:.3e}")
        assert rel <= 1e-5
        got = host(out[It][:, Jt])
        assert_close(got[valid], ref[valid], "bf16", "c5 sampled valid pairs")
        assert np.all(got[~valid] == 0)
        assert torch.isfinite(out).all() and torch.isfinite(acc).all()
        outs[mode] = out.clone()
    # the same kernel on the same blocked panels, in one stream or two
    assert torch.equal(outs["blocked"], outs["packed"])
    del outs


@pytest.mark.parametrize("direction", DIRS)
def test_config5_tile_projection_sampled(direction):
    """tri_mul_block_project on the 3750 x 3750 z tile (7, 7) of the 8 x 8
    grid at N = 30000 (the last 300 tokens padded): the blocked a and b
    panels at sampled (operand row, k) positions, every channel, against the
    oracle's projection of those pairs, to the projection's per-element
    bound (one bf16 rounding of the result; values and gates from x rounded
    once to fp16, 2^-11 |W| |x| and, through the 1/4-Lipschitz logistic,
    2^-13 |W_g| |x| |W x|)."""
    n_total, g = 30000, 8
    b = n_total // g
    row0 = col0 = 7 * b
    say(f"config 5 tile projection: {b}x{b} at ({row0},{col0}) {direction}")
    layer, W = make_layer("bf16", affine=True)
    mask = synth.token_mask(n_total, 300, device="cuda")
    z_tile = synth.pair_tensor(0, dtype="bf16", device="cuda", name="z_tile", shape=(b, b, 128))
    A, B = layer.block_project(z_tile, mask, n_total, row0, col0, direction)
    torch.cuda.synchronize()
    I = sample_index(b, 50, 15, extra=(3449, 3450, 3451, 3700, 3749))   # operand rows
    K = sample_index(b, 50, 16, extra=(3449, 3450, 3451, 3700, 3749))   # contraction index
    Tt, S = -(-b // 256), -(-b // 32)
    c = np.arange(128)[:, None, None]
    i, k = I[None, :, None], K[None, None, :]
    flat = ((c * Tt + i // 256) * S + k // 32) * 8192 + (i % 256) * 32 + k % 32
    fi = torch.as_tensor(flat.reshape(-1), device="cuda")
    got_a = host(A[fi]).reshape(128, len(I), len(K))
    got_b = host(B[fi]).reshape(128, len(I), len(K))
    # pair of operand row i, index k: (row0 + i, col0 + k) outgoing, (row0 + k, col0 + i) incoming
    zi, zk = (K, I) if direction == "incoming" else (I, K)
    It, Kt = torch.as_tensor(zi, device="cuda"), torch.as_tensor(zk, device="cuda")
    zp = host(z_tile[It][:, Kt])                                        # [len(zi)][len(zk)][128]
    mh = host(mask)
    mp = oracle.pair_mask(mh[row0 + zi], mh[col0 + zk])
    ra, rb, _ = oracle.project(zp, mp, W)
    x = oracle.layer_norm(zp, W["ln_in_w"], W["ln_in_b"])
    ax = np.abs(x)
    for got, ref, wv, wg, name in ((got_a, ra, "w_a", "w_ga", "a"), (got_b, rb, "w_b", "w_gb", "b")):
        p = np.abs(oracle.linear(x, W[wv]))
        extra = mp[..., None] * (2.0 ** -13 * (ax @ np.abs(W[wg]).T) * p + 2.0 ** -11 * (ax @ np.abs(W[wv]).T))
        if direction == "incoming":
            ref, extra = ref.transpose(1, 0, 2), extra.transpose(1, 0, 2)
        ref, extra = ref.transpose(2, 0, 1), extra.transpose(2, 0, 1)   # [c][operand row][k]
        bound = 2.0 ** -8 * np.abs(ref) + (1 + 2.0 ** -8) * extra + 1e-5
        mx, rel = errors(got, ref)
        say(f"  {name}: max_abs={mx:.2e} rel_fro={rel:.2e}")
        assert not (np.abs(got - ref) > bound).any(), f"{name}: elements beyond the bound"
        dead = mp == 0 if direction == "outgoing" else (mp == 0).T
        assert np.all(got[:, dead] == 0)


@pytest.mark.parametrize("direction", DIRS)
@pytest.mark.parametrize("N,g,use_ws", [(1024, 2, False), (1024, 4, False), (1000, 4, False), (1024, 2, True),
                                        (1000, 4, True), (1024, 2, "packed"), (1000, 4, "packed")])
def test_block_decomposition_matches_full(direction, N, g, use_ws):
    """The one-GPU stand-in for the paper's ring: split the full problem into
    a g x g grid of tiles, run each tile as g block_accumulate calls (one per
    k-panel, as in the Cannon ring; with use_ws through the repacking entry
    point, or with "packed" through tri_mul_block_repack and
    tri_mul_block_accumulate_packed on two streams) from the same projected
    panels, and compare with the single-call contraction and update."""
    say(f"block == full: N={N} g={g} {direction} ws={use_ws}")
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", device="cuda")
    mask = synth.random_mask(N, 0.9, sub=g).cuda()
    Ap, Bp = layer.project(z, mask, direction)
    Cr = layer.contract(Ap, Bp, N)
    A, B = T.panel_to_dense(Ap, N), T.panel_to_dense(Bp, N)
    out_full = layer.epilogue(Cr, z, mask)
    C_full = T.result_to_dense(Cr, N)
    out_dir = layer(z, mask, direction)
    torch.cuda.synchronize()
    assert torch.equal(out_full, out_dir), "stage calls differ from the one-call entry point"
    bsz = N // g
    ld = (bsz + 7) // 8 * 8
    out_blk = torch.zeros_like(out_full)
    ws = None
    if use_ws:
        n = layer.block_workspace_size(T.BlockView(N, 0, 0, bsz, bsz, 0, bsz, ld, ld, 0, g))
        ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    for r in range(g):
        for c in range(g):
            r0, c0 = r * bsz, c * bsz
            acc = torch.empty((128, bsz, bsz), dtype=torch.float32, device="cuda")
            z_tile = z[r0:r0 + bsz, c0:c0 + bsz].contiguous()
            o_tile = torch.empty((bsz, bsz, 128), dtype=torch.float32, device="cuda")
            aps, bps, views = [], [], []
            for p in range(g):
                k0 = p * bsz
                ap = torch.zeros((128, bsz, ld), dtype=torch.bfloat16, device="cuda")
                bp = torch.zeros((128, bsz, ld), dtype=torch.bfloat16, device="cuda")
                ap[:, :, :bsz] = A[:, r0:r0 + bsz, k0:k0 + bsz]
                bp[:, :, :bsz] = B[:, c0:c0 + bsz, k0:k0 + bsz]
                v = T.BlockView(N, r0, c0, bsz, bsz, k0, bsz, ld, ld, p, g)
                aps.append(ap), bps.append(bp), views.append(v)
                if use_ws != "packed":
                    layer.block_accumulate(v, ap, bp, acc, mask, z_tile, o_tile, ws=ws)
            if use_ws == "packed":
                pacc = torch.full((layer.block_accumulator_size(views[0]) // 4,), float("nan"), device="cuda")
                ring_packed(layer, views, aps, bps, mask, z_tile, o_tile, pacc, [ws, torch.empty_like(ws)])
                acc = T.result_to_dense(pacc, bsz, cols=bsz)
            mx, rel = errors(host(acc), host(C_full[:, r0:r0 + bsz, c0:c0 + bsz]))
            assert rel <= 1e-5, (r, c, rel)
            out_blk[r0:r0 + bsz, c0:c0 + bsz] = o_tile
    torch.cuda.synchronize()
    mx, rel = errors(host(out_blk), host(out_full))
    say(f"  tiles vs full: max_abs={mx:.2e} rel_fro={rel:.2e}")
    assert rel <= 1e-5 and mx <= 1e-3
