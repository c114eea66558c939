"""The ring with panels in the contraction's blocked layout: every device
tile projects its own z tile once (tri_mul_block_project) and the ring steps
contract those panels directly (tri_mul_block_accumulate_blocked).  Checked
against the full update's own stages on the same inputs: the tile panels are
bitwise the corresponding blocks of tri_mul_project's operands, every output
tile equals the repacking ring step's result on the same panel values
bitwise, and the assembled update equals the one-call update up to the fp32
order of the k-panel sums.  Token partitions with unequal and ragged blocks
(tiles of different shapes, sides not multiples of 32 or 256)."""
import numpy as np
import pytest
import torch

from paper_2603_14806_amd import synth
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import errors, host, make_layer, needs_gpu, say
from tests.test_gpu_large import ring_packed

pytestmark = [pytest.mark.gpu, needs_gpu]
DIRS = ("outgoing", "incoming")


def blocks(cuts):
    return [(cuts[i], cuts[i + 1] - cuts[i]) for i in range(len(cuts) - 1)]


def ring_blocked(layer, views, aps, bps, mask, z_tile, out, pacc, reserve_cus=0):
    for v, a, b in zip(views, aps, bps):
        layer.block_accumulate_blocked(v, a, b, pacc, mask, z_tile, out,
                                       reserve_cus=reserve_cus if v.k_index + 1 < v.k_count else 0)


def ring_transposed(layer, views, atps, btps, mask, z_tile, out, pacc, reserve_cus=0):
    for v, a, b in zip(views, atps, btps):
        layer.block_accumulate_transposed(v, a, b, pacc, mask, z_tile, out,
                                          reserve_cus=reserve_cus if v.k_index + 1 < v.k_count else 0)


@pytest.mark.parametrize("direction", DIRS)
@pytest.mark.parametrize("N,cuts", [(1000, (0, 100, 356, 700, 1000)), (77, (0, 33, 77)), (1024, (0, 512, 1024))])
def test_transposed_ring_is_bitwise_the_blocked_ring(direction, N, cuts):
    """Every device projecting its own z tile with the opposite direction
    writes the transposed panels; the ring steps on those
    (tri_mul_block_accumulate_transposed) give the blocked ring's
    accumulator and output bit for bit, for tiles of every shape."""
    say(f"transposed ring: N={N} cuts={cuts} {direction}")
    layer, _ = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", device="cuda")
    mask = synth.random_mask(N, 0.9, sub=len(cuts)).cuda()
    bl = blocks(cuts)
    g = len(bl)
    inc = direction == "incoming"
    other = "outgoing" if inc else "incoming"
    proj, projt = {}, {}
    for x, (r0, nr) in enumerate(bl):
        for y, (c0, nc) in enumerate(bl):
            zt = z[r0:r0 + nr, c0:c0 + nc].contiguous()
            proj[(x, y)] = layer.block_project(zt, mask, N, r0, c0, direction)
            projt[(x, y)] = layer.block_project(zt, mask, N, r0, c0, other)
    for p, (r0, nr) in enumerate(bl):
        for q, (c0, nc) in enumerate(bl):
            z_tile = z[r0:r0 + nr, c0:c0 + nc].contiguous()
            views, aps, bps, atps, btps = [], [], [], [], []
            for r, (k0, nk) in enumerate(bl):
                ld = (nk + 7) // 8 * 8
                views.append(T.BlockView(N, r0, c0, nr, nc, k0, nk, ld, ld, r, g))
                ka, kb = ((r, p), (r, q)) if inc else ((p, r), (q, r))
                aps.append(proj[ka][0]), bps.append(proj[kb][1])
                atps.append(projt[ka][0]), btps.append(projt[kb][1])
            nacc = layer.block_accumulator_size(views[0]) // 4
            o1 = torch.full((nr, nc, 128), float("nan"), device="cuda")
            o2 = torch.full((nr, nc, 128), float("nan"), device="cuda")
            p1 = torch.full((nacc,), float("nan"), device="cuda")
            p2 = torch.full((nacc,), float("nan"), device="cuda")
            ring_blocked(layer, views, aps, bps, mask, z_tile, o1, p1)
            ring_transposed(layer, views, atps, btps, mask, z_tile, o2, p2, reserve_cus=16)
            torch.cuda.synchronize()
            assert torch.equal(T.result_to_dense(p1, nr, cols=nc), T.result_to_dense(p2, nr, cols=nc)), (p, q)
            assert torch.equal(o1, o2), (p, q)
            assert torch.isfinite(o2).all()


@pytest.mark.parametrize("direction", DIRS)
@pytest.mark.parametrize("N,cuts", [(1000, (0, 600, 1000)), (1000, (0, 100, 356, 700, 1000)),
                                    (1024, (0, 512, 1024)), (77, (0, 33, 77))])
def test_blocked_ring_matches_full(direction, N, cuts):
    say(f"blocked ring: N={N} cuts={cuts} {direction}")
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", device="cuda")
    mask = synth.random_mask(N, 0.9, sub=len(cuts)).cuda()
    Ap, Bp = layer.project(z, mask, direction)
    A, B = T.panel_to_dense(Ap, N), T.panel_to_dense(Bp, N)
    Cr = layer.contract(Ap, Bp, N)
    C_full = T.result_to_dense(Cr, N)
    out_full = layer(z, mask, direction)
    torch.cuda.synchronize()
    bl = blocks(cuts)
    g = len(bl)
    inc = direction == "incoming"
    # every device projects its own z tile (x, y) once
    proj = {}
    for x, (r0, nr) in enumerate(bl):
        for y, (c0, nc) in enumerate(bl):
            zt = z[r0:r0 + nr, c0:c0 + nc].contiguous()
            a, b = layer.block_project(zt, mask, N, r0, c0, direction)
            m, k = (nc, nr) if inc else (nr, nc)
            da, db = T.panel_to_dense(a, m, klen=k), T.panel_to_dense(b, m, klen=k)
            # operand rows m, contraction index k: the full operands' block
            ra, ka = (slice(c0, c0 + nc), slice(r0, r0 + nr)) if inc else (slice(r0, r0 + nr), slice(c0, c0 + nc))
            assert torch.equal(da, A[:, ra, ka]) and torch.equal(db, B[:, ra, ka]), (x, y)
            proj[(x, y)] = (a, b)
    torch.cuda.synchronize()
    say("  tile panels equal the full projection's blocks")
    out_blk = torch.zeros_like(out_full)
    for p, (r0, nr) in enumerate(bl):
        for q, (c0, nc) in enumerate(bl):
            z_tile = z[r0:r0 + nr, c0:c0 + nc].contiguous()
            views, aps, bps, rap, rbp = [], [], [], [], []
            for r, (k0, nk) in enumerate(bl):
                ld = (nk + 7) // 8 * 8
                views.append(T.BlockView(N, r0, c0, nr, nc, k0, nk, ld, ld, r, g))
                # outgoing: a from z tile (p, r), b from (q, r); incoming: a from (r, p), b from (r, q)
                aps.append(proj[(r, p) if inc else (p, r)][0])
                bps.append(proj[(r, q) if inc else (q, r)][1])
                ap = torch.zeros((128, nr, ld), dtype=torch.bfloat16, device="cuda")
                bp = torch.zeros((128, nc, ld), dtype=torch.bfloat16, device="cuda")
                ap[:, :, :nk] = A[:, r0:r0 + nr, k0:k0 + nk]
                bp[:, :, :nk] = B[:, c0:c0 + nc, k0:k0 + nk]
                rap.append(ap), rbp.append(bp)
            nacc = layer.block_accumulator_size(views[0]) // 4
            o_blk = torch.full((nr, nc, 128), float("nan"), device="cuda")
            pacc = torch.full((nacc,), float("nan"), device="cuda")
            ring_blocked(layer, views, aps, bps, mask, z_tile, o_blk, pacc, reserve_cus=16)
            o_pk = torch.full((nr, nc, 128), float("nan"), device="cuda")
            pacc2 = torch.full((nacc,), float("nan"), device="cuda")
            wsb = max(layer.block_workspace_size(v) for v in views)
            wss = [torch.empty(wsb, dtype=torch.uint8, device="cuda") for _ in range(2)]
            ring_packed(layer, views, rap, rbp, mask, z_tile, o_pk, pacc2, wss)
            torch.cuda.synchronize()
            acc = T.result_to_dense(pacc, nr, cols=nc)
            assert torch.equal(acc, T.result_to_dense(pacc2, nr, cols=nc)), (p, q)
            assert torch.equal(o_blk, o_pk), (p, q)
            mx, rel = errors(host(acc), host(C_full[:, r0:r0 + nr, c0:c0 + nc]))
            assert rel <= 1e-5, (p, q, rel)
            out_blk[r0:r0 + nr, c0:c0 + nc] = o_blk
    torch.cuda.synchronize()
    mx, rel = errors(host(out_blk), host(out_full))
    say(f"  tiles vs full: max_abs={mx:.2e} rel_fro={rel:.2e}")
    assert rel <= 1e-5 and mx <= 1e-3
    assert torch.isfinite(out_blk).all()


def test_block_project_strided_tile_and_errors():
    """A tile read in place from the full z (ld_z = N > cols), and the
    argument checks of the two entry points."""
    N = 300
    layer, W = make_layer("bf16")
    z = synth.pair_tensor(N, dtype="bf16", device="cuda")
    mask = synth.token_mask(N, 21, device="cuda")
    A, B = (T.panel_to_dense(P, N) for P in layer.project(z, mask, "outgoing"))
    r0, c0, nr, nc = 40, 130, 97, 170
    n = layer.block_panel_size(nr, nc) // 2
    a = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    b = torch.empty_like(a)
    T.tri_mul_block_project(layer.h, z[r0, c0], N, mask, N, r0, c0, nr, nc, T.TRI_MUL_OUTGOING, a, b)
    torch.cuda.synchronize()
    assert torch.equal(T.panel_to_dense(a, nr, klen=nc), A[:, r0:r0 + nr, c0:c0 + nc])
    assert torch.equal(T.panel_to_dense(b, nr, klen=nc), B[:, r0:r0 + nr, c0:c0 + nc])
    # k >= klen of the last k-step is zero
    S = -(-nc // 32)
    full = a.reshape(128, -(-nr // 256), S, 256, 32)[:, :, S - 1, :nr % 256 or 256, nc % 32:]
    assert (full == 0).all()

    def rc(f, *args):
        with pytest.raises(RuntimeError) as e:
            f(*args)
        return str(e.value)
    bad = rc(T.tri_mul_block_project, layer.h, z[r0, c0], nc - 1, mask, N, r0, c0, nr, nc, 0, a, b)
    assert "ld_z" in bad
    assert "exceed" in rc(T.tri_mul_block_project, layer.h, z, N, mask, N, 250, 0, 51, 10, 0, a, b)
    assert "direction" in rc(T.tri_mul_block_project, layer.h, z, N, mask, N, 0, 0, 10, 10, 2, a, b)
    v = T.BlockView(N, 0, 0, 64, 64, 0, 64, 0, 0, 0, 1)    # ld_a / ld_b unused
    acc = torch.empty(layer.block_accumulator_size(T.BlockView(N, 0, 0, 64, 64, 0, 64, 64, 64, 0, 1)) // 4,
                      device="cuda")
    zt = torch.empty((64, 64, 128), dtype=torch.bfloat16, device="cuda")
    ot = torch.empty((64, 64, 128), dtype=torch.float32, device="cuda")
    assert "reserve_cus" in rc(T.tri_mul_block_accumulate_blocked, layer.h, v, a, b, acc, mask, zt, ot, -1)
    assert "z_tile" in rc(T.tri_mul_block_accumulate_blocked, layer.h, v, a, b, acc, mask, None, None, 0)
    f32, _ = make_layer("f32")
    assert "bf16" in rc(T.tri_mul_block_panel_size, f32.h, 10, 10)
