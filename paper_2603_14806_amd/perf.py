"""Algorithmic work and traffic of the kernels (for throughput and roofline
figures).  A multiply-add counts as 2 flops."""

# MI355X published peaks
PEAK_BF16_TFLOPS = 2516.6      # dense bf16 MFMA: 256 CUs x 4096 flop/clk x 2.4 GHz
PEAK_FP32_VALU_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
CUS, BF16_FLOP_PER_CLK_CU = 256, 4096


def bf16_peak_at(mhz):
    """Dense bf16 MFMA peak (TFLOP/s) at a graphics clock of `mhz`."""
    return CUS * BF16_FLOP_PER_CLK_CU * mhz * 1e6 / 1e12


def flops(N, c_z=128, c=128):
    """Per direction: K1 gated a/b projections, K2 contraction, K3 output gate
    and output projection."""
    proj = 2.0 * N * N * c_z * (4 * c)
    contraction = 2.0 * N ** 3 * c
    epi = 2.0 * N * N * (c_z * c_z + c_z * c)
    return {"project": proj, "contract": contraction, "epilogue": epi, "total": proj + contraction + epi}


def bytes_moved(N, c_z=128, c=128, esize=2, out_esize=4):
    """Compulsory HBM bytes per direction of each kernel (each tensor read or
    written once)."""
    ab = 2 * N * N * c * esize
    cbytes = N * N * c * 4
    return {"project": N * N * c_z * esize + ab,
            "contract": ab + cbytes,
            "epilogue": cbytes + N * N * c_z * esize + N * N * c_z * out_esize}


# fp32 vector lane-operations: 256 CUs x 4 SIMDs x 32 lanes per clock x 2.4 GHz
# = 78.6 T/s (an FMA counts once: the published 157.3 TFLOP/s fp32 vector peak
# is this rate of FMAs).  A timing loop of dependent-free fp32 adds on the
# chip ran at 70 T/s (0.89 of it), exp2 and reciprocal at 15.6 and 16.2 T/s:
# a transcendental takes about four lane-operation slots.
PEAK_LANE_OPS = 256 * 4 * 32 * 2.4e9


def backward_layer_work(N, c_z=128, c=128, recompute=True):
    """One direction of the layer backward as the library runs it: the MFMA
    flops of its N^3 products (the recomputed forward contraction unless the
    forward's state is passed in, dA and dB) and the algorithmic HBM bytes of
    its per-pair kernels (per pair: projection recompute 768 B (recompute
    only), epilogue backward 3072 B, projection backward 3328 B, six
    weight-gradient sums 6 x 512 B = 10240 B at c_z = c = 128 with the
    recompute; the products read their transposed operands in place)."""
    mfma = (3 if recompute else 2) * 2.0 * N ** 3 * c
    per_pair = (c_z * 2 + 2 * c * 2 if recompute else 0) \
        + (c * 4 + c_z * 2 + c_z * 4 + c * 2 + c_z * 4 + 4 * 2 * c) \
        + (2 * c * 4 + c_z * 2 + c_z * 4 + c_z * 2 + 5 * 2 * c) + 6 * 4 * c
    return {"mfma_flops": mfma, "hbm_bytes": float(per_pair) * N * N,
            "floor_ms": 1e3 * (mfma / (PEAK_BF16_TFLOPS * 1e12) + per_pair * N * N / (PEAK_HBM_GBS * 1e9))}


# Triangle attention is bound by the vector ALU: the fewest lane-operation
# slots one score of an fp32 online softmax needs -- scale-and-bias FMA,
# running maximum, shift (FMA with log2 e), exp2, running sum, and half a
# bf16 pack for the P V product -- with exp2 taking EXP2_SLOTS slots.
EXP2_SLOTS = 4
TRIATTN_SLOTS = 4.5 + EXP2_SLOTS
TRIATTN_BASIS = (f"{PEAK_LANE_OPS / 1e12:.1f} T lane-ops/s / {TRIATTN_SLOTS} slots per score (FMA scale+bias, max, "
                 f"FMA shift, exp2 at {EXP2_SLOTS} slots, sum, half a bf16 pack)")
