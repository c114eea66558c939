"""Algorithmic work and traffic of the kernels (for throughput and roofline
figures).  A multiply-add counts as 2 flops."""

# MI355X published peaks
PEAK_BF16_TFLOPS = 2516.6      # dense bf16 MFMA: 256 CUs x 4096 flop/clk x 2.4 GHz
PEAK_FP32_VALU_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


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
