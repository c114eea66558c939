"""Seeded synthetic inputs for the triangular multiplicative update.

This module only draws random numbers and rounds them to the storage dtype;
it holds none of the update's arithmetic.  Both the HIP path and the CPU
oracle are fed from it.

Recipe (the paper's workloads are real complexes; seeded Gaussian pair tensors
of the same shapes stand in for them):
  * z ~ N(0, 1) of shape [N][N][c_z], optionally with a per-channel scale
    s ~ U(0.5, 2) (one draw of c_z values);
  * linear weights [out][in] ~ N(0, 1/fan_in) (variance 1/fan_in), no biases;
  * LayerNorm gamma = 1, beta = 0 unless random affine parameters are asked for
    (the tests use them to exercise gamma/beta);
  * token mask uint8 [N] with a suffix of padding tokens set to 0;
  * values drawn in float64 (host) or float32 (device), then rounded to
    nearest-even into float32 or bfloat16.
Each tensor has its own stream: numpy PCG64([seed, stream_id]) on the host,
torch.Generator seeded with seed * 1000 + stream_id on a device.
"""
import numpy as np
import torch

SEED = 2603148060
STREAM = {"z": 1, "w_a": 2, "w_ga": 3, "w_b": 4, "w_gb": 5, "w_g": 6, "w_o": 7,
          "scale": 8, "a_panel": 9, "b_panel": 10, "z_tile": 11,
          "ln_in_w": 12, "ln_in_b": 13, "ln_out_w": 14, "ln_out_b": 15, "dout": 16}

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


def host_rng(name, seed=SEED, sub=0):
    return np.random.Generator(np.random.PCG64([seed, STREAM[name], sub]))


def _round(x64, dtype):
    return torch.from_numpy(np.ascontiguousarray(x64)).to(DTYPES[dtype])


def weights(c_z=128, c=128, dtype="bf16", seed=SEED, affine=False):
    """Layer parameters as CPU tensors of the storage dtype, [out][in] layout."""
    def lin(name, n_out, n_in):
        return _round(host_rng(name, seed).standard_normal((n_out, n_in)) / np.sqrt(n_in), dtype)

    def ln(name_w, name_b, n):
        if not affine:
            return _round(np.ones(n), dtype), _round(np.zeros(n), dtype)
        w = 1.0 + 0.25 * host_rng(name_w, seed).standard_normal(n)
        b = 0.25 * host_rng(name_b, seed).standard_normal(n)
        return _round(w, dtype), _round(b, dtype)

    W = {}
    W["ln_in_w"], W["ln_in_b"] = ln("ln_in_w", "ln_in_b", c_z)
    W["w_a"] = lin("w_a", c, c_z)
    W["w_ga"] = lin("w_ga", c, c_z)
    W["w_b"] = lin("w_b", c, c_z)
    W["w_gb"] = lin("w_gb", c, c_z)
    W["w_g"] = lin("w_g", c_z, c_z)
    W["ln_out_w"], W["ln_out_b"] = ln("ln_out_w", "ln_out_b", c)
    W["w_o"] = lin("w_o", c_z, c)
    return W


def channel_scale(c_z=128, seed=SEED):
    """One draw of c_z per-channel scales s ~ U(0.5, 2)."""
    return host_rng("scale", seed).uniform(0.5, 2.0, size=c_z)


def pair_tensor(N, c_z=128, dtype="bf16", seed=SEED, scale=None, device="cpu",
                name="z", shape=None):
    """z ~ N(0,1) (times an optional per-channel scale) of shape [N][N][c_z]
    (or `shape`), rounded to `dtype`, generated on `device` in row chunks."""
    shape = (N, N, c_z) if shape is None else tuple(shape)
    out = torch.empty(shape, dtype=DTYPES[dtype], device=device)
    rows = shape[0]
    per_row = int(np.prod(shape[1:]))
    chunk = max(1, (1 << 26) // max(1, per_row))
    sc = None if scale is None else np.asarray(scale, dtype=np.float64)
    if torch.device(device).type == "cpu":
        for r0 in range(0, rows, chunk):
            r1 = min(rows, r0 + chunk)
            v = host_rng(name, seed, r0).standard_normal((r1 - r0,) + shape[1:])
            if sc is not None:
                v = v * sc
            out[r0:r1] = _round(v, dtype)
    else:
        gen = torch.Generator(device=device)
        gen.manual_seed(seed * 1000 + STREAM[name])
        sct = None if sc is None else torch.tensor(sc, dtype=torch.float32, device=device)
        for r0 in range(0, rows, chunk):
            r1 = min(rows, r0 + chunk)
            v = torch.randn((r1 - r0,) + shape[1:], generator=gen, device=device,
                            dtype=torch.float32)
            if sct is not None:
                v = v * sct
            out[r0:r1] = v.to(DTYPES[dtype])
    return out


def token_mask(N, n_pad=0, device="cpu"):
    """uint8 [N]: 1 for real tokens, 0 for the last n_pad (padding) tokens."""
    m = torch.ones(N, dtype=torch.uint8, device=device)
    if n_pad:
        m[N - n_pad:] = 0
    return m


def random_mask(N, p_valid=0.8, seed=SEED, sub=0):
    return torch.from_numpy((host_rng("z", seed, 10_000 + sub).random(N) < p_valid)
                            .astype(np.uint8))


# The five workloads of the benchmark table (pair tensors of the paper's
# sizes; the paper's own inputs are real complexes, see the module docstring).
CONFIGS = {
    "c1_fp32_n64": dict(N=64, dtype="f32", n_pad=0, scale=False),
    "c2_bf16_n512_pad51": dict(N=512, dtype="bf16", n_pad=51, scale=False),
    "c3_bf16_n2048_scaled": dict(N=2048, dtype="bf16", n_pad=0, scale=True),
    "c4_bf16_n4096": dict(N=4096, dtype="bf16", n_pad=0, scale=False),
    # one tile of an 8x8 grid at N=30000: tile (7, 7), 8 k-panels of 3750
    "c5_bf16_tile3750_n30000": dict(N=30000, grid=8, tile=(7, 7), dtype="bf16",
                                    n_pad=300, scale=False),
}
