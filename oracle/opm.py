"""fp64 CPU oracle for the outer product mean (Fold-CP, Section 3.5).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module; only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code, constants or helpers with the HIP library.

What it computes (Section 3.5, the equation for z_ijcd): a and b are
linear maps of the MSA features, shape [S][N][D] (sequences, tokens,
channels).  The pair feature of tokens (i, j) is the mean over sequences of
the outer product a_si (x) b_sj, a D x D matrix, which is flattened (index
c * D + d) and linearly projected to c_z channels:

    n_ij   = sum_s m_si m_sj                         (sequences holding both tokens)
    o_ijcd = (1 / n_ij) sum_s m_si m_sj a_sic b_sjd  (o_ij = 0 where n_ij = 0)
    out_ij = W_o vec(o_ij) + b_o                     (W_o: [c_z][D * D], b_o: [c_z])

Readings (the paper writes the mean as 1/|S| and has a single all-reduce
finish a count of the mask): the count is taken per pair, over the sequences
in which both tokens are present (m_si = 1, uint8 MSA mask [S][N]); with every
token present it is |S|, the paper's normalisation.  The projection is a
linear map with bias, applied after the mean.  a and b enter as given; the
mask multiplies them inside the sum (so masked entries never contribute).

Precision: every input is converted exactly to float64 and every step is
float64.  numpy.matmul is the only library primitive (the s-contraction and
the projection), with no blocking or reordering beyond the definition.
"""
import numpy as np

from .trimul import f64


def msa_mask(mask, S, N):
    """The MSA mask as float64 0/1 [S][N] (None: every token present)."""
    if mask is None:
        return np.ones((S, N))
    return (f64(mask) != 0).astype(np.float64)


def pair_counts(mask, S, N):
    """n_ij = sum_s m_si m_sj, the number of sequences holding both tokens."""
    m = msa_mask(mask, S, N)
    return m.T @ m


def outer_sum(a, b, mask):
    """sum_s m_si m_sj a_sic b_sjd as [N_a][N_b][D][D] (a: [S][N_a][D], b: [S][N_b][D];
    mask: ([S][N_a], [S][N_b]) pair of masks or None)."""
    a, b = f64(a), f64(b)
    S, Na, D = a.shape
    Nb = b.shape[1]
    ma = msa_mask(None if mask is None else mask[0], S, Na)
    mb = msa_mask(None if mask is None else mask[1], S, Nb)
    am = (a * ma[..., None]).reshape(S, Na * D)
    bm = (b * mb[..., None]).reshape(S, Nb * D)
    o = am.T @ bm                                   # [(i, c)][(j, d)]
    return o.reshape(Na, D, Nb, D).transpose(0, 2, 1, 3)


def outer_product_mean(a, b, mask, w_o, b_o):
    """The whole op: a, b [S][N][D], mask [S][N] (or None), w_o [c_z][D * D],
    b_o [c_z] -> out [N][N][c_z] (float64)."""
    return outer_product_mean_tile(a, b, mask, w_o, b_o, 0, f64(a).shape[1], 0, f64(b).shape[1])


def outer_product_mean_tile(a, b, mask, w_o, b_o, row0, rows, col0, cols, s0=0, slen=None):
    """The op restricted to tokens i in [row0, row0 + rows), j in [col0, col0 + cols)
    and sequences s in [s0, s0 + slen) (one device's tile of the pair
    representation and the sequences its ring steps bring in)."""
    a, b = f64(a), f64(b)
    S = a.shape[0]
    if slen is None:
        slen = S - s0
    m = msa_mask(mask, S, a.shape[1])
    sl = slice(s0, s0 + slen)
    ai, bj = a[sl, row0:row0 + rows], b[sl, col0:col0 + cols]
    mi, mj = m[sl, row0:row0 + rows], m[sl, col0:col0 + cols]
    o = outer_sum(ai, bj, (mi, mj))                 # [rows][cols][D][D]
    n = mi.T @ mj                                   # [rows][cols]
    inv = np.divide(1.0, n, out=np.zeros_like(n), where=n > 0)
    o = o * inv[:, :, None, None]
    D = ai.shape[2]
    return o.reshape(rows, cols, D * D) @ f64(w_o).T + f64(b_o)
