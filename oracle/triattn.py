"""fp64 CPU oracle for the triangle attention core (Fold-CP, Section 3.2, Eq. 1).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module; only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code, constants or helpers with the HIP library.

What it computes (Eq. 1, attention around the starting node): for every row
i of the pair representation, head h and query pair (i, j),

    s_ijk = (q_ijh . k_ikh) / sqrt(d) + b_hjk      over keys k with m_k = 1
    out_ijh = sum_k softmax_k(s_ijk) v_ikh

q, k, v: [rows][N][H][d] (the projections of z, Eq. 1's proj), b: [H][N][N]
(Eq. 1's tri_bias(z), one value per head and pair (j, k): it does not depend
on the row i, which is what couples the three axes), m: [N] token mask
(Eq. 1's mask_bias: keys with m_k = 0 are excluded, i.e. the bias is -inf).
Readings: if no key is present the output is 0; the softmax is the exact
one (the paper's ring computes it in chunks with a running log-sum-exp and
states that this preserves exact equivalence).

chunked_attention follows the paper's ring: the keys arrive in chunks; each
chunk's partial scores update a running maximum M, a running sum L of
exp(s - M) and an unnormalised output A, rescaled by exp(M_old - M_new);
the final output is A / L.

Precision: every input is converted exactly to float64 and every step is
float64.  numpy.matmul and numpy.exp are the library primitives.
"""
import numpy as np

from .trimul import f64


def key_mask(mask, N):
    """float64 0/1 [N] (None: all present)."""
    if mask is None:
        return np.ones(N)
    return (f64(mask) != 0).astype(np.float64)


def scores(q, k, bias, mask):
    """s[i][h][j][k] = q_ijh . k_ikh / sqrt(d) + b_hjk, -inf on absent keys."""
    q, k, b = f64(q), f64(k), f64(bias)
    d = q.shape[-1]
    s = np.matmul(q.transpose(0, 2, 1, 3), k.transpose(0, 2, 3, 1)) / np.sqrt(d)   # [rows][H][N][N]
    s = s + b[None]
    m = key_mask(mask, k.shape[1])
    return np.where(m[None, None, None, :] != 0, s, -np.inf)


def triangle_attention(q, k, v, bias, mask):
    """out [rows][N][H][d] (float64) by the plain softmax over all keys."""
    s = scores(q, k, bias, mask)
    v = f64(v)
    mx = s.max(axis=-1, keepdims=True)
    ok = np.isfinite(mx)
    p = np.exp(np.where(ok, s - np.where(ok, mx, 0.0), -np.inf))
    den = p.sum(axis=-1, keepdims=True)
    w = np.divide(p, den, out=np.zeros_like(p), where=den > 0)
    out = np.matmul(w, v.transpose(0, 2, 1, 3))                                   # [rows][H][N][d]
    return out.transpose(0, 2, 1, 3)


def chunked_attention(q, k, v, bias, mask, cuts):
    """The same output computed over key chunks [cuts[t], cuts[t+1]) with the
    running log-sum-exp merge of the paper's ring (Section 3.2)."""
    q, k, v, b = f64(q), f64(k), f64(v), f64(bias)
    rows, N, H, d = q.shape
    m = key_mask(mask, N)
    M = np.full((rows, H, N), -np.inf)
    L = np.zeros((rows, H, N))
    A = np.zeros((rows, H, N, d))
    for k0, k1 in zip(cuts[:-1], cuts[1:]):
        s = scores(q, k[:, k0:k1], b[:, :, k0:k1], m[k0:k1])                       # [rows][H][N][nk]
        cm = s.max(axis=-1)
        Mn = np.maximum(M, cm)
        fin = np.isfinite(Mn)
        scale = np.where(fin & np.isfinite(M), np.exp(np.where(np.isfinite(M), M, 0.0) - np.where(fin, Mn, 0.0)), 0.0)
        p = np.exp(np.where(fin[..., None], s - np.where(fin, Mn, 0.0)[..., None], -np.inf))
        L = L * scale + p.sum(axis=-1)
        A = A * scale[..., None] + np.matmul(p, v[:, k0:k1].transpose(0, 2, 1, 3))
        M = Mn
    out = np.divide(A, L[..., None], out=np.zeros_like(A), where=L[..., None] > 0)
    return out.transpose(0, 2, 1, 3)
