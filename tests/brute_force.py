"""Scalar pure-Python brute force of the triangular multiplicative update, for
tiny N only.  It is written straight from the index expressions of Eq. 2
(outgoing: z_nm += sum_k a_nk * b_mk) and Eq. 3 (incoming: z_nm += sum_k
a_kn * b_km) of Section 3.3, with the layer's LayerNorms, gated projections and
output gate written as explicit loops over scalars.  It uses no numpy and
shares nothing with the vectorised oracle, so an index, transpose or dropped
term in either one shows up as a mismatch.
"""
import math

EPS = 1e-5


def _ln(v, gamma, beta):
    n = len(v)
    mu = sum(v) / n
    var = sum((x - mu) * (x - mu) for x in v) / n
    s = math.sqrt(var + EPS)
    return [(v[t] - mu) / s * gamma[t] + beta[t] for t in range(n)]


def _sig(t):
    if t >= 0:
        return 1.0 / (1.0 + math.exp(-t))
    e = math.exp(t)
    return e / (1.0 + e)


def _matvec(W, x):
    return [sum(W[o][d] * x[d] for d in range(len(x))) for o in range(len(W))]


def brute_tri_mul(z, mask, W, direction):
    """z: nested lists [N][N][c_z]; mask: list [N]; W: dict of nested lists.
    Returns nested lists out[N][N][c_z]."""
    N = len(z)
    valid = [1.0 if mask[t] else 0.0 for t in range(N)]
    a = [[None] * N for _ in range(N)]
    b = [[None] * N for _ in range(N)]
    g = [[None] * N for _ in range(N)]
    for i in range(N):
        for j in range(N):
            x = _ln(z[i][j], W["ln_in_w"], W["ln_in_b"])
            m = valid[i] * valid[j]
            pa, qa = _matvec(W["w_ga"], x), _matvec(W["w_a"], x)
            pb, qb = _matvec(W["w_gb"], x), _matvec(W["w_b"], x)
            a[i][j] = [m * _sig(pa[c]) * qa[c] for c in range(len(qa))]
            b[i][j] = [m * _sig(pb[c]) * qb[c] for c in range(len(qb))]
            g[i][j] = [_sig(t) for t in _matvec(W["w_g"], x)]
    hidden = len(W["w_a"])
    out = [[None] * N for _ in range(N)]
    for n in range(N):
        for m_ in range(N):
            if direction == "outgoing":
                C = [sum(a[n][k][c] * b[m_][k][c] for k in range(N)) for c in range(hidden)]
            else:
                C = [sum(a[k][n][c] * b[k][m_][c] for k in range(N)) for c in range(hidden)]
            y = _matvec(W["w_o"], _ln(C, W["ln_out_w"], W["ln_out_b"]))
            mm = valid[n] * valid[m_]
            out[n][m_] = [mm * g[n][m_][d] * y[d] for d in range(len(y))]
    return out
