"""fp64 CPU oracle for the triangular multiplicative update.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this module; only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code, constants or helpers with the HIP library.

What it computes (Fold-CP, Section 3.3, Eq. 2 and Eq. 3):

    outgoing:  C[n, m, c] = sum_k a[n, k, c] * b[m, k, c]
    incoming:  C[n, m, c] = sum_k a[k, n, c] * b[k, m, c]

where a and b are gated linear maps of the pair tensor
z in R^{N x N x c_z} (Section 3.3 names only projections of z and an
element-wise gate; the concrete layer is the usual AlphaFold-family triangle
update that the paper's Boltz models use, written out as mathematics below).  For a pair
(i, j) with pair mask m_ij = m_i * m_j:

    x_ij   = LN_in(z_ij)                               (over c_z, biased var)
    a_ij   = m_ij * sigmoid(W_ga x_ij) * (W_a x_ij)    (c values)
    b_ij   = m_ij * sigmoid(W_gb x_ij) * (W_b x_ij)
    g_ij   = sigmoid(W_g x_ij)                         (c_z values)
    out_ij = m_ij * g_ij * (W_o LN_out(C_ij))          (c_z values)

The function returns the update (the right-hand side of Eq. 2/3 after the
output projection and gate); the residual add z + out is the caller's step.
There is no 1/N normalisation of the k-sum (Eq. 2/3 have none).

Precision: every input is converted exactly to float64 and every step is
float64.  Library primitives used as single steps: numpy.matmul (the linear
maps and the per-channel contraction) and numpy.exp.  No blocking, fusion or
reordering beyond the definition.

Weight layout: linear maps are [out][in] (y = W x), as in torch.nn.Linear.
"""
import numpy as np

EPS = 1e-5

WEIGHT_NAMES = ("ln_in_w", "ln_in_b", "w_a", "w_ga", "w_b", "w_gb", "w_g",
                "ln_out_w", "ln_out_b", "w_o")


def f64(x):
    """Exact conversion of an input array (float32, bfloat16 via torch, ...) to float64."""
    if hasattr(x, "detach"):                       # a CPU torch tensor
        return x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def layer_norm(v, gamma, beta, eps=EPS):
    """LayerNorm over the last axis: (v - mean) / sqrt(var + eps) * gamma + beta,
    with the biased variance (divide by the vector length)."""
    v = f64(v)
    mu = v.mean(axis=-1, keepdims=True)
    d = v - mu
    var = (d * d).mean(axis=-1, keepdims=True)
    return d / np.sqrt(var + eps) * f64(gamma) + f64(beta)


def sigmoid(t):
    """Logistic function 1 / (1 + exp(-t)), evaluated without overflow:
    with e = exp(-|t|), 1 / (1 + e) for t >= 0 and e / (1 + e) for t < 0."""
    t = f64(t)
    e = np.exp(-np.abs(t))
    return np.where(t >= 0, 1.0 / (1.0 + e), e / (1.0 + e))


def pair_mask(mask_rows, mask_cols=None):
    """m_ij = m_i * m_j from per-token masks (nonzero = valid token)."""
    mr = (f64(mask_rows) != 0).astype(np.float64)
    mc = mr if mask_cols is None else (f64(mask_cols) != 0).astype(np.float64)
    return mr[:, None] * mc[None, :]


def linear(x, w):
    """y = W x on the last axis; W is [out][in]."""
    return f64(x) @ f64(w).T


def gated(x, m_pairs, w_gate, w_val):
    """One gated projection of normalised pairs x: m * sigmoid(W_gate x) * (W_val x)."""
    return f64(m_pairs)[..., None] * sigmoid(linear(x, w_gate)) * linear(x, w_val)


def project(z_pairs, m_pairs, W, eps=EPS):
    """Input LayerNorm and the two gated projections plus the output gate for a
    block of pairs (Section 3.3: a, b are gated projections of z).

    z_pairs: [..., c_z]; m_pairs: [...] pair mask.  Returns (a, b, g) with
    a, b: [..., c] and g: [..., c_z]."""
    x = layer_norm(z_pairs, W["ln_in_w"], W["ln_in_b"], eps)
    a = gated(x, m_pairs, W["w_ga"], W["w_a"])
    b = gated(x, m_pairs, W["w_gb"], W["w_b"])
    g = sigmoid(linear(x, W["w_g"]))
    return a, b, g


def contract_outgoing(a_rows, b_rows):
    """Eq. 2: C[n, m, c] = sum_k a[n, k, c] * b[m, k, c].

    a_rows: [n, K, c] (rows n of a), b_rows: [m, K, c].  Returns [n, m, c]."""
    A = np.ascontiguousarray(f64(a_rows).transpose(2, 0, 1))     # [c][n][k]
    B = np.ascontiguousarray(f64(b_rows).transpose(2, 0, 1))     # [c][m][k]
    return (A @ B.transpose(0, 2, 1)).transpose(1, 2, 0)          # [n][m][c]


def contract_incoming(a_cols, b_cols):
    """Eq. 3: C[n, m, c] = sum_k a[k, n, c] * b[k, m, c].

    a_cols: [K, n, c] (columns n of a), b_cols: [K, m, c].  Returns [n, m, c]."""
    A = np.ascontiguousarray(f64(a_cols).transpose(2, 1, 0))     # [c][n][k]
    B = np.ascontiguousarray(f64(b_cols).transpose(2, 1, 0))     # [c][m][k]
    return (A @ B.transpose(0, 2, 1)).transpose(1, 2, 0)


def epilogue(C, g, m_pairs, W, eps=EPS):
    """Output LayerNorm over the hidden channels, output projection, sigmoid
    gate and pair mask: out = m * g * (W_o LN_out(C))."""
    y = linear(layer_norm(C, W["ln_out_w"], W["ln_out_b"], eps), W["w_o"])
    return f64(m_pairs)[..., None] * f64(g) * y


def take_pairs(z, rows=None, cols=None):
    """z[rows][:, cols] as float64, converting only the selected pairs (z may be
    a numpy array or a torch tensor, also on a device)."""
    if hasattr(z, "detach"):
        import torch
        if rows is not None:
            z = z[torch.as_tensor(rows, device=z.device)]
        if cols is not None:
            z = z[:, torch.as_tensor(cols, device=z.device)]
        return f64(z)
    z = np.asarray(z)
    if rows is not None:
        z = z[rows]
    if cols is not None:
        z = z[:, cols]
    return f64(z)


def tri_mul(z, mask, W, direction, rows=None, cols=None, eps=EPS):
    """The whole update for one pair tensor z [N][N][c_z] and token mask [N].

    direction: "outgoing" (Eq. 2) or "incoming" (Eq. 3).  rows / cols select
    the output pairs (index arrays; default all), so large N can be checked on
    a sample.  Returns out[len(rows)][len(cols)][c_z] in float64."""
    mask = f64(mask)
    N = z.shape[0]
    rows = np.arange(N) if rows is None else np.asarray(rows)
    cols = np.arange(N) if cols is None else np.asarray(cols)
    def ln(pairs):
        return layer_norm(pairs, W["ln_in_w"], W["ln_in_b"], eps)

    # each block of pairs gets only the projection the update reads from it
    if direction == "outgoing":
        # a[i, k] for i in rows, all k; b[j, k] for j in cols, all k.
        a = gated(ln(take_pairs(z, rows)), pair_mask(mask[rows], mask), W["w_ga"], W["w_a"])
        b = gated(ln(take_pairs(z, cols)), pair_mask(mask[cols], mask), W["w_gb"], W["w_b"])
        C = contract_outgoing(a, b)
    elif direction == "incoming":
        # a[k, i] for i in rows, all k; b[k, j] for j in cols, all k.
        a = gated(ln(take_pairs(z, None, rows)), pair_mask(mask, mask[rows]), W["w_ga"], W["w_a"])
        b = gated(ln(take_pairs(z, None, cols)), pair_mask(mask, mask[cols]), W["w_gb"], W["w_b"])
        C = contract_incoming(a, b)
    else:
        raise ValueError(f"direction must be 'outgoing' or 'incoming', got {direction!r}")
    m_out = pair_mask(mask[rows], mask[cols])
    g = sigmoid(linear(ln(take_pairs(z, rows, cols)), W["w_g"]))
    return epilogue(C, g, m_out, W, eps)


def projected_panels(z, mask, W, direction, eps=EPS):
    """The channel-major operands of the contraction, A[c][i][k] and B[c][j][k],
    such that C[c] = A[c] @ B[c]^T for either direction:
    outgoing A[c][i][k] = a[i, k, c]; incoming A[c][i][k] = a[k, i, c]."""
    z = f64(z)
    a, b, _ = project(z, pair_mask(mask), W, eps)
    if direction == "outgoing":
        return a.transpose(2, 0, 1), b.transpose(2, 0, 1)
    if direction == "incoming":
        return a.transpose(2, 1, 0), b.transpose(2, 1, 0)
    raise ValueError(direction)


def block_contract(a_panels, b_panels, kmasks, rows=None, cols=None):
    """One device tile of the 2-D pair tiling (Section 2.1.1) accumulated over
    its k-panels, as in the Cannon ring of Section 3.3 where each ring step adds
    the product of the resident a and b blocks into the output block.

    a_panels[p]: [c][R][K_p] (row-panel of a for k-panel p, channel-major),
    b_panels[p]: [c][S][K_p], kmasks[p]: [K_p] token mask of that k range.
    C[i, j, c] = sum_p sum_k a_p[c, i, k] * b_p[c, j, k] * (kmask_p[k] != 0).
    rows / cols select tile rows/cols.  Returns [len(rows)][len(cols)][c]."""
    C = None
    for ap, bp, km in zip(a_panels, b_panels, kmasks):
        ap = f64(ap)
        bp = f64(bp)
        if rows is not None:
            ap = ap[:, rows]
        if cols is not None:
            bp = bp[:, cols]
        keep = (f64(km) != 0).astype(np.float64)
        part = (ap * keep[None, None, :]) @ bp.transpose(0, 2, 1)    # [c][i][j]
        C = part if C is None else C + part
    return C.transpose(1, 2, 0)


def block_epilogue(C_tile, z_tile, row_mask, col_mask, W, eps=EPS):
    """Epilogue of one device tile: the gate comes from the tile's own z and
    the pair mask from the tile's global token indices."""
    m = pair_mask(row_mask, col_mask)
    _, _, g = project(z_tile, m, W, eps)
    return epilogue(C_tile, g, m, W, eps)


# ---------------------------------------------------------------- backward
#
# Gradients of the update for training.  The paper gives every distributed
# module an explicit backward pass that runs the same ring schedule as its
# forward (Section 3.1); for this layer the backward of the contraction is two
# more per-channel products of the same size.  Chain rule of the forward
# above, written out step by step.


def layer_norm_backward(dy, v, gamma, eps=EPS):
    """For y = (v - mu) / sqrt(var + eps) * gamma + beta over the last axis,
    given dL/dy return (dL/dv, dL/dgamma, dL/dbeta), the parameter gradients
    summed over all leading axes."""
    v = f64(v)
    dy = f64(dy)
    mu = v.mean(axis=-1, keepdims=True)
    d = v - mu
    rs = 1.0 / np.sqrt((d * d).mean(axis=-1, keepdims=True) + eps)
    xh = d * rs                                   # the normalised vector
    dxh = dy * f64(gamma)
    dv = rs * (dxh - dxh.mean(axis=-1, keepdims=True) - xh * (dxh * xh).mean(axis=-1, keepdims=True))
    lead = tuple(range(dy.ndim - 1))
    return dv, (dy * xh).sum(axis=lead), dy.sum(axis=lead)


def contract_backward(A, B, dC):
    """Backward of the per-channel contraction C[c] = A[c] @ B[c]^T (the form
    both directions take on the channel-major operands): given dL/dC return
        dA[c] = dC[c] @ B[c],   dB[c] = dC[c]^T @ A[c].
    A: [c][n][K], B: [c][m][K], dC: [c][n][m]."""
    # contiguous copies, as in the forward contraction, so that numpy hands
    # each channel's product to BLAS instead of its strided fallback loop
    A, B, dC = (np.ascontiguousarray(f64(x)) for x in (A, B, dC))
    return dC @ B, dC.transpose(0, 2, 1) @ A


def tri_mul_backward(z, mask, W, direction, dout, eps=EPS):
    """Gradients of sum(out * dout) for the whole update (all pairs).

    Returns a dict: "dz" [N][N][c_z] and one entry per weight name of
    WEIGHT_NAMES (same shapes as the weights; gradients summed over pairs)."""
    z = f64(z)
    dout = f64(dout)
    m = pair_mask(mask)[..., None]
    x = layer_norm(z, W["ln_in_w"], W["ln_in_b"], eps)
    pa, ga = linear(x, W["w_a"]), linear(x, W["w_ga"])
    pb, gb = linear(x, W["w_b"]), linear(x, W["w_gb"])
    sa, sb = sigmoid(ga), sigmoid(gb)
    a, b = m * sa * pa, m * sb * pb
    sg = sigmoid(linear(x, W["w_g"]))
    if direction == "outgoing":
        C = contract_outgoing(a, b)
    elif direction == "incoming":
        C = contract_incoming(a, b)
    else:
        raise ValueError(direction)
    y = layer_norm(C, W["ln_out_w"], W["ln_out_b"], eps)
    u = linear(y, W["w_o"])

    cz, c = u.shape[-1], y.shape[-1]
    g = {}
    du = dout * m * sg                            # out = m * sg * u
    dgg = dout * m * u * sg * (1.0 - sg)          # d/d(W_g x) through the logistic
    g["w_o"] = du.reshape(-1, cz).T @ y.reshape(-1, c)
    dy = du @ f64(W["w_o"])
    dC, g["ln_out_w"], g["ln_out_b"] = layer_norm_backward(dy, C, W["ln_out_w"], eps)

    # contraction: outgoing C = A B^T with A[c][i][k] = a[i][k][c]; incoming
    # with A[c][i][k] = a[k][i][c] -- the same channel-major form.
    dCc = dC.transpose(2, 0, 1)
    if direction == "outgoing":
        dA, dB = contract_backward(a.transpose(2, 0, 1), b.transpose(2, 0, 1), dCc)
        da, db = dA.transpose(1, 2, 0), dB.transpose(1, 2, 0)
    else:
        dA, dB = contract_backward(a.transpose(2, 1, 0), b.transpose(2, 1, 0), dCc)
        da, db = dA.transpose(2, 1, 0), dB.transpose(2, 1, 0)

    dpa, dga = da * m * sa, da * m * pa * sa * (1.0 - sa)
    dpb, dgb = db * m * sb, db * m * pb * sb * (1.0 - sb)
    xf = x.reshape(-1, x.shape[-1])
    for name, d in (("w_a", dpa), ("w_ga", dga), ("w_b", dpb), ("w_gb", dgb), ("w_g", dgg)):
        g[name] = d.reshape(-1, d.shape[-1]).T @ xf
    dx = (dpa @ f64(W["w_a"]) + dga @ f64(W["w_ga"]) + dpb @ f64(W["w_b"]) + dgb @ f64(W["w_gb"])
          + dgg @ f64(W["w_g"]))
    g["dz"], g["ln_in_w"], g["ln_in_b"] = layer_norm_backward(dx, z, W["ln_in_w"], eps)
    return g
