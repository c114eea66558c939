"""Planted mistakes in the fp64 oracles, for checking that the pins catch them.

A pytest plugin (`-p tests.oracle_mutations`): when the environment variable
ORACLE_MUTATION names one of MUTATIONS, the named oracle function is
recompiled from its own source with one substring replaced -- a dropped term,
a wrong sign, a transposed operand, a swapped argument -- before any test
module is imported, and the pin module under test then runs against that
wrong oracle.  tests/test_oracle_mutations.py runs every mutation this way
and requires some pin to fail.  CPU only; nothing here is imported by the
product path or by the unmutated test runs.
"""
import inspect
import os
import textwrap

import pytest

# name: (pin module, oracle module, function, exact source text, replacement)
MUTATIONS = {
    # LayerNorm (both LayerNorms of the layer)
    "ln_unbiased_variance": ("tests/test_oracle.py", "trimul", "layer_norm",
                             "var = (d * d).mean(axis=-1, keepdims=True)",
                             "var = (d * d).sum(axis=-1, keepdims=True) / (v.shape[-1] - 1)"),
    "ln_no_eps": ("tests/test_oracle.py", "trimul", "layer_norm", "np.sqrt(var + eps)", "np.sqrt(var)"),
    "ln_no_bias": ("tests/test_oracle.py", "trimul", "layer_norm", "* f64(gamma) + f64(beta)", "* f64(gamma)"),
    "ln_no_gain": ("tests/test_oracle.py", "trimul", "layer_norm", "* f64(gamma) + f64(beta)", "+ f64(beta)"),
    "ln_mean_not_removed": ("tests/test_oracle.py", "trimul", "layer_norm", "d = v - mu", "d = v"),
    # logistic, linear maps, gating
    "sigmoid_wrong_sign": ("tests/test_oracle.py", "trimul", "sigmoid",
                           "np.where(t >= 0, 1.0 / (1.0 + e), e / (1.0 + e))",
                           "np.where(t >= 0, e / (1.0 + e), 1.0 / (1.0 + e))"),
    "linear_transposed_weights": ("tests/test_oracle.py", "trimul", "linear", "@ f64(w).T", "@ f64(w)"),
    "gate_and_value_swapped": ("tests/test_oracle.py", "trimul", "gated",
                               "sigmoid(linear(x, w_gate)) * linear(x, w_val)",
                               "sigmoid(linear(x, w_val)) * linear(x, w_gate)"),
    "gate_dropped": ("tests/test_oracle.py", "trimul", "gated",
                     "* sigmoid(linear(x, w_gate)) * linear(x, w_val)", "* linear(x, w_val)"),
    "ab_mask_dropped": ("tests/test_oracle.py", "trimul", "gated", "f64(m_pairs)[..., None] * sigmoid", "sigmoid"),
    "pair_mask_or_instead_of_and": ("tests/test_oracle.py", "trimul", "pair_mask",
                                    "return mr[:, None] * mc[None, :]", "return np.maximum(mr[:, None], mc[None, :])"),
    # the contraction (Eq. 2 / Eq. 3)
    "outgoing_b_not_transposed": ("tests/test_oracle.py", "trimul", "contract_outgoing",
                                  "(A @ B.transpose(0, 2, 1))", "(A @ B)"),
    "incoming_reads_rows_of_a": ("tests/test_oracle.py", "trimul", "contract_incoming",
                                 "A = np.ascontiguousarray(f64(a_cols).transpose(2, 1, 0))",
                                 "A = np.ascontiguousarray(f64(a_cols).transpose(2, 0, 1))"),
    "outgoing_a_from_b_weights": ("tests/test_oracle.py", "trimul", "tri_mul",
                                  'pair_mask(mask[rows], mask), W["w_ga"], W["w_a"])',
                                  'pair_mask(mask[rows], mask), W["w_gb"], W["w_b"])'),
    "block_kmask_ignored": ("tests/test_oracle.py", "trimul", "block_contract",
                            "part = (ap * keep[None, None, :]) @ bp.transpose(0, 2, 1)",
                            "part = ap @ bp.transpose(0, 2, 1)"),
    # the epilogue
    "output_layernorm_dropped": ("tests/test_oracle.py", "trimul", "epilogue",
                                 'y = linear(layer_norm(C, W["ln_out_w"], W["ln_out_b"], eps), W["w_o"])',
                                 'y = linear(C, W["w_o"])'),
    "output_projection_transposed": ("tests/test_oracle.py", "trimul", "epilogue",
                                     'eps), W["w_o"])', 'eps), W["w_o"].T)'),
    "output_gate_dropped": ("tests/test_oracle.py", "trimul", "epilogue",
                            "return f64(m_pairs)[..., None] * f64(g) * y", "return f64(m_pairs)[..., None] * y"),
    "output_mask_dropped": ("tests/test_oracle.py", "trimul", "epilogue",
                            "return f64(m_pairs)[..., None] * f64(g) * y", "return f64(g) * y"),
    "gate_from_raw_z_in_update": ("tests/test_oracle.py", "trimul", "tri_mul",
                                  'g = sigmoid(linear(ln(take_pairs(z, rows, cols)), W["w_g"]))',
                                  'g = sigmoid(linear(take_pairs(z, rows, cols), W["w_g"]))'),
    "gate_from_raw_z_in_project": ("tests/test_oracle.py", "trimul", "project",
                                   'g = sigmoid(linear(x, W["w_g"]))', 'g = sigmoid(linear(f64(z_pairs), W["w_g"]))'),
    # backward of the layer
    "ln_backward_variance_term_dropped": ("tests/test_oracle_backward.py", "trimul", "layer_norm_backward",
                                          " - xh * (dxh * xh).mean(axis=-1, keepdims=True))", ")"),
    "ln_backward_mean_term_dropped": ("tests/test_oracle_backward.py", "trimul", "layer_norm_backward",
                                      "dxh - dxh.mean(axis=-1, keepdims=True) - ", "dxh - "),
    "ln_backward_gain_gradient_unnormalised": ("tests/test_oracle_backward.py", "trimul", "layer_norm_backward",
                                               "(dy * xh).sum(axis=lead)", "dy.sum(axis=lead)"),
    "contract_backward_dc_not_transposed": ("tests/test_oracle_backward.py", "trimul", "contract_backward",
                                            "dC.transpose(0, 2, 1) @ A", "dC @ A"),
    "output_gate_derivative_wrong": ("tests/test_oracle_backward.py", "trimul", "tri_mul_backward",
                                     "dgg = dout * m * u * sg * (1.0 - sg)", "dgg = dout * m * u * sg"),
    "a_gate_derivative_wrong": ("tests/test_oracle_backward.py", "trimul", "tri_mul_backward",
                                "da * m * pa * sa * (1.0 - sa)", "da * m * pa * sa"),
    "dx_output_gate_term_dropped": ("tests/test_oracle_backward.py", "trimul", "tri_mul_backward",
                                    '\n          + dgg @ f64(W["w_g"]))', ")"),
    "incoming_gradient_transposed": ("tests/test_oracle_backward.py", "trimul", "tri_mul_backward",
                                     "da, db = dA.transpose(2, 1, 0), dB.transpose(2, 1, 0)",
                                     "da, db = dA.transpose(1, 2, 0), dB.transpose(1, 2, 0)"),
    # triangle attention core
    "attention_scale_dropped": ("tests/test_oracle_triattn.py", "triattn", "scores", " / np.sqrt(d)", ""),
    "attention_bias_transposed": ("tests/test_oracle_triattn.py", "triattn", "scores",
                                  "s = s + b[None]", "s = s + b[None].swapaxes(-1, -2)"),
    "attention_mask_ignored": ("tests/test_oracle_triattn.py", "triattn", "scores",
                               "return np.where(m[None, None, None, :] != 0, s, -np.inf)", "return s"),
    "attention_not_normalised": ("tests/test_oracle_triattn.py", "triattn", "triangle_attention",
                                 "out = np.matmul(w, v", "out = np.matmul(p, v"),
    "chunk_merge_output_not_rescaled": ("tests/test_oracle_triattn.py", "triattn", "chunked_attention",
                                        "A = A * scale[..., None] + ", "A = A + "),
    "chunk_merge_sum_not_rescaled": ("tests/test_oracle_triattn.py", "triattn", "chunked_attention",
                                     "L = L * scale + ", "L = L + "),
    # outer product mean
    "opm_divides_by_all_sequences": ("tests/test_oracle_opm.py", "opm", "outer_product_mean_tile",
                                     "o = o * inv[:, :, None, None]", "o = o / S"),
    "opm_bias_dropped": ("tests/test_oracle_opm.py", "opm", "outer_product_mean_tile", " + f64(b_o)", ""),
    "opm_flatten_order_swapped": ("tests/test_oracle_opm.py", "opm", "outer_sum",
                                  ".transpose(0, 2, 1, 3)", ".transpose(0, 2, 3, 1)"),
    "opm_mask_of_b_ignored": ("tests/test_oracle_opm.py", "opm", "outer_sum",
                              "bm = (b * mb[..., None])", "bm = b"),
}


def apply(name):
    """Recompile the mutated function in its module's namespace and bind it
    there and in the oracle package."""
    import importlib

    import oracle
    _, modname, func, old, new = MUTATIONS[name]
    mod = importlib.import_module(f"oracle.{modname}")
    src = textwrap.dedent(inspect.getsource(getattr(mod, func)))
    if src.count(old) != 1:
        raise pytest.UsageError(f"mutation {name}: {old!r} occurs {src.count(old)} times in {modname}.{func}")
    ns = {}
    exec(compile(src.replace(old, new), f"<mutation {name}>", "exec"), mod.__dict__, ns)
    setattr(mod, func, ns[func])
    if hasattr(oracle, func):
        setattr(oracle, func, ns[func])


def pytest_configure(config):
    name = os.environ.get("ORACLE_MUTATION")
    if name:
        apply(name)
