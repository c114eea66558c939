"""Helpers shared by the GPU parity tests: seeded inputs on the device, the
library wrapper, and the tolerance checks (fp32 path: relative Frobenius
error <= 1e-5; bf16 path: max-abs <= 2e-2 and relative Frobenius <= 5e-3,
both against the fp64 oracle on the checked elements)."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import synth
from paper_2603_14806_amd.trimul import TriMul
from tests.progress import say  # noqa: F401  (re-exported for the tests)

TOL = {"f32": dict(max_abs=None, rel_fro=1e-5), "bf16": dict(max_abs=2e-2, rel_fro=5e-3)}

needs_gpu = pytest.mark.skipif(not torch.cuda.is_available(), reason="no GPU visible")




def errors(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = got - ref
    nref = np.linalg.norm(ref)
    rel = np.linalg.norm(d) / nref if nref > 0 else (0.0 if not np.any(d) else np.inf)
    return float(np.max(np.abs(d))) if d.size else 0.0, float(rel)


def assert_close(got, ref, dtype, what=""):
    mx, rel = errors(got, ref)
    tol = TOL[dtype]
    say(f"  {what}: max_abs={mx:.3e} rel_fro={rel:.3e} n={np.asarray(ref).size}")
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    assert rel <= tol["rel_fro"], f"{what}: relative Frobenius error {rel:.3e} > {tol['rel_fro']}"
    if tol["max_abs"] is not None:
        assert mx <= tol["max_abs"], f"{what}: max-abs error {mx:.3e} > {tol['max_abs']}"


def make_layer(dtype, out_dtype="f32", affine=False, seed=synth.SEED):
    W = synth.weights(128, 128, dtype=dtype, seed=seed, affine=affine)
    return TriMul(W, dtype=dtype, out_dtype=out_dtype), {k: oracle.f64(v) for k, v in W.items()}


def host(t):
    return t.detach().to("cpu").double().numpy()
