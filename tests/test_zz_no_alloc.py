"""tri_mul_update_noalloc, the entry point for callers that cannot allocate
device memory, against tri_mul_outgoing / tri_mul_incoming through the C ABI:
the same kernels with the workspace in the library's device scratch, so the
outputs must be bitwise identical.  Two calls in a row per direction, the
second with a smaller N (the scratch keeps the first call's contents), a
masked ragged size, and the size limit of the scratch."""
import numpy as np
import pytest
import torch

import oracle
from paper_2603_14806_amd import synth
from paper_2603_14806_amd import trimul as T
from tests.gpu_util import assert_close, host, make_layer, needs_gpu, say

pytestmark = [pytest.mark.gpu, needs_gpu]

SCRATCH_BYTES = 256 << 20


def _reference(layer, z, mask, N, direction):
    out = torch.full((N, N, 128), float("nan"), dtype=torch.float32, device="cuda")
    ws, need = layer.workspace(N)
    f = T.tri_mul_outgoing if direction == T.TRI_MUL_OUTGOING else T.tri_mul_incoming
    f(layer.h, z, mask, N, out, ws, need)
    return out


def _noalloc(layer, z, mask, N, direction):
    out = torch.full((N, N, 128), float("nan"), dtype=torch.float32, device="cuda")
    T.tri_mul_update_noalloc(layer.h, z, mask, N, direction, out)
    return out


@pytest.mark.parametrize("direction", [T.TRI_MUL_OUTGOING, T.TRI_MUL_INCOMING])
def test_noalloc_matches_workspace_entry_point(direction):
    layer, W = make_layer("bf16")
    for N, pad in ((512, 51), (300, 17), (33, 0)):   # decreasing sizes, two calls or more in a row
        say(f"no-alloc: N={N} padded={pad} direction={direction}")
        z = synth.pair_tensor(N, dtype="bf16", seed=11 + N, device="cuda")
        mask = synth.token_mask(N, pad, device="cuda") if pad else None
        got = _noalloc(layer, z, mask, N, direction)
        ref = _reference(layer, z, mask, N, direction)
        torch.cuda.synchronize()
        assert torch.isfinite(got).all()
        assert torch.equal(got, ref), f"N={N}: no-alloc output differs from the workspace entry point"
        if N == 33:   # and both agree with the oracle
            name = "outgoing" if direction == T.TRI_MUL_OUTGOING else "incoming"
            m = np.ones(N) if mask is None else host(mask)
            assert_close(host(got), oracle.tri_mul(host(z), m, W, name), "bf16", f"no-alloc N={N} vs oracle")
    layer.close()


def test_noalloc_limits():
    layer, _ = make_layer("bf16")
    assert T.tri_mul_workspace_size(layer.h, 512) <= SCRATCH_BYTES
    assert T.tri_mul_workspace_size(layer.h, 513) > SCRATCH_BYTES
    z = torch.zeros((1, 1, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.zeros((1, 1, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(T.TriMulError) as e:   # rejected on the host, before any launch
        T.tri_mul_update_noalloc(layer.h, z, None, 513, T.TRI_MUL_OUTGOING, out)
    assert e.value.code == T.TRI_MUL_EUNSUPPORTED
    with pytest.raises(T.TriMulError) as e:
        T.tri_mul_update_noalloc(layer.h, z, None, 1, 7, out)
    assert e.value.code == T.TRI_MUL_EINVAL
    layer.close()
