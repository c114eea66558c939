"""Run fp64 oracle calls for the large GPU parity checks in spawned worker
processes (test infrastructure; the workers import only numpy and the oracle,
never torch or the GPU library).

- full output rows of the N = 4096 update: oracle.tri_mul over column chunks,
  each worker reading the pair tensor from a float32 memory-mapped .npy file
  (exact: every bf16 value is a float32 value);
- the layer backward at N = 512: one oracle.tri_mul_backward per direction,
  the two in parallel.
"""
import os
import shutil
import tempfile
from concurrent.futures import ProcessPoolExecutor, as_completed
import multiprocessing as mp

import numpy as np


def _limit_threads(n):
    for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS"):
        os.environ[k] = str(n)


def _rows_chunk(path, mask, W, direction, rows, cols):
    import oracle
    z = np.load(path, mmap_mode="r")
    return oracle.tri_mul(z, mask, W, direction, rows, cols)


def _backward(z, mask, W, direction, dout):
    import oracle
    return oracle.tri_mul_backward(z, mask, W, direction, dout)


def _pool(workers, threads):
    # spawned (not forked) workers: a fresh interpreter without the parent's
    # GPU state; they inherit the thread limit through the environment
    saved = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS", "MKL_NUM_THREADS")}
    _limit_threads(threads)
    try:
        return ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn"))
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v


def scratch_dir(nbytes):
    """A directory with room for nbytes (plus a margin)."""
    for d in (os.environ.get("TMPDIR"), "/dev/shm", tempfile.gettempdir(), os.getcwd()):
        if d and os.path.isdir(d) and os.access(d, os.W_OK) and shutil.disk_usage(d).free > 1.25 * nbytes:
            return d
    raise RuntimeError(f"no scratch directory with {nbytes / 1e9:.1f} GB free")


def tri_mul_rows(z_rows_f32, N, mask, W, directions, rows, chunk=64, workers=15, say=print):
    """oracle.tri_mul(z, mask, W, direction, rows, all columns) for each
    direction, with z given as an iterator of (r0, float32 rows) pieces.
    Returns {direction: [len(rows)][N][c_z] float64}."""
    nbytes = N * N * 128 * 4
    d = tempfile.mkdtemp(prefix="trimul_z_", dir=scratch_dir(nbytes))
    path = os.path.join(d, "z.npy")
    try:
        zm = np.lib.format.open_memmap(path, mode="w+", dtype=np.float32, shape=(N, N, 128))
        for r0, piece in z_rows_f32:
            zm[r0:r0 + piece.shape[0]] = piece
        zm.flush()
        del zm
        say(f"  pair tensor written to {path}")
        out = {d: np.empty((len(rows), N, 128)) for d in directions}
        with _pool(workers, 1) as ex:
            futs = {ex.submit(_rows_chunk, path, mask, W, d, rows, np.arange(c0, min(N, c0 + chunk))): (d, c0)
                    for d in directions for c0 in range(0, N, chunk)}
            for n, f in enumerate(as_completed(futs), 1):
                d, c0 = futs[f]
                r = f.result()
                out[d][:, c0:c0 + r.shape[1]] = r
                if n % 8 == 0 or n == len(futs):
                    say(f"  oracle column chunks done: {n} of {len(futs)}")
        return out
    finally:
        shutil.rmtree(d, ignore_errors=True)


def backward_pair(z, mask, W, dout, directions=("outgoing", "incoming"), threads=8):
    """Start oracle.tri_mul_backward for each direction in its own worker;
    returns the pool and the futures (call .result() on each, then shut the
    pool down)."""
    ex = _pool(len(directions), threads)
    futs = {d: ex.submit(_backward, z, mask, W, d, dout) for d in directions}
    return ex, futs
