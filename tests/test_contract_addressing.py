"""Host-side walk over the contraction kernel's loads (CPU, no GPU).

The bf16 contraction (Section 3.3, Eq. 2 / Eq. 3) streams both operands into
LDS with buffer loads; tri_mul_check_contract_loads runs the kernel's own
addressing functions on the host for one launch shape and counts:
- tiles taken by no (work-group, round) of the persistent grid, or by several;
- loads whose buffer descriptor reaches outside the operand's allocation;
- needed elements (row < rows, k < K) read from a wrong address or not at all.
Every offset is in the lane offset (the scalar offset is 0), so "inside the
descriptor" means inside the allocation whichever offsets the hardware's range
check covers.  The allocation sizes below are written from the layouts'
definitions, not taken from the library.
"""
import pytest

from paper_2603_14806_amd import trimul as T

BLK, ROW, TR = T.TRI_MUL_OPERAND_BLOCKED, T.TRI_MUL_OPERAND_ROW_MAJOR, T.TRI_MUL_OPERAND_TRANSPOSED
SIZES = [1, 33, 300, 3750, 4096]


def ceil(a, b):
    return -(-a // b)


def blocked_bytes(rows, K, nch=128):
    """[nch][ceil(rows/256)][ceil(K/32)][256][32] bf16."""
    return nch * ceil(rows, 256) * ceil(K, 32) * 256 * 32 * 2


def transposed_bytes(rows, K, nch=128):
    """The operand given as X[k][row]: the blocked panel of K rows and `rows` columns."""
    return blocked_bytes(K, rows, nch)


def assert_clean(r, expect_tiles):
    assert r["tiles"] == expect_tiles
    assert r["bad_tiles"] == 0, r
    assert r["bad_desc"] == 0, r
    assert r["bad_elem"] == 0, r
    assert r["elems"] > 0 and r["loads"] > 0


def tiles(M, N, batch=128):
    return ceil(M, 256) * ceil(N, 256) * batch


@pytest.mark.parametrize("n", SIZES)
def test_full_update_blocked_operands(n):
    # outgoing and incoming run the same launch: both panels blocked, M = N = K = n
    b = blocked_bytes(n, n)
    r = T.check_contract_loads(BLK, BLK, n, n, n, a_bytes=b, b_bytes=b, grid=min(256, tiles(n, n)),
                               all_channels=n <= 300)
    assert_clean(r, tiles(n, n))


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("ta,tb", [(0, 1), (1, 1), (1, 0)])
def test_transposed_operands(n, ta, tb):
    # (0, 1): dA = dC B with B read transposed from its panel; (1, 1): the
    # forward from the opposite direction's panels, and dB = dC^T A from the
    # direction's own; (1, 0): dB = dC^T A with A^T given as it is
    a_mode = TR if ta else BLK
    b_mode = TR if tb else BLK
    a_bytes = transposed_bytes(n, n) if ta else blocked_bytes(n, n)
    b_bytes = transposed_bytes(n, n) if tb else blocked_bytes(n, n)
    r = T.check_contract_loads(a_mode, b_mode, n, n, n, a_bytes=a_bytes, b_bytes=b_bytes,
                               grid=min(256, tiles(n, n)), all_channels=n <= 300)
    assert_clean(r, tiles(n, n))


# device-tile views: (rows, cols, klen, ld); the first is one tile of an 8 x 8
# grid at N = 30000 (3750-token panels, ld rounded up to 8)
VIEWS = [(3750, 3750, 3750, 3752), (300, 200, 100, 104), (33, 1, 7, 8), (1, 1, 1, 8), (257, 513, 4096, 4104),
         (256, 256, 32, 32)]


@pytest.mark.parametrize("view", VIEWS)
def test_block_call_row_major_panels(view):
    rows, cols, klen, ld = view
    a_bytes, b_bytes = 128 * rows * ld * 2, 128 * cols * ld * 2
    r = T.check_contract_loads(ROW, ROW, rows, cols, klen, ld, ld, rows * ld, cols * ld, a_bytes=a_bytes,
                               b_bytes=b_bytes, grid=min(256, tiles(rows, cols)), all_channels=rows * cols < 1e5)
    assert_clean(r, tiles(rows, cols))


@pytest.mark.parametrize("view", VIEWS)
def test_block_call_repacked_panels(view):
    rows, cols, klen, _ = view
    r = T.check_contract_loads(BLK, BLK, rows, cols, klen, a_bytes=blocked_bytes(rows, klen),
                               b_bytes=blocked_bytes(cols, klen), grid=min(256, tiles(rows, cols)),
                               all_channels=rows * cols < 1e5)
    assert_clean(r, tiles(rows, cols))


@pytest.mark.parametrize("view", VIEWS)
def test_block_call_transposed_panels(view):
    # the ring step from the panels projected with the opposite direction:
    # A^T with klen rows and `rows` columns, B^T with klen rows and `cols`
    rows, cols, klen, _ = view
    r = T.check_contract_loads(TR, TR, rows, cols, klen, a_bytes=transposed_bytes(rows, klen),
                               b_bytes=transposed_bytes(cols, klen), grid=min(256, tiles(rows, cols)),
                               all_channels=rows * cols < 1e5)
    assert_clean(r, tiles(rows, cols))


@pytest.mark.parametrize("shape", [(1024, 1024, 4096), (100, 257, 37), (3, 5, 1), (9, 2048, 300), (64, 257, 65536)])
def test_outer_product_mean_launches(shape):
    # sums: rows (token, c) = ntok * 32, K = sequences, both operands given
    # transposed (X[s][(token, c)]); counts: rows = tokens, plain panels
    rows, cols, S = shape
    r = T.check_contract_loads(TR, TR, 32 * rows, 32 * cols, S, batch=1, a_bytes=transposed_bytes(32 * rows, S, 1),
                               b_bytes=transposed_bytes(32 * cols, S, 1), grid=min(256, tiles(32 * rows, 32 * cols, 1)))
    assert_clean(r, tiles(32 * rows, 32 * cols, 1))
    r = T.check_contract_loads(BLK, BLK, rows, cols, S, batch=1, a_bytes=blocked_bytes(rows, S, 1),
                               b_bytes=blocked_bytes(cols, S, 1), grid=min(256, tiles(rows, cols, 1)))
    assert_clean(r, tiles(rows, cols, 1))


@pytest.mark.parametrize("grid", [1, 7, 80, 256, 304, 1000])
def test_tile_census_any_grid(grid):
    n = 1000   # 4 x 4 tiles per channel, 2048 tiles
    b = blocked_bytes(n, n)
    r = T.check_contract_loads(BLK, BLK, n, n, n, a_bytes=b, b_bytes=b, grid=min(grid, tiles(n, n)))
    assert_clean(r, tiles(n, n))


def test_short_allocation_is_reported():
    # one 16 KB block short: the last channel's last row tile reaches past the end
    n = 300
    b = blocked_bytes(n, n)
    r = T.check_contract_loads(BLK, BLK, n, n, n, a_bytes=b - 16384, b_bytes=b, grid=tiles(n, n))
    assert r["bad_desc"] > 0
    rows, cols, klen, ld = 300, 200, 100, 104
    r = T.check_contract_loads(ROW, ROW, rows, cols, klen, ld, ld, rows * ld, cols * ld,
                               a_bytes=128 * rows * ld * 2, b_bytes=128 * cols * ld * 2 - 2, grid=4)
    assert r["bad_desc"] > 0


def test_bad_arguments_rejected():
    with pytest.raises(T.TriMulError):
        T.check_contract_loads(ROW, ROW, 10, 10, 100, 96, 104, 960, 1040, a_bytes=1 << 20, b_bytes=1 << 20)
    with pytest.raises(T.TriMulError):
        T.check_contract_loads(ROW, ROW, 10, 10, 100, 1 << 20, 104, 10 << 20, 1040, a_bytes=1 << 30,
                               b_bytes=1 << 20)
    with pytest.raises(T.TriMulError):
        T.check_contract_loads(3, BLK, 10, 10, 10, a_bytes=1 << 20, b_bytes=1 << 20)


# ------------------------------------------------- the result C (pair-blocked)

def result_bytes(rows, cols, nch=128):
    """[rows][ceil(cols/32)][nch][32] fp32 (tri_mul_contract's result layout)."""
    return rows * ceil(cols, 32) * nch * 32 * 4


def assert_clean_result(r, rows, cols, channels_visited):
    assert r["bad_desc"] == 0, r
    assert r["bad_elem"] == 0, r
    assert r["elems"] == rows * cols * channels_visited, r


@pytest.mark.parametrize("n", SIZES)
def test_result_full_update(n):
    # the full update's C, the backward products' dA / dB, the stage call's C
    r = T.check_contract_result(n, n, 128, c_bytes=result_bytes(n, n), all_channels=n <= 33)
    assert_clean_result(r, n, n, 128 if n <= 33 else 2)


@pytest.mark.parametrize("view", VIEWS)
def test_result_packed_accumulator(view):
    # a device tile's packed accumulator (tri_mul_block_accumulator_size)
    rows, cols = view[0], view[1]
    r = T.check_contract_result(rows, cols, 128, c_bytes=result_bytes(rows, cols), all_channels=rows * cols < 1e4)
    assert_clean_result(r, rows, cols, 128 if rows * cols < 1e4 else 2)


@pytest.mark.parametrize("shape", [(1024, 1024), (100, 257), (3, 5)])
def test_result_outer_product_mean(shape):
    rows, cols = shape
    # sums: (token, c) rows and columns, one channel; counts: tokens
    r = T.check_contract_result(32 * rows, 32 * cols, 1, c_bytes=result_bytes(32 * rows, 32 * cols, 1))
    assert_clean_result(r, 32 * rows, 32 * cols, 1)
    r = T.check_contract_result(rows, cols, 1, c_bytes=result_bytes(rows, cols, 1))
    assert_clean_result(r, rows, cols, 1)


def test_result_short_allocation_is_reported():
    n = 300
    r = T.check_contract_result(n, n, 128, c_bytes=result_bytes(n, n) - 4)
    assert r["bad_desc"] > 0
