"""The C-ABI library without a GPU: it loads, exports every symbol declared in
include/mq.h, and its argument validation returns the documented status codes
before anything is launched.  Every call below either fails validation or is
an empty (M == 0 / nnzb == 0) no-op, so the fake pointers are never used."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mq.h")

OK, INVALID, SHAPE, MISALIGNED, WORKSPACE = 0, -1, -2, -3, -4
A = 0x10000          # a 16-byte aligned fake device address (never touched)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mq_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2606_15652_amd as mq
    if not os.path.exists(mq.LIB_PATH):
        from paper_2606_15652_amd import build
        build.build()
    return mq.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(lib, n), f"libmq.so does not export {n}"


def test_status_strings(lib):
    for s in (OK, INVALID, SHAPE, MISALIGNED, WORKSPACE, -5, -99):
        assert lib.mq_status_string(s)
    assert lib.mq_version() >= 100


def test_quantize_act_validation(lib):
    q = lib.mq_quantize_act
    assert q(A, 0, 128, 128, A, A, None) == OK                 # empty input: no-op
    assert q(A, -1, 128, 128, A, A, None) == INVALID
    assert q(A, 4, 100, 128, A, A, None) == SHAPE               # K not a multiple of 128
    assert q(A, 4, 256, 128, A, A, None) == SHAPE               # ldx < K
    assert q(A, 4, 128, 132, A, A, None) == SHAPE               # ldx % 8
    assert q(None, 4, 128, 128, A, A, None) == INVALID
    assert q(A + 2, 4, 128, 128, A, A, None) == MISALIGNED
    assert q(A, 4, 128, 128, A + 8, A, None) == MISALIGNED
    assert q(A, 4, 128, 128, A, A + 1, None) == MISALIGNED


def _gemm(lib, M=4, N=256, K=256, Xq=A, sx=A, Wq=A, sw=A, rp=A, kb=A, nnzb=1, Rq=A, sr=A,
          Y=A, ldy=None, ws=None, ws_bytes=0, variant=0):
    return lib.mq_fused_gemm_variant(variant, M, N, K, Xq, sx, Wq, sw, rp, kb, nnzb, Rq, sr, Y,
                                     N if ldy is None else ldy, ws, ws_bytes, None)


def test_fused_gemm_validation(lib):
    assert _gemm(lib, M=0) == OK
    assert _gemm(lib, M=-1) == INVALID
    assert _gemm(lib, N=200) == SHAPE
    assert _gemm(lib, K=64) == SHAPE
    assert _gemm(lib, K=1 << 21) == SHAPE
    assert _gemm(lib, ldy=128) == SHAPE
    assert _gemm(lib, ldy=260) == SHAPE
    assert _gemm(lib, nnzb=5) == INVALID                       # > NB * KB = 4
    assert _gemm(lib, nnzb=-1) == INVALID
    assert _gemm(lib, Rq=None) == INVALID                      # residual pointers required
    assert _gemm(lib, Xq=None) == INVALID
    assert _gemm(lib, Y=None) == INVALID
    assert _gemm(lib, Wq=A + 4) == MISALIGNED
    assert _gemm(lib, Rq=A + 8) == MISALIGNED
    assert _gemm(lib, kb=A + 2) == MISALIGNED
    assert _gemm(lib, sx=A + 1) == MISALIGNED
    assert _gemm(lib, variant=7) == INVALID
    assert lib.mq_fused_gemm_workspace_size(4, 256, 256) == 0


def test_acc_i32_validation(lib):
    f = lib.mq_fused_gemm_acc_i32
    assert f(0, 0, 256, 256, A, A, A, A, 1, A, A, A, None) == OK
    assert f(0, 4, 256, 256, A, A, A, A, 1, A, None, A, None) == INVALID
    assert f(0, 4, 256, 256, A, A, A, A, 1, A, A + 2, A, None) == MISALIGNED
    assert f(9, 4, 256, 256, A, A, A, A, 1, A, A, A, None) == INVALID        # no such variant


def test_weight_prep_validation(lib):
    assert lib.mq_quantize_weight(A, 256, 200, 256, A, A, A, None) == SHAPE
    assert lib.mq_quantize_weight(A, 256, 256, 255, A, A, A, None) == SHAPE
    assert lib.mq_quantize_weight(A + 4, 256, 256, 256, A, A, A, None) == MISALIGNED
    assert lib.mq_quantize_weight(A, 256, 256, 256, A, A, A + 4, None) == MISALIGNED
    assert lib.mq_select_blocks(A, 2, 2, 5, A, A, None) == INVALID
    assert lib.mq_select_blocks(A, 2, 2, -1, A, A, None) == INVALID
    assert lib.mq_select_blocks(A, 2, 2, 1, A, None, None) == INVALID
    assert lib.mq_quantize_residual(A, 256, 256, 256, A, A, A, A, 9, A, A, None) == INVALID
    assert lib.mq_quantize_residual(A, 256, 256, 256, A, A, A, A, 0, None, None, None) == OK
    assert lib.mq_hessian_diag(A, 0, 128, 128, A, None) == INVALID
    assert lib.mq_block_scores_dhessian(A, 256, 256, 256, A, A, None, A, None) == INVALID


def _lin(lib, M=4, N=256, K=256, X=A, ldx=None, Wq=A, sw=A, rp=A, kb=A, nnzb=1, Rq=A, sr=A,
         Y=A, ldy=None, ws=None, ws_bytes=0):
    return lib.mq_linear(M, N, K, X, K if ldx is None else ldx, Wq, sw, rp, kb, nnzb, Rq, sr, Y,
                         N if ldy is None else ldy, ws, ws_bytes, None)


def test_linear_validation(lib):
    assert _lin(lib, M=0) == OK
    assert _lin(lib, M=-1) == INVALID
    assert _lin(lib, K=200) == SHAPE
    assert _lin(lib, ldx=128) == SHAPE                         # ldx < K
    assert _lin(lib, ldx=260) == SHAPE                         # ldx % 8
    assert _lin(lib, ldy=264 - 16) == SHAPE
    assert _lin(lib, X=None) == INVALID
    assert _lin(lib, X=A + 8) == MISALIGNED
    assert _lin(lib, Rq=None) == INVALID
    assert _lin(lib, Y=None) == INVALID
    # decode sizes need no workspace; larger M need room for the quantised rows
    assert lib.mq_linear_workspace_size(1, 4096, 4096) == 0
    assert lib.mq_linear_workspace_size(4, 4096, 8192) == 0
    need = lib.mq_linear_workspace_size(64, 256, 1024)
    assert need >= 64 * 512 + 2 * 64
    assert _lin(lib, M=64, K=1024, ws=A, ws_bytes=need - 1) == WORKSPACE
    assert _lin(lib, M=64, K=1024, ws=None, ws_bytes=need) == INVALID
    assert _lin(lib, M=64, K=1024, ws=A + 8, ws_bytes=need) == MISALIGNED


def test_repack_validation(lib):
    rw, uw = lib.mq_repack_weights, lib.mq_unpack_weights
    assert rw(256, 200, A, A, 0, None, A, A, None, None, None) == SHAPE
    assert rw(-1, 256, A, A, 0, None, A, A, None, None, None) == INVALID
    assert rw(256, 256, A, A, 5, A, A, A, A, None, None) == INVALID             # nnzb > NB * KB
    assert rw(256, 256, A, A, 1, None, A, A, A, None, None) == INVALID          # residual source missing
    assert rw(256, 256, A, None, 0, None, A, A, None, None, None) == INVALID    # scales: both or neither
    assert rw(256, 256, A + 4, A, 0, None, A, A, None, None, None) == MISALIGNED
    assert rw(256, 256, A, A, 0, None, A + 8, A, None, None, None) == MISALIGNED
    assert rw(256, 256, A, A, 0, None, A, A, None, A + 2, None) == MISALIGNED
    assert uw(256, 256, A + 8, A, 0, None, A, A, None, None) == MISALIGNED     # library side 16-byte
    ra, ua = lib.mq_repack_act, lib.mq_unpack_act
    assert ra(0, 256, A, 128, A, None, None) == OK
    assert ra(4, 256, A, 120, A, None, None) == SHAPE                          # ldq < K/2
    assert ra(4, 256, A, 132, A, None, None) == SHAPE                          # ldq % 8
    assert ra(4, 256, None, 128, A, None, None) == INVALID
    assert ra(4, 256, A, 128, A + 8, None, None) == MISALIGNED
    assert ua(4, 256, A + 8, A, 128, None) == MISALIGNED
    assert ua(-1, 256, A, A, 128, None) == INVALID


def test_noalloc_validation(lib):
    assert lib.mq_scratch_bytes() == 128 << 20
    f = lib.mq_linear_noalloc
    assert f(0, 256, 256, A, 256, A, A, A, A, 1, A, A, A, 256, None) == OK        # empty: no scratch used
    assert f(4, 256, 200, A, 256, A, A, A, A, 1, A, A, A, 256, None) == SHAPE     # K not a multiple of 128
    assert f(65536, 256, 8192, A, 8192, A, A, None, None, 0, None, None, A, 256, None) == -6   # beyond scratch


def test_a8_validation(lib):
    assert lib.mq_quantize_act8(A, 0, 128, 128, A, A, None) == OK
    assert lib.mq_quantize_act8(A, 4, 100, 128, A, A, None) == SHAPE
    assert lib.mq_quantize_act8(A, 4, 128, 128, A + 8, A, None) == MISALIGNED
    g = lib.mq_fused_gemm_a8
    assert g(0, 256, 256, A, A, A, A, A, A, 1, A, A, A, 256, None) == OK
    assert g(4, 200, 256, A, A, A, A, A, A, 1, A, A, A, 256, None) == SHAPE
    assert g(4, 256, 256, A, A, A, A, A, A, 1, A, A, A, 252, None) == SHAPE
    assert g(4, 256, 256, A + 8, A, A, A, A, A, 1, A, A, A, 256, None) == MISALIGNED
    assert g(4, 256, 256, A, None, A, A, A, A, 1, A, A, A, 256, None) == INVALID
    r = lib.mq_fused_gemm_a8_acc_i32
    assert r(4, 256, 256, A, A, A, A, 1, A, None, A, None) == INVALID
    assert lib.mq_repack_act8(4, 256, A, 250, A, None, None) == SHAPE
    assert lib.mq_unpack_act8(4, 256, A + 8, A, 256, None) == MISALIGNED


# AUTO's kernel choice (host logic, no device call): the families and split
# counts the dispatch rules give on the benchmarked and family shapes
PLANS = [
    ((1, 4096, 4096), ("skinny", 1)), ((16, 4096, 4096), ("skinny", 1)), ((32, 4096, 4096), ("skinny", 1)),
    ((33, 4096, 4096), ("medium", 1)), ((256, 4096, 4096), ("medium", 1)), ((512, 4096, 4096), ("medium", 1)),
    ((1536, 4096, 4096), ("tiled", 1)), ((2048, 4096, 4096), ("tiled", 1)), ((4096, 4096, 4096), ("tiled_large", 1)),
    ((512, 5120, 25600), ("tiled", 4)), ((1024, 4096, 14336), ("tiled", 2)), ((768, 5120, 5120), ("tiled", 2)),
    ((2048, 1024, 5120), ("medium", 1)), ((2048, 5120, 5120), ("tiled_large", 1)), ((4096, 14336, 4096), ("tiled_large", 1)),
    ((4096, 384, 4096), ("medium", 1)), ((4096, 384, 14336), ("tiled", 4)),
    ((1024, 4096, 4096), ("medium", 1)), ((1280, 4096, 4096), ("tiled", 1)), ((4096, 5120, 5120), ("tiled_large", 1)),
    ((6144, 4096, 14336), ("tiled_large", 1)), ((768, 25600, 5120), ("tiled_large", 1)),
    ((128, 25600, 5120), ("medium", 1)),
]


@pytest.mark.parametrize("shape,expect", PLANS, ids=[f"M{m}_N{n}_K{k}" for (m, n, k), _ in PLANS])
def test_auto_plan(lib, shape, expect):
    import paper_2606_15652_amd as mq
    M, N, K = shape
    assert mq.plan(M, N, K) == expect
    fam, splits = expect
    ws = lib.mq_fused_gemm_workspace_size(M, N, K)
    if splits > 1:
        assert ws >= splits * M * N * 4          # the partial sums fit the advertised workspace


def test_auto_plan_validation(lib):
    import ctypes as C
    v, s = C.c_int(0), C.c_int(0)
    assert lib.mq_fused_gemm_plan(0, 4096, 4096, C.byref(v), C.byref(s)) == INVALID
    assert lib.mq_fused_gemm_plan(16, 4096, 4096, None, C.byref(s)) == INVALID
    assert lib.mq_fused_gemm_plan(16, 4000, 4096, C.byref(v), C.byref(s)) == SHAPE
    assert lib.mq_fused_gemm_plan(16, 4096, 100, C.byref(v), C.byref(s)) == SHAPE

