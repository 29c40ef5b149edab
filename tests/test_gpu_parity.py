"""GPU parity: libmq's HIP kernels (through the C ABI) against the CPU oracle.

Bars: integer and byte outputs (codes, packed chunks, fp16 scale bits, CSR,
raw int32 accumulators) bit-exact; fp16 outputs within max-abs-rel 2e-3 of the
oracle's fp64 epilogue (norm-relative: max|dY| / max|Y64|).  The fp16
rounding of the output alone contributes up to 2^-11 ~ 4.9e-4, and the fp32
group accumulation a few 2^-24 per group, so the tests also check a tighter
1e-3.  Block scores are fp64 sums taken in a different order on the two sides
and are compared to 1e-12 relative; the selected sets must then coincide
exactly (a tie closer than that at the budget boundary would be reported).
"""
from __future__ import annotations


import numpy as np
import pytest

import oracle as layout    # the device group order, as a permutation of the oracle's row-major packing
import synth
from gpu_util import (B, TIGHT, TOL, _announce, dev, dev_x, gpu_pw, half_bits, host,  # noqa: F401
                      maxabsrel, mq, orc_pw, random_csr, random_operands, tc)

pytestmark = pytest.mark.gpu


# ------------------------------------------------------- activation quant --
ACT_CASES = [(1, 128), (3, 1024), (64, 4096), (257, 384), (5, 28672), (2, 40960), (33, 2048)]


@pytest.mark.parametrize("M,K", ACT_CASES)
def test_act_quant_parity(tc, mq, orc, M, K):
    rng = np.random.default_rng(M * 7919 + K)
    X = synth.gen_act(M, K, 1000 + M + K)
    if M > 2:
        X[1] = (rng.standard_normal(K) * 3).astype(np.float16)      # dense codes
        X[2] = 0                                                    # zero row
    if M > 4:
        X[3, :8] = np.array([0.875, -0.4375, 0.3125, 0.1875, -0.0625, 0.0625, -0.3125, 0.4375])
        X[3, 8:] = 0                                                # exact ties (golden)
        X[4] = (rng.standard_normal(K) * 1e-6).astype(np.float16)   # subnormal halves
    if M > 5:
        X[5, K // 2] = 65504                                        # largest finite half
    Xq, s_x = mq.quantize_act(dev(tc, X))
    Xq_ref, sx_ref = orc.quantize_act(X)
    assert np.array_equal(half_bits(s_x), sx_ref)
    assert np.array_equal(orc.packed_from_act6(host(Xq), K), Xq_ref)


def test_act_quant_exact_ties(tc, mq, orc):
    """Every tie (k + 1/2) s, k = 0..6, both signs, and its fp16 neighbours,
    over 256 scales s = j 2^e with a 7-bit j (so (k + 1/2) s and 7 s are
    halves): the codes are round-half-even, bit-exact against the oracle."""
    rng = np.random.default_rng(77)
    rows = []
    for r in range(256):
        j = int(rng.integers(1, 128))
        e = int(rng.integers(-20, 6))
        s = np.float16(j * 2.0 ** e)
        if not np.isfinite(s) or s == 0 or np.float16(7 * float(s)) != 7 * float(s):
            s = np.float16(0.125)
        row = [np.float16(7 * float(s))]                       # the row maximum: scale s
        for k in range(7):
            t = np.float16((k + 0.5) * float(s))
            assert float(t) == (k + 0.5) * float(s)
            for v in (t, np.nextafter(t, np.float16(0)), np.nextafter(t, np.float16(np.inf))):
                row += [v, -v]
        row = np.array(row, np.float16)
        rows.append(np.concatenate([row, np.zeros(128 - len(row), np.float16)]))
    X = np.stack(rows)
    Xq, s_x = mq.quantize_act(dev(tc, X))
    Xq_ref, sx_ref = orc.quantize_act(X)
    assert np.array_equal(half_bits(s_x), sx_ref)
    assert np.array_equal(orc.packed_from_act6(host(Xq), 128), Xq_ref)


def test_act_quant_strided(tc, mq, orc):
    X = synth.gen_act(9, 640, 5)
    Xbig = np.zeros((9, 1024), np.float16)
    Xbig[:, :640] = X
    Xd = dev(tc, Xbig)[:, :640]
    Xq = tc.empty((9, mq.act_bytes(640)), dtype=tc.uint8, device="cuda")
    s_x = tc.empty((9,), dtype=tc.float16, device="cuda")
    lib = mq.load()
    st = lib.mq_quantize_act(Xd.data_ptr(), 9, 640, 1024, Xq.data_ptr(), s_x.data_ptr(), None)
    tc.cuda.synchronize()
    assert st == 0
    Xq_ref, sx_ref = orc.quantize_act(X)
    assert np.array_equal(orc.packed_from_act6(host(Xq), 640), Xq_ref)
    assert np.array_equal(half_bits(s_x), sx_ref)


# ------------------------------------------------------- weight prep -------
PREP_CASES = [("c1", 1024, 1024, 6, False), ("tall", 2048, 256, 7, False),
              ("wide", 256, 3072, 10, False), ("skew", 2048, 1024, 13, True),
              ("dense100", 384, 512, 12, False), ("none", 512, 384, 0, False)]


def check_prep(tc, mq, orc, W, nnzb, criterion="frob", Xc=None):
    pw = mq.prepare_weight(dev(tc, W), nnzb, criterion=criterion,
                           X_calib=None if Xc is None else dev(tc, Xc))
    ref = orc.prepare_weight(W, nnzb, criterion=criterion, X_calib=Xc)
    tc.cuda.synchronize()
    assert np.array_equal(orc.unblock_rows(host(pw.Wq), W.shape[1]), ref.Wq)
    assert np.array_equal(orc.unblock_scales(half_bits(pw.s_w)), ref.s_w)
    sc = host(pw.score)
    assert np.allclose(sc, ref.score, rtol=1e-12, atol=1e-300)
    # selection: exact unless two scores closer than the comparison tolerance
    # straddle the budget boundary
    rp, kb = host(pw.rowptr), host(pw.kb)
    if not (np.array_equal(rp, ref.rowptr) and np.array_equal(kb, ref.kb)):
        order = np.sort(ref.score.ravel())[::-1]
        gap = abs(order[nnzb - 1] - order[nnzb]) if 0 < nnzb < order.size else np.inf
        pytest.fail(f"selected blocks differ (boundary gap {gap:.3e})")
    assert np.array_equal(host(pw.Rq), ref.Rq)
    assert np.array_equal(half_bits(pw.s_r), ref.s_r)
    return pw, ref


@pytest.mark.parametrize("name,N,K,nnzb,skew", PREP_CASES, ids=[c[0] for c in PREP_CASES])
def test_weight_prep_parity(tc, mq, orc, name, N, K, nnzb, skew):
    seed = 77 + N + K
    des = synth.skew_blocks(N, K, nnzb, seed)[0] if skew else None
    W = synth.gen_weight(N, K, seed, designated=des)
    if name == "dense100":
        nnzb = (N // B) * (K // B)
    check_prep(tc, mq, orc, W, nnzb)


def test_weight_prep_edge_values(tc, mq, orc):
    N, K = 256, 384
    W = synth.gen_weight(N, K, 3)
    W[0, :128] = 0                        # all-zero group -> scale 0
    W[1, 0] = 0.875; W[1, 1:128] = 0.4375  # ties against s = 0.125
    W[2, 128:256] = 1e-9                  # scale underflows in fp16
    W[3, 5] = 7.5                         # a large outlier
    check_prep(tc, mq, orc, W, 3)


def test_dhessian_prep_parity(tc, mq, orc):
    N, K = 1024, 768
    W = synth.gen_weight(N, K, 19)
    rng = np.random.default_rng(2)
    Xc = (rng.standard_normal((256, K)) * rng.uniform(0.1, 5, K)).astype(np.float16)
    h = mq.hessian_diag(dev(tc, Xc))
    assert np.array_equal(host(h), orc.hessian_diag(Xc))    # same sequential order
    check_prep(tc, mq, orc, W, 20, criterion="dhessian", Xc=Xc)


# ------------------------------------------------------------ GEMM ---------
GEMM_CASES = [
    (1, 128, 128, 1), (5, 384, 256, 3), (16, 1024, 1024, 6), (17, 256, 512, 5),
    (32, 640, 384, 0), (33, 256, 256, 4), (64, 1024, 1024, 6), (100, 384, 640, 9),
    (129, 512, 1024, 12), (256, 1024, 2048, 13), (70, 128, 4096, 32), (48, 2304, 256, 18),
    (300, 768, 1024, 10), (257, 512, 512, 16),
]


def _variants(M, N=128):
    vs = ["skinny", "tiled", "medium", "auto"] if M <= 32 else ["tiled", "medium", "auto"]
    if N % 256 == 0:
        vs.append("tiled_large")            # 256 x 256 tiles (AUTO takes them on large problems)
    return vs


@pytest.mark.parametrize("M,N,K,nnzb", GEMM_CASES, ids=[f"M{c[0]}_N{c[1]}_K{c[2]}_r{c[3]}" for c in GEMM_CASES])
def test_gemm_parity_random_codes(tc, mq, orc, M, N, K, nnzb):
    ops = random_operands(M, N, K, nnzb, seed=M * 131 + N * 7 + K + nnzb)
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = ops
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xq_d, sx_d = dev_x(tc, Xq), dev(tc, s_x).view(tc.float16)
    for v in _variants(M, N):
        Tb, Tr = mq.fused_gemm_acc_i32(Xq_d, pw, variant=v)
        Y = mq.fused_gemm(Xq_d, sx_d, pw, variant=v)
        tc.cuda.synchronize()
        assert np.array_equal(host(Tb), Tb_ref), f"{v}: Tb differs"
        assert np.array_equal(host(Tr), Tr_ref), f"{v}: Tr differs"
        err = maxabsrel(Y, Y64)
        assert err <= TIGHT, f"{v}: max-abs-rel {err:.3e}"


# (M, N, K, nnzb): more decode tiles than the workgroups resident at once, so
# each workgroup takes several tiles in turn (the tile count is no multiple of
# the grid); K = 1024 gives every wave one group of a tile, K = 1152 ragged runs
MANY_TILE_CASES = [(1, 65920, 1024, 300), (16, 65920, 1152, 600), (32, 49408, 1024, 250)]


@pytest.mark.parametrize("M,N,K,nnzb", MANY_TILE_CASES, ids=[f"M{c[0]}_N{c[1]}_K{c[2]}" for c in MANY_TILE_CASES])
def test_decode_several_tiles_per_workgroup(tc, mq, orc, M, N, K, nnzb):
    ops = random_operands(M, N, K, nnzb, seed=M * 31 + N + K)
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = ops
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xq_d, sx_d = dev_x(tc, Xq), dev(tc, s_x).view(tc.float16)
    for v in ("skinny", "auto"):
        Tb, Tr = mq.fused_gemm_acc_i32(Xq_d, pw, variant=v)
        Y = mq.fused_gemm(Xq_d, sx_d, pw, variant=v)
        tc.cuda.synchronize()
        assert np.array_equal(host(Tb), Tb_ref), f"{v}: Tb differs"
        assert np.array_equal(host(Tr), Tr_ref), f"{v}: Tr differs"
        err = maxabsrel(Y, Y64)
        assert err <= TIGHT, f"{v}: max-abs-rel {err:.3e}"


def test_linear_decode_several_tiles_per_workgroup(tc, mq, orc):
    """The one-kernel decode path (quantisation fused) with several tiles per
    workgroup: the rows are quantised once and serve every tile."""
    M, N, K, nnzb = 3, 65920, 1024, 300
    _, _, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=4242)
    X = synth.gen_act(M, K, 4243)
    Xq_r, sx_r = orc.quantize_act(X)
    _, _, Y64 = orc.linear(Xq_r, sx_r, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xd = dev(tc, X)
    Y = mq.linear(Xd, pw)
    Xq, s_x = mq.quantize_act(Xd)
    Y2 = mq.fused_gemm(Xq, s_x, pw)
    tc.cuda.synchronize()
    assert maxabsrel(Y, Y64) <= TIGHT
    assert np.array_equal(host(Y.view(tc.int16)), host(Y2.view(tc.int16)))


# ------------------------------------------- whole layer from fp16 X ------
# (M, N, K, nnzb): M <= 4 with M * K <= 32768 take the one-kernel decode path
# (activation quantisation fused into the GEMM), the others quantise first.
LINEAR_CASES = [(1, 256, 128, 1), (2, 512, 1024, 4), (3, 384, 4096, 6), (4, 1024, 8192, 20),
                (1, 256, 32768, 8), (4, 256, 4096, 3), (1, 128, 40960, 2), (5, 256, 1024, 2),
                (64, 512, 2048, 7)]


@pytest.mark.parametrize("M,N,K,nnzb", LINEAR_CASES, ids=[f"M{c[0]}_N{c[1]}_K{c[2]}_r{c[3]}" for c in LINEAR_CASES])
def test_linear_matches_oracle_and_two_step(tc, mq, orc, M, N, K, nnzb):
    """mq_linear from fp16 X: within the bar of the oracle (quantise + layer) and
    bit-identical to mq_quantize_act followed by mq_fused_gemm."""
    _, _, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=M * 977 + K + nnzb)
    X = synth.gen_act(M, K, 7000 + M + K)
    if M > 1:
        X[1] = 0                                                  # zero row: scale 0
    Xq_r, sx_r = orc.quantize_act(X)
    _, _, Y64 = orc.linear(Xq_r, sx_r, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xd = dev(tc, X)
    Y = mq.linear(Xd, pw)
    Xq, s_x = mq.quantize_act(Xd)
    Y2 = mq.fused_gemm(Xq, s_x, pw)
    tc.cuda.synchronize()
    assert maxabsrel(Y, Y64) <= TIGHT
    assert np.array_equal(host(Y.view(tc.int16)), host(Y2.view(tc.int16)))


def test_gemm_quantized_layer_matches_oracle(tc, mq, orc):
    """The whole hot path on a synthetic quantised layer (config-1 recipe)."""
    L = synth.workload("c1_1024")
    W, X = L.weight(), L.act(64)
    ref = orc.prepare_weight(W, L.nnzb)
    Xq_r, sx_r = orc.quantize_act(X)
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq_r, sx_r, ref)
    pw = mq.prepare_weight(dev(tc, W), L.nnzb)
    Y = mq.linear(dev(tc, X), pw)
    Xq, s_x = mq.quantize_act(dev(tc, X))
    for v in ("skinny", "tiled", "tiled_large", "medium"):
        Tb, Tr = mq.fused_gemm_acc_i32(Xq, pw, variant=v)
        assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref)
        assert maxabsrel(mq.fused_gemm(Xq, s_x, pw, variant=v), Y64) <= TIGHT
    assert maxabsrel(Y, Y64) <= TIGHT


def test_gemm_extreme_codes_long_k(tc, mq, orc):
    """All codes -7 or +7 over K = 28672: accumulators at their extreme."""
    M, N, K = 20, 256, 28672
    xc = np.full((M, K), -7, np.int8)
    xc[1::2] = 7
    wc = np.full((N, K), -7, np.int8)
    wc[::3] = 7
    Xq, Wq = orc.pack_codes(xc), orc.pack_codes(wc)
    s_x = np.full(M, np.float16(1).view(np.uint16))
    s_w = np.full((N, K // B), np.float16(2 ** -10).view(np.uint16))
    NB, KB = N // B, K // B
    rowptr = np.array([0, KB, KB], np.int32)           # every block of block row 0
    kb = np.arange(KB, dtype=np.int32)
    Rq = orc.pack_codes(np.full((KB, B, B), -7, np.int8))
    s_r = np.full((KB, B), np.float16(2 ** -12).view(np.uint16))
    sel = np.zeros((NB, KB), bool)
    sel[0] = True
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    assert np.abs(Tb_ref).max() == 49 * K
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    for v in ("skinny", "tiled", "tiled_large", "medium"):
        Tb, Tr = mq.fused_gemm_acc_i32(dev_x(tc, Xq), pw, variant=v)
        Y = mq.fused_gemm(dev_x(tc, Xq), dev(tc, s_x).view(tc.float16), pw, variant=v)
        tc.cuda.synchronize()
        assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref), v
        assert maxabsrel(Y, Y64) <= TIGHT, v


def test_gemm_guard_bands_and_empty(tc, mq, orc):
    """No writes outside Y[:M, :N] (ldy > N, canary rows); M == 0 is a no-op."""
    M, N, K, nnzb = 37, 512, 512, 4
    ops = random_operands(M, N, K, nnzb, seed=5)
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = ops
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xq_d, sx_d = dev_x(tc, Xq), dev(tc, s_x)        # kept alive across the launches
    lib = mq.load()
    for v in (1, 2, 3, 4):
        if v == 1 and M > 32:
            continue
        canary = 12345
        Yfull = tc.full((M + 4, N + 8), canary, dtype=tc.int16, device="cuda")
        Yv = Yfull[2:2 + M]
        st = lib.mq_fused_gemm_variant(v, M, N, K, Xq_d.data_ptr(),
                                       sx_d.data_ptr(), pw.Wq.data_ptr(), pw.s_w.data_ptr(),
                                       pw.rowptr.data_ptr(), pw.kb.data_ptr(), nnzb, pw.Rq.data_ptr(),
                                       pw.s_r.data_ptr(), Yv.data_ptr(), N + 8, None, 0, None)
        tc.cuda.synchronize()
        assert st == 0
        h = host(Yfull)
        assert np.all(h[:2] == canary) and np.all(h[2 + M:] == canary)
        assert np.all(h[2:2 + M, N:] == canary)
    Y = tc.full((1, N), 7, dtype=tc.int16, device="cuda")
    st = lib.mq_fused_gemm(0, N, K, Xq_d.data_ptr(), sx_d.data_ptr(),
                           pw.Wq.data_ptr(), pw.s_w.data_ptr(), pw.rowptr.data_ptr(),
                           pw.kb.data_ptr(), nnzb, pw.Rq.data_ptr(), pw.s_r.data_ptr(),
                           Y.data_ptr(), N, None, 0, None)
    tc.cuda.synchronize()
    assert st == 0 and np.all(host(Y) == 7)


def test_gemm_y_not_16_byte_aligned(tc, mq, orc):
    """Y two bytes past a 16-byte boundary (the tiled kernels then store one
    value a lane instead of staging 16-byte row pieces): the same values, and
    nothing written outside Y[:M, :N]."""
    M, N, K, nnzb = 37, 512, 512, 4
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=6)
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xq_d, sx_d = dev_x(tc, Xq), dev(tc, s_x)
    lib = mq.load()
    ldy, canary = N + 8, 12345
    for v in (2, 3, 4):
        flat = tc.full(((M + 4) * ldy + 8,), canary, dtype=tc.int16, device="cuda")
        base = 2 * ldy + 1                                # elements: 2 bytes past alignment
        assert (flat.data_ptr() + 2 * base) % 16 == 2
        st = lib.mq_fused_gemm_variant(v, M, N, K, Xq_d.data_ptr(), sx_d.data_ptr(), pw.Wq.data_ptr(),
                                       pw.s_w.data_ptr(), pw.rowptr.data_ptr(), pw.kb.data_ptr(), nnzb,
                                       pw.Rq.data_ptr(), pw.s_r.data_ptr(), flat.data_ptr() + 2 * base,
                                       ldy, None, 0, None)
        tc.cuda.synchronize()
        assert st == 0, v
        h = host(flat)
        idx = base + np.arange(M)[:, None] * ldy + np.arange(N)[None, :]
        y = h[idx].view(np.float16).astype(np.float64)
        assert np.abs(y - Y64).max() / np.abs(Y64).max() <= TIGHT, v
        mask = np.ones(h.shape, bool)
        mask[idx.ravel()] = False
        assert np.all(h[mask] == canary), v


def test_gemm_no_residual_null_pointers(tc, mq, orc):
    M, N, K = 40, 256, 384
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, 0, seed=9)
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    Y = tc.empty((M, N), dtype=tc.float16, device="cuda")
    keep = [dev_x(tc, Xq), dev(tc, s_x), dev(tc, layout.block_rows(Wq, K)),
            dev(tc, layout.block_scales(s_w))]               # kept alive across the launches
    lib = mq.load()
    for v in (1, 2, 3, 4):
        st = lib.mq_fused_gemm_variant(v, M, N, K, *[t.data_ptr() for t in keep], None, None, 0,
                                       None, None, Y.data_ptr(), N, None, 0, None)
        tc.cuda.synchronize()
        assert st == 0
        assert maxabsrel(Y, Y64) <= TIGHT
        assert not Tr_ref.any()


def test_gemm_deterministic_and_row_independent(tc, mq, orc):
    M, N, K, nnzb = 48, 512, 1024, 6
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=21)
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    sd = dev(tc, s_x).view(tc.float16)
    for v in ("tiled", "tiled_large", "medium", "skinny"):
        rows = M if v != "skinny" else 16
        Xd = dev_x(tc, Xq[:rows])
        Y1 = host(mq.fused_gemm(Xd, sd[:rows].contiguous(), pw, variant=v).view(tc.int16))
        Y2 = host(mq.fused_gemm(Xd, sd[:rows].contiguous(), pw, variant=v).view(tc.int16))
        assert np.array_equal(Y1, Y2)
        for m in (0, 5, 15):
            Ym = host(mq.fused_gemm(dev_x(tc, Xq[m:m + 1]), sd[m:m + 1].contiguous(), pw,
                                    variant=v).view(tc.int16))
            assert np.array_equal(Ym[0], Y1[m]), (v, m)


# ------------------------------------------------ full workload sizes ------
_prep_cache = {}


def _prepared(tc, mq, orc, layer):
    key = (layer.K, layer.N, layer.seed, layer.nnzb)
    if key not in _prep_cache:
        _prep_cache.clear()
        W = layer.weight()
        ref = orc.prepare_weight(W, layer.nnzb)
        pw = mq.prepare_weight(dev(tc, W), layer.nnzb)
        tc.cuda.synchronize()
        assert np.array_equal(orc.unblock_rows(host(pw.Wq), layer.K), ref.Wq)
        assert np.array_equal(orc.unblock_scales(half_bits(pw.s_w)), ref.s_w)
        assert np.array_equal(host(pw.rowptr), ref.rowptr) and np.array_equal(host(pw.kb), ref.kb)
        assert np.array_equal(host(pw.Rq), ref.Rq) and np.array_equal(half_bits(pw.s_r), ref.s_r)
        des = layer.designated()
        if des is not None:
            assert np.array_equal(ref.mask, des)
        del W
        _prep_cache[key] = (ref, pw)
    return _prep_cache[key]


def _samples(M, N, rowptr, rng, count=3000):
    ms = list(rng.integers(0, M, count))
    ns = list(rng.integers(0, N, count))
    for m in {0, M - 1, min(M - 1, 63), min(M - 1, 64), M // 2}:
        for n in {0, N - 1, 127, 128, min(N - 1, 255), min(N - 1, 256), N // 2}:
            ms.append(m)
            ns.append(n)
    hot = np.flatnonzero(np.diff(rowptr) > 0)       # block rows that carry residual
    for nb in hot[:8]:
        for r in (0, 63, 127):
            ms.append(int(rng.integers(0, M)))
            ns.append(int(nb * B + r))
    return np.array(ms, np.int32), np.array(ns, np.int32)


FULL = [(L.name, M) for L in synth.workloads() for M in L.ms]


@pytest.mark.slow
@pytest.mark.parametrize("name,M", FULL, ids=[f"{n}_M{m}" for n, m in FULL])
def test_full_size_sampled(tc, mq, orc, name, M):
    layer = synth.workload(name)
    ref, pw = _prepared(tc, mq, orc, layer)
    X = layer.act(M)
    Xd = dev(tc, X)
    Xq, s_x = mq.quantize_act(Xd)
    Xq_ref, sx_ref = orc.quantize_act(X)
    assert np.array_equal(orc.packed_from_act6(host(Xq), layer.K), Xq_ref)
    assert np.array_equal(half_bits(s_x), sx_ref)
    rng = np.random.default_rng(M + layer.seed)
    ms, ns = _samples(M, layer.N, ref.rowptr, rng)
    tb_ref, tr_ref, y64 = orc.linear_sampled(Xq_ref, sx_ref, ref, ms, ns)
    Y = mq.fused_gemm(Xq, s_x, pw)                     # the launch bench.py times
    Tb, Tr = mq.fused_gemm_acc_i32(Xq, pw)
    mi, ni = tc.from_numpy(ms).long().cuda(), tc.from_numpy(ns).long().cuda()
    tb, tr = host(Tb[mi, ni]), host(Tr[mi, ni])
    y = Y[mi, ni].float().cpu().numpy().astype(np.float64)
    assert np.array_equal(tb, tb_ref) and np.array_equal(tr, tr_ref)
    # norm-relative bar over the sampled outputs
    den = max(np.abs(y64).max(), 1e-30)
    assert np.abs(y - y64).max() / den <= TIGHT


def test_graph_replay_several_tiles_per_workgroup(tc, mq, orc):
    """The decode kernels whose workgroups take several tiles each (grid sized
    on the host from the kernel's occupancy; fused quantisation at 2 rows,
    staged activations at 16) captured in a HIP graph: every replay equals
    the eager result bit for bit."""
    N, K, nnzb = 65920, 1024, 200
    _, _, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(2, N, K, nnzb, seed=515)
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    X = dev(tc, synth.gen_act(2, K, 516))
    X16 = dev(tc, synth.gen_act(16, K, 517))
    Xq16, sx16 = mq.quantize_act(X16)
    Y = tc.empty((2, N), dtype=tc.float16, device="cuda")
    Y16 = tc.empty((16, N), dtype=tc.float16, device="cuda")
    Y_eager = mq.linear(X, pw).clone()
    Y16_eager = mq.fused_gemm(Xq16, sx16, pw).clone()

    def body():
        mq.linear(X, pw, out=Y)
        mq.fused_gemm(Xq16, sx16, pw, out=Y16)

    body()
    tc.cuda.synchronize()
    g = tc.cuda.CUDAGraph()
    with tc.cuda.graph(g):
        body()
    for rep in range(3):
        Y.zero_()
        Y16.zero_()
        mq.linear(X[:1].contiguous(), pw)            # unrelated eager work in between
        tc.cuda.synchronize()
        g.replay()
        tc.cuda.synchronize()
        assert tc.equal(Y.view(tc.int16), Y_eager.view(tc.int16)), rep
        assert tc.equal(Y16.view(tc.int16), Y16_eager.view(tc.int16)), rep


def test_graph_replay_matches_eager(tc, mq, orc):
    """The hot path captured in a HIP graph: every replay (with eager work and
    synchronisation in between) equals the eager result bit for bit."""
    L = synth.workload("c1_1024")
    pw = mq.prepare_weight(dev(tc, L.weight()), L.nnzb)
    X = dev(tc, L.act(64))
    Xq = tc.empty((64, mq.act_bytes(L.K)), dtype=tc.uint8, device="cuda")
    s_x = tc.empty((64,), dtype=tc.float16, device="cuda")
    Y = tc.empty((64, L.N), dtype=tc.float16, device="cuda")
    Y_eager = mq.linear(X, pw).clone()
    Ys = tc.empty((16, L.N), dtype=tc.float16, device="cuda")
    Xs = X[:16].contiguous()
    Xqs = tc.empty((16, mq.act_bytes(L.K)), dtype=tc.uint8, device="cuda")
    sxs = tc.empty((16,), dtype=tc.float16, device="cuda")
    Ys_eager = mq.linear(Xs, pw).clone()

    def body():
        mq.quantize_act(X, out=(Xq, s_x))
        mq.fused_gemm(Xq, s_x, pw, out=Y)
        mq.quantize_act(Xs, out=(Xqs, sxs))
        mq.fused_gemm(Xqs, sxs, pw, out=Ys)

    body()
    tc.cuda.synchronize()
    g = tc.cuda.CUDAGraph()
    with tc.cuda.graph(g):
        body()
    for rep in range(3):
        Y.zero_()
        Ys.zero_()
        mq.linear(X[:5].contiguous(), pw)            # unrelated eager work in between
        tc.cuda.synchronize()
        g.replay()
        tc.cuda.synchronize()
        assert tc.equal(Y.view(tc.int16), Y_eager.view(tc.int16)), rep
        assert tc.equal(Ys.view(tc.int16), Ys_eager.view(tc.int16)), rep
