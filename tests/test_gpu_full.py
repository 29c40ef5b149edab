"""GPU parity at full workload sizes and through the canonical interchange
layout, against the CPU oracle (bars as in test_gpu_parity).

* Every output of the benched launches that the oracle can recompute in
  seconds: the K = N = 4096 layer at each benched M (AUTO picks the 256 x 256
  tiled kernel at M = 4096, the medium kernel at M = 256 and the decode kernel
  at M <= 32) and the 4096 -> 14336 MLP layer at M = 4096.
* Whole output tiles (first, last and the hottest residual block row) of the
  launches too large to recompute entirely, among them the split-K launch of
  the 5120 -> 1024 layer at M = 2048 and the LLaMA3-70B MLP layers.
* The one-kernel decode call (quantisation inside the GEMM) at the benched
  decode shape.
* Canonical int4 operands converted by mq_repack_weights / mq_repack_act:
  parity is defined on those inputs (the oracle decodes the nibbles itself).
"""
from __future__ import annotations

import numpy as np
import pytest

import synth
from gpu_util import (B, TIGHT, _announce, dev, half_bits, host, maxabsrel, mq, random_csr,  # noqa: F401
                      tc)

pytestmark = pytest.mark.gpu

_prep = {}


def prepared(tc, mq, orc, layer):
    """Oracle and GPU preparation of a layer's weights (checked identical)."""
    key = (layer.K, layer.N, layer.seed, layer.nnzb)
    if key not in _prep:
        _prep.clear()
        W = layer.weight()
        ref = orc.prepare_weight(W, layer.nnzb)
        pw = mq.prepare_weight(dev(tc, W), layer.nnzb)
        tc.cuda.synchronize()
        assert np.array_equal(orc.unblock_rows(host(pw.Wq), layer.K), ref.Wq)
        assert np.array_equal(orc.unblock_scales(half_bits(pw.s_w)), ref.s_w)
        assert np.array_equal(host(pw.rowptr), ref.rowptr) and np.array_equal(host(pw.kb), ref.kb)
        assert np.array_equal(host(pw.Rq), ref.Rq) and np.array_equal(half_bits(pw.s_r), ref.s_r)
        del W
        _prep[key] = (ref, pw)
    return _prep[key]


def run_layer(tc, mq, orc, layer, M):
    ref, pw = prepared(tc, mq, orc, layer)
    X = layer.act(M)
    Xq, s_x = mq.quantize_act(dev(tc, X))
    Xq_ref, sx_ref = orc.quantize_act(X)
    assert np.array_equal(orc.packed_from_act6(host(Xq), layer.K), Xq_ref)
    assert np.array_equal(half_bits(s_x), sx_ref)
    Y = mq.fused_gemm(Xq, s_x, pw)                    # the launch bench.py times (AUTO)
    Tb, Tr = mq.fused_gemm_acc_i32(Xq, pw)            # same kernel family, tiles and splits
    tc.cuda.synchronize()
    return ref, Xq_ref, sx_ref, Y, Tb, Tr


# (the 25600-wide layer at M = 1 and 16: decode workgroups that take several tiles each)
FULL_EXHAUSTIVE = [("c2_4096", 1), ("c2_4096", 16), ("c2_4096", 256), ("c2_4096", 4096),
                   ("c3_up_d10", 4096), ("c4_qo", 32), ("c4_kv", 32), ("c4_up", 1), ("c4_up", 16)]


@pytest.mark.slow
@pytest.mark.parametrize("name,M", FULL_EXHAUSTIVE, ids=[f"{n}_M{m}" for n, m in FULL_EXHAUSTIVE])
def test_full_size_every_output(tc, mq, orc, name, M):
    layer = synth.workload(name)
    ref, Xq_ref, sx_ref, Y, Tb, Tr = run_layer(tc, mq, orc, layer, M)
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq_ref, sx_ref, ref)
    assert np.array_equal(host(Tb), Tb_ref), "Tb differs"
    assert np.array_equal(host(Tr), Tr_ref), "Tr differs"
    assert maxabsrel(Y, Y64) <= TIGHT


def tiles_to_check(M, N, rowptr, T=256):
    """Row and column ranges of the first and last T x T output tiles and of a
    T-row tile over the block row with the most residual blocks."""
    hot = int(np.argmax(np.diff(rowptr)))
    mid = max(0, min(M - T, (M // 2) // T * T))
    return [(0, min(T, M), 0, min(T, N)),
            (max(0, M - T), M, max(0, N - T), N),
            (mid, min(mid + T, M), hot * B, hot * B + B)]


WHOLE_TILES = [("c4_kv", 2048), ("c4_qo", 2048), ("c4_up", 2048), ("c4_down", 2048),
               ("c3_down_d20", 4096), ("c5_up", 8192), ("c5_down", 8192)]


@pytest.mark.slow
@pytest.mark.parametrize("name,M", WHOLE_TILES, ids=[f"{n}_M{m}" for n, m in WHOLE_TILES])
def test_full_size_whole_tiles(tc, mq, orc, name, M):
    layer = synth.workload(name)
    ref, Xq_ref, sx_ref, Y, Tb, Tr = run_layer(tc, mq, orc, layer, M)
    for m0, m1, n0, n1 in tiles_to_check(M, layer.N, ref.rowptr):
        mm, nn = np.meshgrid(np.arange(m0, m1, dtype=np.int32), np.arange(n0, n1, dtype=np.int32),
                             indexing="ij")
        ms, ns = mm.ravel(), nn.ravel()
        tb_ref, tr_ref, y64 = orc.linear_sampled(Xq_ref, sx_ref, ref, ms, ns)
        tile = (slice(m0, m1), slice(n0, n1))
        assert np.array_equal(host(Tb[tile]).ravel(), tb_ref), (m0, n0)
        assert np.array_equal(host(Tr[tile]).ravel(), tr_ref), (m0, n0)
        y = Y[tile].float().cpu().numpy().astype(np.float64).ravel()
        assert np.abs(y - y64).max() / max(np.abs(y64).max(), 1e-30) <= TIGHT, (m0, n0)


def test_split_k_raw_sums(tc, mq, orc):
    """Raw int32 sums of a split-K launch (128 x 128 tiles over K ranges, each
    split walking the CSR from its own first group) are bit-exact."""
    from gpu_util import gpu_pw, orc_pw, random_operands, dev_x
    lib = mq.load()
    for M, N, K, nnzb in ((256, 1024, 2048, 40), (70, 128, 4096, 32), (300, 256, 8192, 64)):
        assert lib.mq_fused_gemm_workspace_size(M, N, K) > 0, "shape must take split-K"
        Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=M + N + K)
        Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
        pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
        Xd = dev_x(tc, Xq)
        for v in ("tiled", "auto"):
            Tb, Tr = mq.fused_gemm_acc_i32(Xd, pw, variant=v)
            Y = mq.fused_gemm(Xd, dev(tc, s_x).view(tc.float16), pw, variant=v)
            tc.cuda.synchronize()
            assert np.array_equal(host(Tb), Tb_ref), (M, N, K, v)
            assert np.array_equal(host(Tr), Tr_ref), (M, N, K, v)
            assert maxabsrel(Y, Y64) <= TIGHT


LINEAR_DECODE = [("c2_4096", 1), ("c2_4096", 2), ("c2_4096", 4), ("c4_up", 1), ("c4_up", 4)]


@pytest.mark.parametrize("name,M", LINEAR_DECODE, ids=[f"{n}_M{m}" for n, m in LINEAR_DECODE])
def test_linear_decode_benched_shape(tc, mq, orc, name, M):
    """mq_linear at decode shapes with the layers' own weights (K = N = 4096,
    the benched layer; 5120 -> 25600, where each workgroup takes several
    tiles): one kernel quantises and multiplies; every output against the
    oracle, bit-identical to quantise-then-GEMM."""
    layer = synth.workload(name)
    ref, pw = prepared(tc, mq, orc, layer)
    X = layer.act(M)
    Xq_ref, sx_ref = orc.quantize_act(X)
    _, _, Y64 = orc.linear(Xq_ref, sx_ref, ref)
    Xd = dev(tc, X)
    assert mq.linear_workspace_bytes(M, layer.N, layer.K) == 0      # the one-kernel path
    Y = mq.linear(Xd, pw)
    Xq, s_x = mq.quantize_act(Xd)
    Y2 = mq.fused_gemm(Xq, s_x, pw)
    tc.cuda.synchronize()
    assert maxabsrel(Y, Y64) <= TIGHT
    assert np.array_equal(host(Y.view(tc.int16)), host(Y2.view(tc.int16)))


# -------------------------------------------------- canonical interchange --
def canonical_operands(orc, M, N, K, nnzb, seed, n_minus8=0):
    """Random canonical int4 operands (codes in [-7, 7]; optionally a few -8
    nibbles in W) and the oracle's folded row-major packing of their codes."""
    rng = np.random.default_rng(seed)
    xc = rng.integers(-7, 8, (M, K)).astype(np.int8)
    wc = rng.integers(-7, 8, (N, K)).astype(np.int8)
    rc = rng.integers(-7, 8, (nnzb, B, B)).astype(np.int8)
    if n_minus8:
        idx = rng.choice(N * K, n_minus8, replace=False)
        wc.reshape(-1)[idx] = -8
    s_x = rng.uniform(0.01, 2.0, M).astype(np.float16).view(np.uint16)
    s_w = rng.uniform(1e-3, 0.05, (N, K // B)).astype(np.float16).view(np.uint16)
    s_r = rng.uniform(1e-4, 5e-3, (nnzb, B)).astype(np.float16).view(np.uint16)
    rowptr, kb, sel = random_csr(N // B, K // B, nnzb, rng)
    canon = dict(Xq=orc.pack_nibbles(xc), Wq=orc.pack_nibbles(wc), Rq=orc.pack_nibbles(rc))
    ref = orc.PackedWeight(N, K, orc.pack_codes(np.maximum(wc, -7)), s_w, rowptr, kb,
                           orc.pack_codes(rc), s_r, None, sel)
    return canon, ref, orc.pack_codes(xc), s_x


@pytest.mark.parametrize("M,N,K,nnzb", [(5, 256, 384, 3), (64, 1024, 1024, 10), (300, 512, 2048, 16),
                                        (1, 4096, 4096, 102)])
def test_canonical_operands_parity(tc, mq, orc, M, N, K, nnzb):
    """Parity on canonical inputs: nibbles -> mq_repack_* -> fused GEMM,
    against the oracle on the same codes; the inverse conversions give the
    canonical bytes back."""
    canon, ref, Xq_fold, s_x = canonical_operands(orc, M, N, K, nnzb, seed=M * 3 + N + K)
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq_fold, s_x, ref)
    pw = mq.repack_weights(dev(tc, canon["Wq"]), dev(tc, ref.s_w).view(tc.float16), dev(tc, ref.rowptr),
                           dev(tc, ref.kb), dev(tc, canon["Rq"]), dev(tc, ref.s_r).view(tc.float16))
    Xq = mq.repack_act(dev(tc, canon["Xq"]))
    sx = dev(tc, s_x).view(tc.float16)
    Tb, Tr = mq.fused_gemm_acc_i32(Xq, pw)
    Y = mq.fused_gemm(Xq, sx, pw)
    tc.cuda.synchronize()
    assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref)
    assert maxabsrel(Y, Y64) <= TIGHT
    # the library layout is the oracle's folded packing in the documented order
    assert np.array_equal(orc.unblock_rows(host(pw.Wq), K), ref.Wq)
    assert np.array_equal(orc.unblock_scales(half_bits(pw.s_w)), ref.s_w)
    assert np.array_equal(host(pw.Rq), ref.Rq)
    assert np.array_equal(orc.packed_from_act6(host(Xq), K), Xq_fold)
    # inverse conversions
    Wq_c, s_w_c, Rq_c = mq.unpack_weights(pw)
    Xq_c = mq.unpack_act(Xq)
    tc.cuda.synchronize()
    assert np.array_equal(host(Wq_c), canon["Wq"]) and np.array_equal(host(Rq_c), canon["Rq"])
    assert np.array_equal(half_bits(s_w_c), ref.s_w)
    assert np.array_equal(host(Xq_c), canon["Xq"])


def test_canonical_minus8_saturates_and_counts(tc, mq, orc):
    """-8 nibbles are stored as -7 (the method's range) and counted."""
    M, N, K, nnzb = 16, 256, 512, 2
    canon, ref, Xq_fold, s_x = canonical_operands(orc, M, N, K, nnzb, seed=4, n_minus8=37)
    Tb_ref, _, _ = orc.linear(Xq_fold, s_x, ref)
    cnt = tc.zeros((1,), dtype=tc.int32, device="cuda")
    pw = mq.repack_weights(dev(tc, canon["Wq"]), dev(tc, ref.s_w).view(tc.float16), dev(tc, ref.rowptr),
                           dev(tc, ref.kb), dev(tc, canon["Rq"]), dev(tc, ref.s_r).view(tc.float16),
                           n_invalid=cnt)
    Tb, _ = mq.fused_gemm_acc_i32(mq.repack_act(dev(tc, canon["Xq"]), n_invalid=cnt), pw)
    tc.cuda.synchronize()
    assert int(cnt.item()) == 37
    assert np.array_equal(host(Tb), Tb_ref)


def test_quantize_act_canonical_codes(tc, mq, orc):
    """mq_quantize_act's codes read back in the canonical layout equal the
    oracle's codes of Eq. (1)."""
    X = synth.gen_act(37, 1280, 99)
    Xq, _ = mq.quantize_act(dev(tc, X))
    Xq_c = mq.unpack_act(Xq)
    tc.cuda.synchronize()
    Xq_ref, _ = orc.quantize_act(X)
    assert np.array_equal(host(Xq_c), orc.pack_nibbles(orc.unpack_codes(Xq_ref, 1280)))


# ------------------------------------------------------ unfused baseline --
@pytest.mark.parametrize("M,N,K,nnzb", [(37, 512, 1024, 9), (256, 1024, 2048, 40), (4096, 4096, 4096, 102),
                                        (1, 256, 512, 8)])
def test_unfused_baseline_matches_oracle(tc, mq, orc, M, N, K, nnzb):
    """The three-kernel baseline (dense GEMM, separate residual GEMM reading Xq
    again, reduce-add) against the oracle's fp64 epilogue, within the output
    bar (its dense output is rounded to fp16 once more); block rows without
    residual blocks equal the dense-only fused call bit for bit."""
    from gpu_util import gpu_pw, orc_pw, random_operands, dev_x
    Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=M + 5 * N + K)
    _, _, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xd, sd = dev_x(tc, Xq), dev(tc, s_x).view(tc.float16)
    Y = mq.unfused_gemm(Xd, sd, pw)
    dense_only = mq.PackedWeight(N, K, pw.Wq, pw.s_w, dev(tc, np.zeros(N // B + 1, np.int32)),
                                 dev(tc, np.zeros(0, np.int32)), pw.Rq[:0], pw.s_r[:0])
    Yd = mq.fused_gemm(Xd, sd, dense_only)
    tc.cuda.synchronize()
    assert maxabsrel(Y, Y64) <= 2e-3
    empty = np.flatnonzero(np.diff(rowptr) == 0)
    cols = (empty[:, None] * B + np.arange(B)[None, :]).ravel()
    assert np.array_equal(host(Y.view(tc.int16))[:, cols], host(Yd.view(tc.int16))[:, cols])


# ------------------------------------------------------------ decode kernel --
DECODE = [(1, 16384, 1024, "full"), (16, 16384, 512, "rand"), (3, 8192, 1280, "full"),
          (17, 8192, 640, "rand"), (32, 16384, 384, "full"), (5, 4096, 128, "full"),
          (1, 4096, 896, "none"), (32, 1024, 2048, "full"), (9, 2048, 28672, "rand")]


def decode_csr(N, K, kind, rng):
    """CSR with every block of some block rows (so each wave of a workgroup
    gets entries, and rows with fewer entries than waves occur), random
    blocks elsewhere; or random only; or none."""
    NB, KB = N // B, K // B
    sel = np.zeros((NB, KB), bool)
    if kind == "full":
        sel[rng.choice(NB, max(1, NB // 8), replace=False)] = True
        sel |= rng.random((NB, KB)) < 0.05
    elif kind == "rand":
        sel = rng.random((NB, KB)) < 0.1
    rowptr = np.zeros(NB + 1, np.int32)
    rowptr[1:] = np.cumsum(sel.sum(1))
    kb = np.concatenate([np.flatnonzero(r) for r in sel]).astype(np.int32) if sel.any() else np.zeros(0, np.int32)
    return rowptr, kb, sel


@pytest.mark.parametrize("M,N,K,kind", DECODE, ids=[f"M{m}_N{n}_K{k}_{c}" for m, n, k, c in DECODE])
def test_decode_kernel_every_output(tc, mq, orc, M, N, K, kind):
    """The decode kernel over its strip counts (1, 2, 4 strips of 16 columns
    per workgroup), row tiles (M <= 16, <= 32), K with fewer groups than
    waves, full and empty block rows: Tb, Tr bit-exact, Y within the bar,
    and mq_linear's one-kernel path (quantisation inside) at M <= 4."""
    from gpu_util import gpu_pw, orc_pw, dev_x
    rng = np.random.default_rng(M * 31 + N + K)
    rowptr, kb, sel = decode_csr(N, K, kind, rng)
    nnzb = int(rowptr[-1])
    Xq = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    s_x = rng.uniform(0.01, 2.0, M).astype(np.float16).view(np.uint16)
    Wq = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    s_w = rng.uniform(1e-3, 0.05, (N, K // B)).astype(np.float16).view(np.uint16)
    Rq = rng.integers(0, 256, (nnzb, B, B // 2), dtype=np.uint8)
    s_r = rng.uniform(1e-4, 5e-3, (nnzb, B)).astype(np.float16).view(np.uint16)
    Tb_ref, Tr_ref, Y64 = orc.linear(Xq, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xd = dev_x(tc, Xq)
    Tb, Tr = mq.fused_gemm_acc_i32(Xd, pw, variant="skinny")
    Y = mq.fused_gemm(Xd, dev(tc, s_x).view(tc.float16), pw, variant="skinny")
    tc.cuda.synchronize()
    assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref)
    assert maxabsrel(Y, Y64) <= TIGHT
    if M <= 4 and M * K // 2 <= 65536:
        X = synth.gen_act(M, K, 11 + M + K)
        Xq_r, sx_r = orc.quantize_act(X)
        _, _, Y64x = orc.linear(Xq_r, sx_r, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
        assert mq.linear_workspace_bytes(M, N, K) == 0
        Yl = mq.linear(dev(tc, X), pw)
        tc.cuda.synchronize()
        assert maxabsrel(Yl, Y64x) <= TIGHT


# ------------------------------------------- concatenated-output operators --
T5 = [("t5_qkv", 32), ("t5_gate_up", 4), ("t5_down", 8), ("t5_o", 8192), ("t5_qkv", 8192),
      ("t5_gate_up", 8192), ("t5_down", 8192)]


@pytest.mark.slow
@pytest.mark.parametrize("name,M", T5, ids=[f"{n}_M{m}" for n, m in T5])
def test_table5_operators(tc, mq, orc, name, M):
    """Qwen3-8B concatenated-output operators at decode and prefill sizes:
    every output at decode M, whole tiles at prefill M."""
    layer = synth.workload(name)
    ref, Xq_ref, sx_ref, Y, Tb, Tr = run_layer(tc, mq, orc, layer, M)
    if M <= 32:
        Tb_ref, Tr_ref, Y64 = orc.linear(Xq_ref, sx_ref, ref)
        assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref)
        assert maxabsrel(Y, Y64) <= TIGHT
        return
    for m0, m1, n0, n1 in tiles_to_check(M, layer.N, ref.rowptr):
        mm, nn = np.meshgrid(np.arange(m0, m1, dtype=np.int32), np.arange(n0, n1, dtype=np.int32),
                             indexing="ij")
        tb_ref, tr_ref, y64 = orc.linear_sampled(Xq_ref, sx_ref, ref, mm.ravel(), nn.ravel())
        tile = (slice(m0, m1), slice(n0, n1))
        assert np.array_equal(host(Tb[tile]).ravel(), tb_ref)
        assert np.array_equal(host(Tr[tile]).ravel(), tr_ref)
        y = Y[tile].float().cpu().numpy().astype(np.float64).ravel()
        assert np.abs(y - y64).max() / max(np.abs(y64).max(), 1e-30) <= TIGHT
