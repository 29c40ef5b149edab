"""GPU parity of the W4A8 variant (per-token INT8 activations) against the
CPU oracle: INT8 codes and scales bit-exact, raw int32 sums bit-exact, fp16
outputs within the bar; the A8 layout round-trips through the canonical int8
codes."""
from __future__ import annotations

import numpy as np
import pytest

import synth
from gpu_util import B, TIGHT, _announce, dev, gpu_pw, half_bits, host, maxabsrel, mq, orc_pw, random_operands, tc  # noqa: F401

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("M,K", [(1, 128), (5, 1024), (64, 4096), (33, 640), (3, 28672)])
def test_quantize_act8_parity(tc, mq, orc, M, K):
    rng = np.random.default_rng(M + K)
    X = synth.gen_act(M, K, 400 + M)
    if M > 2:
        X[1] = 0                                                     # zero row
        X[2, :8] = np.array([127, 0.5, 1.5, 2.5, -0.5, -2.5, 126.5, -127], np.float16)
        X[2, 8:] = 0                                                 # exact ties at s = 1
    if M > 3:
        X[3] = (rng.standard_normal(K) * 1e-6).astype(np.float16)   # subnormal halves
    if M > 4:
        X[4, K // 3] = 65504
    Xq8, s_x = mq.quantize_act8(dev(tc, X))
    codes = mq.unpack_act8(Xq8)
    tc.cuda.synchronize()
    q_ref, s_ref = orc.quantize_act8(X)
    assert np.array_equal(half_bits(s_x), s_ref)
    assert np.array_equal(host(codes), q_ref)


def test_act8_layout_round_trip(tc, mq):
    rng = np.random.default_rng(5)
    codes = rng.integers(-128, 128, (37, 1280)).astype(np.int8)
    codes[0, :256] = np.arange(-128, 128)
    cnt = tc.zeros((1,), dtype=tc.int32, device="cuda")
    Xq8 = mq.repack_act8(dev(tc, codes), n_invalid=cnt)
    back = mq.unpack_act8(Xq8)
    tc.cuda.synchronize()
    want = np.maximum(codes, -127)
    assert np.array_equal(host(back), want)
    assert int(cnt.item()) == int((codes == -128).sum())
    again = mq.repack_act8(back)
    tc.cuda.synchronize()
    assert np.array_equal(host(again), host(Xq8))


A8_CASES = [(1, 256, 384, 3), (5, 1024, 1024, 10), (16, 16384, 512, 40), (17, 2048, 640, 9), (32, 8192, 384, 20),
            (33, 512, 1024, 6), (70, 1024, 2048, 16), (257, 512, 512, 8), (256, 4096, 1024, 30)]


@pytest.mark.parametrize("M,N,K,nnzb", A8_CASES, ids=[f"M{c[0]}_N{c[1]}_K{c[2]}_r{c[3]}" for c in A8_CASES])
def test_gemm_a8_parity(tc, mq, orc, M, N, K, nnzb):
    _, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=M * 5 + N + K)
    codes = np.random.default_rng(M + N).integers(-127, 128, (M, K)).astype(np.int8)
    Tb_ref, Tr_ref, Y64 = orc.linear_a8(codes, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xq8 = mq.repack_act8(dev(tc, codes))
    Tb, Tr = mq.fused_gemm_a8_acc_i32(Xq8, pw)
    Y = mq.fused_gemm_a8(Xq8, dev(tc, s_x).view(tc.float16), pw)
    tc.cuda.synchronize()
    assert np.array_equal(host(Tb), Tb_ref)
    assert np.array_equal(host(Tr), Tr_ref)
    assert maxabsrel(Y, Y64) <= TIGHT


def test_gemm_a8_extreme_codes(tc, mq, orc):
    """+-127 x +-7 over K = 28672, every block of a block row: sums at their extreme."""
    M, N, K = 20, 256, 28672
    xc = np.full((M, K), -127, np.int8)
    xc[1::2] = 127
    wc = np.full((N, K), -7, np.int8)
    wc[::3] = 7
    Wq = orc.pack_codes(wc)
    s_x = np.full(M, np.float16(1).view(np.uint16))
    s_w = np.full((N, K // B), np.float16(2 ** -14).view(np.uint16))
    KB = K // B
    rowptr = np.array([0, KB, KB], np.int32)
    kb = np.arange(KB, dtype=np.int32)
    Rq = orc.pack_codes(np.full((KB, B, B), 7, np.int8))
    s_r = np.full((KB, B), np.float16(2 ** -16).view(np.uint16))
    sel = np.zeros((2, KB), bool)
    sel[0] = True
    Tb_ref, Tr_ref, Y64 = orc.linear_a8(xc, s_x, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
    assert np.abs(Tb_ref).max() == 889 * K
    pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
    Xq8 = mq.repack_act8(dev(tc, xc))
    Tb, Tr = mq.fused_gemm_a8_acc_i32(Xq8, pw)
    Y = mq.fused_gemm_a8(Xq8, dev(tc, s_x).view(tc.float16), pw)
    tc.cuda.synchronize()
    assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref)
    assert maxabsrel(Y, Y64) <= TIGHT


_prep = {}


@pytest.mark.slow
@pytest.mark.parametrize("M", [1, 16, 256, 4096])
def test_gemm_a8_full_size_every_output(tc, mq, orc, M):
    """The W4A8 layer on the K = N = 4096 workload (its weights prepared on
    both sides and checked identical): every output."""
    layer = synth.workload("c2_4096")
    if "c2" not in _prep:
        W = layer.weight()
        ref = orc.prepare_weight(W, layer.nnzb)
        pw = mq.prepare_weight(dev(tc, W), layer.nnzb)
        tc.cuda.synchronize()
        assert np.array_equal(orc.unblock_rows(host(pw.Wq), layer.K), ref.Wq)
        _prep["c2"] = (ref, pw)
    ref, pw = _prep["c2"]
    X = layer.act(M)
    Xq8, s_x = mq.quantize_act8(dev(tc, X))
    Tb, Tr = mq.fused_gemm_a8_acc_i32(Xq8, pw)
    Y = mq.fused_gemm_a8(Xq8, s_x, pw)
    codes = mq.unpack_act8(Xq8)
    tc.cuda.synchronize()
    q_ref, s_ref = orc.quantize_act8(X)
    assert np.array_equal(host(codes), q_ref) and np.array_equal(half_bits(s_x), s_ref)
    Tb_ref, Tr_ref, Y64 = orc.linear_a8(q_ref, s_ref, ref)
    assert np.array_equal(host(Tb), Tb_ref) and np.array_equal(host(Tr), Tr_ref)
    assert maxabsrel(Y, Y64) <= TIGHT
