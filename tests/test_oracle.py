"""Pins for the CPU oracle (no GPU).

Each test ties the oracle to something other than itself: numpy's IEEE half
conversion, exact rational arithmetic, hand-worked fixtures under
tests/golden/, brute-force fp64 / int64 matrix products in numpy, closed-form
invariants of Eq. (1)/(4), and Theorem 4.1 checked by exhaustive subset search.
"""
from __future__ import annotations

import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
B = 128


# ------------------------------------------------------------ helpers ----
def f16(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


def dense_residual(pw, orc):
    """Residual codes and dequantised residual scattered into dense [N, K]."""
    N, K = pw.N, pw.K
    codes = np.zeros((N, K), np.int64)
    deq = np.zeros((N, K), np.float64)
    for nb in range(N // B):
        for p in range(pw.rowptr[nb], pw.rowptr[nb + 1]):
            kb = pw.kb[p]
            c = orc.unpack_codes(pw.Rq[p], B).astype(np.int64)
            codes[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B] = c
            deq[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B] = c * f16(pw.s_r[p])[:, None]
    return codes, deq


def dequant_base(pw, orc):
    codes = orc.unpack_codes(pw.Wq, pw.K).astype(np.float64)
    return codes * np.repeat(f16(pw.s_w), B, axis=1)


def exact_round_half_even(fr: Fraction) -> int:
    fl = fr.numerator // fr.denominator
    rem = fr - fl
    if rem > Fraction(1, 2):
        return fl + 1
    if rem < Fraction(1, 2):
        return fl
    return fl if fl % 2 == 0 else fl + 1


def random_layer(M, N, K, nnzb, seed, orc, dense_codes=False):
    W = synth.gen_weight(N, K, seed)
    pw = orc.prepare_weight(W, nnzb)
    X = synth.gen_act(M, K, seed)
    if dense_codes:   # spread the activations so that most codes are non-zero
        X = (np.random.default_rng(seed).standard_normal((M, K)) * 3).astype(np.float16)
    Xq, s_x = orc.quantize_act(X)
    return W, X, pw, Xq, s_x


# --------------------------------------------------------------- fp16 ----
def test_f16_to_f32_all_bit_patterns(orc):
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = orc.f16_bits_to_f32(bits)
    ref = bits.view(np.float16).astype(np.float32)
    finite = np.isfinite(ref)
    assert np.array_equal(got[finite].view(np.uint32), ref[finite].view(np.uint32))
    assert np.all(np.isnan(got[np.isnan(ref)]))
    assert np.array_equal(np.isinf(got), np.isinf(ref))


def test_f32_to_f16_matches_numpy(orc):
    rng = np.random.default_rng(1)
    # wide exponent range, including subnormal halves and overflow
    mant = rng.random(200000).astype(np.float32) + np.float32(1)
    expo = rng.integers(-30, 18, 200000)
    x = (mant * np.exp2(expo).astype(np.float32)) * rng.choice([-1, 1], 200000).astype(np.float32)
    # exact ties between adjacent halves: (h_i + h_{i+1}) / 2 is exact in fp32
    h = np.arange(0, 0x7BFF, dtype=np.uint16)
    lo = h.view(np.float16).astype(np.float32)
    hi = (h + 1).view(np.float16).astype(np.float32)
    ties = (lo + hi) / np.float32(2)
    edge = np.array([0.0, -0.0, 65504, 65519.99, 65520, 70000, 2**-24, 2**-25,
                     1.5 * 2**-25, 2**-14, 6e-8, 5.96e-8, 1e-10], np.float32)
    allx = np.concatenate([x, ties, -ties, edge, -edge])
    got = orc.f32_to_f16_bits(allx)
    with np.errstate(over="ignore"):
        ref = allx.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


# ------------------------------------------------------ packed layout ----
def _read_layout():
    cases, cur = [], {}
    for line in open(os.path.join(GOLDEN, "pack_layout.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, val = line.split(":", 1)
        cur[key] = val.split()
        if key == "bytes":
            cases.append(cur)
            cur = {}
    return cases


@pytest.mark.parametrize("case", _read_layout(), ids=lambda c: " ".join(c["codes"])[:20])
def test_pack_layout_golden(orc, case):
    """Hand-worked chunks: packing gives the fixture's bytes, both decoders
    (C and numpy) give the codes back."""
    codes = np.array([int(v) for v in case["codes"]], np.int8)[None, :]
    want = bytes(int(b, 16) for b in case["bytes"])
    packed = orc.pack_codes(codes)
    assert packed.tobytes() == want
    buf = np.frombuffer(want, np.uint8)[None, :]
    assert orc.unpack_codes(buf, 16)[0].tolist() == codes[0].tolist()
    import ctypes
    ptr = buf.ctypes.data_as(ctypes.c_void_p)
    assert [orc.lib().orc_unpack_code(ptr, k) for k in range(16)] == codes[0].tolist()


def test_pack_layout_invariants(orc):
    """Round trip of random codes; every byte pattern decodes to [-7, 7] with
    the C and numpy decoders agreeing; the fold masks partition the third
    word's data bits."""
    rng = np.random.default_rng(11)
    codes = rng.integers(-7, 8, (9, 512)).astype(np.int8)
    assert np.array_equal(orc.unpack_codes(orc.pack_codes(codes), 512), codes)
    raw = rng.integers(0, 256, (4, 64), dtype=np.uint8)
    dec = orc.unpack_codes(raw, 128)
    assert dec.min() >= -7 and dec.max() <= 7
    import ctypes
    for r in range(4):
        ptr = raw[r].ctypes.data_as(ctypes.c_void_p)
        assert [orc.lib().orc_unpack_code(ptr, k) for k in range(128)] == dec[r].tolist()
    # re-packing a decoded random pattern reproduces it except for sign bits
    # of zero codes (the only redundancy of the encoding)
    assert np.array_equal(orc.unpack_codes(orc.pack_codes(dec), 128), dec)
    za, zb, z2 = orc._zero_bits(0), orc._zero_bits(1), orc._zero_bits(2)
    assert za & zb == 0 and (za | zb) == (~z2 & 0xFFFFFFFF)
    # each code lands in its own chunk position: a single non-zero code moves
    # exactly one decoded position
    for k in (0, 5, 10, 15, 16, 31, 127):
        one = np.zeros((1, 128), np.int8)
        one[0, k] = -5
        assert np.flatnonzero(orc.unpack_codes(orc.pack_codes(one), 128)[0]).tolist() == [k]


# ------------------------------------------------------- quantiser -------
def _read_ties():
    cases, cur = [], {}
    for line in open(os.path.join(GOLDEN, "quant_ties.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, val = line.split(":", 1)
        cur[key] = val.split()
        if key == "q":
            cases.append(cur)
            cur = {}
    return cases


@pytest.mark.parametrize("case", _read_ties(), ids=lambda c: " ".join(c["x"])[:24])
def test_quantizer_golden_ties(orc, case):
    x = np.array([float(v) for v in case["x"]], np.float16)[None, :]
    pad = -x.shape[1] % 16                      # the packed layout holds chunks of 16 codes
    xq, s = orc.quantize_act(np.concatenate([x, np.zeros((1, pad), np.float16)], axis=1))
    assert float(f16(s)[0]) == float(case["s"][0])
    codes = orc.unpack_codes(xq, xq.shape[1] * 2)[0][: len(case["q"])]
    assert codes.tolist() == [int(v) for v in case["q"]]


def test_act_quant_exact_rational(orc):
    """Every code equals the exactly rounded (Fraction) quotient x / s."""
    rng = np.random.default_rng(7)
    X = (rng.standard_normal((6, 256)) * np.array([[1], [30], [1e-3], [200], [1e-6], [5]])).astype(np.float16)
    X[2, 5] = 0
    Xq, s_x = orc.quantize_act(X)
    codes = orc.unpack_codes(Xq, 256)
    for m in range(6):
        amax = np.abs(X[m].astype(np.float32)).max()
        s_ref = np.float16(np.float32(amax) / np.float32(7))
        assert s_x[m] == s_ref.view(np.uint16)
        s = Fraction(float(s_ref))
        for k in range(256):
            if s == 0:
                assert codes[m, k] == 0
                continue
            q = exact_round_half_even(Fraction(float(X[m, k])) / s)
            assert codes[m, k] == max(-7, min(7, q)), (m, k)


def test_act_quant_zero_row_and_bounds(orc):
    X = np.zeros((3, 128), np.float16)
    X[1] = np.linspace(-5, 5, 128).astype(np.float16)
    X[2, 0] = np.float16(65504)
    Xq, s_x = orc.quantize_act(X)
    assert s_x[0] == 0 and not Xq[0].any()
    codes = orc.unpack_codes(Xq, 128)
    assert codes.min() >= -7 and codes.max() <= 7
    # |x - s q| <= s/2 on every element (Eq. 1 rounding bound)
    s = f16(s_x)
    err = np.abs(X.astype(np.float64) - s[:, None] * codes)
    assert np.all(err <= s[:, None] / 2 * (1 + 1e-12) + 0.0)


def test_weight_quant_groups(orc):
    rng = np.random.default_rng(3)
    N, K = 128, 512
    W = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    W[5, 130] = 0.9            # an outlier only affects its own (row, group)
    W[7, 256:384] = 0          # an all-zero group
    Wq, s_w, R = orc.quantize_weight(W)
    codes = orc.unpack_codes(Wq, K)
    for n in range(N):
        for g in range(K // B):
            v = W[n, g * B:(g + 1) * B]
            s_ref = np.float16(np.abs(v).max() / np.float32(7))
            assert s_w[n, g] == s_ref.view(np.uint16)
    assert s_w[7, 2] == 0 and not codes[7, 256:384].any()
    # R = W - s q with one fp32 rounding (s q exact)
    deq = (codes.astype(np.float32) * np.repeat(f16(s_w), B, axis=1).astype(np.float32))
    assert np.array_equal(R, W - deq)
    # exact-rational rounding of a sample of entries
    s_full = np.repeat(f16(s_w), B, axis=1)
    for (n, k) in rng.integers(0, [N, K], size=(300, 2)):
        s = s_full[n, k]
        if s == 0:
            continue
        fr = Fraction(float(W[n, k])) / Fraction(float(s))
        assert codes[n, k] == max(-7, min(7, exact_round_half_even(fr)))


def test_weight_quant_near_ties_exact(orc):
    """Entries one fp32 ulp either side of every half-integer tie t * s: the
    codes equal exact-rational rounding (an fp32 quotient by an fp16 scale never
    lands on a tie unless the exact quotient is one)."""
    rng = np.random.default_rng(12)
    rows = []
    for _ in range(64):
        s = np.float32(np.float16(rng.uniform(0.003, 0.2)))
        row = np.zeros(B, np.float32)
        row[0] = np.float32(7) * s                 # sets the scale back to s
        if np.float16(row[0] / np.float32(7)) != np.float16(s):
            continue
        j = 1
        for t in np.arange(-6.5, 7, 1.0):
            ts = np.float32(t) * s                 # exact: <= 15 significant bits
            for w in (ts, np.nextafter(ts, np.float32(np.inf)), np.nextafter(ts, np.float32(-np.inf))):
                row[j] = w
                j += 1
        rows.append(row)
    W = np.stack(rows)
    Wq, s_w, _ = orc.quantize_weight(W)
    codes = orc.unpack_codes(Wq, B)
    s_all = f16(s_w)[:, 0]
    for n in range(W.shape[0]):
        for k in range(B):
            fr = Fraction(float(W[n, k])) / Fraction(float(s_all[n]))
            assert codes[n, k] == max(-7, min(7, exact_round_half_even(fr))), (n, k)


# ------------------------------------------------ golden tiny layer ------
def _read_tiny():
    d = {}
    for line in open(os.path.join(GOLDEN, "tiny_layer.txt")):
        line = line.split("#", 1)[0].strip()
        if line:
            k, v = line.split(":", 1)
            d[k.strip()] = v.strip()
    return d


def _sparse(s):
    out = {}
    for tok in s.split():
        i, v = tok.split(":")
        out[int(i)] = float(v)
    return out


def test_golden_tiny_layer(orc):
    d = _read_tiny()
    X = np.zeros((1, B), np.float16)
    for i, v in _sparse(d["x_nonzero"]).items():
        X[0, i] = v
    W = np.zeros((B, B), np.float32)
    for i, v in _sparse(d["w_row0_nonzero"]).items():
        W[0, i] = v
    pw = orc.prepare_weight(W, 1)
    Xq, s_x = orc.quantize_act(X)
    assert f16(s_x)[0] == float(d["s_x"])
    xc = orc.unpack_codes(Xq, B)[0]
    assert {i: int(v) for i, v in enumerate(xc) if v} == {i: int(v) for i, v in _sparse(d["xq_nonzero"]).items()}
    assert f16(pw.s_w)[0, 0] == float(d["s_w_row0"])
    wc = orc.unpack_codes(pw.Wq, B)[0]
    assert {i: int(v) for i, v in enumerate(wc) if v} == {i: int(v) for i, v in _sparse(d["wq_row0_nonzero"]).items()}
    assert pw.score[0, 0] == float(d["score"])
    assert pw.nnzb == 1 and pw.kb.tolist() == [0]
    assert f16(pw.s_r)[0, 0] == float(d["s_r_row0"])
    rc = orc.unpack_codes(pw.Rq[0], B)[0]
    assert {i: int(v) for i, v in enumerate(rc) if v} == {i: int(v) for i, v in _sparse(d["rq_row0_nonzero"]).items()}
    Tb, Tr, Y = orc.linear(Xq, s_x, pw)
    assert Tb[0, 0] == int(d["Tb00"]) and Tr[0, 0] == int(d["Tr00"])
    assert Y[0, 0] == float(d["Y00"])
    assert np.all(Y[0, 1:] == 0)
    pw0 = orc.prepare_weight(W, 0)
    _, Tr0, Y0 = orc.linear(Xq, s_x, pw0)
    assert Y0[0, 0] == float(d["Y00_base_only"]) and not Tr0.any()


# ------------------------------------------- linear layer vs brute force --
@pytest.mark.parametrize("M,N,K,pct", [(1, 128, 128, 100), (3, 256, 256, 25),
                                       (17, 384, 256, 50), (5, 256, 384, 0),
                                       (2, 128, 512, 100)])
@pytest.mark.parametrize("dense", [False, True])
def test_linear_vs_bruteforce(orc, M, N, K, pct, dense):
    nnzb = synth.budget(N, K, pct)
    W, X, pw, Xq, s_x = random_layer(M, N, K, nnzb, 11 + M + N + K, orc, dense_codes=dense)
    Tb, Tr, Y = orc.linear(Xq, s_x, pw)
    xc = orc.unpack_codes(Xq, K).astype(np.int64)
    wc = orc.unpack_codes(pw.Wq, K).astype(np.int64)
    rcodes, rdeq = dense_residual(pw, orc)
    assert np.array_equal(Tb, xc @ wc.T)
    assert np.array_equal(Tr, xc @ rcodes.T)
    # fp64 product of the dequantised operands: Q(X) [Q(W) + M (.) Q(R)]^T
    Wmq = dequant_base(pw, orc) + rdeq
    Yref = (xc * f16(s_x)[:, None]) @ Wmq.T
    scale = max(np.abs(Yref).max(), 1e-300)
    assert np.abs(Y - Yref).max() <= 1e-12 * scale
    if pct == 0:
        assert not Tr.any()
    if dense:
        assert np.count_nonzero(xc) > xc.size // 2


def test_linear_density0_is_plain_w4a4(orc):
    W, X, pw0, Xq, s_x = random_layer(4, 256, 256, 0, 5, orc, dense_codes=True)
    _, _, pw1, _, _ = random_layer(4, 256, 256, 2, 5, orc, dense_codes=True)
    Tb0, Tr0, Y0 = orc.linear(Xq, s_x, pw0)
    Tb1, Tr1, Y1 = orc.linear(Xq, s_x, pw1)
    assert not Tr0.any() and np.array_equal(Tb0, Tb1)   # base is budget-independent
    # plain W4A4: s_x * sum_g s_w A_b, computed here group by group in numpy
    xc = orc.unpack_codes(Xq, 256).astype(np.int64)
    wc = orc.unpack_codes(pw0.Wq, 256).astype(np.int64)
    ref = np.zeros_like(Y0)
    for g in range(2):
        ab = xc[:, g * B:(g + 1) * B] @ wc[:, g * B:(g + 1) * B].T
        ref += ab * f16(pw0.s_w)[:, g][None, :]
    ref *= f16(s_x)[:, None]
    assert np.abs(Y0 - ref).max() <= 1e-12 * np.abs(ref).max()
    # linearity of Eq. (4): T(rho) = Tb + Tr, and Tr only on selected blocks
    assert Tr1.any()


def test_linear_sampled_matches_full(orc):
    W, X, pw, Xq, s_x = random_layer(9, 384, 256, 3, 21, orc, dense_codes=True)
    Tb, Tr, Y = orc.linear(Xq, s_x, pw)
    rng = np.random.default_rng(0)
    ms = rng.integers(0, 9, 200)
    ns = rng.integers(0, 384, 200)
    tb, tr, y = orc.linear_sampled(Xq, s_x, pw, ms, ns)
    assert np.array_equal(tb, Tb[ms, ns]) and np.array_equal(tr, Tr[ms, ns])
    assert np.array_equal(y, Y[ms, ns])


def test_int32_range_extremes(orc):
    """All codes at +-7 over a long K: accumulators stay exact and in int32."""
    K, N, M = 28672, 128, 2
    codes = np.full((M, K), 7, np.int8)
    codes[1] = -7
    Xq = orc.pack_codes(codes)
    s_x = np.full(M, np.float16(1).view(np.uint16))
    W = np.full((N, K), 0.7, np.float32)
    pw = orc.prepare_weight(W, 0)
    Tb, Tr, Y = orc.linear(Xq, s_x, pw)
    assert Tb[0, 0] == 49 * K and Tb[1, 0] == -49 * K and not Tr.any()


# ---------------------------------------- residual / reconstruction ------
def test_reconstruction_improves(orc):
    N, K = 512, 512
    W = synth.gen_weight(N, K, 99)
    for pct in (10, 50, 100):
        pw = orc.prepare_weight(W, synth.budget(N, K, pct))
        base = dequant_base(pw, orc)
        _, rdeq = dense_residual(pw, orc)
        R = W.astype(np.float64) - base
        e_base = np.linalg.norm(W - base)
        e_mq = np.linalg.norm(W - (base + rdeq))
        assert e_mq < e_base
        # entrywise on selected blocks: |R - Q(R)| <= |R| (0 is on the grid)
        sel = np.repeat(np.repeat(pw.mask, B, 0), B, 1)
        assert np.all(np.abs(R - rdeq)[sel] <= np.abs(R)[sel] + 1e-15)
        assert np.all(rdeq[~sel] == 0)
        # memory overhead of the residual = selected fraction of the base bytes
        assert pw.Rq.nbytes / pw.Wq.nbytes == pytest.approx(pw.nnzb / pw.mask.size)


def test_residual_quant_is_eq1_per_block_row(orc):
    N, K = 256, 384
    W = synth.gen_weight(N, K, 8)
    pw = orc.prepare_weight(W, 3)
    _, _, R = orc.quantize_weight(W)
    for nb in range(N // B):
        for p in range(pw.rowptr[nb], pw.rowptr[nb + 1]):
            kb = pw.kb[p]
            blk = R[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B]
            for r in range(0, B, 17):
                s_ref = np.float16(np.abs(blk[r]).max() / np.float32(7))
                assert pw.s_r[p, r] == s_ref.view(np.uint16)
                codes = orc.unpack_codes(pw.Rq[p, r:r + 1], B)[0]
                qf = np.clip(np.rint(blk[r] / np.float32(s_ref)), -7, 7)
                assert np.array_equal(codes, qf.astype(np.int8))


# ------------------------------------------------------------- selection --
def test_scores_and_topk_bruteforce(orc):
    N, K = 640, 768
    W = synth.gen_weight(N, K, 4)
    Wq, s_w, R = orc.quantize_weight(W)
    score = orc.block_scores_frob(R)
    ref = (R.astype(np.float64) ** 2).reshape(N // B, B, K // B, B).sum(axis=(1, 3))
    assert np.allclose(score, ref, rtol=1e-12, atol=0)
    for nnzb in (0, 1, 7, 30):
        rowptr, kb, mask = orc.select_topk(score, nnzb)
        order = np.lexsort((np.arange(score.size), -score.ravel()))
        want = np.zeros(score.size, bool)
        want[order[:nnzb]] = True
        assert np.array_equal(mask.ravel(), want)
        # CSR validity: ascending kb per row, counts match the mask
        assert rowptr[0] == 0 and rowptr[-1] == nnzb
        for nb in range(N // B):
            row = kb[rowptr[nb]:rowptr[nb + 1]]
            assert np.all(np.diff(row) > 0)
            assert set(row.tolist()) == set(np.flatnonzero(want.reshape(N // B, -1)[nb]).tolist())


def test_topk_ties_lower_index_wins(orc):
    score = np.array([[1.0, 3.0, 3.0], [3.0, 0.0, 3.0]])
    rowptr, kb, mask = orc.select_topk(score, 2)
    assert mask.tolist() == [[False, True, True], [False, False, False]]
    rowptr, kb, mask = orc.select_topk(score, 3)
    assert mask.tolist() == [[False, True, True], [True, False, False]]
    assert rowptr.tolist() == [0, 2, 3] and kb.tolist() == [1, 2, 0]
    with pytest.raises(ValueError):
        orc.select_topk(score, 7)


def test_skewed_generator_selects_designated(orc):
    """Residual-norm selection returns exactly the designated skew blocks."""
    N, K = 2048, 1024
    nnzb = synth.budget(N, K, 10)
    des, n_hot = synth.skew_blocks(N, K, nnzb, 1234)
    W = synth.gen_weight(N, K, 1234, designated=des)
    pw = orc.prepare_weight(W, nnzb)
    assert np.array_equal(pw.mask, des)
    assert n_hot == round(0.8 * nnzb)


# ------------------------------------- Algorithm 1 / Theorem 4.1 ---------
def _surrogate(R, h, rdeq_full, sel_blocks, NB, KB):
    E = R.copy()
    for b in sel_blocks:
        nb, kb = divmod(b, KB)
        E[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B] -= rdeq_full[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B]
    return float(np.sum(h[None, :] * E ** 2))


def _all_block_qr(R, orc):
    """Q(R) of every block (Eq. 1 per block row), dense fp64."""
    N, K = R.shape
    out = np.zeros((N, K))
    for nb in range(N // B):
        for kb in range(K // B):
            blk = np.ascontiguousarray(R[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B])
            for r in range(B):
                s = np.float16(np.abs(blk[r]).max() / np.float32(7))
                if s == 0:
                    continue
                q = np.clip(np.rint(blk[r] / np.float32(s)), -7, 7)
                out[nb * B + r, kb * B:(kb + 1) * B] = q * float(s)
    return out


def test_dhessian_topk_optimal_for_diagonal_surrogate(orc):
    """Theorem 4.1: top-K by S_B minimises sum_ij h_j (R - M_S (.) Q(R))^2."""
    N, K = 384, 384                         # 9 blocks
    rng = np.random.default_rng(5)
    W = synth.gen_weight(N, K, 77)
    X = (rng.standard_normal((64, K)) * rng.uniform(0.1, 3, K)).astype(np.float16)
    _, _, R = orc.quantize_weight(W)
    h = orc.hessian_diag(X)
    # h_j = (2/T) sum_t X_tj^2, checked directly
    assert np.allclose(h, 2 / 64 * (X.astype(np.float64) ** 2).sum(0), rtol=1e-12)
    S = orc.block_scores_dhessian(R, h)
    qr = _all_block_qr(R.astype(np.float64), orc)
    NB, KB = N // B, K // B
    for b in range(NB * KB):   # S_B = [L(0) - L({B})]_+ on the surrogate
        d = _surrogate(R.astype(np.float64), h, qr, [], NB, KB) - _surrogate(R.astype(np.float64), h, qr, [b], NB, KB)
        assert S.ravel()[b] == pytest.approx(max(d, 0.0), rel=1e-9, abs=1e-18)
    for Kb in (1, 2, 3, 4):
        best = min(itertools.combinations(range(NB * KB), Kb),
                   key=lambda s: _surrogate(R.astype(np.float64), h, qr, s, NB, KB))
        _, _, mask = orc.select_topk(S, Kb)
        sel = tuple(np.flatnonzero(mask.ravel()))
        assert _surrogate(R.astype(np.float64), h, qr, sel, NB, KB) == pytest.approx(
            _surrogate(R.astype(np.float64), h, qr, best, NB, KB), rel=1e-12)


def test_dhessian_exact_when_offdiagonal_zero(orc):
    """App. A: with orthogonal activation columns (O = 0) the Delta-Hessian
    top-K equals the exhaustive optimum of the exact output distortion."""
    N, K = 256, 384                         # 6 blocks
    rng = np.random.default_rng(9)
    W = synth.gen_weight(N, K, 31)
    T = K
    X = np.zeros((T, K), np.float16)        # token t only touches channel t
    X[np.arange(K), np.arange(K)] = rng.uniform(0.2, 4.0, K).astype(np.float16)
    Xd = X.astype(np.float64)
    assert np.count_nonzero(Xd.T @ Xd - np.diag(np.diag(Xd.T @ Xd))) == 0
    _, _, R = orc.quantize_weight(W)
    h = orc.hessian_diag(X)
    S = orc.block_scores_dhessian(R, h)
    qr = _all_block_qr(R.astype(np.float64), orc)
    NB, KB = N // B, K // B

    def exact(sel):
        E = R.astype(np.float64).copy()
        for b in sel:
            nb, kb = divmod(b, KB)
            E[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B] -= qr[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B]
        return 2 / T * np.linalg.norm(Xd @ E.T) ** 2

    for Kb in (1, 2, 3):
        best = min(itertools.combinations(range(NB * KB), Kb), key=exact)
        _, _, mask = orc.select_topk(S, Kb)
        sel = tuple(np.flatnonzero(mask.ravel()))
        assert exact(sel) == pytest.approx(exact(best), rel=1e-12)


def test_planted_mistakes_are_caught(orc):
    """The brute-force pins fail for plausible oracle mistakes (planted here,
    on the CPU, in numpy restatements of the oracle's output)."""
    W, X, pw, Xq, s_x = random_layer(3, 256, 256, 2, 17, orc, dense_codes=True)
    Tb, Tr, Y = orc.linear(Xq, s_x, pw)
    xc = orc.unpack_codes(Xq, 256).astype(np.int64)
    wc = orc.unpack_codes(pw.Wq, 256).astype(np.int64)
    rcodes, rdeq = dense_residual(pw, orc)
    Yref = (xc * f16(s_x)[:, None]) @ (dequant_base(pw, orc) + rdeq).T
    tol = 1e-12 * np.abs(Yref).max()
    # dropped residual term
    assert np.abs((Y - (xc * f16(s_x)[:, None]) @ rdeq.T) - Yref).max() > tol
    # transposed residual block (rows <-> columns inside a block)
    rdeq_t = rdeq.copy()
    for nb in range(2):
        for kb in range(2):
            blk = rdeq_t[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B]
            rdeq_t[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B] = blk.T
    assert np.abs((xc * f16(s_x)[:, None]) @ (dequant_base(pw, orc) + rdeq_t).T - Yref).max() > tol
    # swapped element order
    wsw = np.empty_like(wc)
    wsw[:, 0::2], wsw[:, 1::2] = wc[:, 1::2], wc[:, 0::2]
    assert not np.array_equal(xc @ wsw.T, Tb)
    # sign error on the residual
    assert not np.array_equal(xc @ (-rcodes).T, Tr)


# ------------------------------------------ canonical nibbles, device order --
def _read_pairs(name, last):
    cases, cur = [], {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, val = line.split(":", 1)
        cur[key] = val.split()
        if key == last:
            cases.append(cur)
            cur = {}
    return cases


@pytest.mark.parametrize("case", _read_pairs("nibble_layout.txt", "bytes"),
                         ids=lambda c: " ".join(c["codes"]))
def test_nibble_layout_golden(orc, case):
    """Hand-worked canonical bytes: packing gives them, unpacking gives the codes."""
    codes = np.array([int(v) for v in case["codes"]], np.int8)[None, :]
    want = bytes(int(b, 16) for b in case["bytes"])
    assert orc.pack_nibbles(codes).tobytes() == want
    assert orc.unpack_nibbles(np.frombuffer(want, np.uint8)[None, :], codes.shape[1]).tolist() == codes.tolist()


def test_nibble_layout_invariants(orc):
    """Round trips over every byte value; each code only moves its own nibble;
    the folded and canonical layouts hold the same codes (-8 saturating)."""
    allb = np.arange(256, dtype=np.uint8)[None, :]
    codes = orc.unpack_nibbles(allb, 512)
    assert codes.min() == -8 and codes.max() == 7
    assert np.array_equal(orc.pack_nibbles(codes), allb)
    # a byte's low nibble is k = 2j, its high nibble k = 2j + 1 (numpy restatement)
    assert np.array_equal(codes[0, 0::2], ((allb[0] & 15).astype(np.int16) ^ 8) - 8)
    assert np.array_equal(codes[0, 1::2], ((allb[0] >> 4).astype(np.int16) ^ 8) - 8)
    for k in (0, 1, 2, 7, 126, 127):
        one = np.zeros((1, 128), np.int8)
        one[0, k] = -3
        b = orc.pack_nibbles(one)
        assert np.flatnonzero(b[0]).tolist() == [k // 2]
        assert np.flatnonzero(orc.unpack_nibbles(b, 128)[0]).tolist() == [k]
    rng = np.random.default_rng(3)
    raw = rng.integers(0, 256, (5, 256), dtype=np.uint8)
    fold = orc.folded_from_nibbles(raw, 512)
    assert np.array_equal(orc.unpack_codes(fold, 512), np.maximum(orc.unpack_nibbles(raw, 512), -7))
    assert np.array_equal(orc.unpack_codes_c(fold, 512), orc.unpack_codes(fold, 512))


def _device_order_golden():
    rows, pieces, scales = None, [], []
    for line in open(os.path.join(GOLDEN, "device_order.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, val = line.split(":", 1)
        v = [int(x) for x in val.split()]
        if key == "rows":
            rows = v[0]
        elif key == "K":
            K = v[0]
        elif key == "piece":
            pieces.append(v)
        elif key == "scale":
            scales.append(v)
    return rows, K, pieces, scales


def test_device_order_golden(orc):
    """block_rows / block_scales (the permutation every GPU parity test applies
    at the boundary) against the hand-worked offsets of the documented
    formulas, and their inverses."""
    R, K, pieces, scales = _device_order_golden()
    G = K // B
    rm = np.zeros((R, K // 2), np.uint8)
    for r in range(R):
        for g in range(G):
            rm[r, 64 * g:64 * (g + 1)] = 16 * (r + 1) + g + np.arange(64) % 2
    dev = orc.block_rows(rm, K).reshape(-1)
    assert len(pieces) == R * G
    for r, g, off in pieces:
        assert np.array_equal(dev[off:off + 64], rm[r, 64 * g:64 * (g + 1)]), (r, g, off)
    assert np.array_equal(orc.unblock_rows(dev.reshape(R, K // 2), K), rm)
    s = (np.arange(R * G, dtype=np.uint16) * 7 + 1).reshape(R, G)
    ds = orc.block_scales(s).reshape(-1)
    assert len(scales) == R * G
    for n, g, el in scales:
        assert ds[el] == s[n, g], (n, g, el)
    assert np.array_equal(orc.unblock_scales(ds.reshape(R, G)), s)


def test_device_order_formula_random(orc):
    """The same formulas at larger, ragged sizes by direct indexing."""
    rng = np.random.default_rng(8)
    for R, K in ((37, 640), (130, 1024), (1, 128)):
        rm = rng.integers(0, 256, (R, K // 2), dtype=np.uint8)
        dev = orc.block_rows(rm, K).reshape(-1)
        for _ in range(200):
            r, g = int(rng.integers(R)), int(rng.integers(K // B))
            off = (g * R + r) * 64
            assert np.array_equal(dev[off:off + 64], rm[r, 64 * g:64 * g + 64])
        s = rng.integers(0, 65536, (R, K // B)).astype(np.uint16)
        ds = orc.block_scales(s).reshape(-1)
        for _ in range(200):
            n, g = int(rng.integers(R)), int(rng.integers(K // B))
            assert ds[g * R + n] == s[n, g]


def _act_layout_golden():
    M = K = None
    cases = []
    for line in open(os.path.join(GOLDEN, "act_operand_layout.txt")):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        key, val = line.split(":", 1)
        if key == "M":
            M = int(val)
        elif key == "K":
            K = int(val)
        else:
            code, nz = val.split("|")
            r, k, q = (int(x) for x in code.split())
            cases.append((r, k, q, {int(a): int(b) for a, b in (t.split(":") for t in nz.split())}))
    return M, K, cases


def test_act_operand_layout_golden(orc):
    """pack_act6 / unpack_act6 (the activation operand layout every GPU test
    compares the quantiser's output with) against hand-worked bytes."""
    M, K, cases = _act_layout_golden()
    for r, k, q, nz in cases:
        codes = np.zeros((M, K), np.int8)
        codes[r, k] = q
        dev = orc.pack_act6(codes).reshape(-1)
        assert dev.size == M * K * 3 // 4
        got = {int(i): int(dev[i]) for i in np.nonzero(dev)[0]}
        assert got == nz, (r, k, q, got)
        back, bad = orc.unpack_act6(dev, K)
        assert bad == 0 and np.array_equal(back, codes)


def test_act_operand_layout_matches_unfolded_chunks(orc):
    """Each quarter's six words are the unfolded words (o0, o1, o2) of the two
    folded chunks of the same 32 codes in the packed layout (whose decoder the
    pack-layout pins fix), and every field decodes back to its code."""
    rng = np.random.default_rng(12)
    for M, K in ((5, 384), (1, 128), (33, 1024)):
        codes = rng.integers(-7, 8, (M, K)).astype(np.int8)
        dev = orc.pack_act6(codes).reshape(-1)
        packed = orc.pack_codes(codes)
        za = sum(1 << (6 * e + b) for e in range(16) for b in (3, 4) if (6 * e + b) < 32)
        zb = sum(1 << (6 * e + b - 32) for e in range(16) for b in (3, 4) if 32 <= (6 * e + b) < 64)
        G = K // B
        for _ in range(40):
            r, g, j = int(rng.integers(M)), int(rng.integers(G)), int(rng.integers(4))
            mo = (g * M + r) * 64 + 16 * j
            to = G * M * 64 + (g * M + r) * 32 + 8 * j
            d = np.concatenate([dev[mo:mo + 16], dev[to:to + 8]]).view("<u4").astype(np.uint64)
            F = sum(int(d[w]) << (32 * w) for w in range(6))
            for h in range(2):
                c = (128 * g + 32 * j + 16 * h) // 16
                p0, p1 = (int(x) for x in packed[r, 8 * c:8 * c + 8].view("<u4"))
                o = (p0 & ~za & 0xFFFFFFFF) | ((p1 & ~zb & 0xFFFFFFFF) << 32) | (((p0 & za) | (p1 & zb)) << 64)
                assert (F >> (96 * h)) & ((1 << 96) - 1) == o, (M, K, r, g, j, h)
            for e in range(32):
                f = (F >> (6 * e)) & 63
                v = -(f & 7) if f & 32 else f & 7
                assert v == codes[r, 128 * g + 32 * j + e]
        back, bad = orc.unpack_act6(dev, K)
        assert bad == 0 and np.array_equal(back, codes)
        assert np.array_equal(orc.packed_from_act6(dev, K), packed)


def test_act_operand_layout_counts_non_codes(orc):
    """A field with an exponent bit set is not a code: unpack_act6 counts it."""
    M, K = 2, 128
    dev = orc.pack_act6(np.zeros((M, K), np.int8)).reshape(-1).copy()
    dev[0] |= 0x08                      # bit 3 of field 0 (exponent) of row 0
    dev[M * 64] |= 0x80                # tail plane, row 0, group 0, quarter 0: d4 bit 7 = F bit 135 (field 22, bit 3)
    _, bad = orc.unpack_act6(dev, K)
    assert bad == 2
    with pytest.raises(ValueError):
        orc.packed_from_act6(dev, K)


def test_hessian_constant_against_exact_distortion(orc):
    """App. A: the exact output distortion L(S) = (2/N) ||X E_S^T||_F^2 (its own
    constant, computed by a matrix product) equals the diagonal surrogate
    sum h_j E_ij^2 built from the oracle's h when the columns of X are
    orthogonal, in absolute value; and L(0) - L(S) is the sum of the oracle's
    Delta-Hessian scores of S.  A wrong factor in h (which the top-K ranking
    cannot see) fails here."""
    N, K = 256, 256
    rng = np.random.default_rng(21)
    W = synth.gen_weight(N, K, 44)
    T = K
    X = np.zeros((T, K), np.float16)
    X[np.arange(K), np.arange(K)] = rng.uniform(0.2, 4.0, K).astype(np.float16)
    Xd = X.astype(np.float64)
    _, _, R = orc.quantize_weight(W)
    h = orc.hessian_diag(X)
    S = orc.block_scores_dhessian(R, h)
    qr = _all_block_qr(R.astype(np.float64), orc)
    KB = K // B

    def err(sel):
        E = R.astype(np.float64).copy()
        for b in sel:
            nb, kb = divmod(b, KB)
            E[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B] -= qr[nb * B:(nb + 1) * B, kb * B:(kb + 1) * B]
        return E

    for sel in ((), (0,), (1, 2), (0, 1, 2, 3)):
        E = err(sel)
        exact = 2.0 / T * np.linalg.norm(Xd @ E.T) ** 2
        surrogate = float((h[None, :] * E ** 2).sum())
        assert surrogate == pytest.approx(exact, rel=1e-12)
        gain = 2.0 / T * np.linalg.norm(Xd @ R.astype(np.float64).T) ** 2 - exact
        assert gain == pytest.approx(sum(S.ravel()[b] for b in sel), rel=1e-9, abs=1e-15)


# ------------------------------------------------------------ W4A8 layer --
def test_quant8_golden_ties(orc):
    """Hand-worked INT8 codes (q_max = 127, round half to even)."""
    for case in _read_pairs("quant8_ties.txt", "q"):
        x = np.array([float(v) for v in case["x"]], np.float16)
        want = [int(v) for v in case["q"]]
        X = np.zeros((1, 128), np.float16)
        X[0, :len(x)] = x
        q, s = orc.quantize_act8(X)
        assert q[0, :len(x)].tolist() == want
        assert not q[0, len(x):].any()


def test_quant8_exact_rational(orc):
    """Every INT8 code equals round-half-even of the exact quotient x / s by the
    stored fp16 scale (Python Fraction), with s = fp16(fp32(max|x|) / 127)."""
    rng = np.random.default_rng(12)
    X = (rng.standard_normal((6, 256)) * rng.uniform(0.01, 50, (6, 1))).astype(np.float16)
    X[1, :7] = [0.5, 1.5, 2.5, 3.5, -0.5, -1.5, -2.5]
    X[1, 7] = 127
    X[2] = 0
    q, s = orc.quantize_act8(X)
    for m in range(X.shape[0]):
        amax = float(np.abs(X[m].astype(np.float32)).max())
        sf = float(np.float16(np.float32(amax) / np.float32(127)))
        assert f16(s[m]) == sf
        for k in range(X.shape[1]):
            want = 0 if sf == 0 else max(-127, min(127, exact_round_half_even(
                Fraction(float(X[m, k])) / Fraction(sf))))
            assert q[m, k] == want, (m, k, float(X[m, k]), sf)


def test_linear_a8_vs_bruteforce(orc):
    """W4A8 layer: int64 sums and the fp64 epilogue against a numpy product of
    the dequantised operands."""
    W = synth.gen_weight(256, 384, 8)
    pw = orc.prepare_weight(W, 3)
    X = synth.gen_act(9, 384, 8)
    q, s = orc.quantize_act8(X)
    Tb, Tr, Y = orc.linear_a8(q, s, pw)
    xc = q.astype(np.int64)
    wc = orc.unpack_codes(pw.Wq, 384).astype(np.int64)
    rcodes, rdeq = dense_residual(pw, orc)
    assert np.array_equal(Tb, xc @ wc.T)
    assert np.array_equal(Tr, xc @ rcodes.T)
    Yref = (xc * f16(s)[:, None]) @ (dequant_base(pw, orc) + rdeq).T
    assert np.abs(Y - Yref).max() <= 1e-12 * np.abs(Yref).max()
    assert np.abs(q).max() == 127


def test_linear_a8_reduces_to_a4_on_4bit_codes(orc):
    """With activation codes inside [-7, 7], the W4A8 layer computes exactly
    what the W4A4 layer computes on the same codes (packed 4-bit)."""
    W = synth.gen_weight(256, 512, 21)
    pw = orc.prepare_weight(W, 4)
    rng = np.random.default_rng(2)
    codes = rng.integers(-7, 8, (5, 512)).astype(np.int8)
    s = np.full(5, np.float16(0.25).view(np.uint16))
    a8 = orc.linear_a8(codes, s, pw)
    a4 = orc.linear(orc.pack_codes(codes), s, pw)
    for u, v in zip(a8, a4):
        assert np.array_equal(u, v)


def test_linear_a8_int32_range(orc):
    """+-127 x +-7 over K = 28672 stays inside int32 (|T| = 889 K)."""
    K, N = 28672, 128
    codes = np.full((2, K), 127, np.int8)
    codes[1] = -127
    wc = np.full((N, K), -7, np.int8)
    pw = orc.PackedWeight(N, K, orc.pack_codes(wc), np.full((N, K // B), 0x3c00, np.uint16),
                          np.zeros(N // B + 1, np.int32), np.zeros(0, np.int32),
                          np.zeros((0, B, B // 2), np.uint8), np.zeros((0, B), np.uint16), None, None)
    Tb, _, _ = orc.linear_a8(codes, np.full(2, 0x3c00, np.uint16), pw)
    assert Tb[0, 0] == -889 * K and Tb[1, 0] == 889 * K
