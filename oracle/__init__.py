"""CPU oracle (test infrastructure): numpy front end of ``mq_oracle.c``.

Only the test-suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never does, and this
package imports nothing from it: the two sides share only the seeded input
generator in ``synth``.

Every function returns fresh numpy arrays; fp16 quantities are returned as
their raw ``uint16`` bit patterns (compare bit-for-bit) unless noted.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mq_oracle.c")
_LIB = os.path.join(_HERE, "libmq_oracle.so")
BLOCK = 128

_CFLAGS = ["-O3", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
           "-shared", "-fPIC", "-std=c11", "-Wall"]


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (always when ``force``)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", *_CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        _lib = C.CDLL(build())
        P = C.c_void_p
        i, i64 = C.c_int, C.c_int64
        sig = {
            "orc_num_threads": (i, []),
            "orc_f32_to_f16": (C.c_uint16, [C.c_float]),
            "orc_f16_to_f32": (C.c_float, [C.c_uint16]),
            "orc_f32_to_f16_array": (None, [P, P, i64]),
            "orc_f16_to_f32_array": (None, [P, P, i64]),
            "orc_pack_codes": (None, [P, i, i, P]),
            "orc_unpack_codes": (None, [P, i, i, P]),
            "orc_pack_nibbles": (None, [P, i, i, P]),
            "orc_unpack_nibbles": (None, [P, i, i, P]),
            "orc_pack_act6": (None, [P, i, i, P]),
            "orc_unpack_act6": (i64, [P, i, i, P]),
            "orc_unpack_code": (i, [P, i]),
            "orc_quantize_act": (None, [P, i, i, i, P, P]),
            "orc_quantize_weight": (None, [P, i, i, P, P, P]),
            "orc_block_scores_frob": (None, [P, i, i, P]),
            "orc_hessian_diag": (None, [P, i, i, P]),
            "orc_block_scores_dhessian": (None, [P, i, i, P, P]),
            "orc_select_topk": (C.c_int, [P, i, i, i, P, P, P]),
            "orc_quantize_residual": (None, [P, i, i, P, P, i, P, P]),
            "orc_linear": (i64, [i, i, i, P, P, P, P, P, P, i, P, P, P, P, P]),
            "orc_linear_sampled": (i64, [i, i, i, P, P, P, P, P, P, i, P, P,
                                         i64, P, P, P, P, P]),
            "orc_quantize_act8": (None, [P, i, i, i, P, P]),
            "orc_linear_a8": (i64, [i, i, i, P, P, P, P, P, P, i, P, P, P, P, P]),
            "orc_linear_a8_sampled": (i64, [i, i, i, P, P, P, P, P, P, i, P, P,
                                            i64, P, P, P, P, P]),
        }
        for name, (res, args) in sig.items():
            f = getattr(_lib, name)
            f.restype = res
            f.argtypes = args
    return _lib


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle expects C-contiguous arrays"
    return a.ctypes.data


def num_threads() -> int:
    return int(lib().orc_num_threads())


# ---------------------------------------------------------------- fp16 ----
def f32_to_f16_bits(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().orc_f32_to_f16_array(_p(x), _p(out), x.size)
    return out


def f16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, np.float32)
    lib().orc_f16_to_f32_array(_p(h), _p(out), h.size)
    return out


def _zero_bits(w: int) -> int:
    """Always-zero bits of 32-bit word w of a chunk's 96-bit field word (the
    two middle bits, 6e+3 and 6e+4, of every 6-bit field e)."""
    z = 0
    for e in range(16):
        for b in (3, 4):
            bit = 6 * e + b
            if bit // 32 == w:
                z |= 1 << (bit % 32)
    return z


def unpack_codes(packed: np.ndarray, K: int) -> np.ndarray:
    """Signed int8 codes [rows, K] from packed rows [rows, K/2] (pure numpy
    restatement of the chunk layout documented in mq_oracle.c; tests only).
    Chunk c of a row (bytes 8c..8c+7, little-endian words P0, P1) holds codes
    16c..16c+15; the 96-bit field word is (P0 & ~ZA, P1 & ~ZB,
    (P0 & ZA) | (P1 & ZB)) and code e is the sign-magnitude field at bit 6e."""
    p = np.ascontiguousarray(packed, dtype=np.uint8).reshape(-1, K // 2)
    words = p.reshape(p.shape[0], K // 16, 2, 4).astype(np.uint64)
    w = words[..., 0] | (words[..., 1] << 8) | (words[..., 2] << 16) | (words[..., 3] << 24)
    p0, p1 = w[..., 0], w[..., 1]
    za, zb = np.uint64(_zero_bits(0)), np.uint64(_zero_bits(1))
    full = np.uint64(0xFFFFFFFF)
    o = [p0 & (full ^ za), p1 & (full ^ zb), (p0 & za) | (p1 & zb)]
    big = o[0] | (o[1] << np.uint64(32))          # bits 0..63 of the field word
    out = np.empty((p.shape[0], K // 16, 16), np.int8)
    for e in range(16):
        lo = 6 * e
        if lo + 6 <= 64:
            f = (big >> np.uint64(lo)) & np.uint64(63)
        else:                                     # fields 11..15 start in word 2 or straddle
            f = ((o[1] >> np.uint64(lo - 32)) | (o[2] << np.uint64(64 - lo))) & np.uint64(63) \
                if lo < 64 else (o[2] >> np.uint64(lo - 64)) & np.uint64(63)
        mag = (f & np.uint64(7)).astype(np.int8)
        out[..., e] = np.where((f & np.uint64(32)) != 0, -mag, mag)
    return out.reshape(p.shape[0], K)


def pack_codes(codes: np.ndarray) -> np.ndarray:
    """Packed rows [rows, K/2] of int codes [rows, K] in [-7, 7] (oracle C)."""
    q = np.ascontiguousarray(codes, dtype=np.int8)
    q2 = q.reshape(-1, q.shape[-1])
    if np.abs(q2.astype(np.int16)).max(initial=0) > 7:
        raise ValueError("codes must lie in [-7, 7]")
    out = np.empty((q2.shape[0], q2.shape[1] // 2), np.uint8)
    lib().orc_pack_codes(_p(q2), q2.shape[0], q2.shape[1], _p(out))
    return out.reshape(*q.shape[:-1], q.shape[-1] // 2)


def unpack_codes_c(packed: np.ndarray, K: int) -> np.ndarray:
    """Signed int8 codes [rows, K] of folded packed rows [rows, K/2] (oracle C)."""
    p = np.ascontiguousarray(packed, np.uint8).reshape(-1, K // 2)
    out = np.empty((p.shape[0], K), np.int8)
    lib().orc_unpack_codes(_p(p), p.shape[0], K, _p(out))
    return out


# ---------------------------------------------------- canonical nibbles ----
# The interchange layout of the library's boundary: two's-complement 4-bit
# codes, two per byte, even k in the low nibble, rows in k order.
def pack_nibbles(codes: np.ndarray) -> np.ndarray:
    """Canonical nibble rows [rows, K/2] of int codes [rows, K] in [-8, 7]."""
    q = np.ascontiguousarray(codes, dtype=np.int8)
    q2 = q.reshape(-1, q.shape[-1])
    if q2.size and (q2.min() < -8 or q2.max() > 7):
        raise ValueError("codes must lie in [-8, 7]")
    out = np.empty((q2.shape[0], q2.shape[1] // 2), np.uint8)
    lib().orc_pack_nibbles(_p(q2), q2.shape[0], q2.shape[1], _p(out))
    return out.reshape(*q.shape[:-1], q.shape[-1] // 2)


def unpack_nibbles(packed: np.ndarray, K: int) -> np.ndarray:
    """Signed codes [rows, K] in [-8, 7] of canonical nibble rows [rows, K/2]."""
    p = np.ascontiguousarray(packed, np.uint8).reshape(-1, K // 2)
    out = np.empty((p.shape[0], K), np.int8)
    lib().orc_unpack_nibbles(_p(p), p.shape[0], K, _p(out))
    return out


def folded_from_nibbles(packed: np.ndarray, K: int) -> np.ndarray:
    """Canonical nibble rows -> the oracle's folded rows (row-major), codes
    of -8 saturated to -7 (the codes the library's repacking produces)."""
    q = np.maximum(unpack_nibbles(packed, K), -7)
    return pack_codes(q).reshape(np.asarray(packed).shape)


# ------------------------------------------------------- device layout ----
# The oracle works on row-major packed rows ([rows, K/2], row r's 64-byte
# group pieces in K order) and row-major scales ([N, K/128]).  The GPU library
# stores the same bytes group-major, so that every 128-row x 128-code tile is
# one contiguous 8 KB run and the tiles of neighbouring row blocks are
# neighbours in memory:
#   packed rows: piece (row r, group g) at byte (g rows + r) 64;
#   weight scales: s_w[n, g] at element g N + n.
# These helpers are that permutation and its inverse (tests only).
def block_rows(packed: np.ndarray, K: int) -> np.ndarray:
    """Row-major packed rows [rows, K/2] -> device group-major order (same shape)."""
    p = np.ascontiguousarray(packed, np.uint8).reshape(-1, K // 2)
    rows, G = p.shape[0], K // BLOCK
    return np.ascontiguousarray(p.reshape(rows, G, 64).transpose(1, 0, 2)).reshape(rows, K // 2)


def unblock_rows(dev: np.ndarray, K: int) -> np.ndarray:
    """Device group-major order -> row-major packed rows [rows, K/2]."""
    d = np.ascontiguousarray(dev, np.uint8).reshape(-1, K // 2)
    rows, G = d.shape[0], K // BLOCK
    return np.ascontiguousarray(d.reshape(G, rows, 64).transpose(1, 0, 2)).reshape(rows, K // 2)


def block_scales(s_w: np.ndarray) -> np.ndarray:
    """Row-major weight scales [N, K/128] -> device order [K/128, N]
    (returned with shape [N, K/128])."""
    s = np.ascontiguousarray(s_w)
    N, G = s.shape
    return np.ascontiguousarray(s.T).reshape(N, G)


def unblock_scales(dev: np.ndarray) -> np.ndarray:
    d = np.ascontiguousarray(dev)
    N, G = d.shape
    return np.ascontiguousarray(d.reshape(G, N).T)


# The activation operand layout the library's quantiser writes (3K/4 bytes
# a row; oracle C, from the field definition): a main plane and a tail plane
# per 128-code group, holding the unfolded 6-bit fields of each 32-code quarter.
def pack_act6(codes: np.ndarray) -> np.ndarray:
    """Activation operand layout [M, 3K/4] of int codes [M, K] in [-7, 7]."""
    q = np.ascontiguousarray(codes, dtype=np.int8)
    M, K = q.shape
    if np.abs(q.astype(np.int16)).max(initial=0) > 7:
        raise ValueError("codes must lie in [-7, 7]")
    out = np.empty((M, 3 * K // 4), np.uint8)
    lib().orc_pack_act6(_p(q), M, K, _p(out))
    return out


def unpack_act6(dev: np.ndarray, K: int):
    """Codes [M, K] of the activation operand layout, and the number of
    fields that are not codes (non-zero exponent bits)."""
    d = np.ascontiguousarray(dev, np.uint8).reshape(-1)
    M = d.size // (3 * K // 4)
    out = np.empty((M, K), np.int8)
    bad = lib().orc_unpack_act6(_p(d), M, K, _p(out))
    return out, int(bad)


def act6_from_packed(packed: np.ndarray, K: int) -> np.ndarray:
    """Row-major folded packed rows [M, K/2] -> activation operand layout."""
    return pack_act6(unpack_codes_c(packed, K))


def packed_from_act6(dev: np.ndarray, K: int) -> np.ndarray:
    """Activation operand layout -> row-major folded packed rows [M, K/2]
    (raises if a field is not a code)."""
    q, bad = unpack_act6(dev, K)
    if bad:
        raise ValueError(f"{bad} fields of the activation operand layout are not codes")
    return pack_codes(q)


# ------------------------------------------------------- quantisation ----
def quantize_act(X: np.ndarray):
    """Per-token INT4 of fp16 X [M, K] -> (Xq uint8 [M, K/2], s_x bits [M])."""
    X = np.ascontiguousarray(X, dtype=np.float16)
    M, K = X.shape
    Xq = np.empty((M, K // 2), np.uint8)
    s_x = np.empty(M, np.uint16)
    lib().orc_quantize_act(_p(X.view(np.uint16)), M, K, K, _p(Xq), _p(s_x))
    return Xq, s_x


def quantize_weight(W: np.ndarray, want_residual: bool = True):
    """Base INT4 (group 128) of fp32 W [N, K] -> (Wq [N,K/2], s_w bits [N,K/128], R fp32)."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    N, K = W.shape
    Wq = np.empty((N, K // 2), np.uint8)
    s_w = np.empty((N, K // BLOCK), np.uint16)
    R = np.empty((N, K), np.float32) if want_residual else None
    lib().orc_quantize_weight(_p(W), N, K, _p(Wq), _p(s_w), _p(R))
    return Wq, s_w, R


def block_scores_frob(R: np.ndarray) -> np.ndarray:
    R = np.ascontiguousarray(R, dtype=np.float32)
    N, K = R.shape
    out = np.empty((N // BLOCK, K // BLOCK), np.float64)
    lib().orc_block_scores_frob(_p(R), N, K, _p(out))
    return out


def hessian_diag(X: np.ndarray) -> np.ndarray:
    X = np.ascontiguousarray(X, dtype=np.float16)
    T, K = X.shape
    h = np.empty(K, np.float64)
    lib().orc_hessian_diag(_p(X.view(np.uint16)), T, K, _p(h))
    return h


def block_scores_dhessian(R: np.ndarray, h: np.ndarray) -> np.ndarray:
    R = np.ascontiguousarray(R, dtype=np.float32)
    h = np.ascontiguousarray(h, dtype=np.float64)
    N, K = R.shape
    out = np.empty((N // BLOCK, K // BLOCK), np.float64)
    lib().orc_block_scores_dhessian(_p(R), N, K, _p(h), _p(out))
    return out


def select_topk(score: np.ndarray, nnzb: int):
    """-> (rowptr int32 [NB+1], kb int32 [nnzb], mask bool [NB, KB])."""
    score = np.ascontiguousarray(score, dtype=np.float64)
    NB, KB = score.shape
    rowptr = np.empty(NB + 1, np.int32)
    kb = np.empty(max(nnzb, 1), np.int32)
    mask = np.empty(NB * KB, np.uint8)
    rc = lib().orc_select_topk(_p(score), NB, KB, nnzb, _p(rowptr), _p(kb), _p(mask))
    if rc != 0:
        raise ValueError("bad block budget")
    return rowptr, kb[:nnzb].copy(), mask.reshape(NB, KB).astype(bool)


def quantize_residual(R: np.ndarray, rowptr: np.ndarray, kb: np.ndarray):
    """-> (Rq uint8 [nnzb, 128, 64], s_r bits [nnzb, 128])."""
    R = np.ascontiguousarray(R, dtype=np.float32)
    N, K = R.shape
    nnzb = int(rowptr[-1])
    Rq = np.zeros((max(nnzb, 1), BLOCK, BLOCK // 2), np.uint8)
    s_r = np.zeros((max(nnzb, 1), BLOCK), np.uint16)
    rowptr = np.ascontiguousarray(rowptr, np.int32)
    kb = np.ascontiguousarray(kb if len(kb) else np.zeros(1, np.int32), np.int32)
    lib().orc_quantize_residual(_p(R), N, K, _p(rowptr), _p(kb), nnzb, _p(Rq), _p(s_r))
    return Rq[:nnzb].copy(), s_r[:nnzb].copy()


@dataclass
class PackedWeight:
    """The kernel's weight operands in canonical layout (oracle-produced)."""
    N: int
    K: int
    Wq: np.ndarray        # uint8 [N, K/2]
    s_w: np.ndarray       # fp16 bits [N, K/128]
    rowptr: np.ndarray    # int32 [N/128 + 1]
    kb: np.ndarray        # int32 [nnzb]
    Rq: np.ndarray        # uint8 [nnzb, 128, 64]
    s_r: np.ndarray       # fp16 bits [nnzb, 128]
    score: np.ndarray     # fp64 [N/128, K/128]
    mask: np.ndarray      # bool [N/128, K/128]

    @property
    def nnzb(self) -> int:
        return int(self.rowptr[-1])


def prepare_weight(W: np.ndarray, nnzb: int, criterion: str = "frob",
                   X_calib: Optional[np.ndarray] = None) -> PackedWeight:
    """Alg. 1 end to end: base quantisation, residual, block scores, top-K,
    residual quantisation.  ``criterion``: "frob" (||R_B||_F^2) or "dhessian"."""
    Wq, s_w, R = quantize_weight(W)
    if criterion == "frob":
        score = block_scores_frob(R)
    elif criterion == "dhessian":
        score = block_scores_dhessian(R, hessian_diag(X_calib))
    else:
        raise ValueError(criterion)
    rowptr, kb, mask = select_topk(score, nnzb)
    Rq, s_r = quantize_residual(R, rowptr, kb)
    N, K = W.shape
    return PackedWeight(N, K, Wq, s_w, rowptr, kb, Rq, s_r, score, mask)


# ------------------------------------------------------- linear layer ----
def _lin_args(Xq, s_x, pw: PackedWeight):
    M = Xq.shape[0]
    nnzb = pw.nnzb
    z32 = np.zeros(1, np.int32)
    Rq = pw.Rq if nnzb else np.zeros((1, BLOCK, BLOCK // 2), np.uint8)
    s_r = pw.s_r if nnzb else np.zeros((1, BLOCK), np.uint16)
    kb = pw.kb if nnzb else z32
    keep = (np.ascontiguousarray(Xq), np.ascontiguousarray(s_x, np.uint16),
            np.ascontiguousarray(pw.Wq), np.ascontiguousarray(pw.s_w),
            np.ascontiguousarray(pw.rowptr, np.int32), np.ascontiguousarray(kb, np.int32),
            np.ascontiguousarray(Rq), np.ascontiguousarray(s_r))
    return M, keep, nnzb


def linear(Xq: np.ndarray, s_x: np.ndarray, pw: PackedWeight):
    """Full layer -> (Tb int64 [M,N], Tr int64 [M,N], Y64 fp64 [M,N])."""
    M, k, nnzb = _lin_args(Xq, s_x, pw)
    N, K = pw.N, pw.K
    Tb = np.empty((M, N), np.int64)
    Tr = np.empty((M, N), np.int64)
    Y = np.empty((M, N), np.float64)
    ovf = lib().orc_linear(M, N, K, *[_p(a) for a in k[:6]], nnzb, _p(k[6]), _p(k[7]),
                           _p(Tb), _p(Tr), _p(Y))
    if ovf:
        raise OverflowError(f"{ovf} accumulators exceed int32")
    return Tb, Tr, Y


def linear_sampled(Xq: np.ndarray, s_x: np.ndarray, pw: PackedWeight,
                   ms: np.ndarray, ns: np.ndarray):
    """Selected outputs (ms[i], ns[i]) -> (Tb, Tr, Y64) 1-D arrays."""
    M, k, nnzb = _lin_args(Xq, s_x, pw)
    ms = np.ascontiguousarray(ms, np.int32)
    ns = np.ascontiguousarray(ns, np.int32)
    cnt = ms.size
    Tb = np.empty(cnt, np.int64)
    Tr = np.empty(cnt, np.int64)
    Y = np.empty(cnt, np.float64)
    ovf = lib().orc_linear_sampled(M, pw.N, pw.K, *[_p(a) for a in k[:6]], nnzb,
                                   _p(k[6]), _p(k[7]), cnt, _p(ms), _p(ns),
                                   _p(Tb), _p(Tr), _p(Y))
    if ovf:
        raise OverflowError(f"{ovf} accumulators exceed int32")
    return Tb, Tr, Y


# ---------------------------------------------------------- W4A8 layer ----
def quantize_act8(X: np.ndarray):
    """Per-token INT8 of fp16 X [M, K] (q_max = 127) -> (codes int8 [M, K], s_x bits [M])."""
    X = np.ascontiguousarray(X, dtype=np.float16)
    M, K = X.shape
    q = np.empty((M, K), np.int8)
    s_x = np.empty(M, np.uint16)
    lib().orc_quantize_act8(_p(X.view(np.uint16)), M, K, K, _p(q), _p(s_x))
    return q, s_x


def linear_a8(Xq8: np.ndarray, s_x: np.ndarray, pw: PackedWeight):
    """W4A8 layer from int8 activation codes -> (Tb int64, Tr int64, Y64 fp64) [M, N]."""
    Xq8 = np.ascontiguousarray(Xq8, np.int8)
    M, k, nnzb = _lin_args(np.zeros((Xq8.shape[0], 1), np.uint8), s_x, pw)
    N, K = pw.N, pw.K
    Tb = np.empty((M, N), np.int64)
    Tr = np.empty((M, N), np.int64)
    Y = np.empty((M, N), np.float64)
    ovf = lib().orc_linear_a8(M, N, K, _p(Xq8), *[_p(a) for a in k[1:6]], nnzb, _p(k[6]), _p(k[7]),
                              _p(Tb), _p(Tr), _p(Y))
    if ovf:
        raise OverflowError(f"{ovf} accumulators exceed int32")
    return Tb, Tr, Y


def linear_a8_sampled(Xq8: np.ndarray, s_x: np.ndarray, pw: PackedWeight,
                      ms: np.ndarray, ns: np.ndarray):
    Xq8 = np.ascontiguousarray(Xq8, np.int8)
    M, k, nnzb = _lin_args(np.zeros((Xq8.shape[0], 1), np.uint8), s_x, pw)
    ms = np.ascontiguousarray(ms, np.int32)
    ns = np.ascontiguousarray(ns, np.int32)
    cnt = ms.size
    Tb = np.empty(cnt, np.int64)
    Tr = np.empty(cnt, np.int64)
    Y = np.empty(cnt, np.float64)
    ovf = lib().orc_linear_a8_sampled(M, pw.N, pw.K, _p(Xq8), *[_p(a) for a in k[1:6]], nnzb,
                                      _p(k[6]), _p(k[7]), cnt, _p(ms), _p(ns), _p(Tb), _p(Tr), _p(Y))
    if ovf:
        raise OverflowError(f"{ovf} accumulators exceed int32")
    return Tb, Tr, Y
