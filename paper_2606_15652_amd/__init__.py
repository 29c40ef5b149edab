"""Python binding of libmq (MosaicQuant fused W4A4 + sparse-residual GEMM on
MI355X / gfx950).

Argument marshalling only: every function checks tensor dtypes, devices and
layouts, then calls the C ABI declared in ``include/mq.h`` with raw device
pointers and the current torch stream.  All arithmetic runs in libmq's HIP
kernels; there is no fallback.  Importing the package does not load the
library; the first call does, and raises if ``libmq.so`` has not been built
(``python -m paper_2606_15652_amd.build``) or no GPU is visible.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmq.so")

MQ_OK = 0
VARIANTS = {"auto": 0, "skinny": 1, "tiled": 2, "tiled_large": 3, "medium": 4}
BLOCK = 128

_P = C.c_void_p
_I = C.c_int
_SIG = {
    "mq_status_string": (C.c_char_p, [_I]),
    "mq_version": (_I, []),
    "mq_quantize_act": (_I, [_P, _I, _I, _I, _P, _P, _P]),
    "mq_fused_gemm_workspace_size": (C.c_size_t, [_I, _I, _I]),
    "mq_fused_gemm_plan": (_I, [_I, _I, _I, _P, _P]),
    "mq_fused_gemm": (_I, [_I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P, _P, _P, _I, _P,
                          C.c_size_t, _P]),
    "mq_linear_workspace_size": (C.c_size_t, [_I, _I, _I]),
    "mq_linear": (_I, [_I, _I, _I, _P, _I, _P, _P, _P, _P, _I, _P, _P, _P, _I, _P,
                      C.c_size_t, _P]),
    "mq_fused_gemm_variant": (_I, [_I, _I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P, _P, _P, _I,
                                  _P, C.c_size_t, _P]),
    "mq_fused_gemm_acc_i32": (_I, [_I, _I, _I, _I, _P, _P, _P, _P, _I, _P, _P, _P, _P]),
    "mq_quantize_weight": (_I, [_P, _I, _I, _I, _P, _P, _P, _P]),
    "mq_hessian_diag": (_I, [_P, _I, _I, _I, _P, _P]),
    "mq_block_scores_dhessian": (_I, [_P, _I, _I, _I, _P, _P, _P, _P, _P]),
    "mq_select_blocks": (_I, [_P, _I, _I, _I, _P, _P, _P]),
    "mq_quantize_residual": (_I, [_P, _I, _I, _I, _P, _P, _P, _P, _I, _P, _P, _P]),
    "mq_unfused_workspace_size": (C.c_size_t, [_I, _I, _I]),
    "mq_unfused_gemm": (_I, [_I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P, _P, _P, _I, _P,
                            C.c_size_t, _P]),
    "mq_quantize_act8": (_I, [_P, _I, _I, _I, _P, _P, _P]),
    "mq_fused_gemm_a8": (_I, [_I, _I, _I, _P, _P, _P, _P, _P, _P, _I, _P, _P, _P, _I, _P]),
    "mq_fused_gemm_a8_acc_i32": (_I, [_I, _I, _I, _P, _P, _P, _P, _I, _P, _P, _P, _P]),
    "mq_repack_act8": (_I, [_I, _I, _P, _I, _P, _P, _P]),
    "mq_unpack_act8": (_I, [_I, _I, _P, _P, _I, _P]),
    "mq_scratch_bytes": (C.c_size_t, []),
    "mq_linear_noalloc": (_I, [_I, _I, _I, _P, _I, _P, _P, _P, _P, _I, _P, _P, _P, _I, _P]),
    "mq_repack_weights": (_I, [_I, _I, _P, _P, _I, _P, _P, _P, _P, _P, _P]),
    "mq_unpack_weights": (_I, [_I, _I, _P, _P, _I, _P, _P, _P, _P, _P]),
    "mq_repack_act": (_I, [_I, _I, _P, _I, _P, _P, _P]),
    "mq_unpack_act": (_I, [_I, _I, _P, _P, _I, _P]),
}

_lib: Optional[C.CDLL] = None


class MQError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = load().mq_status_string(status).decode()
        super().__init__(f"{fn} failed with status {status}: {msg}")
        self.status = status


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load libmq.so (once) and declare its signatures."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise ImportError(f"libmq.so not found at {path}; build it with "
                              "`python -m paper_2606_15652_amd.build` (hipcc, gfx950)")
        lib = C.CDLL(path)
        for name, (res, args) in _SIG.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


# ------------------------------------------------------------------ utils --
def _torch():
    import torch
    return torch


def _stream(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t, dtype, name, ndim=None):
    torch = _torch()
    if t is None:
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D, got shape {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check(fn, status):
    if status != MQ_OK:
        raise MQError(fn, status)


def _need_out(t, shape, dtype, name):
    """A caller-provided output: CUDA, contiguous rows, the exact shape."""
    _need(t, dtype, name, len(shape))
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def _scratch(nbytes, device, stream, given=None, name="workspace"):
    """Workspace for one launch on `stream`.  A caller-provided tensor is
    checked for size; an allocated one is tied to `stream` when that is not
    torch's current stream, so that the caching allocator does not hand it
    out again while the launch still uses it."""
    torch = _torch()
    if nbytes == 0:
        return None
    if given is not None:
        _need(given, torch.uint8, name)
        if given.numel() < nbytes:
            raise ValueError(f"{name} needs {nbytes} bytes, got {given.numel()}")
        return given
    buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
    if stream is not None and stream != torch.cuda.current_stream(device):
        buf.record_stream(stream)
    return buf


# -------------------------------------------------------------- hot path --
def act_bytes(K: int) -> int:
    """Bytes per row of INT4 activation codes in the library's operand layout (3K/4)."""
    return 3 * K // 4


def quantize_act(X, out=None, stream=None):
    """Per-token INT4 quantisation of fp16 X [M, K] -> (Xq uint8 [M, 3K/4] in
    the operand layout, s_x fp16 [M])."""
    torch = _torch()
    _need(X, torch.float16, "X", 2)
    M, K = X.shape
    if out is None:
        Xq = torch.empty((M, act_bytes(K)), dtype=torch.uint8, device=X.device)
        s_x = torch.empty((M,), dtype=torch.float16, device=X.device)
    else:
        Xq, s_x = out
        _need_out(Xq, (M, act_bytes(K)), torch.uint8, "out[0] (Xq)")
        _need_out(s_x, (M,), torch.float16, "out[1] (s_x)")
    _check("mq_quantize_act", load().mq_quantize_act(_ptr(X), M, K, X.stride(0), _ptr(Xq),
                                                     _ptr(s_x), _stream(stream)))
    return Xq, s_x


@dataclass
class PackedWeight:
    """Device-resident operands of one MosaicQuant linear layer, in the
    library's storage order (include/mq.h): Wq's N*K/2 bytes group-major
    (piece (row n, group g) at (g N + n) 64), s_w's N*K/128 values [K/128][N]."""
    N: int
    K: int
    Wq: "object"          # uint8, N*K/2 bytes held as [N, K/2], group order
    s_w: "object"         # fp16, N*K/128 values held as [N, K/128], order [K/128][N]
    rowptr: "object"      # int32 [N/128 + 1]
    kb: "object"          # int32 [nnzb] (may be empty)
    Rq: "object"          # uint8 [nnzb, 128, 64]
    s_r: "object"         # fp16 [nnzb, 128]
    score: "object" = None

    @property
    def nnzb(self) -> int:
        return int(self.kb.numel())

    @property
    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in
                   (self.Wq, self.s_w, self.rowptr, self.kb, self.Rq, self.s_r))


def _res_ptrs(pw: PackedWeight):
    if pw.nnzb == 0:
        return None, None, None, None
    return _ptr(pw.rowptr), _ptr(pw.kb), _ptr(pw.Rq), _ptr(pw.s_r)


def plan(M: int, N: int, K: int):
    """(kernel family name, K splits) that the AUTO variant takes for an
    M x N x K layer (host logic only; no device needed)."""
    v, sp = C.c_int(0), C.c_int(0)
    _check("mq_fused_gemm_plan", load().mq_fused_gemm_plan(M, N, K, C.byref(v), C.byref(sp)))
    name = {code: n for n, code in VARIANTS.items()}[v.value]
    return name, sp.value


def fused_gemm(Xq, s_x, pw: PackedWeight, out=None, variant: str = "auto", stream=None,
               workspace=None):
    """Y fp16 [M, N] = s_x * (Xq Wq^T scaled per group + sparse residual term)."""
    torch = _torch()
    _need(Xq, torch.uint8, "Xq", 2)
    _need(s_x, torch.float16, "s_x", 1)
    M = Xq.shape[0]
    if Xq.shape[1] != act_bytes(pw.K) or s_x.shape[0] != M:
        raise ValueError("Xq / s_x shapes do not match the weight")
    Y = out if out is not None else torch.empty((M, pw.N), dtype=torch.float16, device=Xq.device)
    if out is not None:
        _need_out(Y, (M, pw.N), torch.float16, "out")
    rp, kb, rq, sr = _res_ptrs(pw)
    lib = load()
    ws = lib.mq_fused_gemm_workspace_size(M, pw.N, pw.K)
    wbuf = _scratch(ws, Xq.device, stream, workspace)
    _check("mq_fused_gemm", lib.mq_fused_gemm_variant(
        VARIANTS[variant], M, pw.N, pw.K, _ptr(Xq), _ptr(s_x), _ptr(pw.Wq), _ptr(pw.s_w),
        rp, kb, pw.nnzb, rq, sr, _ptr(Y), Y.stride(0), _ptr(wbuf), ws, _stream(stream)))
    return Y


def unfused_gemm(Xq, s_x, pw: PackedWeight, out=None, stream=None, workspace=None):
    """The three-kernel baseline (dense GEMM, separate residual GEMM,
    reduce-add) on the same operands as fused_gemm; Y fp16 [M, N]."""
    torch = _torch()
    _need(Xq, torch.uint8, "Xq", 2)
    _need(s_x, torch.float16, "s_x", 1)
    M = Xq.shape[0]
    if Xq.shape[1] != act_bytes(pw.K) or s_x.shape[0] != M:
        raise ValueError("Xq / s_x shapes do not match the weight")
    Y = out if out is not None else torch.empty((M, pw.N), dtype=torch.float16, device=Xq.device)
    if out is not None:
        _need_out(Y, (M, pw.N), torch.float16, "out")
    rp, kb, rq, sr = _res_ptrs(pw)
    lib = load()
    ws = lib.mq_unfused_workspace_size(M, pw.N, pw.K)
    wbuf = _scratch(ws, Xq.device, stream, workspace)
    _check("mq_unfused_gemm", lib.mq_unfused_gemm(
        M, pw.N, pw.K, _ptr(Xq), _ptr(s_x), _ptr(pw.Wq), _ptr(pw.s_w), rp, kb, pw.nnzb, rq, sr,
        _ptr(Y), Y.stride(0), _ptr(wbuf), ws, _stream(stream)))
    return Y


def fused_gemm_acc_i32(Xq, pw: PackedWeight, variant: str = "auto", stream=None):
    """Raw exact integer sums (Tb, Tr) int32 [M, N] of the same main loop."""
    torch = _torch()
    _need(Xq, torch.uint8, "Xq", 2)
    M = Xq.shape[0]
    if Xq.shape[1] != act_bytes(pw.K):
        raise ValueError("Xq shape does not match the weight")
    Tb = torch.empty((M, pw.N), dtype=torch.int32, device=Xq.device)
    Tr = torch.empty((M, pw.N), dtype=torch.int32, device=Xq.device)
    rp, kb, rq, _ = _res_ptrs(pw)
    _check("mq_fused_gemm_acc_i32", load().mq_fused_gemm_acc_i32(
        VARIANTS[variant], M, pw.N, pw.K, _ptr(Xq), _ptr(pw.Wq), rp, kb, pw.nnzb, rq,
        _ptr(Tb), _ptr(Tr), _stream(stream)))
    return Tb, Tr


# ------------------------------------------------------- W4A8 variant --
def quantize_act8(X, out=None, stream=None):
    """Per-token INT8 quantisation of fp16 X [M, K] -> (Xq8 uint8 [M, 3K/2] in
    the A8 layout, s_x fp16 [M])."""
    torch = _torch()
    _need(X, torch.float16, "X", 2)
    M, K = X.shape
    if out is None:
        Xq8 = torch.empty((M, 3 * K // 2), dtype=torch.uint8, device=X.device)
        s_x = torch.empty((M,), dtype=torch.float16, device=X.device)
    else:
        Xq8, s_x = out
        _need_out(Xq8, (M, 3 * K // 2), torch.uint8, "out[0] (Xq8)")
        _need_out(s_x, (M,), torch.float16, "out[1] (s_x)")
    _check("mq_quantize_act8", load().mq_quantize_act8(_ptr(X), M, K, X.stride(0), _ptr(Xq8),
                                                       _ptr(s_x), _stream(stream)))
    return Xq8, s_x


def fused_gemm_a8(Xq8, s_x, pw: PackedWeight, out=None, stream=None):
    """W4A8 layer: Y fp16 [M, N] from INT8 activation codes (A8 layout)."""
    torch = _torch()
    _need(Xq8, torch.uint8, "Xq8", 2)
    _need(s_x, torch.float16, "s_x", 1)
    M = Xq8.shape[0]
    if Xq8.shape[1] * 2 != 3 * pw.K or s_x.shape[0] != M:
        raise ValueError("Xq8 / s_x shapes do not match the weight")
    Y = out if out is not None else torch.empty((M, pw.N), dtype=torch.float16, device=Xq8.device)
    if out is not None:
        _need_out(Y, (M, pw.N), torch.float16, "out")
    rp, kb, rq, sr = _res_ptrs(pw)
    _check("mq_fused_gemm_a8", load().mq_fused_gemm_a8(
        M, pw.N, pw.K, _ptr(Xq8), _ptr(s_x), _ptr(pw.Wq), _ptr(pw.s_w), rp, kb, pw.nnzb, rq, sr,
        _ptr(Y), Y.stride(0), _stream(stream)))
    return Y


def fused_gemm_a8_acc_i32(Xq8, pw: PackedWeight, stream=None):
    torch = _torch()
    _need(Xq8, torch.uint8, "Xq8", 2)
    M = Xq8.shape[0]
    Tb = torch.empty((M, pw.N), dtype=torch.int32, device=Xq8.device)
    Tr = torch.empty((M, pw.N), dtype=torch.int32, device=Xq8.device)
    rp, kb, rq, _ = _res_ptrs(pw)
    _check("mq_fused_gemm_a8_acc_i32", load().mq_fused_gemm_a8_acc_i32(
        M, pw.N, pw.K, _ptr(Xq8), _ptr(pw.Wq), rp, kb, pw.nnzb, rq, _ptr(Tb), _ptr(Tr), _stream(stream)))
    return Tb, Tr


def unpack_act8(Xq8, stream=None):
    """A8 layout -> canonical int8 codes [M, K]."""
    torch = _torch()
    _need(Xq8, torch.uint8, "Xq8", 2)
    M, K = Xq8.shape[0], Xq8.shape[1] * 2 // 3
    Xc = torch.empty((M, K), dtype=torch.int8, device=Xq8.device)
    _check("mq_unpack_act8", load().mq_unpack_act8(M, K, _ptr(Xq8), _ptr(Xc), K, _stream(stream)))
    return Xc


def repack_act8(Xc, n_invalid=None, stream=None):
    """Canonical int8 codes [M, K] -> A8 layout."""
    torch = _torch()
    _need(Xc, torch.int8, "Xc", 2)
    M, K = Xc.shape
    Xq8 = torch.empty((M, 3 * K // 2), dtype=torch.uint8, device=Xc.device)
    if n_invalid is not None:
        _need(n_invalid, torch.int32, "n_invalid", 1)
    _check("mq_repack_act8", load().mq_repack_act8(M, K, _ptr(Xc), Xc.stride(0), _ptr(Xq8),
                                                   _ptr(n_invalid), _stream(stream)))
    return Xq8


def linear_workspace_bytes(M: int, N: int, K: int) -> int:
    return int(load().mq_linear_workspace_size(M, N, K))


def linear(X, pw: PackedWeight, out=None, workspace=None, stream=None):
    """The whole hot path from fp16 X [M, K]: quantisation and the fused GEMM
    (one kernel at decode sizes), Y fp16 [M, N]."""
    torch = _torch()
    _need(X, torch.float16, "X", 2)
    M, K = X.shape
    if K != pw.K:
        raise ValueError("X does not match the weight")
    Y = out if out is not None else torch.empty((M, pw.N), dtype=torch.float16, device=X.device)
    if out is not None:
        _need_out(Y, (M, pw.N), torch.float16, "out")
    rp, kb, rq, sr = _res_ptrs(pw)
    lib = load()
    ws = lib.mq_linear_workspace_size(M, pw.N, pw.K)
    wbuf = _scratch(ws, X.device, stream, workspace)
    _check("mq_linear", lib.mq_linear(
        M, pw.N, pw.K, _ptr(X), X.stride(0), _ptr(pw.Wq), _ptr(pw.s_w), rp, kb, pw.nnzb, rq, sr,
        _ptr(Y), Y.stride(0), _ptr(wbuf), ws, _stream(stream)))
    return Y


# ------------------------------------------------------ layout conversion --
def repack_weights(Wq_c, s_w_c, rowptr, kb, Rq_c, s_r, n_invalid=None, stream=None) -> PackedWeight:
    """Canonical int4 weights (two's-complement nibbles, even k low; Wq_c
    uint8 [N, K/2], s_w_c fp16 [N, K/128], Rq_c uint8 [nnzb, 128, 64]) ->
    a PackedWeight in the library layout.  ``n_invalid``: optional int32 [1]
    device counter that receives the number of -8 nibbles (stored as -7)."""
    torch = _torch()
    _need(Wq_c, torch.uint8, "Wq_c", 2)
    _need(s_w_c, torch.float16, "s_w_c", 2)
    N, K = Wq_c.shape[0], Wq_c.shape[1] * 2
    nnzb = int(kb.numel())
    Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=Wq_c.device)
    s_w = torch.empty((N, K // BLOCK), dtype=torch.float16, device=Wq_c.device)
    Rq = torch.empty((max(nnzb, 1), BLOCK, BLOCK // 2), dtype=torch.uint8, device=Wq_c.device)
    if nnzb:
        _need(Rq_c, torch.uint8, "Rq_c", 3)
    if n_invalid is not None:
        _need(n_invalid, torch.int32, "n_invalid", 1)
    _check("mq_repack_weights", load().mq_repack_weights(
        N, K, _ptr(Wq_c), _ptr(s_w_c), nnzb, _ptr(Rq_c) if nnzb else None, _ptr(Wq), _ptr(s_w),
        _ptr(Rq) if nnzb else None, _ptr(n_invalid), _stream(stream)))
    return PackedWeight(N, K, Wq, s_w, rowptr, kb, Rq[:nnzb], s_r)


def unpack_weights(pw: PackedWeight, stream=None):
    """Library layout -> canonical (Wq_c [N, K/2], s_w_c [N, K/128], Rq_c [nnzb, 128, 64])."""
    torch = _torch()
    dev = pw.Wq.device
    Wq_c = torch.empty((pw.N, pw.K // 2), dtype=torch.uint8, device=dev)
    s_w_c = torch.empty((pw.N, pw.K // BLOCK), dtype=torch.float16, device=dev)
    Rq_c = torch.empty((max(pw.nnzb, 1), BLOCK, BLOCK // 2), dtype=torch.uint8, device=dev)
    _check("mq_unpack_weights", load().mq_unpack_weights(
        pw.N, pw.K, _ptr(pw.Wq), _ptr(pw.s_w), pw.nnzb, _ptr(pw.Rq) if pw.nnzb else None,
        _ptr(Wq_c), _ptr(s_w_c), _ptr(Rq_c) if pw.nnzb else None, _stream(stream)))
    return Wq_c, s_w_c, Rq_c[:pw.nnzb]


def repack_act(Xq_c, n_invalid=None, stream=None):
    """Canonical int4 activation rows uint8 [M, K/2] -> library operand layout [M, 3K/4]."""
    torch = _torch()
    _need(Xq_c, torch.uint8, "Xq_c", 2)
    M, K = Xq_c.shape[0], Xq_c.shape[1] * 2
    Xq = torch.empty((M, act_bytes(K)), dtype=torch.uint8, device=Xq_c.device)
    if n_invalid is not None:
        _need(n_invalid, torch.int32, "n_invalid", 1)
    _check("mq_repack_act", load().mq_repack_act(M, K, _ptr(Xq_c), Xq_c.stride(0), _ptr(Xq),
                                                 _ptr(n_invalid), _stream(stream)))
    return Xq


def unpack_act(Xq, stream=None):
    """Library-layout activation codes uint8 [M, 3K/4] -> canonical rows [M, K/2]."""
    torch = _torch()
    _need(Xq, torch.uint8, "Xq", 2)
    M, K = Xq.shape[0], Xq.shape[1] * 4 // 3
    if Xq.shape[1] != act_bytes(K) or K % 128:
        raise ValueError("Xq is not in the operand layout of a K divisible by 128")
    Xq_c = torch.empty((M, K // 2), dtype=torch.uint8, device=Xq.device)
    _check("mq_unpack_act", load().mq_unpack_act(M, K, _ptr(Xq), _ptr(Xq_c), K // 2, _stream(stream)))
    return Xq_c


# --------------------------------------------------- weight preparation --
def quantize_weight(W, with_score: bool = True, stream=None):
    """fp32 W [N, K] -> (Wq uint8 [N, K/2], s_w fp16 [N, K/128], score fp64 [N/128, K/128])."""
    torch = _torch()
    _need(W, torch.float32, "W", 2)
    N, K = W.shape
    Wq = torch.empty((N, K // 2), dtype=torch.uint8, device=W.device)
    s_w = torch.empty((N, K // BLOCK), dtype=torch.float16, device=W.device)
    score = torch.empty((N // BLOCK, K // BLOCK), dtype=torch.float64, device=W.device) if with_score else None
    _check("mq_quantize_weight", load().mq_quantize_weight(
        _ptr(W), N, K, W.stride(0), _ptr(Wq), _ptr(s_w), _ptr(score), _stream(stream)))
    return Wq, s_w, score


def hessian_diag(X, stream=None):
    torch = _torch()
    _need(X, torch.float16, "X", 2)
    T, K = X.shape
    h = torch.empty((K,), dtype=torch.float64, device=X.device)
    _check("mq_hessian_diag", load().mq_hessian_diag(_ptr(X), T, K, X.stride(0), _ptr(h),
                                                     _stream(stream)))
    return h


def block_scores_dhessian(W, Wq, s_w, h, stream=None):
    torch = _torch()
    _need(W, torch.float32, "W", 2)
    N, K = W.shape
    score = torch.empty((N // BLOCK, K // BLOCK), dtype=torch.float64, device=W.device)
    _check("mq_block_scores_dhessian", load().mq_block_scores_dhessian(
        _ptr(W), N, K, W.stride(0), _ptr(Wq), _ptr(s_w), _ptr(h), _ptr(score), _stream(stream)))
    return score


def select_blocks(score, nnzb: int, stream=None):
    """Top-nnzb blocks of fp64 score [NB, KB] -> (rowptr int32 [NB+1], kb int32 [nnzb])."""
    torch = _torch()
    _need(score, torch.float64, "score", 2)
    NB, KB = score.shape
    rowptr = torch.empty((NB + 1,), dtype=torch.int32, device=score.device)
    kb = torch.empty((max(nnzb, 1),), dtype=torch.int32, device=score.device)
    _check("mq_select_blocks", load().mq_select_blocks(_ptr(score), NB, KB, nnzb, _ptr(rowptr),
                                                       _ptr(kb), _stream(stream)))
    return rowptr, kb[:nnzb]


def quantize_residual(W, Wq, s_w, rowptr, kb, stream=None):
    torch = _torch()
    _need(W, torch.float32, "W", 2)
    N, K = W.shape
    nnzb = int(kb.numel())
    Rq = torch.empty((max(nnzb, 1), BLOCK, BLOCK // 2), dtype=torch.uint8, device=W.device)
    s_r = torch.empty((max(nnzb, 1), BLOCK), dtype=torch.float16, device=W.device)
    _check("mq_quantize_residual", load().mq_quantize_residual(
        _ptr(W), N, K, W.stride(0), _ptr(Wq), _ptr(s_w), _ptr(rowptr),
        _ptr(kb) if nnzb else None, nnzb, _ptr(Rq), _ptr(s_r), _stream(stream)))
    return Rq[:nnzb], s_r[:nnzb]


def prepare_weight(W, nnzb: int, criterion: str = "frob", X_calib=None, stream=None) -> PackedWeight:
    """Offline MosaicQuant packing of fp32 W [N, K] on the GPU (Alg. 1):
    base INT4, block scores, top-nnzb selection, residual INT4."""
    Wq, s_w, score = quantize_weight(W, with_score=(criterion == "frob"), stream=stream)
    if criterion == "dhessian":
        if X_calib is None:
            raise ValueError("dhessian selection needs calibration activations")
        score = block_scores_dhessian(W, Wq, s_w, hessian_diag(X_calib, stream), stream)
    elif criterion != "frob":
        raise ValueError(criterion)
    rowptr, kb = select_blocks(score, nnzb, stream)
    Rq, s_r = quantize_residual(W, Wq, s_w, rowptr, kb, stream)
    N, K = W.shape
    return PackedWeight(N, K, Wq, s_w, rowptr, kb, Rq, s_r, score)
