"""Shared fixtures and helpers of the GPU parity tests: device transfers,
the library's storage order applied to oracle-packed operands (a permutation
pinned by the oracle tests), random operands and the fp16 error measure."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle as layout    # the device group order, as a permutation of the oracle's row-major packing

B = 128
TOL = 2e-3
TIGHT = 1e-3


@pytest.fixture(autouse=True)
def _announce(request):
    sys.__stderr__.write(f"\n[gpu-case] {request.node.nodeid}\n")
    sys.__stderr__.flush()
    yield


@pytest.fixture(scope="module")
def tc():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


@pytest.fixture(scope="module")
def mq(tc):
    import paper_2606_15652_amd as m
    m.load()
    return m


def dev(tc, a):
    return tc.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    return t.cpu().numpy()


def half_bits(t):
    import torch
    return t.cpu().view(torch.int16).numpy().view(np.uint16)


def maxabsrel(Y, Y64):
    Yf = Y.float().cpu().numpy().astype(np.float64)
    den = np.abs(Y64).max()
    return float(np.abs(Yf - Y64).max() / den) if den > 0 else float(np.abs(Yf).max())


# ------------------------------------------------------------------ data ----
def random_csr(NB, KB, nnzb, rng):
    sel = np.zeros(NB * KB, bool)
    sel[rng.choice(NB * KB, size=nnzb, replace=False)] = True
    sel = sel.reshape(NB, KB)
    rowptr = np.zeros(NB + 1, np.int32)
    rowptr[1:] = np.cumsum(sel.sum(1))
    kb = np.concatenate([np.flatnonzero(r) for r in sel]).astype(np.int32) if nnzb else np.zeros(0, np.int32)
    return rowptr, kb, sel


def random_operands(M, N, K, nnzb, seed):
    """Uniform random packed operands: every byte pattern is valid (each 8-byte
    chunk decodes to 16 codes in [-7, 7], the sign-only pattern being 0)."""
    rng = np.random.default_rng(seed)
    NB, KB = N // B, K // B
    Xq = rng.integers(0, 256, (M, K // 2), dtype=np.uint8)
    s_x = rng.uniform(0.01, 2.0, M).astype(np.float16).view(np.uint16)
    Wq = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    s_w = rng.uniform(1e-3, 0.05, (N, KB)).astype(np.float16).view(np.uint16)
    rowptr, kb, sel = random_csr(NB, KB, nnzb, rng)
    Rq = rng.integers(0, 256, (nnzb, B, B // 2), dtype=np.uint8)
    s_r = rng.uniform(1e-4, 5e-3, (nnzb, B)).astype(np.float16).view(np.uint16)
    return Xq, s_x, Wq, s_w, rowptr, kb, sel, Rq, s_r


def orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r):
    return orc.PackedWeight(N, K, Wq, s_w, rowptr, kb, Rq, s_r, None, sel)


def dev_x(tc, Xq):
    """Row-major packed activations -> the library's operand layout on the GPU."""
    return dev(tc, layout.act6_from_packed(Xq, Xq.shape[1] * 2))


def gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r):
    import torch
    return mq.PackedWeight(N, K, dev(tc, layout.block_rows(Wq, K)),
                           dev(tc, layout.block_scales(s_w)).view(torch.float16),
                           dev(tc, rowptr), dev(tc, kb),
                           dev(tc, Rq), dev(tc, s_r).view(torch.float16))


