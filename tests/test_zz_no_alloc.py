"""The scratch-free entry point mq_linear_noalloc, called through the C ABI:
bit-identical to mq_linear (same kernels, the workspace taken from the
library's device scratch array instead of the caller), on two calls in a row
with the second smaller, including shapes whose workspace holds split-K
partial sums; and a shape beyond the scratch array is refused without a
launch."""
from __future__ import annotations

import numpy as np
import pytest

import synth
from gpu_util import B, TIGHT, _announce, dev, gpu_pw, host, maxabsrel, mq, orc_pw, random_operands, tc  # noqa: F401

pytestmark = pytest.mark.gpu

SCRATCH_LIMIT = -6


def call_noalloc(lib, X, pw, Y):
    rp, kb, rq, sr = (pw.rowptr.data_ptr(), pw.kb.data_ptr(), pw.Rq.data_ptr(), pw.s_r.data_ptr()) \
        if pw.nnzb else (None, None, None, None)
    return lib.mq_linear_noalloc(X.shape[0], pw.N, pw.K, X.data_ptr(), X.stride(0), pw.Wq.data_ptr(),
                                 pw.s_w.data_ptr(), rp, kb, pw.nnzb, rq, sr, Y.data_ptr(), Y.stride(0), None)


# (M, N, K, nnzb): first a shape with split-K partials and quantised rows in
# the scratch, then a smaller one; a decode shape needing no scratch; the
# benched prefill shape
SEQUENCES = [[(300, 1024, 2048, 40), (70, 512, 1024, 9)],
             [(4096, 4096, 4096, 102), (256, 1024, 4096, 20)],
             [(1, 2048, 1024, 12), (40, 256, 2048, 5)]]


@pytest.mark.parametrize("seq", SEQUENCES, ids=["splitk_then_smaller", "prefill_then_smaller", "decode_then_small"])
def test_noalloc_matches_linear_two_calls(tc, mq, orc, seq):
    lib = mq.load()
    for M, N, K, nnzb in seq:
        assert lib.mq_linear_workspace_size(M, N, K) <= lib.mq_scratch_bytes()
        _, _, Wq, s_w, rowptr, kb, sel, Rq, s_r = random_operands(M, N, K, nnzb, seed=M + 3 * N + K)
        X = synth.gen_act(M, K, 900 + M)
        Xq_r, sx_r = orc.quantize_act(X)
        _, _, Y64 = orc.linear(Xq_r, sx_r, orc_pw(orc, N, K, Wq, s_w, rowptr, kb, sel, Rq, s_r))
        pw = gpu_pw(tc, mq, N, K, Wq, s_w, rowptr, kb, Rq, s_r)
        Xd = dev(tc, X)
        Y_ref = mq.linear(Xd, pw)
        Y = tc.full((M, N), 7, dtype=tc.float16, device="cuda")
        st = call_noalloc(lib, Xd, pw, Y)
        tc.cuda.synchronize()
        assert st == 0, lib.mq_status_string(st)
        assert np.array_equal(host(Y.view(tc.int16)), host(Y_ref.view(tc.int16))), (M, N, K)
        assert maxabsrel(Y, Y64) <= TIGHT


def test_noalloc_refuses_beyond_scratch(tc, mq):
    lib = mq.load()
    M, N, K = 65536, 256, 8192                       # quantised rows alone: 256 MiB
    assert lib.mq_linear_workspace_size(M, N, K) > lib.mq_scratch_bytes()
    X = tc.empty((1, 1), dtype=tc.float16, device="cuda")   # never read: refused before any launch
    st = lib.mq_linear_noalloc(M, N, K, X.data_ptr(), K, X.data_ptr(), X.data_ptr(), None, None, 0,
                               None, None, X.data_ptr(), N, None)
    assert st == SCRATCH_LIMIT
