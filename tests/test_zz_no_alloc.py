"""xgemm_run_noalloc: the allocation-free variant of xgemm_run (scratch in a
static per-GPU array).  Through the C ABI, against xgemm_run's output (the
same plan and kernels, so the same bits) and the oracle, on two calls in a
row, the second with a smaller input; the device's free memory does not
change across the calls."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import CODE, check_close, check_exact, to_device
from paper_2609_16389_amd import workloads as wl
from paper_2609_16389_amd import xgemm as xg

pytestmark = pytest.mark.gpu


def _plan_scratch(M, N, K, dtype):
    """Workspace bytes of xgemm_run's plan for these (aligned) arguments."""
    band = xg.xgemm_select_band(M, N, K, CODE[dtype], 256)
    return band, xg.xgemm_workspace_bytes(M, N, K, 256, band.body)


def _call(fn, h, M, N, K, dA, dB, C, dtype, s):
    rc = fn(h, M, N, K, dA.data_ptr(), dA.stride(0), dB.data_ptr(), dB.stride(0), C.data_ptr(), N, CODE[dtype], s)
    return rc


@pytest.mark.parametrize("cases", [
    # split-k plans (partials in the scratch array), the second smaller
    [(1024, 1024, 16384, "bf16", 301), (512, 512, 8192, "bf16", 302)],
    # operand copies (N or K odd: B, or both, copied into the scratch array)
    [(1000, 1001, 1024, "fp16", 303), (300, 203, 777, "fp16", 304)],
], ids=["split_k", "packed"])
def test_noalloc_matches_xgemm_run(cases):
    oracle.build(force=False)
    h = xg.xgemm_create()
    try:
        s = torch.cuda.current_stream().cuda_stream
        data = []
        for M, N, K, dtype, seed in cases:
            A, B = wl.make_inputs(M, N, K, dtype, "uniform", seed)
            C_ref, S = oracle.gemm(A, B, dtype)
            data.append((M, N, K, dtype, to_device(A, dtype), to_device(B, dtype), C_ref, S))
        # the scratch array is really used: split partials or copies
        for M, N, K, dtype, *_ in data:
            band, ws = _plan_scratch(M, N, K, dtype)
            assert 0 < ws <= xg.XGEMM_NOALLOC_SCRATCH_BYTES or (N % 8 or K % 8), (M, N, K, band, ws)
        outs = [torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda") for M, N, *_ in data]
        torch.cuda.synchronize()
        free0, _ = torch.cuda.mem_get_info()
        for (M, N, K, dtype, dA, dB, _, _), C in zip(data, outs):
            assert _call(xg.xgemm_run_noalloc, h, M, N, K, dA, dB, C, dtype, s) == xg.XGEMM_OK, \
                xg.xgemm_last_error(h)
            torch.cuda.synchronize()
        free1, _ = torch.cuda.mem_get_info()
        assert free1 == free0, "device free memory changed by %d bytes" % (free0 - free1)
        for (M, N, K, dtype, dA, dB, C_ref, S), C in zip(data, outs):
            ref = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
            assert _call(xg.xgemm_run, h, M, N, K, dA, dB, ref, dtype, s) == xg.XGEMM_OK
            torch.cuda.synchronize()
            got = C.cpu().numpy()
            check_exact(got, ref.cpu().numpy().astype(np.float64), "noalloc vs xgemm_run %dx%dx%d" % (M, N, K))
            check_close(got, C_ref, S, "noalloc vs oracle %dx%dx%d" % (M, N, K))
    finally:
        torch.cuda.synchronize()
        xg.xgemm_destroy(h)


def test_noalloc_rejects_calls_beyond_the_scratch():
    """A call whose plan needs more scratch than the static array holds
    fails with XGEMM_ERR_INVALID_ARG before anything is enqueued; the
    buffers are sized for the call, and C is left as it was."""
    M, N, K = 4096, 4097, 4096        # N odd: B copied, 4096 x 4104 x 2 bytes = 32 MiB
    M2, N2, K2 = 8192, 8193, 8192     # B copy 8192 x 8200 x 2 bytes = 128 MiB, above 64 MiB
    h = xg.xgemm_create()
    try:
        s = torch.cuda.current_stream().cuda_stream
        A = torch.zeros((M2, K2), dtype=torch.bfloat16, device="cuda")
        B = torch.zeros((K2, N2), dtype=torch.bfloat16, device="cuda")
        C = torch.full((M2, N2), 5.0, dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        rc = xg.xgemm_run_noalloc(h, M2, N2, K2, A.data_ptr(), K2, B.data_ptr(), N2, C.data_ptr(), N2,
                                  xg.XGEMM_BF16, s)
        assert rc == xg.XGEMM_ERR_INVALID_ARG
        assert "scratch" in xg.xgemm_last_error(h)
        torch.cuda.synchronize()
        assert torch.all(C == 5.0)
        # a call that fits still runs on the same handle (zeros in, zeros out)
        rc = xg.xgemm_run_noalloc(h, M, N, K, A.data_ptr(), K2, B.data_ptr(), N2, C.data_ptr(), N2,
                                  xg.XGEMM_BF16, s)
        assert rc == xg.XGEMM_OK, xg.xgemm_last_error(h)
        torch.cuda.synchronize()
        assert torch.all(C[:M, :N] == 0.0) and torch.all(C[:, N:] == 5.0) and torch.all(C[M:] == 5.0)
    finally:
        xg.xgemm_destroy(h)
