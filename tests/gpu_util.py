"""Helpers for the GPU parity tests: move stored bit patterns to the device,
call the library through its C ABI, and apply the acceptance bound
|C_gpu - C_ref| <= 1e-4 * sum_k |a_ik * b_kj| elementwise."""
import numpy as np
import torch

from paper_2609_16389_amd import xgemm as xg

REL_TOL = 1e-4

TORCH_DT = {"bf16": torch.bfloat16, "fp16": torch.float16}
CODE = {"bf16": xg.XGEMM_BF16, "fp16": xg.XGEMM_FP16}


def to_device(bits: np.ndarray, dtype: str, ld: int | None = None, offset: int = 0,
              pad: int | None = None) -> torch.Tensor:
    """uint16 bit patterns (rows x cols) -> a device tensor view with row stride
    ``ld`` (>= cols; padding filled with ``pad``, by default a large value,
    that must never be read) starting ``offset`` elements into its
    allocation."""
    rows, cols = bits.shape
    ld = max(cols, 1) if ld is None else ld
    pad = (0x7BFF if dtype == "fp16" else 0x7F7F) if pad is None else pad
    buf = np.full(offset + rows * ld + 1, pad, dtype=np.uint16)
    if rows and cols:
        buf[offset:offset + rows * ld].reshape(rows, ld)[:, :cols] = bits
    t = torch.from_numpy(buf.view(np.int16)).to("cuda").view(TORCH_DT[dtype])
    return t.as_strided((rows, cols), (ld, 1), offset)


def run_gpu(A_bits, B_bits, dtype, config=None, out=None, lda=None, ldb=None, offset=0, pad=None):
    """C = A*B on the GPU through xgemm_run / xgemm_run_config; returns fp32 numpy."""
    A = to_device(A_bits, dtype, lda, offset, pad)
    B = to_device(B_bits, dtype, ldb, offset, pad)
    C = xg.gemm(A, B, out=out, config=config)
    torch.cuda.synchronize()
    return C.cpu().numpy()


def empty_out(M, N, ldc=None, offset=0, fill=float("nan")):
    """A float32 output view (M x N, row stride ldc) pre-filled with ``fill``."""
    ldc = max(N, 1) if ldc is None else ldc
    t = torch.full((offset + M * ldc + 1,), fill, dtype=torch.float32, device="cuda")
    return t.as_strided((M, N), (ldc, 1), offset)


def check_close(C_gpu: np.ndarray, C_ref: np.ndarray, S: np.ndarray, what: str = ""):
    C_gpu = np.asarray(C_gpu, dtype=np.float64)
    assert C_gpu.shape == C_ref.shape
    assert np.all(np.isfinite(C_gpu)), "%s: non-finite output" % what
    err = np.abs(C_gpu - C_ref)
    bad = err > REL_TOL * S
    if bad.any():
        i, j = np.argwhere(bad)[0]
        raise AssertionError("%s: %d elements out of tolerance; first at (%d, %d): gpu=%r ref=%r S=%r"
                             % (what, int(bad.sum()), i, j, C_gpu[i, j], C_ref[i, j], S[i, j]))


def check_exact(C_gpu: np.ndarray, C_ref: np.ndarray, what: str = ""):
    C_gpu = np.asarray(C_gpu, dtype=np.float64)
    bad = C_gpu != C_ref
    if bad.any():
        i, j = np.argwhere(bad)[0]
        raise AssertionError("%s: %d elements differ; first at (%d, %d): gpu=%r ref=%r"
                             % (what, int(bad.sum()), i, j, C_gpu[i, j], C_ref[i, j]))


def config(tile, split=1, group_m=4, stream_k=0):
    return xg.xgemm_config(tile=tile, split_k=split, group_m=group_m, stream_k=stream_k)
