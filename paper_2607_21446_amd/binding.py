"""Thin Python binding of libkroquant.so (include/kroquant.h).

Argument marshalling only: every step of the quantizer runs in the HIP
kernels of the library.  torch supplies device memory and the current HIP
stream.  There is no fallback: if the library is missing the first call raises.
"""
from __future__ import annotations

import ctypes
import os
from functools import lru_cache

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkroquant.so")

STATUS = {
    0: "KQ_SUCCESS", 1: "KQ_ERROR_INVALID_VALUE", 2: "KQ_ERROR_NULL_POINTER", 3: "KQ_ERROR_MISALIGNED",
    4: "KQ_ERROR_UNSUPPORTED", 5: "KQ_ERROR_SINGULAR", 6: "KQ_ERROR_HIP",
}

EXPORTED = (
    "kq_quantize", "kq_quantize_exact", "kq_quantize_packed", "kq_pack_factors", "kq_quantize_lu",
    "kq_smoothquant_quantize", "kq_hadamard32_quantize", "kq_fwht_quantize", "kq_mxfp4_quantize", "kq_mxfp4_gemm",
    "kq_mxfp4_gemm_bf16",
    "kq_stream_floor", "kq_stream_probe", "kq_timestamp",
    "kq_e2m1_encode", "kq_weight_transform", "kq_factors_inverse_transpose", "kq_lu_to_factors",
    "kq_calib_workspace_size", "kq_calib_reference", "kq_calib_step", "kq_calibrate",
    "kq_calib_step_noalloc",
    "kq_status_string", "kq_last_error_detail", "kq_version",
)


class KQError(RuntimeError):
    def __init__(self, status: int, detail: str, call: str):
        self.status = status
        self.name = STATUS.get(status, f"status {status}")
        self.detail = detail
        super().__init__(f"{call}: {self.name}: {detail}")


@lru_cache(maxsize=1)
def lib() -> ctypes.CDLL:
    """Load libkroquant.so (built in-tree by __graft_entry__.build())."""
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"libkroquant.so not found at {_LIB_PATH}; build it first "
                          "(python -m paper_2607_21446_amd._build)")
    L = ctypes.CDLL(_LIB_PATH)
    P, I64, I, F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    L.kq_quantize.argtypes = [P, I64, I64, P, P, I, I, I64, P, P, P, P]
    L.kq_quantize_exact.argtypes = [P, I64, I64, P, P, I, I, I64, P, P, P, P]
    L.kq_quantize_packed.argtypes = [P, I64, I64, P, P, I, I, I64, P, P, P, P, P]
    L.kq_pack_factors.argtypes = [P, P, I, I, I64, P, P]
    L.kq_quantize_lu.argtypes = [P, I64, I64, P, I, I64, P, P, P, P, P]
    L.kq_smoothquant_quantize.argtypes = [P, I64, I64, P, P, P, P, P]
    L.kq_hadamard32_quantize.argtypes = [P, I64, I64, P, P, P, P]
    L.kq_fwht_quantize.argtypes = [P, I64, I64, P, P, P, P]
    L.kq_mxfp4_gemm.argtypes = [P, P, I64, P, P, I64, I64, P, I64, I, P]
    L.kq_mxfp4_gemm_bf16.argtypes = [P, P, I64, P, P, I64, I64, P, I64, P]
    L.kq_mxfp4_quantize.argtypes = [P, I64, I64, P, P, P]
    L.kq_stream_floor.argtypes = [P, I64, I64, P, P, P]
    L.kq_stream_probe.argtypes = [P, I64, I64, P, P, I, I, I64, P]
    L.kq_e2m1_encode.argtypes = [P, I64, I, P, P]
    L.kq_weight_transform.argtypes = [P, I64, I64, P, P, I, I, I64, P, P, P, P]
    L.kq_factors_inverse_transpose.argtypes = [P, P, I, I, I64, P, P]
    L.kq_lu_to_factors.argtypes = [P, I, I64, P, P]
    L.kq_calib_workspace_size.argtypes = [I64, I64, I64, I, I64, ctypes.POINTER(ctypes.c_size_t)]
    L.kq_calib_reference.argtypes = [P, I64, I64, P, I64, P, P]
    L.kq_calib_step.argtypes = [P, I64, I64, P, I64, P, P, I, I64, P, P, P, P, P, I, F, P, ctypes.c_size_t, P]
    L.kq_calibrate.argtypes = [P, I64, I64, P, I64, P, P, I, I64, I, F, P, P, ctypes.c_size_t, P]
    L.kq_calib_step_noalloc.argtypes = [P, I64, I64, P, I64, P, P, I, I64, P, P, P, P, P, I, F, P]
    L.kq_timestamp.argtypes = [P, P]
    for name in EXPORTED[:23]:
        getattr(L, name).restype = ctypes.c_int
    L.kq_status_string.argtypes = [I]
    L.kq_status_string.restype = ctypes.c_char_p
    L.kq_last_error_detail.argtypes = []
    L.kq_last_error_detail.restype = ctypes.c_char_p
    L.kq_version.argtypes = []
    L.kq_version.restype = ctypes.c_int
    return L


def _check(status: int, call: str):
    if status != 0:
        raise KQError(status, lib().kq_last_error_detail().decode(), call)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _need(t, dtype, name, device=True):
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if device and not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _size(t, numel, name, device=None):
    """A caller-supplied buffer must hold exactly the elements the call reads
    or writes (an undersized one would be accessed out of bounds) and sit on
    the device of the input."""
    if t.numel() != numel:
        raise ValueError(f"{name} holds {t.numel()} elements, the call needs {numel}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the input on {device}")


def _matrix(X, name="X"):
    if X.dim() != 2:
        raise ValueError(f"{name} must be a 2-D [rows, columns] tensor, got shape {tuple(X.shape)}")
    return X.shape


def _outputs(X, codes, scales, y, want_y):
    M, d = _matrix(X)
    if codes is None:
        codes = torch.empty((M, d // 2), dtype=torch.uint8, device=X.device)
    if scales is None:
        scales = torch.empty((M, d // 32), dtype=torch.uint8, device=X.device)
    if y is None and want_y:
        y = torch.empty((M, d), dtype=torch.float32, device=X.device)
    # on X's device (the public calls require X to be a device tensor)
    _need(codes, torch.uint8, "codes", device=False)
    _need(scales, torch.uint8, "scales", device=False)
    _size(codes, M * (d // 2), "codes", X.device)
    _size(scales, M * (d // 32), "scales", X.device)
    if y is not None:
        _need(y, torch.float32, "y", device=False)
        _size(y, M * d, "y", X.device)
    return codes, scales, y


def _pairs(A, B, device=None):
    """Factor pairs A [nfac, a, a], B [nfac, b, b]: returns (a, b, nfac)."""
    a, b = A.shape[-1], B.shape[-1]
    if A.dim() < 2 or A.shape[-2] != a or B.dim() < 2 or B.shape[-2] != b:
        raise ValueError(f"A and B must be [nfac, a, a] and [nfac, b, b], got {tuple(A.shape)}, {tuple(B.shape)}")
    nfac = A.numel() // (a * a)
    if B.numel() != nfac * b * b:
        raise ValueError(f"A holds {nfac} factors of {a}x{a}, B {B.numel() / (b * b):g} of {b}x{b}")
    if device is not None and (A.device != device or B.device != device):
        raise ValueError(f"A ({A.device}) and B ({B.device}) must be on the input's device {device}")
    return a, b, nfac


def _kron(fn, name, X, A, B, codes, scales, y, want_y, stream):
    _need(X, torch.bfloat16, "X")
    _need(A, torch.float32, "A")
    _need(B, torch.float32, "B")
    a, b, nfac = _pairs(A, B, X.device)
    codes, scales, y = _outputs(X, codes, scales, y, want_y)
    M, d = X.shape
    _check(fn(_ptr(X), M, d, _ptr(A), _ptr(B), a, b, nfac, _ptr(codes), _ptr(scales), _ptr(y),
              _stream(stream)), name)
    return codes, scales, y


def quantize(X, A, B, codes=None, scales=None, y=None, want_y=False, stream=None):
    """KroQuant quantizer kq_quantize (matrix-core path): X bf16 [M, d];
    A [nfac, a, a] and B [nfac, b, b] fp32 device tensors.
    Returns (codes, scales, y or None)."""
    return _kron(lib().kq_quantize, "kq_quantize", X, A, B, codes, scales, y, want_y, stream)


def quantize_exact(X, A, B, codes=None, scales=None, y=None, want_y=False, stream=None):
    """kq_quantize_exact: the same quantizer with the fixed-order fp32
    evaluation on the vector ALUs."""
    return _kron(lib().kq_quantize_exact, "kq_quantize_exact", X, A, B, codes, scales, y, want_y, stream)


PACK_BYTES_PER_FACTOR = 6160


def pack_factors(A, B, kpack=None, stream=None):
    """kq_pack_factors: materialised K = A (x) B terms for the matrix cores
    (offline, once per layer).  Returns a uint8 device tensor."""
    _need(A, torch.float32, "A")
    _need(B, torch.float32, "B")
    a, b, nfac = _pairs(A, B, A.device)
    if kpack is None:
        kpack = torch.empty(nfac * PACK_BYTES_PER_FACTOR, dtype=torch.uint8, device=A.device)
    _need(kpack, torch.uint8, "kpack")
    _size(kpack, nfac * PACK_BYTES_PER_FACTOR, "kpack", A.device)
    _check(lib().kq_pack_factors(_ptr(A), _ptr(B), a, b, nfac, _ptr(kpack), _stream(stream)), "kq_pack_factors")
    return kpack


def quantize_packed(X, A, B, kpack, codes=None, scales=None, y=None, want_y=False, stream=None):
    """kq_quantize_packed: kq_quantize with K read from kpack."""
    _need(X, torch.bfloat16, "X")
    _need(A, torch.float32, "A")
    _need(B, torch.float32, "B")
    _need(kpack, torch.uint8, "kpack")
    a, b, nfac = _pairs(A, B, X.device)
    _size(kpack, nfac * PACK_BYTES_PER_FACTOR, "kpack", X.device)
    codes, scales, y = _outputs(X, codes, scales, y, want_y)
    M, d = X.shape
    _check(lib().kq_quantize_packed(_ptr(X), M, d, _ptr(A), _ptr(B), a, b, nfac, _ptr(kpack), _ptr(codes),
                                    _ptr(scales), _ptr(y), _stream(stream)), "kq_quantize_packed")
    return codes, scales, y


def quantize_lu(X, lu, a=4, codes=None, scales=None, y=None, y16=None, want_y=False, want_y16=False,
                stream=None):
    """kq_quantize_lu: K2-form factors, lu fp32 [nfac, 5, 3] = (a_k, b_k, c_k)
    of G_1..G_5, decoded on chip; a = number of rows of A (1, 2, 4 or 8).
    Returns (codes, scales, y or None, y16 or None); y16 is bf16 [M, d]."""
    _need(X, torch.bfloat16, "X")
    _need(lu, torch.float32, "lu")
    if lu.numel() % 15 or lu.numel() == 0:
        raise ValueError("lu must hold 15 parameters per factor pair")
    nfac = lu.numel() // 15
    _size(lu, nfac * 15, "lu", X.device)
    codes, scales, y = _outputs(X, codes, scales, y, want_y)
    M, d = X.shape
    if y16 is None and want_y16:
        y16 = torch.empty((M, d), dtype=torch.bfloat16, device=X.device)
    if y16 is not None:
        _need(y16, torch.bfloat16, "y16")
        _size(y16, M * d, "y16", X.device)
    _check(lib().kq_quantize_lu(_ptr(X), M, d, _ptr(lu), a, nfac, _ptr(codes), _ptr(scales), _ptr(y), _ptr(y16),
                                _stream(stream)), "kq_quantize_lu")
    return codes, scales, y, y16


def smoothquant(X, mult, codes=None, scales=None, y=None, want_y=False, stream=None):
    """SmoothQuant comparator kq_smoothquant_quantize; mult fp32 [d] = 1/s."""
    _need(X, torch.bfloat16, "X")
    _need(mult, torch.float32, "mult")
    codes, scales, y = _outputs(X, codes, scales, y, want_y)
    M, d = X.shape
    _size(mult, d, "mult", X.device)
    _check(lib().kq_smoothquant_quantize(_ptr(X), M, d, _ptr(mult), _ptr(codes), _ptr(scales), _ptr(y),
                                         _stream(stream)), "kq_smoothquant_quantize")
    return codes, scales, y


def hadamard32(X, codes=None, scales=None, y=None, want_y=False, stream=None):
    """Hadamard-32 comparator kq_hadamard32_quantize."""
    _need(X, torch.bfloat16, "X")
    codes, scales, y = _outputs(X, codes, scales, y, want_y)
    M, d = X.shape
    _check(lib().kq_hadamard32_quantize(_ptr(X), M, d, _ptr(codes), _ptr(scales), _ptr(y), _stream(stream)),
           "kq_hadamard32_quantize")
    return codes, scales, y


def fwht(X, codes=None, scales=None, y=None, want_y=False, stream=None):
    """Full-row FWHT comparator kq_fwht_quantize (d a power of two)."""
    _need(X, torch.bfloat16, "X")
    codes, scales, y = _outputs(X, codes, scales, y, want_y)
    M, d = X.shape
    _check(lib().kq_fwht_quantize(_ptr(X), M, d, _ptr(codes), _ptr(scales), _ptr(y), _stream(stream)),
           "kq_fwht_quantize")
    return codes, scales, y


def mxfp4_gemm(a_codes, a_scales, b_codes, b_scales, C=None, accumulate=False, stream=None, out_dtype=None):
    """kq_mxfp4_gemm: C[M, N] (+)= deq(A) deq(B)^T for MXFP4 operands (codes
    uint8 [rows, K/2], scales uint8 [rows, K/32]).  Returns C (fp32; with
    out_dtype=torch.bfloat16 or a bf16 C, kq_mxfp4_gemm_bf16: the product
    rounded to bf16, no accumulate)."""
    for t, name in ((a_codes, "a_codes"), (a_scales, "a_scales"), (b_codes, "b_codes"), (b_scales, "b_scales")):
        _need(t, torch.uint8, name)
    _matrix(a_codes, "a_codes")
    _matrix(b_codes, "b_codes")
    M, N, K = a_codes.shape[0], b_codes.shape[0], 2 * a_codes.shape[1]
    if b_codes.shape[1] * 2 != K or a_scales.shape != (M, K // 32) or b_scales.shape != (N, K // 32):
        raise ValueError("operand shapes do not match")
    dev = a_codes.device
    if any(t.device != dev for t in (a_scales, b_codes, b_scales)):
        raise ValueError("all operands must be on one device")
    if C is None:
        C = torch.empty((M, N), dtype=out_dtype or torch.float32, device=dev)
    if tuple(C.shape) != (M, N) or C.device != dev:
        raise ValueError(f"C must be [{M}, {N}] on {dev}, got {tuple(C.shape)} on {C.device}")
    if C.dtype == torch.bfloat16:
        _need(C, torch.bfloat16, "C")
        if accumulate:
            raise ValueError("the bf16 output has no accumulate mode")
        _check(lib().kq_mxfp4_gemm_bf16(_ptr(a_codes), _ptr(a_scales), M, _ptr(b_codes), _ptr(b_scales), N, K, _ptr(C),
                                        C.stride(0), _stream(stream)), "kq_mxfp4_gemm_bf16")
        return C
    _need(C, torch.float32, "C")
    _check(lib().kq_mxfp4_gemm(_ptr(a_codes), _ptr(a_scales), M, _ptr(b_codes), _ptr(b_scales), N, K, _ptr(C),
                               C.stride(0), int(accumulate), _stream(stream)), "kq_mxfp4_gemm")
    return C


def mxfp4(X, codes=None, scales=None, stream=None):
    """Plain MXFP4 kq_mxfp4_quantize."""
    _need(X, torch.bfloat16, "X")
    codes, scales, _ = _outputs(X, codes, scales, None, False)
    M, d = X.shape
    _check(lib().kq_mxfp4_quantize(_ptr(X), M, d, _ptr(codes), _ptr(scales), _stream(stream)),
           "kq_mxfp4_quantize")
    return codes, scales


def stream_floor(X, out16=None, out1=None, stream=None):
    """kq_stream_floor: the quantizers' traffic with no arithmetic (a timing aid)."""
    _need(X, torch.bfloat16, "X")
    out16, out1, _ = _outputs(X, out16, out1, None, False)
    M, d = X.shape
    _check(lib().kq_stream_floor(_ptr(X), M, d, _ptr(out16), _ptr(out1), _stream(stream)), "kq_stream_floor")
    return out16, out1


def timestamp(dst, index=0, stream=None):
    """kq_timestamp: enqueue a store of the 100 MHz device real-time counter
    into dst[index] (dst a device int64 tensor; a timing aid)."""
    if not (isinstance(dst, torch.Tensor) and dst.is_cuda and dst.dtype == torch.int64 and dst.is_contiguous()):
        raise TypeError("timestamp: dst must be a contiguous device int64 tensor")
    if not 0 <= index < dst.numel():
        raise ValueError(f"timestamp: index {index} outside dst of {dst.numel()} entries")
    _check(lib().kq_timestamp(ctypes.c_void_p(dst.data_ptr() + 8 * int(index)), _stream(stream)), "kq_timestamp")


TIMESTAMP_HZ = 100_000_000  # rate of the counter kq_timestamp stores


def stream_probe(X, waves=1, units=1, groups=0, out16=None, out1=None, stream=None):
    """kq_stream_probe: kq_stream_floor's traffic in another launch shape (a timing aid)."""
    _need(X, torch.bfloat16, "X")
    out16, out1, _ = _outputs(X, out16, out1, None, False)
    M, d = X.shape
    _check(lib().kq_stream_probe(_ptr(X), M, d, _ptr(out16), _ptr(out1), int(waves), int(units), int(groups),
                                 _stream(stream)), "kq_stream_probe")
    return out16, out1


def e2m1_encode(v, s, codes=None, stream=None):
    """Element encode kq_e2m1_encode: v fp32 [n] -> codes uint8 [n/2]."""
    _need(v, torch.float32, "v")
    n = v.numel()
    if codes is None:
        codes = torch.empty(n // 2, dtype=torch.uint8, device=v.device)
    _need(codes, torch.uint8, "codes")
    _size(codes, n // 2, "codes", v.device)
    _check(lib().kq_e2m1_encode(_ptr(v), n, int(s), _ptr(codes), _stream(stream)), "kq_e2m1_encode")
    return codes


def weight_transform(W, A_host, B_host, W_out=None, codes=None, scales=None, quantize=True, stream=None):
    """Offline weight side kq_weight_transform: W bf16 [o, d] on the device;
    A_host, B_host CPU fp32 tensors (forward factors).  Synchronizes."""
    _need(W, torch.bfloat16, "W")
    A_host = A_host.detach().to("cpu", torch.float32).contiguous()
    B_host = B_host.detach().to("cpu", torch.float32).contiguous()
    a, b, nfac = _pairs(A_host, B_host)
    o, d = _matrix(W, "W")
    if W_out is None:
        W_out = torch.empty((o, d), dtype=torch.float32, device=W.device)
    _need(W_out, torch.float32, "W_out")
    _size(W_out, o * d, "W_out", W.device)
    if quantize:
        codes, scales, _ = _outputs(W, codes, scales, None, False)
    _check(lib().kq_weight_transform(_ptr(W), o, d, _ptr(A_host), _ptr(B_host), a, b, nfac, _ptr(W_out),
                                     _ptr(codes), _ptr(scales), _stream(stream)), "kq_weight_transform")
    return W_out, codes, scales


def factors_inverse_transpose(A, B):
    """Host helper kq_factors_inverse_transpose on CPU fp32 tensors."""
    A = A.detach().to("cpu", torch.float32).contiguous()
    B = B.detach().to("cpu", torch.float32).contiguous()
    a, b, nfac = _pairs(A, B)
    Ait, Bit = torch.empty_like(A), torch.empty_like(B)
    _check(lib().kq_factors_inverse_transpose(_ptr(A), _ptr(B), a, b, nfac, _ptr(Ait), _ptr(Bit)),
           "kq_factors_inverse_transpose")
    return Ait, Bit


def lu_to_factors(abc, a):
    """Host helper kq_lu_to_factors: abc CPU fp32 [nfac, 5, 3] -> (A, B)."""
    abc = abc.detach().to("cpu", torch.float32).contiguous()
    if abc.numel() % 15 or abc.numel() == 0:
        raise ValueError("abc must hold 15 parameters per factor pair")
    nfac = abc.numel() // 15
    b = 32 // a
    A = torch.empty((nfac, a, a), dtype=torch.float32)
    B = torch.empty((nfac, b, b), dtype=torch.float32)
    _check(lib().kq_lu_to_factors(_ptr(abc), int(a), nfac, _ptr(A), _ptr(B)), "kq_lu_to_factors")
    return A, B


def status_string(status: int) -> str:
    return lib().kq_status_string(int(status)).decode()


def version() -> int:
    return int(lib().kq_version())


# ------------------------------------------------------------ calibration

def hadamard_lu(nfac, device="cuda"):
    """LU parameters of the Hadamard initialisation (Sec. 3.2): a = b = 1/sqrt(2),
    c = 1 for every factor; fp32 [nfac, 5, 3] on ``device``."""
    lu = torch.empty((nfac, 5, 3), dtype=torch.float32)
    lu[..., 0] = 2.0 ** -0.5
    lu[..., 1] = 2.0 ** -0.5
    lu[..., 2] = 1.0
    return lu.to(device)


def calib_workspace(R, o, d, a=4, nfac=1, device="cuda"):
    """Device workspace of kq_calib_step / kq_calibrate for these sizes."""
    n = ctypes.c_size_t(0)
    _check(lib().kq_calib_workspace_size(R, o, d, a, nfac, ctypes.byref(n)), "kq_calib_workspace_size")
    return torch.empty(int(n.value), dtype=torch.uint8, device=device)


def calib_reference(X, W, Yneg=None, stream=None):
    """kq_calib_reference: Yneg = -(X W^T), fp32 [R, o]."""
    _need(X, torch.bfloat16, "X")
    _need(W, torch.bfloat16, "W")
    R, d = _matrix(X)
    o = _matrix(W, "W")[0]
    if W.shape[1] != d or W.device != X.device:
        raise ValueError("X and W must have the same number of columns and sit on one device")
    if Yneg is None:
        Yneg = torch.empty((R, o), dtype=torch.float32, device=X.device)
    _need(Yneg, torch.float32, "Yneg")
    _size(Yneg, R * o, "Yneg", X.device)
    _check(lib().kq_calib_reference(_ptr(X), R, d, _ptr(W), o, _ptr(Yneg), _stream(stream)), "kq_calib_reference")
    return Yneg


def _calib_shapes(X, W, Yneg, lu):
    R, d = _matrix(X)
    o = _matrix(W, "W")[0]
    if W.shape[1] != d or W.device != X.device:
        raise ValueError("X and W must have the same number of columns and sit on one device")
    _need(Yneg, torch.float32, "Yneg")
    _size(Yneg, R * o, "Yneg", X.device)
    if lu.numel() % 15 or lu.numel() == 0:
        raise ValueError("lu must hold 15 parameters per factor pair")
    _size(lu, lu.numel(), "lu", X.device)
    return R, d, o, lu.numel() // 15


def calib_step(X, W, Yneg, lu, lambdas, a=4, workspace=None, adam=None, grad=None, losses=None, stream=None):
    """kq_calib_step: losses (fp64 [4]: L_out, L_A, L_W, L) and gradient (fp32
    [nfac, 5, 3]) of the calibration objective at ``lu``; with
    ``adam = (m, v, t, lr)`` (t >= 1) also one Adam update of ``lu`` in place.
    ``lambdas``: device fp32 [2].  Returns (losses, grad)."""
    _need(X, torch.bfloat16, "X")
    _need(W, torch.bfloat16, "W")
    _need(Yneg, torch.float32, "Yneg")
    _need(lu, torch.float32, "lu")
    _need(lambdas, torch.float32, "lambdas")
    R, d, o, nfac = _calib_shapes(X, W, Yneg, lu)
    _size(lambdas, 2, "lambdas", X.device)
    if workspace is None:
        workspace = calib_workspace(R, o, d, a, nfac, X.device)
    _need(workspace, torch.uint8, "workspace")
    if grad is None:
        grad = torch.empty((nfac, 5, 3), dtype=torch.float32, device=X.device)
    if losses is None:
        losses = torch.empty(4, dtype=torch.float64, device=X.device)
    _need(grad, torch.float32, "grad")
    _size(grad, nfac * 15, "grad", X.device)
    _need(losses, torch.float64, "losses")
    _size(losses, 4, "losses", X.device)
    m = v = None
    t, lr = 0, 0.0
    if adam is not None:
        m, v, t, lr = adam
        for buf, name in ((m, "adam m"), (v, "adam v")):
            _need(buf, torch.float32, name)
            _size(buf, nfac * 15, name, X.device)
    _check(lib().kq_calib_step(_ptr(X), R, d, _ptr(W), o, _ptr(Yneg), _ptr(lu), a, nfac, _ptr(lambdas), _ptr(grad),
                               _ptr(losses), _ptr(m), _ptr(v), int(t), float(lr), _ptr(workspace),
                               workspace.numel(), _stream(stream)), "kq_calib_step")
    return losses, grad


CALIB_NOALLOC_MAX_BYTES = 64 << 20


def calib_step_noalloc(X, W, Yneg, lu, lambdas, a=4, adam=None, grad=None, losses=None, stream=None):
    """kq_calib_step_noalloc: kq_calib_step on the library's own per-GPU
    scratch (no workspace argument, no allocation inside the call; for sizes
    whose workspace fits CALIB_NOALLOC_MAX_BYTES).  ``grad`` and ``losses``
    are allocated here when not given (pass them to allocate nothing).
    Returns (losses, grad)."""
    _need(X, torch.bfloat16, "X")
    _need(W, torch.bfloat16, "W")
    _need(lu, torch.float32, "lu")
    _need(lambdas, torch.float32, "lambdas")
    R, d, o, nfac = _calib_shapes(X, W, Yneg, lu)
    _size(lambdas, 2, "lambdas", X.device)
    if grad is None:
        grad = torch.empty((nfac, 5, 3), dtype=torch.float32, device=X.device)
    if losses is None:
        losses = torch.empty(4, dtype=torch.float64, device=X.device)
    _need(grad, torch.float32, "grad")
    _size(grad, nfac * 15, "grad", X.device)
    _need(losses, torch.float64, "losses")
    _size(losses, 4, "losses", X.device)
    m = v = None
    t, lr = 0, 0.0
    if adam is not None:
        m, v, t, lr = adam
        for buf, name in ((m, "adam m"), (v, "adam v")):
            _need(buf, torch.float32, name)
            _size(buf, nfac * 15, name, X.device)
    _check(lib().kq_calib_step_noalloc(_ptr(X), R, d, _ptr(W), o, _ptr(Yneg), _ptr(lu), a, nfac, _ptr(lambdas),
                                       _ptr(grad), _ptr(losses), _ptr(m), _ptr(v), int(t), float(lr),
                                       _stream(stream)), "kq_calib_step_noalloc")
    return losses, grad


def calibrate(X, W, lu=None, a=4, per_block=True, steps=100, lr=1e-2, Yneg=None, workspace=None, stream=None):
    """kq_calibrate: the per-layer optimisation of Sec. 3.3 (automatic lambdas
    at the start, ``steps`` Adam steps of rate ``lr``), from the Hadamard
    initialisation unless ``lu`` is given (updated in place).  Returns (lu,
    losses fp64 [steps + 2, 4])."""
    _need(X, torch.bfloat16, "X")
    _need(W, torch.bfloat16, "W")
    R, d = _matrix(X)
    if lu is None:
        lu = hadamard_lu(d // 32 if per_block else 1, X.device)
    _need(lu, torch.float32, "lu")
    if Yneg is None:
        Yneg = calib_reference(X, W, stream=stream)
    R, d, o, nfac = _calib_shapes(X, W, Yneg, lu)
    if workspace is None:
        workspace = calib_workspace(R, o, d, a, nfac, X.device)
    _need(workspace, torch.uint8, "workspace")
    losses = torch.empty((steps + 2, 4), dtype=torch.float64, device=X.device)
    _check(lib().kq_calibrate(_ptr(X), R, d, _ptr(W), o, _ptr(Yneg), _ptr(lu), a, nfac, int(steps), float(lr),
                              _ptr(losses), _ptr(workspace), workspace.numel(), _stream(stream)), "kq_calibrate")
    return lu, losses
