"""Python binding of libfp8train (include/fp8train.h).

Argument marshalling only: every step runs in the HIP library.  Arrays are
torch tensors on the GPU (uint8 for FP8 codes, uint16 for FP16 codes, float32
for IEEE inputs); work goes onto torch's current HIP stream unless a stream is
given.  A call that the library rejects raises Fp8tError.  There is no CPU
fallback: if the library is not built, every call raises.
"""
import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libfp8train.so")

OK, EINVAL, EWORKSPACE, EHIP = 0, -1, -2, -3
SRC_F32, SRC_FP16 = 0, 1
EXACT, FAST = 0, 1

_lib = None


class Fp8tError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn}: {status_string(status)} (status {status})")
        self.status = status


def lib():
    """The loaded library.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run `python -m paper_1812_08011_amd.build` "
                "or __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        i32, i64, u64, f32, vp, sz = (ctypes.c_int, ctypes.c_int64, ctypes.c_uint64,
                                      ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t)
        L.fp8_quantize.restype = i32
        L.fp8_quantize.argtypes = [vp, i32, f32, vp, i64, vp]
        L.fp16_quantize.restype = i32
        L.fp16_quantize.argtypes = [vp, vp, i64, vp]
        L.chunk_gemm.restype = i32
        L.chunk_gemm.argtypes = [i32, i32, i64, i64, i64, i64, vp, i64, vp, i64, vp, i64,
                                 i32, vp, sz, vp]
        L.chunk_gemm_noalloc.restype = i32
        L.chunk_gemm_noalloc.argtypes = [i32, i32, i64, i64, i64, i64, vp, i64, vp, i64, vp, i64,
                                         i32, vp]
        L.chunk_gemm_workspace_size.restype = sz
        L.chunk_gemm_workspace_size.argtypes = [i32, i32, i64, i64, i64, i64, i32]
        L.chunk_gemm_fp8.restype = i32
        L.chunk_gemm_fp8.argtypes = [i32, i32, i64, i64, i64, i64, vp, i64, vp, i64, vp, i64,
                                     vp, i64, f32, i32, vp, sz, vp]
        L.chunk_gemm_fp8_workspace_size.restype = sz
        L.chunk_gemm_fp8_workspace_size.argtypes = [i32, i32, i64, i64, i64, i64, i32]
        L.chunk_gemm_sr.restype = i32
        L.chunk_gemm_sr.argtypes = [i32, i32, i64, i64, i64, i64, vp, i64, vp, i64, vp, i64,
                                    u64, u64, vp, sz, vp]
        L.chunk_gemm_sr_workspace_size.restype = sz
        L.chunk_gemm_sr_workspace_size.argtypes = [i32, i32, i64, i64, i64, i64]
        L.chunk_gemm_p16.restype = i32
        L.chunk_gemm_p16.argtypes = [i32, i32, i64, i64, i64, i64, vp, i64, vp, i64, vp, i64,
                                     vp, sz, vp]
        L.chunk_gemm_p16_workspace_size.restype = sz
        L.chunk_gemm_p16_workspace_size.argtypes = [i32, i32, i64, i64, i64, i64]
        L.relu_codes.restype = i32
        L.relu_codes.argtypes = [vp, i32, vp, i64, vp]
        L.relu_backward_fp8.restype = i32
        L.relu_backward_fp8.argtypes = [vp, vp, vp, i64, f32, vp]
        L.mse_grad_fp16.restype = i32
        L.mse_grad_fp16.argtypes = [vp, vp, vp, i64, f32, vp]
        L.conv2d_fwd_fp8.restype = i32
        L.conv2d_fwd_fp8.argtypes = [vp, i64, i64, i64, i64, i64, i64, i64, i64, vp, i64, i64,
                                     vp, i64, vp, sz, vp]
        L.conv2d_wgrad_fp8.restype = i32
        L.conv2d_wgrad_fp8.argtypes = list(L.conv2d_fwd_fp8.argtypes)
        L.conv2d_workspace_size.restype = sz
        L.conv2d_workspace_size.argtypes = [i32, i64, i64, i64, i64, i64, i64, i64, i64, i64,
                                            i64]
        L.col2im_fp16.restype = i32
        L.col2im_fp16.argtypes = [vp, i64, i64, i64, i64, i64, i64, i64, i64, vp, vp]
        L.adam_update.restype = i32
        L.adam_update.argtypes = [vp, vp, vp, vp, vp, i64, f32, f32, f32, f32, f32, u64, u64,
                                  u64, vp]
        L.sr_weight_update.restype = i32
        L.sr_weight_update.argtypes = [vp, vp, vp, vp, i64, f32, f32, f32, u64, u64, vp]
        L.fp8t_status_string.restype = ctypes.c_char_p
        L.fp8t_status_string.argtypes = [i32]
        _lib = L
    return _lib


def status_string(status):
    return lib().fp8t_status_string(int(status)).decode()


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(fn, status):
    if status != OK:
        raise Fp8tError(fn, status)


def fp8_quantize(src, dst, scale=1.0, stream=None):
    """dst (uint8, FP8 codes) = Q8(src * scale); src float32 or uint16 FP16 codes."""
    import torch
    if src.dtype == torch.float32:
        fmt = SRC_F32
    elif src.dtype == torch.uint16:
        fmt = SRC_FP16
    else:
        raise TypeError("fp8_quantize: src must be float32 or uint16 (FP16 codes)")
    if dst.dtype != torch.uint8 or dst.numel() != src.numel():
        raise TypeError("fp8_quantize: dst must be uint8 with as many elements as src")
    if not (src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("fp8_quantize: tensors must be contiguous")
    _check("fp8_quantize", lib().fp8_quantize(_ptr(src), fmt, float(scale), _ptr(dst),
                                               src.numel(), _stream(stream)))
    return dst


def fp16_quantize(src, dst, stream=None):
    """dst (uint16, FP16 codes) = round-to-nearest-even of float32 src."""
    import torch
    if src.dtype != torch.float32 or dst.dtype != torch.uint16 or dst.numel() != src.numel():
        raise TypeError("fp16_quantize: float32 src, uint16 dst of the same size")
    if not (src.is_contiguous() and dst.is_contiguous()):
        raise ValueError("fp16_quantize: tensors must be contiguous")
    _check("fp16_quantize", lib().fp16_quantize(_ptr(src), _ptr(dst), src.numel(),
                                                 _stream(stream)))
    return dst


def chunk_gemm_workspace_size(trans_a, trans_b, M, N, K, CL, mode):
    return int(lib().chunk_gemm_workspace_size(int(trans_a), int(trans_b), int(M), int(N),
                                               int(K), int(CL), int(mode)))


def chunk_gemm(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, mode=EXACT,
               workspace=None, workspace_bytes=0, stream=None):
    """The C-ABI call with the same argument order; A, B, C, workspace are
    tensors (or raw device addresses)."""
    _check("chunk_gemm", lib().chunk_gemm(int(trans_a), int(trans_b), int(M), int(N), int(K),
                                          int(CL), _ptr(A), int(lda), _ptr(B), int(ldb),
                                          _ptr(C), int(ldc), int(mode), _ptr(workspace),
                                          int(workspace_bytes), _stream(stream)))
    return C


def chunk_gemm_noalloc(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, mode=EXACT,
                       stream=None):
    """The C-ABI call with the same argument order (no workspace: the
    library's static scratch holds shared tiles' chunk sums)."""
    _check("chunk_gemm_noalloc",
           lib().chunk_gemm_noalloc(int(trans_a), int(trans_b), int(M), int(N), int(K), int(CL),
                                    _ptr(A), int(lda), _ptr(B), int(ldb), _ptr(C), int(ldc),
                                    int(mode), _stream(stream)))
    return C


def chunk_gemm_fp8_workspace_size(trans_a, trans_b, M, N, K, CL, mode):
    return int(lib().chunk_gemm_fp8_workspace_size(int(trans_a), int(trans_b), int(M), int(N),
                                                   int(K), int(CL), int(mode)))


def chunk_gemm_fp8(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, C8, ldc8, scale=1.0,
                   mode=EXACT, workspace=None, workspace_bytes=0, stream=None):
    """The C-ABI call with the same argument order; C may be None (FP8 result
    only)."""
    _check("chunk_gemm_fp8",
           lib().chunk_gemm_fp8(int(trans_a), int(trans_b), int(M), int(N), int(K), int(CL),
                                _ptr(A), int(lda), _ptr(B), int(ldb), _ptr(C), int(ldc), _ptr(C8),
                                int(ldc8), float(scale), int(mode), _ptr(workspace),
                                int(workspace_bytes), _stream(stream)))
    return C8


def chunk_gemm_sr_workspace_size(trans_a, trans_b, M, N, K, CL):
    return int(lib().chunk_gemm_sr_workspace_size(int(trans_a), int(trans_b), int(M), int(N),
                                                  int(K), int(CL)))


def chunk_gemm_sr(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, seed, offset=0,
                  workspace=None, workspace_bytes=0, stream=None):
    """The C-ABI call with the same argument order (stochastic rounding after
    every FP16 addition)."""
    _check("chunk_gemm_sr",
           lib().chunk_gemm_sr(int(trans_a), int(trans_b), int(M), int(N), int(K), int(CL),
                               _ptr(A), int(lda), _ptr(B), int(ldb), _ptr(C), int(ldc),
                               int(seed), int(offset), _ptr(workspace), int(workspace_bytes),
                               _stream(stream)))
    return C


def sr_weight_update(w, g, v, w8, n, lr, momentum, weight_decay, seed, offset, stream=None):
    """The C-ABI call with the same argument order; w, g, v, w8 are tensors
    (v, w8 may be None)."""
    _check("sr_weight_update",
           lib().sr_weight_update(_ptr(w), _ptr(g), _ptr(v), _ptr(w8), int(n), float(lr),
                                  float(momentum), float(weight_decay), int(seed), int(offset),
                                  _stream(stream)))
    return w


def adam_update(w, g, m, v, w8, n, lr, beta1, beta2, eps, weight_decay, t, seed, offset,
                stream=None):
    """The C-ABI call with the same argument order; w8 may be None."""
    _check("adam_update",
           lib().adam_update(_ptr(w), _ptr(g), _ptr(m), _ptr(v), _ptr(w8), int(n), float(lr),
                             float(beta1), float(beta2), float(eps), float(weight_decay), int(t),
                             int(seed), int(offset), _stream(stream)))
    return w


def chunk_gemm_p16_workspace_size(trans_a, trans_b, M, N, K, CL):
    return int(lib().chunk_gemm_p16_workspace_size(int(trans_a), int(trans_b), int(M), int(N),
                                                   int(K), int(CL)))


def chunk_gemm_p16(trans_a, trans_b, M, N, K, CL, A, lda, B, ldb, C, ldc, workspace=None,
                   workspace_bytes=0, stream=None):
    """The C-ABI call with the same argument order (FP16-code operands)."""
    _check("chunk_gemm_p16",
           lib().chunk_gemm_p16(int(trans_a), int(trans_b), int(M), int(N), int(K), int(CL),
                                _ptr(A), int(lda), _ptr(B), int(ldb), _ptr(C), int(ldc),
                                _ptr(workspace), int(workspace_bytes), _stream(stream)))
    return C


def relu_codes(x, fmt, y, n, stream=None):
    """ReLU on FP8 (fmt 8) or FP16 (fmt 16) codes; y may be x."""
    _check("relu_codes", lib().relu_codes(_ptr(x), int(fmt), _ptr(y), int(n), _stream(stream)))
    return y


def relu_backward_fp8(d, z, e, n, scale=1.0, stream=None):
    _check("relu_backward_fp8", lib().relu_backward_fp8(_ptr(d), _ptr(z), _ptr(e), int(n),
                                                        float(scale), _stream(stream)))
    return e


def mse_grad_fp16(y, t, e, n, scale, stream=None):
    _check("mse_grad_fp16", lib().mse_grad_fp16(_ptr(y), _ptr(t), _ptr(e), int(n), float(scale),
                                                _stream(stream)))
    return e


def conv2d_workspace_size(wgrad, N, H, W, C, KH, KW, pad, stride, Cout, CL):
    return int(lib().conv2d_workspace_size(int(wgrad), int(N), int(H), int(W), int(C), int(KH),
                                           int(KW), int(pad), int(stride), int(Cout), int(CL)))


def conv2d_fwd_fp8(X, N, H, W, C, KH, KW, pad, stride, Wt, Cout, CL, Y, ldy, workspace=None,
                   workspace_bytes=0, stream=None):
    _check("conv2d_fwd_fp8",
           lib().conv2d_fwd_fp8(_ptr(X), int(N), int(H), int(W), int(C), int(KH), int(KW),
                                int(pad), int(stride), _ptr(Wt), int(Cout), int(CL), _ptr(Y),
                                int(ldy), _ptr(workspace), int(workspace_bytes), _stream(stream)))
    return Y


def conv2d_wgrad_fp8(X, N, H, W, C, KH, KW, pad, stride, dY, Cout, CL, dW, lddw, workspace=None,
                     workspace_bytes=0, stream=None):
    _check("conv2d_wgrad_fp8",
           lib().conv2d_wgrad_fp8(_ptr(X), int(N), int(H), int(W), int(C), int(KH), int(KW),
                                  int(pad), int(stride), _ptr(dY), int(Cout), int(CL), _ptr(dW),
                                  int(lddw), _ptr(workspace), int(workspace_bytes),
                                  _stream(stream)))
    return dW


def col2im_fp16(cols, N, H, W, C, KH, KW, pad, stride, dX, stream=None):
    _check("col2im_fp16",
           lib().col2im_fp16(_ptr(cols), int(N), int(H), int(W), int(C), int(KH), int(KW),
                             int(pad), int(stride), _ptr(dX), _stream(stream)))
    return dX
