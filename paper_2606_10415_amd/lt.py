"""ctypes binding of liblt.so (the gfx950 HIP kernels behind the C ABI of include/lt.h).

Argument marshalling only: every function has the name and argument order of
its C counterpart, accepts device tensors (``torch.Tensor`` on a ROCm device)
or raw integer device pointers, passes torch's current stream unless a stream
is given, and raises ``LtError`` when the library returns a non-LT_OK status.
There is no fallback: if liblt.so is missing, importing this module fails.
"""

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblt.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "lt.h")

LT_OK = 0
LT_ERR_INVALID_ARG = 1
LT_ERR_UNSUPPORTED = 2
LT_ERR_WORKSPACE = 3
LT_ERR_HIP = 4


class LtError(RuntimeError):
    def __init__(self, status, func, detail):
        self.status = status
        super().__init__(f"{func}: {status_string(status)}: {detail}")


if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_10415_amd.build` "
                      "(the HIP library is required, there is no fallback path)")

# liblt.so needs libamdhip64.so.7.  The PyTorch wheel bundles its own copy of
# the HIP runtime; if liblt were loaded first, the system copy would be mapped
# and torch would later map a second runtime, so device pointers from torch
# would be foreign to liblt's runtime.  Loading torch first makes the dynamic
# linker reuse torch's runtime for liblt (same soname).
try:
    import torch  # noqa: F401
except ImportError:   # plain C-ABI use without PyTorch: the system runtime is the only one
    torch = None

_lib = ctypes.CDLL(LIB_PATH)


def _hip_runtimes():
    try:
        with open("/proc/self/maps") as f:
            return sorted({ln.split()[-1] for ln in f if "libamdhip64" in ln})
    except OSError:
        return []


if len(_hip_runtimes()) > 1:
    raise ImportError("two HIP runtimes are mapped in this process: " + ", ".join(_hip_runtimes()) +
                      "; import torch before anything that loads /opt/rocm's libamdhip64")

_i64 = ctypes.c_int64
_int = ctypes.c_int
_f32 = ctypes.c_float
_vp = ctypes.c_void_p
_sz = ctypes.c_size_t

_lib.lt_status_string.restype = ctypes.c_char_p
_lib.lt_status_string.argtypes = [_int]
_lib.lt_last_error.restype = ctypes.c_char_p
_lib.lt_last_error.argtypes = []
_lib.lt_version.restype = _int
_lib.lt_version.argtypes = []
_lib.lt_gemm_f16.restype = _int
_lib.lt_gemm_f16.argtypes = [_int, _int, _i64, _i64, _i64, _f32, _vp, _i64, _vp, _i64, _f32, _vp, _i64, _vp]
_lib.lt_gemm_f16_res.restype = _int
_lib.lt_gemm_f16_res.argtypes = [_int, _int, _i64, _i64, _i64, _f32, _vp, _i64, _vp, _i64, _f32, _vp, _i64,
                                 _vp, _i64, _vp]
_lib.lt_attn_fwd.restype = _int
_lib.lt_attn_fwd.argtypes = [_vp, _vp, _vp, _i64, _i64, _vp, _i64, _vp, _int, _int, _int, _int, _int,
                             _f32, _int, _vp]
_lib.lt_attn_bwd_workspace_size.restype = _sz
_lib.lt_attn_bwd_workspace_size.argtypes = [_int, _int, _int, _int, _int, _int]
_lib.lt_attn_bwd.restype = _int
_lib.lt_attn_bwd.argtypes = [_vp, _vp, _vp, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _vp, _vp, _i64, _i64,
                             _vp, _sz, _int, _int, _int, _int, _int, _f32, _int, _vp]
_lib.lt_attn_p_size.restype = _sz
_lib.lt_attn_p_size.argtypes = [_int, _int, _int, _int]
_lib.lt_attn_fwd_p.restype = _int
_lib.lt_attn_fwd_p.argtypes = [_vp, _vp, _vp, _i64, _i64, _vp, _i64, _vp, _vp, _sz, _int, _int, _int,
                               _int, _int, _f32, _int, _vp]
_lib.lt_attn_bwd_p_workspace_size.restype = _sz
_lib.lt_attn_bwd_p_workspace_size.argtypes = [_int, _int, _int, _int, _int]
_lib.lt_attn_bwd_p.restype = _int
_lib.lt_attn_bwd_p.argtypes = [_vp, _vp, _vp, _i64, _i64, _vp, _vp, _i64, _vp, _vp, _sz, _vp, _vp, _vp,
                               _i64, _i64, _vp, _sz, _int, _int, _int, _int, _int, _f32, _int, _vp]
_lib.lt_swiglu_fwd.restype = _int
_lib.lt_swiglu_fwd.argtypes = [_vp, _vp, _i64, _i64, _vp]
_lib.lt_swiglu_bwd.restype = _int
_lib.lt_swiglu_bwd.argtypes = [_vp, _vp, _vp, _i64, _i64, _vp]
_lib.lt_gemm_f16_bias.restype = _int
_lib.lt_gemm_f16_bias.argtypes = [_int, _int, _i64, _i64, _i64, ctypes.c_float, _vp, _i64, _vp, _i64,
                                  ctypes.c_float, _vp, _i64, _vp, _vp, _i64, _vp]
_lib.lt_gemm_f16_workspace_size.restype = _sz
_lib.lt_gemm_f16_workspace_size.argtypes = [_int, _int, _i64, _i64, _i64]
_lib.lt_gemm_f16_ws.restype = _int
_lib.lt_gemm_f16_ws.argtypes = [_int, _int, _i64, _i64, _i64, ctypes.c_float, _vp, _i64, _vp, _i64,
                                ctypes.c_float, _vp, _i64, _vp, _vp, _i64, _vp, _sz, _vp]
_lib.lt_gemm_f16_noalloc.restype = _int
_lib.lt_gemm_f16_noalloc.argtypes = [_int, _int, _i64, _i64, _i64, ctypes.c_float, _vp, _i64, _vp,
                                     _i64, ctypes.c_float, _vp, _i64, _vp, _vp, _i64, _vp]
LT_GEMM_NOALLOC_SCRATCH_BYTES = 64 << 20
_lib.lt_bias_grad_workspace_size.restype = ctypes.c_size_t
_lib.lt_bias_grad_workspace_size.argtypes = [_i64, _i64]
_lib.lt_bias_grad_f16.restype = _int
_lib.lt_bias_grad_f16.argtypes = [_vp, _i64, _i64, _i64, _vp, _vp, ctypes.c_size_t, _vp]
_lib.lt_gemm_gu_swiglu_f16.restype = _int
_lib.lt_gemm_gu_swiglu_f16.argtypes = [_vp, _i64, _vp, _i64, _vp, _i64, _vp, _i64, _i64, _i64, _i64, _vp]
_lib.lt_gemm_swiglu_bwd_f16.restype = _int
_lib.lt_gemm_swiglu_bwd_f16.argtypes = [_vp, _i64, _vp, _i64, _vp, _i64, _vp, _i64, _i64, _i64, _i64,
                                        _vp]
_lib.lt_rmsnorm_fwd.restype = _int
_lib.lt_rmsnorm_fwd.argtypes = [_vp, _i64, _vp, _vp, _i64, _vp, _i64, _i64, _f32, _vp]
_lib.lt_rmsnorm_bwd_workspace_size.restype = _sz
_lib.lt_rmsnorm_bwd_workspace_size.argtypes = [_i64, _i64]
_lib.lt_rmsnorm_bwd.restype = _int
_lib.lt_rmsnorm_bwd.argtypes = [_vp, _i64, _vp, _i64, _vp, _vp, _vp, _i64, _vp, _i64, _vp, _vp, _sz,
                                _i64, _i64, _vp]
_lib.lt_rope_table.restype = _int
_lib.lt_rope_table.argtypes = [_vp, _int, _int, ctypes.c_double, _vp]
_lib.lt_rope_f16.restype = _int
_lib.lt_rope_f16.argtypes = [_vp, _i64, _int, _int, _int, _int, _vp, _int, _vp]


def status_string(status):
    return _lib.lt_status_string(int(status)).decode()


def last_error():
    return _lib.lt_last_error().decode()


def lt_version():
    return _lib.lt_version()


def _ptr(x):
    """Device address of a tensor (must live on a GPU) or a raw integer pointer / None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not getattr(x, "is_cuda", False):
        raise TypeError("liblt takes device tensors (or raw device pointers), got a host tensor")
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status, func):
    if status != LT_OK:
        raise LtError(status, func, last_error())


def lt_gemm_f16(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, C, ldc, stream=None):
    _check(_lib.lt_gemm_f16(int(transA), int(transB), int(M), int(N), int(K), float(alpha), _ptr(A),
                            int(lda), _ptr(B), int(ldb), float(beta), _ptr(C), int(ldc),
                            _stream(stream)), "lt_gemm_f16")


def lt_gemm_f16_res(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, C, ldc, stream=None):
    _check(_lib.lt_gemm_f16_res(int(transA), int(transB), int(M), int(N), int(K), float(alpha), _ptr(A),
                                int(lda), _ptr(B), int(ldb), float(beta), _ptr(R), int(ldr), _ptr(C),
                                int(ldc), _stream(stream)), "lt_gemm_f16_res")


def lt_attn_fwd(Q, K, V, q_row_stride, kv_row_stride, O, o_row_stride, LSE, B, S, Hq, Hkv, D, scale,
                causal, stream=None):
    _check(_lib.lt_attn_fwd(_ptr(Q), _ptr(K), _ptr(V), int(q_row_stride), int(kv_row_stride), _ptr(O),
                            int(o_row_stride), _ptr(LSE), int(B), int(S), int(Hq), int(Hkv), int(D),
                            float(scale), int(causal), _stream(stream)), "lt_attn_fwd")


def lt_attn_bwd_workspace_size(B, S, Hq, Hkv, D, causal):
    return int(_lib.lt_attn_bwd_workspace_size(int(B), int(S), int(Hq), int(Hkv), int(D),
                                               int(causal)))


def lt_attn_bwd(Q, K, V, q_row_stride, kv_row_stride, O, dO, o_row_stride, LSE, dQ, dK, dV,
                dq_row_stride, dkv_row_stride, workspace, ws_bytes, B, S, Hq, Hkv, D, scale, causal,
                stream=None):
    _check(_lib.lt_attn_bwd(_ptr(Q), _ptr(K), _ptr(V), int(q_row_stride), int(kv_row_stride), _ptr(O),
                            _ptr(dO), int(o_row_stride), _ptr(LSE), _ptr(dQ), _ptr(dK), _ptr(dV),
                            int(dq_row_stride), int(dkv_row_stride), _ptr(workspace), int(ws_bytes),
                            int(B), int(S), int(Hq), int(Hkv), int(D), float(scale), int(causal),
                            _stream(stream)), "lt_attn_bwd")


def lt_attn_p_size(B, S, Hq, causal):
    return int(_lib.lt_attn_p_size(int(B), int(S), int(Hq), int(causal)))


def lt_attn_fwd_p(Q, K, V, q_row_stride, kv_row_stride, O, o_row_stride, LSE, P, p_bytes, B, S, Hq,
                  Hkv, D, scale, causal, stream=None):
    _check(_lib.lt_attn_fwd_p(_ptr(Q), _ptr(K), _ptr(V), int(q_row_stride), int(kv_row_stride),
                              _ptr(O), int(o_row_stride), _ptr(LSE), _ptr(P), int(p_bytes), int(B),
                              int(S), int(Hq), int(Hkv), int(D), float(scale), int(causal),
                              _stream(stream)), "lt_attn_fwd_p")


def lt_attn_bwd_p_workspace_size(B, S, Hq, Hkv, D):
    return int(_lib.lt_attn_bwd_p_workspace_size(int(B), int(S), int(Hq), int(Hkv), int(D)))


def lt_attn_bwd_p(Q, K, V, q_row_stride, kv_row_stride, O, dO, o_row_stride, LSE, P, p_bytes, dQ, dK,
                  dV, dq_row_stride, dkv_row_stride, workspace, ws_bytes, B, S, Hq, Hkv, D, scale,
                  causal, stream=None):
    _check(_lib.lt_attn_bwd_p(_ptr(Q), _ptr(K), _ptr(V), int(q_row_stride), int(kv_row_stride),
                              _ptr(O), _ptr(dO), int(o_row_stride), _ptr(LSE), _ptr(P), int(p_bytes),
                              _ptr(dQ), _ptr(dK), _ptr(dV), int(dq_row_stride),
                              int(dkv_row_stride), _ptr(workspace), int(ws_bytes), int(B), int(S),
                              int(Hq), int(Hkv), int(D), float(scale), int(causal),
                              _stream(stream)), "lt_attn_bwd_p")


def lt_swiglu_fwd(GU, A, T, F, stream=None):
    _check(_lib.lt_swiglu_fwd(_ptr(GU), _ptr(A), int(T), int(F), _stream(stream)), "lt_swiglu_fwd")


def lt_swiglu_bwd(dA, GU, dGU, T, F, stream=None):
    _check(_lib.lt_swiglu_bwd(_ptr(dA), _ptr(GU), _ptr(dGU), int(T), int(F), _stream(stream)),
           "lt_swiglu_bwd")


def lt_gemm_f16_bias(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                     stream=None):
    _check(_lib.lt_gemm_f16_bias(int(transA), int(transB), int(M), int(N), int(K), float(alpha),
                                 _ptr(A), int(lda), _ptr(B), int(ldb), float(beta), _ptr(R),
                                 int(ldr), _ptr(bias), _ptr(C), int(ldc), _stream(stream)),
           "lt_gemm_f16_bias")


def lt_gemm_f16_workspace_size(transA, transB, M, N, K):
    return int(_lib.lt_gemm_f16_workspace_size(int(transA), int(transB), int(M), int(N), int(K)))


def lt_gemm_f16_ws(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                   workspace, ws_bytes, stream=None):
    _check(_lib.lt_gemm_f16_ws(int(transA), int(transB), int(M), int(N), int(K), float(alpha),
                               _ptr(A), int(lda), _ptr(B), int(ldb), float(beta), _ptr(R), int(ldr),
                               _ptr(bias), _ptr(C), int(ldc), _ptr(workspace), int(ws_bytes),
                               _stream(stream)), "lt_gemm_f16_ws")


def lt_gemm_f16_noalloc(transA, transB, M, N, K, alpha, A, lda, B, ldb, beta, R, ldr, bias, C, ldc,
                        stream=None):
    _check(_lib.lt_gemm_f16_noalloc(int(transA), int(transB), int(M), int(N), int(K), float(alpha),
                                    _ptr(A), int(lda), _ptr(B), int(ldb), float(beta), _ptr(R),
                                    int(ldr), _ptr(bias), _ptr(C), int(ldc), _stream(stream)),
           "lt_gemm_f16_noalloc")


def lt_bias_grad_workspace_size(T, N):
    return int(_lib.lt_bias_grad_workspace_size(int(T), int(N)))


def lt_bias_grad_f16(dY, lddy, T, N, db, workspace, ws_bytes, stream=None):
    _check(_lib.lt_bias_grad_f16(_ptr(dY), int(lddy), int(T), int(N), _ptr(db), _ptr(workspace),
                                 int(ws_bytes), _stream(stream)), "lt_bias_grad_f16")


def lt_gemm_gu_swiglu_f16(X, ldx, Wgu, ldw, GU, ldgu, A, lda, T, H, F, stream=None):
    _check(_lib.lt_gemm_gu_swiglu_f16(_ptr(X), int(ldx), _ptr(Wgu), int(ldw), _ptr(GU), int(ldgu),
                                      _ptr(A), int(lda), int(T), int(H), int(F), _stream(stream)),
           "lt_gemm_gu_swiglu_f16")


def lt_gemm_swiglu_bwd_f16(dY, lddy, Wd, ldwd, GU, ldgu, dGU, lddgu, T, H, F, stream=None):
    _check(_lib.lt_gemm_swiglu_bwd_f16(_ptr(dY), int(lddy), _ptr(Wd), int(ldwd), _ptr(GU),
                                       int(ldgu), _ptr(dGU), int(lddgu), int(T), int(H), int(F),
                                       _stream(stream)), "lt_gemm_swiglu_bwd_f16")


def lt_rmsnorm_fwd(X, ldx, W, Y, ldy, RSTD, T, H, eps, stream=None):
    _check(_lib.lt_rmsnorm_fwd(_ptr(X), int(ldx), _ptr(W), _ptr(Y), int(ldy), _ptr(RSTD), int(T),
                               int(H), float(eps), _stream(stream)), "lt_rmsnorm_fwd")


def lt_rmsnorm_bwd_workspace_size(T, H):
    return int(_lib.lt_rmsnorm_bwd_workspace_size(int(T), int(H)))


def lt_rmsnorm_bwd(dY, lddy, X, ldx, W, RSTD, R, ldr, dX, lddx, dW, workspace, ws_bytes, T, H,
                   stream=None):
    _check(_lib.lt_rmsnorm_bwd(_ptr(dY), int(lddy), _ptr(X), int(ldx), _ptr(W), _ptr(RSTD),
                               _ptr(R), int(ldr), _ptr(dX), int(lddx), _ptr(dW), _ptr(workspace),
                               int(ws_bytes), int(T), int(H), _stream(stream)), "lt_rmsnorm_bwd")


def lt_rope_table(CS, S, D, base, stream=None):
    _check(_lib.lt_rope_table(_ptr(CS), int(S), int(D), float(base), _stream(stream)),
           "lt_rope_table")


def lt_rope_f16(X, row_stride, B, S, heads, D, CS, inverse, stream=None):
    _check(_lib.lt_rope_f16(_ptr(X), int(row_stride), int(B), int(S), int(heads), int(D), _ptr(CS),
                            int(inverse), _stream(stream)), "lt_rope_f16")


def declared_functions():
    """Names of the functions include/lt.h declares (used by the export test)."""
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lt_[a-z0-9_]+)\s*\(", text)))
