"""ctypes binding of libunisvq (argument marshalling only).

Every function takes torch tensors that already live on the GPU, passes their
device pointers and the current HIP stream to the C ABI declared in
``include/unisvq.h``, and raises on a non-zero status.  All compute happens in
the library's HIP kernels; there is no host or PyTorch fallback.  If the
library has not been built the first call raises ``UniSVQLibraryMissing``.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libunisvq.so")

F16, BF16, F32 = 0, 1, 2
GROUP, DIM, ROW_BLOCK = 128, 4, 16

STATUS = {0: "UNISVQ_OK", -1: "UNISVQ_EINVAL", -2: "UNISVQ_ESHAPE", -3: "UNISVQ_EUNSUP",
          -4: "UNISVQ_EALIGN", -5: "UNISVQ_EHIP", -6: "UNISVQ_EWORKSPACE", -7: "UNISVQ_ESCRATCH"}

EXPORTS = ("unisvq_version", "unisvq_status_string", "unisvq_packed_bytes", "unisvq_pack",
           "unisvq_unpack", "unisvq_gemv", "unisvq_gemv_batched", "unisvq_gemm_workspace_bytes",
           "unisvq_gemm", "unisvq_codes_bytes", "unisvq_shared_affine_bytes", "unisvq_pack_shared",
           "unisvq_unpack_shared", "unisvq_gemv_shared", "unisvq_gemv_shared_batched", "unisvq_gemm_shared",
           "unisvq_gemm_fold_workspace_bytes", "unisvq_gemm_shared_fold",
           "unisvq_quantize", "unisvq_rht", "unisvq_var_codes_bytes", "unisvq_var_affine_bytes",
           "unisvq_var_pack", "unisvq_var_unpack", "unisvq_var_gemv", "unisvq_var_gemv_batched",
           "unisvq_var_gemm_workspace_bytes", "unisvq_var_gemm", "unisvq_ldlq_workspace_bytes", "unisvq_ldlq",
           "unisvq_ldl_workspace_bytes", "unisvq_ldl",
           "unisvq_gemv_rht_batched", "unisvq_read_sink_words", "unisvq_read_bytes", "unisvq_noalloc_scratch_bytes",
           "unisvq_gemm_noalloc", "unisvq_gemm_batched_workspace_bytes", "unisvq_gemm_batched")
# format variants: (bits, d) pairs served by the unisvq_var_* entry points
VARIANTS = ((3, 4), (2, 8), (3, 8))
MAX_BATCH = 8


class GemvProblem(ctypes.Structure):
    """Mirror of unisvq_gemv_problem."""
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("packed", ctypes.c_void_p),
                ("x", ctypes.c_void_p), ("y", ctypes.c_void_p)]


class GemvSharedProblem(ctypes.Structure):
    """Mirror of unisvq_gemv_shared_problem."""
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("affine_groups", ctypes.c_int64),
                ("packed_codes", ctypes.c_void_p), ("packed_affine", ctypes.c_void_p),
                ("x", ctypes.c_void_p), ("y", ctypes.c_void_p)]


class ByteRange(ctypes.Structure):
    """Mirror of unisvq_byte_range."""
    _fields_ = [("ptr", ctypes.c_void_p), ("bytes", ctypes.c_int64)]


class UniSVQLibraryMissing(RuntimeError):
    pass


class UniSVQError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} returned {STATUS.get(status, status)}: {_status_string(status)}")


_lib = None


def load():
    """Load libunisvq.so (once) and declare its C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise UniSVQLibraryMissing(
            f"{LIB_PATH} is missing: build it with `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(LIB_PATH)
    i64, p, i32, sz = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.unisvq_version.argtypes = []
    lib.unisvq_version.restype = i32
    lib.unisvq_status_string.argtypes = [i32]
    lib.unisvq_status_string.restype = ctypes.c_char_p
    lib.unisvq_packed_bytes.argtypes = [i64, i64]
    lib.unisvq_packed_bytes.restype = sz
    lib.unisvq_pack.argtypes = [i64, i64, p, p, p, p, p, p]
    lib.unisvq_pack.restype = i32
    lib.unisvq_unpack.argtypes = [i64, i64, p, p, p, p, p]
    lib.unisvq_unpack.restype = i32
    lib.unisvq_gemv.argtypes = [i64, i64, p, i64, p, i32, p, i32, p]
    lib.unisvq_gemv.restype = i32
    lib.unisvq_gemv_batched.argtypes = [ctypes.POINTER(GemvProblem), i32, i64, i32, i32, p]
    lib.unisvq_gemv_batched.restype = i32
    lib.unisvq_gemv_rht_batched.argtypes = [ctypes.POINTER(GemvProblem), i32, i64, i32, i32,
                                            ctypes.POINTER(ctypes.c_void_p), p]
    lib.unisvq_gemv_rht_batched.restype = i32
    lib.unisvq_gemm_workspace_bytes.argtypes = [i64, i64, i64, i32]
    lib.unisvq_gemm_workspace_bytes.restype = sz
    lib.unisvq_gemm.argtypes = [i64, i64, p, i64, p, i32, p, i32, p, sz, p]
    lib.unisvq_gemm.restype = i32
    lib.unisvq_codes_bytes.argtypes = [i64, i64]
    lib.unisvq_codes_bytes.restype = sz
    lib.unisvq_shared_affine_bytes.argtypes = [i64, i64]
    lib.unisvq_shared_affine_bytes.restype = sz
    lib.unisvq_pack_shared.argtypes = [i64, i64, i64, p, p, p, p, p, p, p]
    lib.unisvq_pack_shared.restype = i32
    lib.unisvq_unpack_shared.argtypes = [i64, i64, i64, p, p, p, p, p, p]
    lib.unisvq_unpack_shared.restype = i32
    lib.unisvq_gemv_shared.argtypes = [i64, i64, i64, p, p, i64, p, i32, p, i32, p]
    lib.unisvq_gemv_shared.restype = i32
    lib.unisvq_gemv_shared_batched.argtypes = [ctypes.POINTER(GemvSharedProblem), i32, i64, i32, i32, p]
    lib.unisvq_gemv_shared_batched.restype = i32
    lib.unisvq_gemm_shared.argtypes = [i64, i64, i64, p, p, i64, p, i32, p, i32, p, sz, p]
    lib.unisvq_gemm_shared.restype = i32
    lib.unisvq_gemm_shared_fold.argtypes = lib.unisvq_gemm_shared.argtypes
    lib.unisvq_gemm_shared_fold.restype = i32
    lib.unisvq_gemm_fold_workspace_bytes.argtypes = [i64, i64, i64]
    lib.unisvq_gemm_fold_workspace_bytes.restype = sz
    lib.unisvq_quantize.argtypes = [i64, i64, p, p, p, i64, p, p]
    lib.unisvq_quantize.restype = i32
    lib.unisvq_rht.argtypes = [i64, i64, p, i32, p, i32, p, i32, p]
    lib.unisvq_rht.restype = i32
    lib.unisvq_var_codes_bytes.argtypes = [i64, i64, i32, i32]
    lib.unisvq_var_codes_bytes.restype = sz
    lib.unisvq_var_affine_bytes.argtypes = [i64, i64, i32, i32]
    lib.unisvq_var_affine_bytes.restype = sz
    lib.unisvq_var_pack.argtypes = [i64, i64, i32, i32, i64, p, p, p, p, p, p, p]
    lib.unisvq_var_pack.restype = i32
    lib.unisvq_var_unpack.argtypes = [i64, i64, i32, i32, i64, p, p, p, p, p, p]
    lib.unisvq_var_unpack.restype = i32
    lib.unisvq_var_gemv.argtypes = [i64, i64, i32, i32, i64, p, p, i64, p, i32, p, i32, p]
    lib.unisvq_var_gemv.restype = i32
    lib.unisvq_var_gemv_batched.argtypes = [ctypes.POINTER(GemvSharedProblem), i32, i32, i32, i64, i32, i32, p]
    lib.unisvq_var_gemv_batched.restype = i32
    lib.unisvq_var_gemm_workspace_bytes.argtypes = [i64, i64, i64, i32]
    lib.unisvq_var_gemm_workspace_bytes.restype = sz
    lib.unisvq_var_gemm.argtypes = [i64, i64, i32, i32, i64, p, p, i64, p, i32, p, i32, p, sz, p]
    lib.unisvq_var_gemm.restype = i32
    lib.unisvq_ldlq_workspace_bytes.argtypes = [i64, i64]
    lib.unisvq_ldlq_workspace_bytes.restype = sz
    lib.unisvq_ldlq.argtypes = [i64, i64, p, p, p, p, i64, p, p, sz, p]
    lib.unisvq_ldlq.restype = i32
    lib.unisvq_ldl_workspace_bytes.argtypes = [i64]
    lib.unisvq_ldl_workspace_bytes.restype = sz
    lib.unisvq_ldl.argtypes = [i64, p, p, p, p, p, sz, p]
    lib.unisvq_ldl.restype = i32
    lib.unisvq_gemm_batched_workspace_bytes.argtypes = [ctypes.POINTER(GemvProblem), i32, i64, i32]
    lib.unisvq_gemm_batched_workspace_bytes.restype = sz
    lib.unisvq_gemm_batched.argtypes = [ctypes.POINTER(GemvProblem), i32, i64, i32, i32, p, sz, p]
    lib.unisvq_gemm_batched.restype = i32
    lib.unisvq_noalloc_scratch_bytes.argtypes = []
    lib.unisvq_noalloc_scratch_bytes.restype = sz
    lib.unisvq_gemm_noalloc.argtypes = [i64, i64, p, i64, p, i32, p, i32, p]
    lib.unisvq_gemm_noalloc.restype = i32
    lib.unisvq_read_sink_words.argtypes = [ctypes.POINTER(ByteRange), i32]
    lib.unisvq_read_sink_words.restype = i64
    lib.unisvq_read_bytes.argtypes = [ctypes.POINTER(ByteRange), i32, i32, p, i64, p]
    lib.unisvq_read_bytes.restype = i32
    _lib = lib
    return lib


def _status_string(status: int) -> str:
    try:
        return load().unisvq_status_string(status).decode()
    except UniSVQLibraryMissing:  # pragma: no cover
        return "?"


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise UniSVQError(fn, status)


def _torch():
    import torch
    return torch


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dtype_code(t) -> int:
    torch = _torch()
    codes = {torch.float16: F16, torch.bfloat16: BF16, torch.float32: F32}
    if t not in codes:
        raise TypeError(f"unsupported dtype {t}")
    return codes[t]


def _need_cuda(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("libunisvq takes device tensors only")


def _nbytes(t) -> int:
    return t.numel() * t.element_size()


def _need_buffer(t, need: int, what: str, exact: bool = False):
    """A device buffer of at least (exactly, if `exact`) `need` contiguous bytes:
    the kernels take their address ranges from the shape arguments, so a short
    or strided tensor would be read or written out of bounds."""
    if t is None:
        raise ValueError(f"{what} is required")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    have = _nbytes(t)
    if (have != need) if exact else (have < need):
        raise ValueError(f"{what} holds {have} bytes, expected {'' if exact else 'at least '}{need}")


def _activations(x, K: int):
    """x as a contiguous [M][K] fp16/bf16 view (a 1-D x is one or more rows)."""
    torch = _torch()
    if x.dim() == 2:
        if x.shape[1] != K:
            raise ValueError(f"x has {x.shape[1]} columns, the weights K = {K}")
        x2 = x
    else:
        if x.numel() == 0 or x.numel() % K:
            raise ValueError(f"x holds {x.numel()} elements, not a multiple of K = {K}")
        x2 = x.reshape(-1, K)
    if not x2.is_contiguous():
        raise ValueError("x must be contiguous")
    if x2.dtype not in (torch.float16, torch.bfloat16):
        raise TypeError(f"activations must be fp16 or bf16, got {x2.dtype}")
    return x2


def _output(out, M: int, N: int, out_dtype, like):
    """The caller's out (checked: contiguous, M*N elements, fp16/bf16/fp32) or a new [M][N] tensor."""
    torch = _torch()
    if out is None:
        return torch.empty((M, N), dtype=out_dtype or like.dtype, device=like.device)
    _dtype_code(out.dtype)
    if not out.is_contiguous():
        raise ValueError("out must be contiguous")
    if out.numel() != M * N:
        raise ValueError(f"out holds {out.numel()} elements, the product has M*N = {M * N}")
    return out


def version() -> int:
    return load().unisvq_version()


def packed_bytes(N: int, K: int) -> int:
    return load().unisvq_packed_bytes(N, K)


def _canonical(codes, A, B, N: int, K: int, pairs: int, d: int = DIM):
    """Shapes of canonical codes [N][K] (uint8) and of `pairs` (A, B) pairs (fp16 d x d and d)."""
    torch = _torch()
    if codes.dtype != torch.uint8 or tuple(codes.shape) != (N, K):
        raise ValueError(f"codes must be uint8 [{N}][{K}]")
    if A.dtype != torch.float16 or A.numel() != pairs * d * d:
        raise ValueError(f"A must hold {pairs} fp16 {d}x{d} matrices")
    if B.dtype != torch.float16 or B.numel() != pairs * d:
        raise ValueError(f"B must hold {pairs} fp16 {d}-vectors")


def pack(codes, A, B, out=None, bad_codes=None, stream=None):
    """codes uint8 [N][K]; A fp16 [N][K/128][4][4]; B fp16 [N][K/128][4] -> packed uint8 bytes."""
    torch = _torch()
    _need_cuda(codes, A, B, out, bad_codes)
    N, K = codes.shape
    _canonical(codes, A, B, N, K, N * (K // GROUP))
    if out is None:
        out = torch.empty(packed_bytes(N, K), dtype=torch.uint8, device=codes.device)
    _need_buffer(out, packed_bytes(N, K), "out")
    _check("unisvq_pack", load().unisvq_pack(N, K, _ptr(codes.contiguous()), _ptr(A.contiguous()),
                                             _ptr(B.contiguous()), _ptr(out), _ptr(bad_codes),
                                             _stream(stream)))
    return out


def unpack(packed, N: int, K: int, stream=None):
    """Inverse of pack: returns (codes uint8, A fp16, B fp16) device tensors."""
    torch = _torch()
    _need_cuda(packed)
    _need_buffer(packed, packed_bytes(N, K), "packed", exact=True)
    dev = packed.device
    codes = torch.empty((N, K), dtype=torch.uint8, device=dev)
    A = torch.empty((N, K // GROUP, DIM, DIM), dtype=torch.float16, device=dev)
    B = torch.empty((N, K // GROUP, DIM), dtype=torch.float16, device=dev)
    _check("unisvq_unpack", load().unisvq_unpack(N, K, _ptr(packed), _ptr(codes), _ptr(A), _ptr(B),
                                                 _stream(stream)))
    return codes, A, B


def _product(fn_name, N, K, packed, x, out, out_dtype, stream, extra=()):
    _need_cuda(packed, x, out)
    _need_buffer(packed, packed_bytes(N, K), "packed", exact=True)
    x2 = _activations(x, K)
    M = x2.shape[0]
    out = _output(out, M, N, out_dtype, x2)
    fn = getattr(load(), fn_name)
    _check(fn_name, fn(N, K, _ptr(packed), M, _ptr(x2), _dtype_code(x2.dtype), _ptr(out),
                       _dtype_code(out.dtype), *extra, _stream(stream)))
    return out


def gemv(packed, N: int, K: int, x, out=None, out_dtype=None, stream=None):
    """y[M][N] = x[M][K] . W_hat^T for 1 <= M <= 4 (decode-phase kernel)."""
    return _product("unisvq_gemv", N, K, packed, x, out, out_dtype, stream)


def gemv_batched(problems, out_dtype=None, stream=None):
    """Several independent decode products in one launch.

    problems: sequence of (packed, N, K, x, out-or-None); all x share M and dtype.
    Returns the list of outputs."""
    torch = _torch()
    if not 1 <= len(problems) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} problems per call")
    arr = (GemvProblem * len(problems))()
    outs, M, xdt = [], None, None
    for i, (packed, N, K, x, out) in enumerate(problems):
        _need_cuda(packed, x, out)
        _need_buffer(packed, packed_bytes(N, K), "packed", exact=True)
        x2 = _activations(x, K)
        if M is None:
            M, xdt = x2.shape[0], x2.dtype
        if x2.shape[0] != M or x2.dtype != xdt:
            raise ValueError("all problems need the same token count and activation dtype")
        out = _output(out, M, N, out_dtype, x2)
        outs.append(out)
        arr[i] = GemvProblem(N, K, packed.data_ptr(), x2.data_ptr(), out.data_ptr())
    ydt = {o.dtype for o in outs}
    if len(ydt) != 1:
        raise ValueError("all outputs need the same dtype")
    _check("unisvq_gemv_batched", load().unisvq_gemv_batched(arr, len(problems), M, _dtype_code(xdt),
                                                             _dtype_code(outs[0].dtype), _stream(stream)))
    return outs


def gemv_rht_batched(problems, out_dtype=None, stream=None):
    """Decode products of a rotated layer with the input-side transform fused in
    (Eq. 5): y_i = ((x_i diag(s_i)) H / sqrt(K)) W_rot,i^T.

    problems: sequence of (packed, N, K, x, signs, out-or-None); x in the
    original basis, signs int8 [K]; every K the same (4096 or 8192).
    Returns the list of outputs."""
    torch = _torch()
    if not 1 <= len(problems) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} problems per call")
    arr = (GemvProblem * len(problems))()
    sgn = (ctypes.c_void_p * len(problems))()
    outs, M, xdt = [], None, None
    for i, (packed, N, K, x, signs, out) in enumerate(problems):
        _need_cuda(packed, x, signs, out)
        _need_buffer(packed, packed_bytes(N, K), "packed", exact=True)
        _need_buffer(signs, K, "signs", exact=True)
        x2 = _activations(x, K)
        if M is None:
            M, xdt = x2.shape[0], x2.dtype
        if x2.shape[0] != M or x2.dtype != xdt:
            raise ValueError("all problems need the same token count and activation dtype")
        out = _output(out, M, N, out_dtype, x2)
        outs.append(out)
        arr[i] = GemvProblem(N, K, packed.data_ptr(), x2.data_ptr(), out.data_ptr())
        sgn[i] = signs.data_ptr()
    ydt = {o.dtype for o in outs}
    if len(ydt) != 1:
        raise ValueError("all outputs need the same dtype")
    _check("unisvq_gemv_rht_batched", load().unisvq_gemv_rht_batched(arr, len(problems), M, _dtype_code(xdt),
                                                                     _dtype_code(outs[0].dtype), sgn,
                                                                     _stream(stream)))
    return outs


def gemm_workspace_bytes(N: int, K: int, M: int, x_dtype=None) -> int:
    """Workspace bytes unisvq_gemm needs (x_dtype: torch dtype, default bf16)."""
    code = BF16 if x_dtype is None else _dtype_code(x_dtype)
    return load().unisvq_gemm_workspace_bytes(N, K, M, code)


def _workspace(workspace, need: int, like):
    """The caller's workspace (contiguous, at least `need` bytes) or a new one; and its size."""
    torch = _torch()
    if workspace is None:
        if not need:
            return None, 0
        workspace = torch.empty(need, dtype=torch.uint8, device=like.device)
    _need_cuda(workspace)
    _need_buffer(workspace, need, "workspace")
    return workspace, _nbytes(workspace)


def gemm(packed, N: int, K: int, x, out=None, out_dtype=None, workspace=None, stream=None):
    """y[M][N] = x[M][K] . W_hat^T for any M (prefill kernel)."""
    M = _activations(x, K).shape[0]
    workspace, ws_bytes = _workspace(workspace, gemm_workspace_bytes(N, K, M, x.dtype), x)
    return _product("unisvq_gemm", N, K, packed, x, out, out_dtype, stream,
                    extra=(_ptr(workspace), ws_bytes))


def noalloc_scratch_bytes() -> int:
    return int(load().unisvq_noalloc_scratch_bytes())


def gemm_noalloc(packed, N: int, K: int, x, out=None, out_dtype=None, stream=None):
    """unisvq_gemm with the library's fixed scratch as the workspace (the C
    call allocates nothing; pass `out` to keep this wrapper from allocating
    the output)."""
    return _product("unisvq_gemm_noalloc", N, K, packed, x, out, out_dtype, stream)


def gemm_batched(problems, out_dtype=None, workspace=None, stream=None):
    """Several independent products (same M and dtypes), each as unisvq_gemm:
    one launch (plus one reduction launch above 32 tokens when K is split).
    problems: sequence of (packed, N, K, x, out-or-None).
    Returns the list of outputs."""
    if not 1 <= len(problems) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} problems per call")
    arr = (GemvProblem * len(problems))()
    outs, M, xdt = [], None, None
    for i, (packed, N, K, x, out) in enumerate(problems):
        _need_cuda(packed, x, out)
        _need_buffer(packed, packed_bytes(N, K), "packed", exact=True)
        x2 = _activations(x, K)
        if M is None:
            M, xdt = x2.shape[0], x2.dtype
        if x2.shape[0] != M or x2.dtype != xdt:
            raise ValueError("all problems need the same token count and activation dtype")
        out = _output(out, M, N, out_dtype, x2)
        outs.append(out)
        arr[i] = GemvProblem(N, K, packed.data_ptr(), x2.data_ptr(), out.data_ptr())
    if len({o.dtype for o in outs}) != 1:
        raise ValueError("all outputs need the same dtype")
    lib = load()
    need = lib.unisvq_gemm_batched_workspace_bytes(arr, len(problems), M, _dtype_code(xdt))
    workspace, wb = _workspace(workspace, need, outs[0])
    _check("unisvq_gemm_batched", lib.unisvq_gemm_batched(arr, len(problems), M, _dtype_code(xdt),
                                                          _dtype_code(outs[0].dtype), _ptr(workspace), wb,
                                                          _stream(stream)))
    return outs


# ------------------------------------------------ row-shared affine parameters

def codes_bytes(N: int, K: int) -> int:
    return load().unisvq_codes_bytes(N, K)


def shared_affine_bytes(K: int, affine_groups: int) -> int:
    return load().unisvq_shared_affine_bytes(K, affine_groups)


def pack_shared(codes, A, B, out_codes=None, out_affine=None, bad_codes=None, stream=None):
    """codes uint8 [N][K]; A fp16 [Ga][4][4]; B fp16 [Ga][4] (Ga = 1 or K/128)
    -> (packed codes, packed shared affine block), uint8 device tensors."""
    torch = _torch()
    _need_cuda(codes, A, B, out_codes, out_affine, bad_codes)
    N, K = codes.shape
    Ga = A.shape[0]
    _canonical(codes, A, B, N, K, Ga)
    if out_codes is None:
        out_codes = torch.empty(codes_bytes(N, K), dtype=torch.uint8, device=codes.device)
    if out_affine is None:
        out_affine = torch.empty(max(shared_affine_bytes(K, Ga), 16), dtype=torch.uint8, device=codes.device)
    _need_buffer(out_codes, codes_bytes(N, K), "out_codes")
    _need_buffer(out_affine, shared_affine_bytes(K, Ga), "out_affine")
    _check("unisvq_pack_shared", load().unisvq_pack_shared(
        N, K, Ga, _ptr(codes.contiguous()), _ptr(A.contiguous()), _ptr(B.contiguous()), _ptr(out_codes),
        _ptr(out_affine), _ptr(bad_codes), _stream(stream)))
    return out_codes, out_affine


def unpack_shared(packed_codes, packed_affine, N: int, K: int, affine_groups: int, stream=None):
    """Inverse of pack_shared: (codes uint8 [N][K], A fp16 [Ga][4][4], B fp16 [Ga][4])."""
    torch = _torch()
    _need_cuda(packed_codes, packed_affine)
    _need_buffer(packed_codes, codes_bytes(N, K), "packed_codes", exact=True)
    _need_buffer(packed_affine, shared_affine_bytes(K, affine_groups), "packed_affine")
    dev = packed_codes.device
    codes = torch.empty((N, K), dtype=torch.uint8, device=dev)
    A = torch.empty((affine_groups, DIM, DIM), dtype=torch.float16, device=dev)
    B = torch.empty((affine_groups, DIM), dtype=torch.float16, device=dev)
    _check("unisvq_unpack_shared", load().unisvq_unpack_shared(
        N, K, affine_groups, _ptr(packed_codes), _ptr(packed_affine), _ptr(codes), _ptr(A), _ptr(B),
        _stream(stream)))
    return codes, A, B


def _shared_operands(packed_codes, packed_affine, N, K, affine_groups):
    _need_buffer(packed_codes, codes_bytes(N, K), "packed_codes", exact=True)
    need = shared_affine_bytes(K, affine_groups)
    if not need:
        raise ValueError(f"affine_groups must be 1 or K/128 = {K // GROUP}, got {affine_groups}")
    _need_buffer(packed_affine, need, "packed_affine")


def _shared_product(fn_name, N, K, affine_groups, packed_codes, packed_affine, x, out, out_dtype, stream,
                    extra=()):
    _need_cuda(packed_codes, packed_affine, x, out)
    _shared_operands(packed_codes, packed_affine, N, K, affine_groups)
    x2 = _activations(x, K)
    M = x2.shape[0]
    out = _output(out, M, N, out_dtype, x2)
    fn = getattr(load(), fn_name)
    _check(fn_name, fn(N, K, affine_groups, _ptr(packed_codes), _ptr(packed_affine), M, _ptr(x2),
                       _dtype_code(x2.dtype), _ptr(out), _dtype_code(out.dtype), *extra, _stream(stream)))
    return out


def gemv_shared(packed_codes, packed_affine, N: int, K: int, affine_groups: int, x, out=None, out_dtype=None,
                stream=None):
    """Decode-phase product with codes-only weights and row-shared pairs (M <= 4)."""
    return _shared_product("unisvq_gemv_shared", N, K, affine_groups, packed_codes, packed_affine, x, out,
                           out_dtype, stream)


def gemv_shared_batched(problems, out_dtype=None, stream=None):
    """problems: sequence of (packed_codes, packed_affine, N, K, affine_groups, x, out-or-None)."""
    torch = _torch()
    if not 1 <= len(problems) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} problems per call")
    arr = (GemvSharedProblem * len(problems))()
    outs, M, xdt = [], None, None
    for i, (pc, pa, N, K, ga, x, out) in enumerate(problems):
        _need_cuda(pc, pa, x, out)
        _shared_operands(pc, pa, N, K, ga)
        x2 = _activations(x, K)
        if M is None:
            M, xdt = x2.shape[0], x2.dtype
        if x2.shape[0] != M or x2.dtype != xdt:
            raise ValueError("all problems need the same token count and activation dtype")
        out = _output(out, M, N, out_dtype, x2)
        outs.append(out)
        arr[i] = GemvSharedProblem(N, K, ga, pc.data_ptr(), pa.data_ptr(), x2.data_ptr(), out.data_ptr())
    if len({o.dtype for o in outs}) != 1:
        raise ValueError("all outputs need the same dtype")
    _check("unisvq_gemv_shared_batched", load().unisvq_gemv_shared_batched(
        arr, len(problems), M, _dtype_code(xdt), _dtype_code(outs[0].dtype), _stream(stream)))
    return outs


def gemm_shared(packed_codes, packed_affine, N: int, K: int, affine_groups: int, x, out=None, out_dtype=None,
                workspace=None, stream=None):
    """Prefill product with codes-only weights and row-shared pairs (any M)."""
    M = _activations(x, K).shape[0]
    workspace, ws_bytes = _workspace(workspace, gemm_workspace_bytes(N, K, M, x.dtype), x)
    return _shared_product("unisvq_gemm_shared", N, K, affine_groups, packed_codes, packed_affine, x, out,
                           out_dtype, stream, extra=(_ptr(workspace), ws_bytes))


def gemm_fold_workspace_bytes(N: int, K: int, M: int) -> int:
    return int(load().unisvq_gemm_fold_workspace_bytes(N, K, M))


def gemm_shared_fold(packed_codes, packed_affine, N: int, K: int, affine_groups: int, x, out=None,
                     out_dtype=None, workspace=None, stream=None):
    """Prefill product with row-shared pairs through the Eq. 9 fold (any M)."""
    M = _activations(x, K).shape[0]
    workspace, ws_bytes = _workspace(workspace, gemm_fold_workspace_bytes(N, K, M), x)
    return _shared_product("unisvq_gemm_shared_fold", N, K, affine_groups, packed_codes, packed_affine, x, out,
                           out_dtype, stream, extra=(_ptr(workspace), ws_bytes))


# ------------------------------------------------ nearest-codeword quantiser

def quantize(W, A, B, affine_groups: int = 0, out=None, stream=None):
    """Codes uint8 [N][K] of the nearest codeword per vector of W (fp32 [N][K]).
    affine_groups 0: A/B per (row, group); 1 or K/128: row-shared pairs."""
    torch = _torch()
    _need_cuda(W, A, B, out)
    N, K = W.shape
    if W.dtype != torch.float32:
        raise TypeError("W must be fp32")
    pairs = N * (K // GROUP) if affine_groups == 0 else affine_groups
    _canonical(torch.empty((N, K), dtype=torch.uint8, device="meta"), A, B, N, K, pairs)
    if out is None:
        out = torch.empty((N, K), dtype=torch.uint8, device=W.device)
    _need_buffer(out, N * K, "out", exact=True)
    _check("unisvq_quantize", load().unisvq_quantize(N, K, _ptr(W.contiguous()), _ptr(A.contiguous()),
                                                     _ptr(B.contiguous()), affine_groups, _ptr(out),
                                                     _stream(stream)))
    return out


# ------------------------------------------------ randomized Hadamard transform

def rht(x, signs, mode: str, out=None, out_dtype=None, stream=None):
    """mode 'in': (x diag(signs)) H / sqrt(n); mode 'out': (x H / sqrt(n)) diag(signs).
    x [M][n] (fp16, bf16 or fp32), signs int8 [n] (+-1)."""
    _need_cuda(x, signs, out)
    x2 = x if x.dim() == 2 else x.reshape(1, -1)
    if not x2.is_contiguous():
        raise ValueError("x must be contiguous")
    M, n = x2.shape
    _need_buffer(signs, n, "signs", exact=True)
    out = _output(out, M, n, out_dtype, x2)
    _check("unisvq_rht", load().unisvq_rht(n, M, _ptr(x2), _dtype_code(x2.dtype), _ptr(signs.contiguous()),
                                           0 if mode == "in" else 1, _ptr(out), _dtype_code(out.dtype),
                                           _stream(stream)))
    return out


# ------------------------------------------------ format variants (b-bit codes, d-dim vectors)

def var_codes_bytes(N: int, K: int, bits: int, d: int) -> int:
    return load().unisvq_var_codes_bytes(N, K, bits, d)


def var_affine_bytes(K: int, affine_groups: int, bits: int, d: int) -> int:
    return load().unisvq_var_affine_bytes(K, affine_groups, bits, d)


def var_pack(codes, A, B, bits: int, d: int, out_codes=None, out_affine=None, bad_codes=None, stream=None):
    """codes uint8 [N][K] (0..2^bits-1); A fp16 [Ga][d][d]; B fp16 [Ga][d]
    -> (packed variant codes, packed shared affine block), uint8 device tensors."""
    torch = _torch()
    _need_cuda(codes, A, B, out_codes, out_affine, bad_codes)
    N, K = codes.shape
    Ga = A.shape[0]
    _canonical(codes, A, B, N, K, Ga, d)
    if out_codes is None:
        out_codes = torch.empty(max(var_codes_bytes(N, K, bits, d), 16), dtype=torch.uint8, device=codes.device)
    if out_affine is None:
        out_affine = torch.empty(max(var_affine_bytes(K, Ga, bits, d), 16), dtype=torch.uint8, device=codes.device)
    _need_buffer(out_codes, var_codes_bytes(N, K, bits, d), "out_codes")
    _need_buffer(out_affine, var_affine_bytes(K, Ga, bits, d), "out_affine")
    _check("unisvq_var_pack", load().unisvq_var_pack(
        N, K, bits, d, Ga, _ptr(codes.contiguous()), _ptr(A.contiguous()), _ptr(B.contiguous()), _ptr(out_codes),
        _ptr(out_affine), _ptr(bad_codes), _stream(stream)))
    return out_codes, out_affine


def var_unpack(packed_codes, packed_affine, N: int, K: int, bits: int, d: int, affine_groups: int, stream=None):
    """Inverse of var_pack: (codes uint8 [N][K], A fp16 [Ga][d][d], B fp16 [Ga][d])."""
    torch = _torch()
    _need_cuda(packed_codes, packed_affine)
    _var_operands(packed_codes, packed_affine, N, K, bits, d, affine_groups)
    dev = packed_codes.device
    codes = torch.empty((N, K), dtype=torch.uint8, device=dev)
    A = torch.empty((affine_groups, d, d), dtype=torch.float16, device=dev)
    B = torch.empty((affine_groups, d), dtype=torch.float16, device=dev)
    _check("unisvq_var_unpack", load().unisvq_var_unpack(
        N, K, bits, d, affine_groups, _ptr(packed_codes), _ptr(packed_affine), _ptr(codes), _ptr(A), _ptr(B),
        _stream(stream)))
    return codes, A, B


def _var_operands(packed_codes, packed_affine, N, K, bits, d, affine_groups):
    need_c = var_codes_bytes(N, K, bits, d)
    need_a = var_affine_bytes(K, affine_groups, bits, d)
    if not need_c or not need_a:
        raise ValueError(f"unsupported variant (bits={bits}, d={d}, affine_groups={affine_groups}) or shape")
    _need_buffer(packed_codes, need_c, "packed_codes")
    _need_buffer(packed_affine, need_a, "packed_affine")


def _var_product(fn_name, N, K, bits, d, affine_groups, packed_codes, packed_affine, x, out, out_dtype, stream,
                 extra=()):
    _need_cuda(packed_codes, packed_affine, x, out)
    _var_operands(packed_codes, packed_affine, N, K, bits, d, affine_groups)
    x2 = _activations(x, K)
    M = x2.shape[0]
    out = _output(out, M, N, out_dtype, x2)
    fn = getattr(load(), fn_name)
    _check(fn_name, fn(N, K, bits, d, affine_groups, _ptr(packed_codes), _ptr(packed_affine), M, _ptr(x2),
                       _dtype_code(x2.dtype), _ptr(out), _dtype_code(out.dtype), *extra, _stream(stream)))
    return out


def var_gemv(packed_codes, packed_affine, N: int, K: int, bits: int, d: int, affine_groups: int, x, out=None,
             out_dtype=None, stream=None):
    """Decode-phase product with variant weights (M <= 4)."""
    return _var_product("unisvq_var_gemv", N, K, bits, d, affine_groups, packed_codes, packed_affine, x, out,
                        out_dtype, stream)


def var_gemv_batched(problems, bits: int, d: int, out_dtype=None, stream=None):
    """problems: list of dicts with packed_codes, packed_affine, N, K, affine_groups, x (same M and dtype), and
    optionally out; one launch.  Returns the list of outputs."""
    torch = _torch()
    if not 1 <= len(problems) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} problems per launch")
    arr = (GemvSharedProblem * len(problems))()
    outs = []
    M = None
    for i, pr in enumerate(problems):
        _need_cuda(pr["packed_codes"], pr["packed_affine"], pr["x"], pr.get("out"))
        _var_operands(pr["packed_codes"], pr["packed_affine"], pr["N"], pr["K"], bits, d, pr["affine_groups"])
        x = _activations(pr["x"], pr["K"])
        if M is None:
            M, xdt = x.shape[0], x.dtype
        if x.shape[0] != M or x.dtype != xdt:
            raise ValueError("all problems need the same token count and activation dtype")
        out = _output(pr.get("out"), M, pr["N"], out_dtype, x)
        outs.append(out)
        arr[i] = GemvSharedProblem(pr["N"], pr["K"], pr["affine_groups"], _ptr(pr["packed_codes"]),
                                   _ptr(pr["packed_affine"]), _ptr(x), _ptr(out))
    if len({o.dtype for o in outs}) != 1:
        raise ValueError("all outputs need the same dtype")
    _check("unisvq_var_gemv_batched", load().unisvq_var_gemv_batched(
        arr, len(problems), bits, d, M, _dtype_code(xdt), _dtype_code(outs[0].dtype), _stream(stream)))
    return outs


def var_gemm_workspace_bytes(N: int, K: int, M: int, x_dtype=None) -> int:
    """Workspace bytes unisvq_var_gemm needs (x_dtype: torch dtype, default bf16)."""
    code = BF16 if x_dtype is None else _dtype_code(x_dtype)
    return load().unisvq_var_gemm_workspace_bytes(N, K, M, code)


def var_gemm(packed_codes, packed_affine, N: int, K: int, bits: int, d: int, affine_groups: int, x, out=None,
             out_dtype=None, workspace=None, stream=None):
    """Prefill product with variant weights (any M)."""
    M = _activations(x, K).shape[0]
    workspace, wb = _workspace(workspace, var_gemm_workspace_bytes(N, K, M, x.dtype), x)
    return _var_product("unisvq_var_gemm", N, K, bits, d, affine_groups, packed_codes, packed_affine, x, out,
                        out_dtype, stream, extra=(_ptr(workspace), wb))


# ------------------------------------------------ LDLQ (Eq. 7)

def ldl_workspace_bytes(K: int) -> int:
    return load().unisvq_ldl_workspace_bytes(K)


def ldl(H, out=None, with_d: bool = True, workspace=None, stream=None):
    """H = U D U^T (fp64 [K][K], symmetric positive definite; the upper
    triangle is read) with U unit upper block triangular and D block diagonal
    (4 x 4 blocks): the factor ldlq() takes.  `out` may be H itself (in place).
    Returns (U, D [K/4][4][4] or None, info): info is a device int32 [1], 0 or
    1 + the first pivot block found not positive definite."""
    torch = _torch()
    _need_cuda(H, out, workspace)
    if H.dtype != torch.float64 or H.dim() != 2 or H.shape[0] != H.shape[1]:
        raise ValueError("H must be fp64 [K][K]")
    if not H.is_contiguous():
        raise ValueError("H must be contiguous")
    K = H.shape[0]
    if out is None:
        out = torch.empty((K, K), dtype=torch.float64, device=H.device)
    if out.dtype != torch.float64:
        raise ValueError("out must be fp64")
    _need_buffer(out, K * K * 8, "out", exact=True)
    D = torch.empty((K // 4, 4, 4), dtype=torch.float64, device=H.device) if with_d else None
    info = torch.empty(1, dtype=torch.int32, device=H.device)
    workspace, wb = _workspace(workspace, ldl_workspace_bytes(K), H)
    _check("unisvq_ldl", load().unisvq_ldl(K, _ptr(H), _ptr(out), _ptr(D), _ptr(info), _ptr(workspace), wb,
                                            _stream(stream)))
    return out, D, info


def ldlq_workspace_bytes(N: int, K: int) -> int:
    return load().unisvq_ldlq_workspace_bytes(N, K)


def ldlq(W, U, A, B, affine_groups: int = 0, out=None, workspace=None, stream=None):
    """LDLQ codes of fp32 W [N][K] with the feedback factor U (fp64 [K][K], unit
    upper block triangular, from H = U D U^T); A/B as quantize().  Returns
    codes uint8 [N][K]."""
    torch = _torch()
    _need_cuda(W, U, A, B, out, workspace)
    N, K = W.shape
    if W.dtype != torch.float32 or U.dtype != torch.float64 or U.numel() != K * K:
        raise ValueError(f"W must be fp32 [N][K] and U fp64 [{K}][{K}]")
    pairs = N * (K // GROUP) if affine_groups == 0 else affine_groups
    _canonical(torch.empty((N, K), dtype=torch.uint8, device="meta"), A, B, N, K, pairs)
    if out is None:
        out = torch.empty((N, K), dtype=torch.uint8, device=W.device)
    _need_buffer(out, N * K, "out", exact=True)
    workspace, wb = _workspace(workspace, ldlq_workspace_bytes(N, K), W)
    _check("unisvq_ldlq", load().unisvq_ldlq(N, K, _ptr(W.contiguous()), _ptr(U.contiguous()), _ptr(A.contiguous()),
                                              _ptr(B.contiguous()), affine_groups, _ptr(out), _ptr(workspace), wb,
                                              _stream(stream)))
    return out


# ------------------------------------------------ bandwidth reference

def read_bytes(buffers, store: bool = True, sink=None, stream=None):
    """Plain read of the given device tensors (contiguous, 16-byte multiples)
    in one launch.  With `store`, returns the sink (uint32 words as int32, one
    per wavefront) whose XOR equals the XOR of every 32-bit word read;
    without it nothing is written and None is returned."""
    torch = _torch()
    _need_cuda(sink, *buffers)
    if not 1 <= len(buffers) <= MAX_BATCH:
        raise ValueError(f"1..{MAX_BATCH} buffers per call")
    arr = (ByteRange * len(buffers))()
    for i, t in enumerate(buffers):
        if not t.is_contiguous():
            raise ValueError("buffers must be contiguous")
        arr[i] = ByteRange(t.data_ptr(), _nbytes(t))
    if not store:
        _check("unisvq_read_bytes", load().unisvq_read_bytes(arr, len(buffers), 0, None, 0, _stream(stream)))
        return None
    words = load().unisvq_read_sink_words(arr, len(buffers))
    if sink is None:
        sink = torch.empty(max(words, 1), dtype=torch.int32, device=buffers[0].device)
    _need_buffer(sink, 4 * words, "sink")
    _check("unisvq_read_bytes", load().unisvq_read_bytes(arr, len(buffers), 1, _ptr(sink), sink.numel(),
                                                         _stream(stream)))
    return sink
