"""UniSVQ fp64 CPU oracle -- TEST INFRASTRUCTURE ONLY.

Thin ctypes wrapper around ``oracle.c``: a plain, slow, obviously correct
implementation of the UniSVQ inference product (Sec. 3.1 Eq. 4 decode, Sec.
3.2.3 Eq. 8 stacking along the input dimension, Sec. 2.1 Eq. 1 product) and of
the packed byte format.  Only ``tests/``, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  It
shares no code with the HIP library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with the host C compiler (gcc)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-pthread",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    i64, p = ctypes.c_int64, ctypes.c_void_p
    lib.oracle_half_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_half_to_double.restype = ctypes.c_double
    lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
    lib.oracle_bf16_to_double.restype = ctypes.c_double
    lib.oracle_half_array_to_double.argtypes = [p, p, i64]
    lib.oracle_half_array_to_double.restype = None
    lib.oracle_bf16_array_to_double.argtypes = [p, p, i64]
    lib.oracle_bf16_array_to_double.restype = None
    lib.oracle_packed_bytes.argtypes = [i64, i64]
    lib.oracle_packed_bytes.restype = i64
    lib.oracle_pack.argtypes = [i64, i64, p, p, p, p]
    lib.oracle_pack.restype = i64
    lib.oracle_unpack.argtypes = [i64, i64, p, p, p, p]
    lib.oracle_unpack.restype = ctypes.c_int
    lib.oracle_decode.argtypes = [i64, i64, p, p, p, p]
    lib.oracle_decode.restype = ctypes.c_int
    lib.oracle_decode_packed_rows.argtypes = [i64, i64, p, i64, i64, p]
    lib.oracle_decode_packed_rows.restype = ctypes.c_int
    lib.oracle_matmul_rows.argtypes = [i64, i64, p, i64, p, i64, p, p, ctypes.c_int]
    lib.oracle_matmul_rows.restype = ctypes.c_int
    lib.oracle_codes_packed_bytes.argtypes = [i64, i64]
    lib.oracle_codes_packed_bytes.restype = i64
    lib.oracle_pack_codes.argtypes = [i64, i64, p, p]
    lib.oracle_pack_codes.restype = i64
    lib.oracle_unpack_codes.argtypes = [i64, i64, p, p]
    lib.oracle_unpack_codes.restype = ctypes.c_int
    lib.oracle_matmul_shared_rows.argtypes = [i64, i64, p, i64, p, p, i64, p, i64, p, p, ctypes.c_int]
    lib.oracle_matmul_shared_rows.restype = ctypes.c_int
    lib.oracle_quantize.argtypes = [i64, i64, p, p, p, i64, p]
    lib.oracle_quantize.restype = ctypes.c_int
    lib.oracle_hadamard_factor.argtypes = [i64, p]
    lib.oracle_hadamard_factor.restype = ctypes.c_int
    lib.oracle_hadamard.argtypes = [i64, p]
    lib.oracle_hadamard.restype = ctypes.c_int
    lib.oracle_rht.argtypes = [i64, i64, p, p, ctypes.c_int, p]
    lib.oracle_rht.restype = ctypes.c_int
    ci = ctypes.c_int
    lib.oracle_var_codes_bytes.argtypes = [i64, i64, ci]
    lib.oracle_var_codes_bytes.restype = i64
    lib.oracle_var_pack_codes.argtypes = [i64, i64, ci, ci, p, p]
    lib.oracle_var_pack_codes.restype = i64
    lib.oracle_var_unpack_codes.argtypes = [i64, i64, ci, ci, p, p]
    lib.oracle_var_unpack_codes.restype = ci
    lib.oracle_var_affine_bytes.argtypes = [i64, i64, ci]
    lib.oracle_var_affine_bytes.restype = i64
    lib.oracle_var_pack_affine.argtypes = [i64, i64, ci, p, p, p]
    lib.oracle_var_pack_affine.restype = ci
    lib.oracle_var_unpack_affine.argtypes = [i64, i64, ci, p, p, p]
    lib.oracle_var_unpack_affine.restype = ci
    lib.oracle_var_decode.argtypes = [i64, i64, ci, p, i64, p, p, p]
    lib.oracle_var_decode.restype = ci
    lib.oracle_var_matmul_rows.argtypes = [i64, i64, ci, ci, p, i64, p, p, i64, p, i64, p, p, ci]
    lib.oracle_var_matmul_rows.restype = ci
    lib.oracle_ldlq.argtypes = [i64, i64, p, p, p, p, i64, p, p, ci]
    lib.oracle_ldlq.restype = ci
    _lib = lib
    return lib


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"], "oracle arrays must be C-contiguous"
    return ctypes.c_void_p(a.ctypes.data)


def _bits16(a: np.ndarray) -> np.ndarray:
    """fp16 / bf16-bit arrays are passed as raw uint16 bits."""
    if a.dtype == np.float16:
        return np.ascontiguousarray(a).view(np.uint16)
    assert a.dtype == np.uint16, a.dtype
    return np.ascontiguousarray(a)


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> int:
    if rc < 0:
        raise OracleError(f"{what} failed with status {rc}")
    return rc


def half_to_double(bits: np.ndarray) -> np.ndarray:
    lib = _load()
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(b.shape, dtype=np.float64)
    lib.oracle_half_array_to_double(_ptr(b), _ptr(out), b.size)
    return out


def bf16_to_double(bits: np.ndarray) -> np.ndarray:
    lib = _load()
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    out = np.empty(b.shape, dtype=np.float64)
    lib.oracle_bf16_array_to_double(_ptr(b), _ptr(out), b.size)
    return out


def packed_bytes(N: int, K: int) -> int:
    return _check(_load().oracle_packed_bytes(N, K), "packed_bytes")


def pack(Q: np.ndarray, A: np.ndarray, B: np.ndarray):
    """Pack canonical arrays; returns (packed uint8 bytes, number of codes > 3)."""
    lib = _load()
    N, K = Q.shape
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    Ab, Bb = _bits16(A), _bits16(B)
    assert Ab.shape == (N, K // 128, 4, 4) and Bb.shape == (N, K // 128, 4)
    out = np.empty(packed_bytes(N, K), dtype=np.uint8)
    bad = _check(lib.oracle_pack(N, K, _ptr(Q), _ptr(Ab), _ptr(Bb), _ptr(out)), "pack")
    return out, int(bad)


def unpack(packed: np.ndarray, N: int, K: int):
    """Inverse of pack: returns (Q uint8, A fp16, B fp16)."""
    lib = _load()
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    assert packed.size == packed_bytes(N, K)
    Q = np.empty((N, K), dtype=np.uint8)
    A = np.empty((N, K // 128, 4, 4), dtype=np.uint16)
    B = np.empty((N, K // 128, 4), dtype=np.uint16)
    _check(lib.oracle_unpack(N, K, _ptr(packed), _ptr(Q), _ptr(A), _ptr(B)), "unpack")
    return Q, A.view(np.float16), B.view(np.float16)


def decode(Q: np.ndarray, A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """fp64 dequantised weights W_hat [N][K] from canonical arrays."""
    lib = _load()
    N, K = Q.shape
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    Ab, Bb = _bits16(A), _bits16(B)
    W = np.empty((N, K), dtype=np.float64)
    _check(lib.oracle_decode(N, K, _ptr(Q), _ptr(Ab), _ptr(Bb), _ptr(W)), "decode")
    return W


def decode_packed_rows(packed: np.ndarray, N: int, K: int, r0: int, r1: int) -> np.ndarray:
    lib = _load()
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    W = np.empty((r1 - r0, K), dtype=np.float64)
    _check(lib.oracle_decode_packed_rows(N, K, _ptr(packed), r0, r1, _ptr(W)), "decode_packed_rows")
    return W


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def matmul(packed: np.ndarray, N: int, K: int, X: np.ndarray, rows=None, threads: int | None = None):
    """Y = X * W_hat^T in fp64 from packed bytes.

    X is [M][K] (any float dtype; converted exactly to fp64).  With ``rows``
    given, only those output columns are computed and Y is [M][len(rows)].
    """
    lib = _load()
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    assert packed.size == packed_bytes(N, K)
    X = np.ascontiguousarray(X, dtype=np.float64)
    if X.ndim == 1:
        X = X[None, :]
    M = X.shape[0]
    assert X.shape[1] == K
    if threads is None:
        threads = default_threads()
    if rows is None:
        Y = np.empty((M, N), dtype=np.float64)
        _check(lib.oracle_matmul_rows(N, K, _ptr(packed), M, _ptr(X), N, None, _ptr(Y), threads),
               "matmul")
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        Y = np.empty((M, r.size), dtype=np.float64)
        _check(lib.oracle_matmul_rows(N, K, _ptr(packed), M, _ptr(X), r.size, _ptr(r), _ptr(Y),
                                      threads), "matmul_rows")
    return Y


# ------------------------------------------------ row-shared affine parameters

def codes_packed_bytes(N: int, K: int) -> int:
    """Bytes of the codes-only format: 2 bits per weight, nothing else."""
    return _check(_load().oracle_codes_packed_bytes(N, K), "codes_packed_bytes")


def pack_codes(Q: np.ndarray):
    """Codes-only packing; returns (packed uint8 bytes, number of codes > 3)."""
    lib = _load()
    N, K = Q.shape
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    out = np.empty(codes_packed_bytes(N, K), dtype=np.uint8)
    bad = _check(lib.oracle_pack_codes(N, K, _ptr(Q), _ptr(out)), "pack_codes")
    return out, int(bad)


def unpack_codes(packed: np.ndarray, N: int, K: int) -> np.ndarray:
    lib = _load()
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    assert packed.size == codes_packed_bytes(N, K)
    Q = np.empty((N, K), dtype=np.uint8)
    _check(lib.oracle_unpack_codes(N, K, _ptr(packed), _ptr(Q)), "unpack_codes")
    return Q


def matmul_shared(packed_codes: np.ndarray, N: int, K: int, As: np.ndarray, Bs: np.ndarray, X: np.ndarray,
                  rows=None, threads: int | None = None):
    """Y = X * W_hat^T in fp64 where every row decodes with the shared pairs
    As [Ga][4][4], Bs [Ga][4] (Ga = 1: one pair for the matrix; Ga = K/128: one
    per group)."""
    lib = _load()
    packed_codes = np.ascontiguousarray(packed_codes, dtype=np.uint8)
    assert packed_codes.size == codes_packed_bytes(N, K)
    Ab, Bb = _bits16(As), _bits16(Bs)
    Ga = Ab.shape[0]
    assert Ab.shape == (Ga, 4, 4) and Bb.shape == (Ga, 4)
    X = np.ascontiguousarray(X, dtype=np.float64)
    if X.ndim == 1:
        X = X[None, :]
    M = X.shape[0]
    assert X.shape[1] == K
    if threads is None:
        threads = default_threads()
    if rows is None:
        Y = np.empty((M, N), dtype=np.float64)
        _check(lib.oracle_matmul_shared_rows(N, K, _ptr(packed_codes), Ga, _ptr(Ab), _ptr(Bb), M, _ptr(X), N,
                                             None, _ptr(Y), threads), "matmul_shared")
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        Y = np.empty((M, r.size), dtype=np.float64)
        _check(lib.oracle_matmul_shared_rows(N, K, _ptr(packed_codes), Ga, _ptr(Ab), _ptr(Bb), M, _ptr(X),
                                             r.size, _ptr(r), _ptr(Y), threads), "matmul_shared_rows")
    return Y


# ------------------------------------------------ nearest-codeword quantiser

def quantize(W: np.ndarray, A: np.ndarray, B: np.ndarray, shared: bool = False) -> np.ndarray:
    """Codes of the nearest codeword A q + B per vector of W (fp32 [N][K]).

    A/B per (row, group) ([N][K/128][4][4] / [N][K/128][4]), or with
    ``shared`` row-shared ([Ga][4][4] / [Ga][4], Ga = 1 or K/128).  Distances
    in fp64 with a fixed operation order; ties to the lowest index
    q0 + 4 q1 + 16 q2 + 64 q3."""
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.float32)
    N, K = W.shape
    Ab, Bb = _bits16(A), _bits16(B)
    Ga = Ab.shape[0] if shared else 0
    Q = np.empty((N, K), dtype=np.uint8)
    _check(lib.oracle_quantize(N, K, _ptr(W), _ptr(Ab), _ptr(Bb), Ga, _ptr(Q)), "quantize")
    return Q


# ------------------------------------------------ randomized Hadamard transform

def hadamard_factor(n: int) -> dict:
    """The construction used for order n: n = 2^k * m (m = 1, or m = q + 1 with
    q = p^e a prime power = 3 mod 4)."""
    out = np.zeros(5, dtype=np.int64)
    _check(_load().oracle_hadamard_factor(n, _ptr(out)), "hadamard_factor")
    return dict(zip(("k", "m", "q", "p", "e"), (int(v) for v in out)))


def hadamard(n: int) -> np.ndarray:
    """The +-1 Hadamard matrix of order n (int8)."""
    H = np.empty((n, n), dtype=np.int8)
    _check(_load().oracle_hadamard(n, _ptr(H)), "hadamard")
    return H


def rht(X: np.ndarray, signs: np.ndarray, mode: str) -> np.ndarray:
    """mode 'in': (X diag(s)) H / sqrt(n)  (x S_V V);  mode 'out': (X H / sqrt(n)) diag(s)  (y U S_U)."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    if X.ndim == 1:
        X = X[None, :]
    M, n = X.shape
    s = np.ascontiguousarray(signs, dtype=np.int8)
    assert s.shape == (n,)
    Y = np.empty_like(X)
    _check(_load().oracle_rht(n, M, _ptr(X), _ptr(s), 0 if mode == "in" else 1, _ptr(Y)), "rht")
    return Y


# ------------------------------------------------ format variants (b = 2, 3; d = 4, 8)

def var_codes_bytes(N: int, K: int, bits: int) -> int:
    """Bytes of the variant codes-only format: bits per weight, nothing else."""
    return _check(_load().oracle_var_codes_bytes(N, K, bits), "var_codes_bytes")


def var_pack_codes(Q: np.ndarray, bits: int, d: int):
    """Variant codes-only packing; returns (packed bytes, number of codes >= 2^bits)."""
    N, K = Q.shape
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    out = np.empty(var_codes_bytes(N, K, bits), dtype=np.uint8)
    bad = _check(_load().oracle_var_pack_codes(N, K, bits, d, _ptr(Q), _ptr(out)), "var_pack_codes")
    return out, int(bad)


def var_unpack_codes(packed: np.ndarray, N: int, K: int, bits: int, d: int) -> np.ndarray:
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    assert packed.size == var_codes_bytes(N, K, bits)
    Q = np.empty((N, K), dtype=np.uint8)
    _check(_load().oracle_var_unpack_codes(N, K, bits, d, _ptr(packed), _ptr(Q)), "var_unpack_codes")
    return Q


def var_affine_bytes(K: int, Ga: int, d: int) -> int:
    return _check(_load().oracle_var_affine_bytes(K, Ga, d), "var_affine_bytes")


def var_pack_affine(As: np.ndarray, Bs: np.ndarray, K: int) -> np.ndarray:
    """Shared affine block (lane and row views) of As [Ga][d][d], Bs [Ga][d]."""
    Ab, Bb = _bits16(As), _bits16(Bs)
    Ga, d = Ab.shape[0], Ab.shape[1]
    assert Ab.shape == (Ga, d, d) and Bb.shape == (Ga, d)
    out = np.empty(var_affine_bytes(K, Ga, d), dtype=np.uint8)
    _check(_load().oracle_var_pack_affine(K, Ga, d, _ptr(Ab), _ptr(Bb), _ptr(out)), "var_pack_affine")
    return out


def var_unpack_affine(block: np.ndarray, K: int, Ga: int, d: int):
    """Inverse of var_pack_affine (raises if the two views disagree)."""
    block = np.ascontiguousarray(block, dtype=np.uint8)
    assert block.size == var_affine_bytes(K, Ga, d)
    A = np.empty((Ga, d, d), dtype=np.uint16)
    B = np.empty((Ga, d), dtype=np.uint16)
    _check(_load().oracle_var_unpack_affine(K, Ga, d, _ptr(block), _ptr(A), _ptr(B)), "var_unpack_affine")
    return A.view(np.float16), B.view(np.float16)


def var_decode(Q: np.ndarray, As: np.ndarray, Bs: np.ndarray) -> np.ndarray:
    """fp64 W_hat [N][K] from canonical codes and shared pairs As [Ga][d][d], Bs [Ga][d]."""
    N, K = Q.shape
    Q = np.ascontiguousarray(Q, dtype=np.uint8)
    Ab, Bb = _bits16(As), _bits16(Bs)
    Ga, d = Ab.shape[0], Ab.shape[1]
    W = np.empty((N, K), dtype=np.float64)
    _check(_load().oracle_var_decode(N, K, d, _ptr(Q), Ga, _ptr(Ab), _ptr(Bb), _ptr(W)), "var_decode")
    return W


def var_matmul(packed_codes: np.ndarray, N: int, K: int, bits: int, As: np.ndarray, Bs: np.ndarray,
               X: np.ndarray, rows=None, threads: int | None = None):
    """Y = X * W_hat^T in fp64 from variant codes-only bytes and shared pairs."""
    packed_codes = np.ascontiguousarray(packed_codes, dtype=np.uint8)
    assert packed_codes.size == var_codes_bytes(N, K, bits)
    Ab, Bb = _bits16(As), _bits16(Bs)
    Ga, d = Ab.shape[0], Ab.shape[1]
    assert Ab.shape == (Ga, d, d) and Bb.shape == (Ga, d)
    X = np.ascontiguousarray(X, dtype=np.float64)
    if X.ndim == 1:
        X = X[None, :]
    M = X.shape[0]
    assert X.shape[1] == K
    if threads is None:
        threads = default_threads()
    lib = _load()
    if rows is None:
        Y = np.empty((M, N), dtype=np.float64)
        _check(lib.oracle_var_matmul_rows(N, K, bits, d, _ptr(packed_codes), Ga, _ptr(Ab), _ptr(Bb), M, _ptr(X),
                                          N, None, _ptr(Y), threads), "var_matmul")
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        Y = np.empty((M, r.size), dtype=np.float64)
        _check(lib.oracle_var_matmul_rows(N, K, bits, d, _ptr(packed_codes), Ga, _ptr(Ab), _ptr(Bb), M, _ptr(X),
                                          r.size, _ptr(r), _ptr(Y), threads), "var_matmul_rows")
    return Y


# ------------------------------------------------ LDLQ (Eq. 7)

def regularised(H: np.ndarray, mu: float = 0.01) -> np.ndarray:
    """H + mu I (the Tikhonov term of Sec. 4.2, mu = 0.01)."""
    return np.asarray(H, dtype=np.float64) + mu * np.eye(H.shape[0])


def ldl_blocks(H: np.ndarray, d: int = 4):
    """H = U D U^T with U unit upper block triangular (d x d identity blocks on
    the diagonal) and D block diagonal, from a Cholesky factorisation (library
    routine) of H with its index order reversed: reversed(H) = C C^T gives
    H = R R^T with R = reversed(C) upper triangular; U = R diag(R_jj)^-1 and
    D_j = R_jj R_jj^T.  Returns (U [K][K], D [K/d][d][d])."""
    H = np.asarray(H, dtype=np.float64)
    K = H.shape[0]
    C = np.linalg.cholesky(H[::-1, ::-1])
    R = C[::-1, ::-1]
    U = np.empty_like(R)
    D = np.empty((K // d, d, d))
    for j in range(K // d):
        s = slice(d * j, d * (j + 1))
        Rjj = R[s, s]
        U[:, s] = np.linalg.solve(Rjj.T, R[:, s].T).T  # R[:, s] Rjj^-1
        U[s, s] = np.eye(d)  # Rjj Rjj^-1, exactly
        D[j] = Rjj @ Rjj.T
    return np.ascontiguousarray(U), D


def ldlq(W: np.ndarray, U: np.ndarray, A: np.ndarray, B: np.ndarray, shared: bool = False, threads: int | None = None):
    """LDLQ codes (Eq. 7) of fp32 W [N][K] with the feedback factor U (fp64
    [K][K], from ldl_blocks) and pairs as for quantize().  Returns (codes uint8
    [N][K], errors W - W_hat fp64 [N][K])."""
    lib = _load()
    W = np.ascontiguousarray(W, dtype=np.float32)
    N, K = W.shape
    U = np.ascontiguousarray(U, dtype=np.float64)
    assert U.shape == (K, K)
    Ab, Bb = _bits16(A), _bits16(B)
    Ga = Ab.shape[0] if shared else 0
    Q = np.empty((N, K), dtype=np.uint8)
    E = np.empty((N, K), dtype=np.float64)
    if threads is None:
        threads = default_threads()
    _check(lib.oracle_ldlq(N, K, _ptr(W), _ptr(U), _ptr(Ab), _ptr(Bb), Ga, _ptr(Q), _ptr(E), threads), "ldlq")
    return Q, E
