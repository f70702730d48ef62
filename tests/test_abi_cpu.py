"""Host-only checks of the C ABI: the library loads, exports every function
declared in include/unisvq.h, and rejects bad arguments before any HIP call
(every call here fails validation, so no kernel is ever launched)."""
import ctypes
import os
import re

import pytest

import paper_2606_10520_amd.unisvq as u

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "unisvq.h")

pytestmark = pytest.mark.skipif(not os.path.exists(u.LIB_PATH), reason="libunisvq.so not built")

OK, EINVAL, ESHAPE, EUNSUP, EALIGN, EHIP, EWS, ESCRATCH = 0, -1, -2, -3, -4, -5, -6, -7
GOOD = 0x10000  # 16-byte aligned stand-in address; never dereferenced (validation fails first)


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(unisvq_[a-z_]+)\s*\(", text)))


def test_header_declares_the_documented_entry_points():
    assert set(header_functions()) == set(u.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(u.LIB_PATH)
    for name in header_functions():
        assert hasattr(lib, name), name


def test_version_and_status_strings():
    lib = u.load()
    assert lib.unisvq_version() == 1
    for st in (OK, EINVAL, ESHAPE, EUNSUP, EALIGN, EHIP, EWS, ESCRATCH):
        assert lib.unisvq_status_string(st)
    assert lib.unisvq_status_string(12345) == b"unknown status"


@pytest.mark.parametrize("N,K,expect", [
    (16, 128, 1152), (4096, 4096, 4096 * 4096 // 4 + 4096 * 32 * 40), (11008, 4096, 25_362_432),
    (15, 128, 0), (16, 100, 0), (0, 128, 0), (16, 0, 0), (-16, 128, 0),
])
def test_packed_bytes(N, K, expect):
    assert u.load().unisvq_packed_bytes(N, K) == expect


def test_pack_validation():
    lib = u.load()
    assert lib.unisvq_pack(16, 128, None, GOOD, GOOD, GOOD, None, None) == EINVAL
    assert lib.unisvq_pack(16, 128, GOOD, GOOD, GOOD, None, None, None) == EINVAL
    assert lib.unisvq_pack(17, 128, GOOD, GOOD, GOOD, GOOD, None, None) == ESHAPE
    assert lib.unisvq_pack(16, 130, GOOD, GOOD, GOOD, GOOD, None, None) == ESHAPE
    assert lib.unisvq_pack(16, 128, GOOD, GOOD, GOOD, GOOD + 8, None, None) == EALIGN
    assert lib.unisvq_pack(16, 128, GOOD, GOOD + 1, GOOD, GOOD, None, None) == EALIGN
    assert lib.unisvq_pack(16, 128, GOOD, GOOD, GOOD, GOOD, GOOD + 2, None) == EALIGN
    assert lib.unisvq_unpack(16, 128, None, GOOD, GOOD, GOOD, None) == EINVAL
    assert lib.unisvq_unpack(32, 64, GOOD, GOOD, GOOD, GOOD, None) == ESHAPE
    assert lib.unisvq_unpack(16, 128, GOOD + 4, GOOD, GOOD, GOOD, None) == EALIGN


@pytest.mark.parametrize("fn", ["gemv", "gemm"])
def test_product_validation(fn):
    lib = u.load()

    def call(N=64, K=256, packed=GOOD, M=1, x=GOOD, xt=u.F16, y=GOOD, yt=u.F16, ws_bytes=0):
        if fn == "gemv":
            return lib.unisvq_gemv(N, K, packed, M, x, xt, y, yt, None)
        return lib.unisvq_gemm(N, K, packed, M, x, xt, y, yt, None, ws_bytes, None)

    assert call(packed=None) == EINVAL
    assert call(x=None) == EINVAL
    assert call(y=None) == EINVAL
    assert call(M=0) == EINVAL
    assert call(M=-3) == EINVAL
    assert call(xt=u.F32) == EINVAL  # activations must be fp16 or bf16
    assert call(xt=7) == EINVAL
    assert call(yt=9) == EINVAL
    assert call(N=8) == ESHAPE
    assert call(N=40) == ESHAPE
    assert call(K=200) == ESHAPE
    assert call(K=64) == ESHAPE
    assert call(packed=GOOD + 8) == EALIGN
    assert call(x=GOOD + 2) == EALIGN
    assert call(y=GOOD + 1) == EALIGN
    assert call(y=GOOD + 2, yt=u.F32) == EALIGN
    if fn == "gemv":
        # more tokens than the matrix-vector kernel takes; checked before launch
        assert call(M=5, packed=None) == EINVAL
        assert lib.unisvq_gemv(64, 256, GOOD, 5, GOOD, u.F16, GOOD, u.F16, None) == EUNSUP


def test_batched_validation():
    lib = u.load()
    P = u.GemvProblem

    def arr(*ps):
        a = (P * len(ps))()
        for i, q in enumerate(ps):
            a[i] = q
        return a

    good = P(64, 256, GOOD, GOOD, GOOD)
    assert lib.unisvq_gemv_batched(None, 1, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_batched(arr(good), 0, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_batched(arr(*[good] * 9), 9, 1, u.F16, u.F16, None) == EUNSUP
    # any bad descriptor fails the whole call before launch
    assert lib.unisvq_gemv_batched(arr(good, P(64, 256, None, GOOD, GOOD)), 2, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_batched(arr(good, P(40, 256, GOOD, GOOD, GOOD)), 2, 1, u.F16, u.F16, None) == ESHAPE
    assert lib.unisvq_gemv_batched(arr(P(64, 256, GOOD + 4, GOOD, GOOD), good), 2, 1, u.F16, u.F16, None) == EALIGN
    assert lib.unisvq_gemv_batched(arr(good, good), 2, 0, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_batched(arr(good, good), 2, 5, u.F16, u.F16, None) == EUNSUP
    assert lib.unisvq_gemv_batched(arr(good), 1, 1, u.F32, u.F16, None) == EINVAL


def test_rht_batched_validation():
    """The fused input-transform product: descriptors as unisvq_gemv_batched,
    plus one sign vector per problem and K = 4096 or 8192 for all of them."""
    import ctypes
    lib = u.load()
    P = u.GemvProblem

    def arr(*ps):
        a = (P * len(ps))()
        for i, q in enumerate(ps):
            a[i] = q
        return a

    def sg(*ptrs):
        a = (ctypes.c_void_p * len(ptrs))()
        for i, v in enumerate(ptrs):
            a[i] = v
        return a

    good = P(64, 4096, GOOD, GOOD, GOOD)
    f = lib.unisvq_gemv_rht_batched
    assert f(None, 1, 1, u.F16, u.F16, sg(GOOD), None) == EINVAL
    assert f(arr(good), 1, 1, u.F16, u.F16, None, None) == EINVAL
    assert f(arr(good, good), 2, 1, u.F16, u.F16, sg(GOOD, None), None) == EINVAL
    assert f(arr(good), 0, 1, u.F16, u.F16, sg(GOOD), None) == EINVAL
    assert f(arr(*[good] * 9), 9, 1, u.F16, u.F16, sg(*[GOOD] * 9), None) == EUNSUP
    assert f(arr(P(64, 11008 // 128 * 128, GOOD, GOOD, GOOD)), 1, 1, u.F16, u.F16, sg(GOOD), None) == EUNSUP
    assert f(arr(P(64, 2048, GOOD, GOOD, GOOD)), 1, 1, u.F16, u.F16, sg(GOOD), None) == EUNSUP
    assert f(arr(good, P(64, 8192, GOOD, GOOD, GOOD)), 2, 1, u.F16, u.F16, sg(GOOD, GOOD), None) == EUNSUP
    assert f(arr(good), 1, 5, u.F16, u.F16, sg(GOOD), None) == EUNSUP
    assert f(arr(P(40, 4096, GOOD, GOOD, GOOD)), 1, 1, u.F16, u.F16, sg(GOOD), None) == ESHAPE
    assert f(arr(P(64, 4096, GOOD + 4, GOOD, GOOD)), 1, 1, u.F16, u.F16, sg(GOOD), None) == EALIGN
    assert f(arr(good), 1, 1, u.F32, u.F16, sg(GOOD), None) == EINVAL


def test_gemm_workspace():
    lib = u.load()
    ws = lib.unisvq_gemm_workspace_bytes
    # bf16: fp16 copy of the activations plus one fp32 scale per token (each rounded up to 256 B);
    # M = 2048 fills the GPU with output tiles, so there is no split along K
    assert ws(4096, 4096, 2048, u.BF16) == 2048 * 4096 * 2 + 2048 * 4
    assert ws(4096, 4096, 2048, u.F16) == 0
    # above 16 tokens the size covers the tiled fp16 copy (16-token tiles): 33 tokens take 48 rows,
    # 17 take 32; up to 16 the row-major copy of the small-batch kernel
    assert ws(64, 256, 33, u.BF16) == 48 * 256 * 2 + 256
    assert ws(64, 256, 32, u.BF16) == 32 * 256 * 2 + 256
    assert ws(64, 256, 17, u.BF16) == 32 * 256 * 2 + 256
    assert ws(64, 256, 15, u.BF16) == 15 * 256 * 2 + 256
    assert ws(16, 128, 1, u.BF16) == 256 + 256
    assert ws(16, 128, 1, u.F16) == 0
    assert ws(15, 128, 1, u.BF16) == 0
    assert ws(16, 128, 0, u.BF16) == 0
    assert ws(16, 128, 1, u.F32) == 0
    # up to 16 tokens the small-batch kernel needs nothing; from 17 to 32 the
    # size also covers the tiled product (the launch's width picks the kernel);
    # a product with few output tiles is split along K: fp32 partials for every split
    assert ws(64, 1024, 16, u.F16) == 0
    for m in (17, 32, 33):
        assert ws(64, 1024, m, u.F16) > 0 and ws(64, 1024, m, u.F16) % (m * 64 * 4) == 0
    split = ws(64, 1024, 100, u.F16)
    assert split > 0 and split % (100 * 64 * 4) == 0
    # (the bf16 pre-pass's fp16 copy for the tiled kernel: 100 tokens padded to 112)
    assert ws(64, 1024, 100, u.BF16) == split + 112 * 1024 * 2 + 512
    # bf16 activations need it; so does a split product with fp16 activations
    need = ws(64, 256, 4, u.BF16)
    assert lib.unisvq_gemm(64, 256, GOOD, 4, GOOD, u.BF16, GOOD, u.F16, None, need, None) == EWS
    assert lib.unisvq_gemm(64, 256, GOOD, 4, GOOD, u.BF16, GOOD, u.F16, GOOD, need - 1, None) == EWS
    assert lib.unisvq_gemm(64, 256, GOOD, 4, GOOD, u.BF16, GOOD, u.F16, GOOD + 8, need, None) == EALIGN
    assert lib.unisvq_gemm(64, 1024, GOOD, 100, GOOD, u.F16, GOOD, u.F16, None, 0, None) == EWS
    # bf16 activations: K up to 65536
    assert lib.unisvq_gemm(16, 65664, GOOD, 4, GOOD, u.BF16, GOOD, u.F16, GOOD, 1 << 30, None) == EUNSUP


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(u, "_lib", None)
    monkeypatch.setattr(u, "LIB_PATH", str(tmp_path / "libunisvq.so"))
    with pytest.raises(u.UniSVQLibraryMissing):
        u.load()


# ------------------------------------------------ row-shared affine parameters

@pytest.mark.parametrize("N,K,expect", [(16, 128, 512), (4096, 4096, 4096 * 4096 // 4), (11008, 4096, 11_272_192),
                                        (15, 128, 0), (16, 100, 0), (0, 128, 0)])
def test_codes_bytes(N, K, expect):
    assert u.load().unisvq_codes_bytes(N, K) == expect


@pytest.mark.parametrize("K,ga,expect", [(128, 1, 80), (128, 1, 80), (4096, 1, 80), (4096, 32, 16 * 80),
                                         (384, 3, 2 * 80), (11008, 86, 43 * 80), (4096, 2, 0), (4096, 0, 0),
                                         (100, 1, 0), (0, 1, 0)])
def test_shared_affine_bytes(K, ga, expect):
    assert u.load().unisvq_shared_affine_bytes(K, ga) == expect


def test_pack_shared_validation():
    lib = u.load()
    assert lib.unisvq_pack_shared(16, 256, 1, None, GOOD, GOOD, GOOD, GOOD, None, None) == EINVAL
    assert lib.unisvq_pack_shared(16, 256, 1, GOOD, GOOD, GOOD, GOOD, None, None, None) == EINVAL
    assert lib.unisvq_pack_shared(16, 256, 3, GOOD, GOOD, GOOD, GOOD, GOOD, None, None) == EINVAL
    assert lib.unisvq_pack_shared(17, 256, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None, None) == ESHAPE
    assert lib.unisvq_pack_shared(16, 256, 2, GOOD, GOOD, GOOD, GOOD + 8, GOOD, None, None) == EALIGN
    assert lib.unisvq_pack_shared(16, 256, 2, GOOD, GOOD, GOOD, GOOD, GOOD + 4, None, None) == EALIGN
    assert lib.unisvq_unpack_shared(16, 256, 5, GOOD, GOOD, GOOD, GOOD, GOOD, None) == EINVAL
    assert lib.unisvq_unpack_shared(16, 250, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None) == ESHAPE
    assert lib.unisvq_unpack_shared(16, 256, 1, GOOD, GOOD + 2, GOOD, GOOD, GOOD, None) == EALIGN


@pytest.mark.parametrize("fn", ["gemv", "gemm"])
def test_shared_product_validation(fn):
    lib = u.load()

    def call(N=64, K=256, ga=1, pc=GOOD, pa=GOOD, M=1, x=GOOD, xt=u.F16, y=GOOD, yt=u.F16, ws_bytes=0):
        if fn == "gemv":
            return lib.unisvq_gemv_shared(N, K, ga, pc, pa, M, x, xt, y, yt, None)
        return lib.unisvq_gemm_shared(N, K, ga, pc, pa, M, x, xt, y, yt, None, ws_bytes, None)

    assert call(pc=None) == EINVAL
    assert call(pa=None) == EINVAL
    assert call(x=None) == EINVAL
    assert call(M=0) == EINVAL
    assert call(ga=3) == EINVAL
    assert call(ga=0) == EINVAL
    assert call(xt=u.F32) == EINVAL
    assert call(N=60) == ESHAPE
    assert call(K=200) == ESHAPE
    assert call(pc=GOOD + 8) == EALIGN
    assert call(pa=GOOD + 8) == EALIGN
    assert call(y=GOOD + 1) == EALIGN
    if fn == "gemv":
        assert call(M=5) == EUNSUP
    else:
        # bf16 activations need the workspace; none given
        assert call(xt=u.BF16, M=64) == EWS
        assert call(xt=u.BF16, K=65664, M=64) == EUNSUP


def test_shared_batched_validation():
    lib = u.load()
    arr = (u.GemvSharedProblem * 2)()
    arr[0] = u.GemvSharedProblem(64, 256, 1, GOOD, GOOD, GOOD, GOOD)
    arr[1] = u.GemvSharedProblem(64, 256, 5, GOOD, GOOD, GOOD, GOOD)
    assert lib.unisvq_gemv_shared_batched(arr, 2, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_shared_batched(arr, 0, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_shared_batched(None, 1, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_gemv_shared_batched(arr, 9, 1, u.F16, u.F16, None) == EUNSUP


def test_quantize_validation():
    lib = u.load()
    assert lib.unisvq_quantize(16, 128, None, GOOD, GOOD, 0, GOOD, None) == EINVAL
    assert lib.unisvq_quantize(16, 128, GOOD, GOOD, GOOD, 0, None, None) == EINVAL
    assert lib.unisvq_quantize(16, 256, GOOD, GOOD, GOOD, 3, GOOD, None) == EINVAL
    assert lib.unisvq_quantize(15, 128, GOOD, GOOD, GOOD, 0, GOOD, None) == ESHAPE
    assert lib.unisvq_quantize(16, 120, GOOD, GOOD, GOOD, 1, GOOD, None) == ESHAPE
    assert lib.unisvq_quantize(16, 128, GOOD + 4, GOOD, GOOD, 0, GOOD, None) == EALIGN
    assert lib.unisvq_quantize(16, 128, GOOD, GOOD + 1, GOOD, 0, GOOD, None) == EALIGN
    assert lib.unisvq_quantize(16, 128, GOOD, GOOD, GOOD, 0, GOOD + 2, None) == EALIGN


def test_rht_validation():
    lib = u.load()
    assert lib.unisvq_rht(4096, 1, None, u.F16, GOOD, 0, GOOD + 0x100000, u.F16, None) == EINVAL
    assert lib.unisvq_rht(4096, 1, GOOD, u.F16, None, 0, GOOD + 0x100000, u.F16, None) == EINVAL
    assert lib.unisvq_rht(4096, 0, GOOD, u.F16, GOOD, 0, GOOD + 0x100000, u.F16, None) == EINVAL
    assert lib.unisvq_rht(4096, 1, GOOD, u.F16, GOOD, 2, GOOD + 0x100000, u.F16, None) == EINVAL
    assert lib.unisvq_rht(4096, 1, GOOD, 7, GOOD, 0, GOOD + 0x100000, u.F16, None) == EINVAL
    assert lib.unisvq_rht(4096, 1, GOOD, u.F16, GOOD, 0, GOOD + 1000, u.F16, None) == EINVAL  # overlap
    assert lib.unisvq_rht(4096, 1, GOOD + 1, u.F16, GOOD, 0, GOOD + 0x100000, u.F16, None) == EALIGN
    assert lib.unisvq_rht(4096, 1, GOOD, u.F16, GOOD, 0, GOOD + 0x100002, u.F32, None) == EALIGN
    # orders without a supported construction, or beyond the LDS row
    assert lib.unisvq_rht(100, 1, GOOD, u.F16, GOOD, 0, GOOD + 0x100000, u.F16, None) == EUNSUP
    assert lib.unisvq_rht(65536, 1, GOOD, u.F16, GOOD, 0, GOOD + 0x100000, u.F16, None) == EUNSUP


# ---- format variants (b-bit codes, d-dimensional vectors) ----

@pytest.mark.parametrize("bits,d,N,K,expect", [
    (3, 4, 16, 128, 768), (2, 8, 16, 128, 512), (3, 8, 4096, 4096, 4096 * 4096 * 3 // 8),
    (2, 4, 16, 128, 0), (4, 4, 16, 128, 0), (3, 6, 16, 128, 0), (3, 8, 15, 128, 0), (3, 8, 16, 100, 0)])
def test_var_codes_bytes(bits, d, N, K, expect):
    assert u.load().unisvq_var_codes_bytes(N, K, bits, d) == expect


@pytest.mark.parametrize("bits,d,K,ga,expect", [
    (3, 4, 128, 1, 160), (3, 4, 384, 3, 320), (2, 8, 4096, 1, 576), (2, 8, 11008, 86, 43 * 576),
    (3, 8, 4096, 32, 16 * 576), (2, 4, 4096, 1, 0), (3, 8, 4096, 2, 0), (3, 8, 100, 1, 0)])
def test_var_affine_bytes(bits, d, K, ga, expect):
    assert u.load().unisvq_var_affine_bytes(K, ga, bits, d) == expect


def test_var_pack_validation():
    lib = u.load()
    assert lib.unisvq_var_pack(16, 256, 3, 8, 1, None, GOOD, GOOD, GOOD, GOOD, None, None) == EINVAL
    assert lib.unisvq_var_pack(16, 256, 2, 4, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None, None) == EUNSUP
    assert lib.unisvq_var_pack(16, 256, 4, 8, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None, None) == EUNSUP
    assert lib.unisvq_var_pack(16, 256, 3, 8, 3, GOOD, GOOD, GOOD, GOOD, GOOD, None, None) == EINVAL
    assert lib.unisvq_var_pack(17, 256, 3, 8, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None, None) == ESHAPE
    assert lib.unisvq_var_pack(16, 256, 3, 8, 2, GOOD, GOOD, GOOD, GOOD + 8, GOOD, None, None) == EALIGN
    assert lib.unisvq_var_pack(16, 256, 3, 8, 2, GOOD, GOOD, GOOD, GOOD, GOOD + 4, None, None) == EALIGN
    assert lib.unisvq_var_unpack(16, 256, 3, 4, 5, GOOD, GOOD, GOOD, GOOD, GOOD, None) == EINVAL
    assert lib.unisvq_var_unpack(16, 250, 3, 4, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None) == ESHAPE
    assert lib.unisvq_var_unpack(16, 256, 2, 4, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None) == EUNSUP
    assert lib.unisvq_var_unpack(16, 256, 3, 4, 1, GOOD, GOOD + 2, GOOD, GOOD, GOOD, None) == EALIGN


@pytest.mark.parametrize("fn", ["gemv", "gemm"])
def test_var_product_validation(fn):
    lib = u.load()

    def call(N=64, K=256, bits=3, d=8, ga=1, pc=GOOD, pa=GOOD, M=1, x=GOOD, xt=u.F16, y=GOOD, yt=u.F16,
             ws_bytes=0):
        if fn == "gemv":
            return lib.unisvq_var_gemv(N, K, bits, d, ga, pc, pa, M, x, xt, y, yt, None)
        return lib.unisvq_var_gemm(N, K, bits, d, ga, pc, pa, M, x, xt, y, yt, None, ws_bytes, None)

    assert call(pc=None) == EINVAL
    assert call(pa=None) == EINVAL
    assert call(M=0) == EINVAL
    assert call(ga=3) == EINVAL
    assert call(xt=u.F32) == EINVAL
    assert call(bits=2, d=4) == EUNSUP
    assert call(bits=1) == EUNSUP
    assert call(d=16) == EUNSUP
    assert call(N=60) == ESHAPE
    assert call(K=200) == ESHAPE
    assert call(pc=GOOD + 8) == EALIGN
    assert call(pa=GOOD + 8) == EALIGN
    assert call(y=GOOD + 1) == EALIGN
    if fn == "gemv":
        assert call(M=5) == EUNSUP
    else:
        assert call(xt=u.BF16, M=64) == EWS
        assert call(xt=u.BF16, K=65664, M=64) == EUNSUP
        # every M goes to the tiled kernel: a small product splits K and needs partials
        assert call(M=8, K=4096) == EWS


def test_var_batched_validation():
    lib = u.load()
    arr = (u.GemvSharedProblem * 2)()
    arr[0] = u.GemvSharedProblem(64, 256, 1, GOOD, GOOD, GOOD, GOOD)
    arr[1] = u.GemvSharedProblem(64, 256, 5, GOOD, GOOD, GOOD, GOOD)
    assert lib.unisvq_var_gemv_batched(arr, 2, 3, 8, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_var_gemv_batched(arr, 1, 2, 4, 1, u.F16, u.F16, None) == EUNSUP
    assert lib.unisvq_var_gemv_batched(arr, 0, 3, 8, 1, u.F16, u.F16, None) == EINVAL
    assert lib.unisvq_var_gemv_batched(arr, 9, 3, 8, 1, u.F16, u.F16, None) == EUNSUP


def test_var_gemm_workspace():
    lib = u.load()
    # bf16 copy of x plus per-token scales, and K-split partials when the tiles cannot fill the GPU
    assert lib.unisvq_var_gemm_workspace_bytes(4096, 4096, 2048, u.F16) == 0
    assert lib.unisvq_var_gemm_workspace_bytes(4096, 4096, 2048, u.BF16) == 2048 * 4096 * 2 + 2048 * 4
    assert lib.unisvq_var_gemm_workspace_bytes(4096, 4096, 16, u.F16) > 0
    assert lib.unisvq_var_gemm_workspace_bytes(4096, 100, 16, u.F16) == 0


def test_ldlq_validation():
    lib = u.load()
    need = lib.unisvq_ldlq_workspace_bytes(16, 256)
    assert need == 16 * 256 * 8 + 16 * 128 * 8
    assert lib.unisvq_ldlq_workspace_bytes(15, 256) == 0
    assert lib.unisvq_ldlq(16, 256, None, GOOD, GOOD, GOOD, 0, GOOD, GOOD, need, None) == EINVAL
    assert lib.unisvq_ldlq(16, 256, GOOD, None, GOOD, GOOD, 0, GOOD, GOOD, need, None) == EINVAL
    assert lib.unisvq_ldlq(16, 256, GOOD, GOOD, GOOD, GOOD, 3, GOOD, GOOD, need, None) == EINVAL
    assert lib.unisvq_ldlq(16, 200, GOOD, GOOD, GOOD, GOOD, 0, GOOD, GOOD, need, None) == ESHAPE
    assert lib.unisvq_ldlq(16, 256, GOOD + 4, GOOD, GOOD, GOOD, 0, GOOD, GOOD, need, None) == EALIGN
    assert lib.unisvq_ldlq(16, 256, GOOD, GOOD + 8, GOOD, GOOD, 0, GOOD, GOOD, need, None) == EALIGN
    assert lib.unisvq_ldlq(16, 256, GOOD, GOOD, GOOD, GOOD, 0, GOOD + 2, GOOD, need, None) == EALIGN
    assert lib.unisvq_ldlq(16, 256, GOOD, GOOD, GOOD, GOOD, 0, GOOD, None, need, None) == EWS
    assert lib.unisvq_ldlq(16, 256, GOOD, GOOD, GOOD, GOOD, 0, GOOD, GOOD, need - 8, None) == EWS
    assert lib.unisvq_ldlq(16, 256, GOOD, GOOD, GOOD, GOOD, 0, GOOD, GOOD + 8, need, None) == EALIGN


def test_ldl_validation():
    lib = u.load()
    K = 256
    need = lib.unisvq_ldl_workspace_bytes(K)
    assert need == K * 64 * 8 + 256 * 8
    for bad in (0, 64, 200, 32768 + 128):
        assert lib.unisvq_ldl_workspace_bytes(bad) == 0
    H = GOOD
    U = H + K * K * 8
    D = U + K * K * 8
    info = D + K * 4 * 8
    ws = info + 256

    def call(K=K, H=H, U=U, D=D, info=info, ws=ws, wb=need):
        return lib.unisvq_ldl(K, H, U, D, info, ws, wb, None)

    assert call(H=None) == EINVAL
    assert call(U=None) == EINVAL
    for bad in (0, 64, 200, 32768 + 128):
        assert call(K=bad) == ESHAPE
    assert call(H=H + 8) == EALIGN
    assert call(U=U + 8) == EALIGN
    assert call(D=D + 4) == EALIGN
    assert call(info=info + 2) == EALIGN
    assert call(U=H + 128) == EINVAL  # overlaps H without being H
    assert call(D=H + 64) == EINVAL
    assert call(D=U + K * K * 8 - 8) == EINVAL
    assert call(info=U + 4) == EINVAL
    assert call(ws=None) == EWS
    assert call(wb=need - 8) == EWS
    assert call(ws=ws + 8) == EALIGN


def test_fold_workspace_and_validation():
    lib = u.load()
    ws = lib.unisvq_gemm_fold_workspace_bytes
    # M = 2048 at 4096 x 4096: no K split; tiled copy + scales + bias terms
    assert ws(4096, 4096, 2048) == 2048 * 4096 * 2 + 2 * 2048 * 4
    # 33 tokens take 48 rows of the tiled copy; the small product splits K
    small = ws(64, 1024, 33)
    assert small > 48 * 1024 * 2 + 2 * 256 and (small - 48 * 1024 * 2 - 2 * 256) % (33 * 64 * 4) == 0
    assert ws(60, 1024, 1) == 0 and ws(64, 1000, 1) == 0 and ws(64, 1024, 0) == 0

    def call(N=64, K=256, ga=1, M=4, xt=u.F16, wsp=GOOD, ws_bytes=1 << 20):
        return lib.unisvq_gemm_shared_fold(N, K, ga, GOOD, GOOD, M, GOOD, xt, GOOD, u.F16, wsp, ws_bytes, None)

    assert call(M=0) == EINVAL
    assert call(ga=3) == EINVAL
    assert call(xt=u.F32) == EINVAL
    assert call(N=60) == ESHAPE
    assert call(K=200) == ESHAPE
    assert call(wsp=None) == EWS
    assert call(ws_bytes=ws(64, 256, 4) - 1) == EWS
    assert call(wsp=GOOD + 4) == EALIGN


def test_binding_checks_buffers_against_the_shape():
    """The kernels take their address ranges from N, K and M, so the binding
    rejects short, strided or mistyped tensors before any call (checked with
    host tensors: the helpers look only at shape, dtype and layout)."""
    torch = pytest.importorskip("torch")
    N, K = 32, 256
    need = u.packed_bytes(N, K)
    u._need_buffer(torch.empty(need, dtype=torch.uint8), need, "packed", exact=True)
    with pytest.raises(ValueError):
        u._need_buffer(torch.empty(need - 1, dtype=torch.uint8), need, "packed", exact=True)
    with pytest.raises(ValueError):
        u._need_buffer(torch.empty(need + 16, dtype=torch.uint8), need, "packed", exact=True)
    with pytest.raises(ValueError):
        u._need_buffer(torch.empty(2 * need, dtype=torch.uint8)[::2], need, "packed")
    with pytest.raises(ValueError):
        u._need_buffer(None, need, "workspace")
    # activations: K columns, contiguous, fp16/bf16
    assert u._activations(torch.empty(3, K, dtype=torch.float16), K).shape == (3, K)
    assert u._activations(torch.empty(2 * K, dtype=torch.bfloat16), K).shape == (2, K)
    for bad in (torch.empty(3, K + 128, dtype=torch.float16), torch.empty(K + 1, dtype=torch.float16),
                torch.empty(K, 3, dtype=torch.float16).t()):
        with pytest.raises(ValueError):
            u._activations(bad, K)
    with pytest.raises(TypeError):
        u._activations(torch.empty(1, K, dtype=torch.float32), K)
    # outputs: M*N elements, contiguous, fp16/bf16/fp32
    like = torch.empty(1, K, dtype=torch.float16)
    assert u._output(None, 3, N, None, like).shape == (3, N)
    assert u._output(torch.empty(3 * N, dtype=torch.float32), 3, N, None, like).numel() == 3 * N
    with pytest.raises(ValueError):
        u._output(torch.empty(3 * N - 1, dtype=torch.float16), 3, N, None, like)
    with pytest.raises(ValueError):
        u._output(torch.empty(N, 3, dtype=torch.float16).t(), 3, N, None, like)
    with pytest.raises(TypeError):
        u._output(torch.empty(3 * N, dtype=torch.int32), 3, N, None, like)
    # canonical codes and pairs
    q = torch.zeros(N, K, dtype=torch.uint8)
    u._canonical(q, torch.zeros(N, 2, 4, 4, dtype=torch.float16), torch.zeros(N, 2, 4, dtype=torch.float16),
                 N, K, N * 2)
    with pytest.raises(ValueError):
        u._canonical(q, torch.zeros(N, 2, 4, 4, dtype=torch.float16), torch.zeros(N, 1, 4, dtype=torch.float16),
                     N, K, N * 2)


def test_read_bytes_validation():
    lib = u.load()
    R = u.ByteRange
    one = (R * 1)(R(GOOD, 4096))
    two = (R * 2)(R(GOOD, 32768 * 3), R(GOOD, 16))
    assert lib.unisvq_read_sink_words(one, 1) == 2
    assert lib.unisvq_read_sink_words(two, 2) == 2 * 13
    assert lib.unisvq_read_bytes(None, 1, 1, GOOD, 8, None) == EINVAL
    assert lib.unisvq_read_bytes(one, 0, 1, GOOD, 8, None) == EINVAL
    assert lib.unisvq_read_bytes(one, 1, 1, None, 8, None) == EINVAL
    assert lib.unisvq_read_bytes(one, 9, 1, GOOD, 8, None) == EUNSUP
    assert lib.unisvq_read_bytes(one, 1, 1, GOOD + 2, 8, None) == EALIGN
    assert lib.unisvq_read_bytes(two, 2, 1, GOOD, 25, None) == EWS
    for st in (0, 1):
        for bad in (R(GOOD, 4100), R(GOOD, -16), R(None, 4096), R(GOOD, 2 ** 31)):
            assert lib.unisvq_read_bytes((R * 1)(bad), 1, st, GOOD, 8, None) == EINVAL
        assert lib.unisvq_read_bytes((R * 1)(R(GOOD + 8, 4096)), 1, st, GOOD, 8, None) == EALIGN


def test_gemm_noalloc_validation():
    """The no-allocation product checks its arguments like unisvq_gemm and
    refuses, before any HIP call, a product whose workspace exceeds the fixed
    scratch."""
    lib = u.load()
    cap = lib.unisvq_noalloc_scratch_bytes()
    assert cap == 32 << 20
    f = lib.unisvq_gemm_noalloc
    assert f(64, 256, None, 4, GOOD, u.F16, GOOD, u.F16, None) == EINVAL
    assert f(64, 256, GOOD, 0, GOOD, u.F16, GOOD, u.F16, None) == EINVAL
    assert f(60, 256, GOOD, 4, GOOD, u.F16, GOOD, u.F16, None) == ESHAPE
    assert f(64, 256, GOOD + 8, 4, GOOD, u.F16, GOOD, u.F16, None) == EALIGN
    assert f(64, 256, GOOD, 4, GOOD, 7, GOOD, u.F16, None) == EINVAL
    assert f(64, 70016, GOOD, 4, GOOD, u.BF16, GOOD, u.F16, None) == EUNSUP
    # bf16 activations: the fp16 copy alone (1024 x 16384 x 2 bytes) exceeds 32 MiB
    assert lib.unisvq_gemm_workspace_bytes(4096, 16384, 1024, u.BF16) > cap
    assert f(4096, 16384, GOOD, 1024, GOOD, u.BF16, GOOD, u.F16, None) == ESCRATCH
    assert lib.unisvq_status_string(ESCRATCH).startswith(b"product needs more")


def test_gemm_batched_validation():
    lib = u.load()
    P = u.GemvProblem
    two = (P * 2)(P(4096, 4096, GOOD, GOOD, GOOD), P(1024, 4096, GOOD, GOOD, GOOD))
    f = lib.unisvq_gemm_batched
    assert f(None, 1, 16, u.F16, u.F16, None, 0, None) == EINVAL
    assert f(two, 0, 16, u.F16, u.F16, None, 0, None) == EINVAL
    assert f(two, 9, 16, u.F16, u.F16, None, 0, None) == EUNSUP
    assert f(two, 2, 0, u.F16, u.F16, None, 0, None) == EINVAL
    bad = (P * 2)(P(4096, 4096, GOOD, GOOD, GOOD), P(1000, 4096, GOOD, GOOD, GOOD))
    assert f(bad, 2, 16, u.F16, u.F16, None, 0, None) == ESHAPE
    mis = (P * 2)(P(4096, 4096, GOOD, GOOD, GOOD), P(1024, 4096, GOOD, GOOD + 8, GOOD))
    assert f(mis, 2, 16, u.F16, u.F16, None, 0, None) == EALIGN
    # fp16 activations at <= 32 tokens need no workspace; bf16 needs one slice per problem
    assert lib.unisvq_gemm_batched_workspace_bytes(two, 2, 16, u.F16) == 0
    need = lib.unisvq_gemm_batched_workspace_bytes(two, 2, 16, u.BF16)
    singles = [lib.unisvq_gemm_workspace_bytes(N, 4096, 16, u.BF16) for N in (4096, 1024)]
    assert need == sum(-(-s // 256) * 256 for s in singles) > 0
    assert f(two, 2, 16, u.BF16, u.F16, None, need, None) == EWS
    assert f(two, 2, 16, u.BF16, u.F16, GOOD, need - 1, None) == EWS
    assert f(two, 2, 16, u.BF16, u.F16, GOOD + 8, need, None) == EALIGN
    assert lib.unisvq_gemm_batched_workspace_bytes(two, 2, 16, 9) == 0
