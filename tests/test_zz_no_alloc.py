"""The no-allocation product (unisvq_gemm_noalloc), called through the C ABI,
gives what unisvq_gemm gives with a caller workspace -- the same kernels and
summation order, so bit for bit -- on two calls in a row, the second with a
smaller input (the scratch keeps the first call's contents)."""
import ctypes

import numpy as np
import pytest

from paper_2606_10520_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_10520_amd.unisvq as u
    u.load()  # raises if the library is missing: no fallback
    return u


def half_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(DEV)


def packed_layer(u, N, K, seed):
    Q, A, B = wl.gen_weights(N, K, seed=seed)
    pk = u.pack(torch.from_numpy(Q).to(DEV), half_dev(A), half_dev(B))
    torch.cuda.synchronize()
    return pk


def call_noalloc(u, pk, N, K, x, y):
    stream = torch.cuda.current_stream().cuda_stream
    st = u.load().unisvq_gemm_noalloc(N, K, ctypes.c_void_p(pk.data_ptr()), x.shape[0], ctypes.c_void_p(x.data_ptr()),
                                      u.BF16 if x.dtype == torch.bfloat16 else u.F16, ctypes.c_void_p(y.data_ptr()),
                                      u.F32 if y.dtype == torch.float32 else u.F16, ctypes.c_void_p(stream))
    assert st == 0, u.STATUS.get(st, st)


# (first call, second smaller call): bf16 activations use the scratch for the
# fp16 copy (tiled above 32 tokens) and, at few tokens, the K-split partials;
# fp16 activations at 80 tokens only for the partials
@pytest.mark.parametrize("dtype,first,second", [
    ("bf16", (4096, 4096, 300), (1024, 4096, 70)),
    ("f16", (4096, 11008, 80), (2048, 4096, 70)),
    ("bf16", (11008, 4096, 64), (4096, 4096, 16)),
])
def test_noalloc_equals_workspace_path(lib, dtype, first, second):
    u = lib
    for i, (N, K, M) in enumerate((first, second)):
        assert u.gemm_workspace_bytes(N, K, M, torch.bfloat16 if dtype == "bf16" else torch.float16) \
            <= u.noalloc_scratch_bytes()
        pk = packed_layer(u, N, K, seed=100 + i)
        xb = wl.gen_activations(M, K, seed=200 + i, dtype=dtype)
        x = torch.from_numpy(xb.view(np.int16)).view(torch.bfloat16 if dtype == "bf16" else torch.float16).to(DEV)
        ref = u.gemm(pk, N, K, x, out_dtype=torch.float32)
        y = torch.full((M, N), 12345.0, dtype=torch.float32, device=DEV)
        call_noalloc(u, pk, N, K, x, y)
        y16 = torch.empty((M, N), dtype=torch.float16, device=DEV)
        call_noalloc(u, pk, N, K, x, y16)
        torch.cuda.synchronize()
        assert torch.equal(y, ref), (N, K, M)
        assert torch.equal(y16, ref.to(torch.float16)), (N, K, M)


def test_noalloc_rejects_products_beyond_the_scratch(lib):
    u = lib
    N, K, M = 4096, 16384, 1024
    pk = torch.zeros(u.packed_bytes(N, K), dtype=torch.uint8, device=DEV)
    x = torch.zeros((M, K), dtype=torch.bfloat16, device=DEV)
    y = torch.zeros((M, N), dtype=torch.float16, device=DEV)
    with pytest.raises(u.UniSVQError) as e:
        u.gemm_noalloc(pk, N, K, x, out=y)
    assert e.value.status == -7
