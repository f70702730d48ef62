"""GPU parity of the Eq. 9 fold for row-shared pairs (unisvq_gemm_shared_fold)
against the fp64 oracle, which decodes every weight and multiplies plainly."""
import numpy as np
import pytest

import oracle
from paper_2606_10520_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"
u = None


@pytest.fixture(scope="module", autouse=True)
def lib():
    global u
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_10520_amd.unisvq as mod
    mod.load()  # raises if the library is missing: no fallback
    u = mod
    yield mod


def half_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(DEV)


def x_dev(bits, dtype):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.float16 if dtype == "f16" else torch.bfloat16).to(DEV)


def x_f64(bits, dtype):
    return oracle.half_to_double(bits) if dtype == "f16" else oracle.bf16_to_double(bits)


def rel_err(y, ref):
    return float(np.abs(y.astype(np.float64) - ref).max() / max(np.abs(ref).max(), 1e-300))


def run(N, K, M, Ga, dtype, seed, out=torch.float32, x_bits=None):
    Q, A, B = wl.gen_shared_weights(N, K, Ga, seed=seed)
    xb = wl.gen_activations(M, K, seed=wl.activation_seed(seed, M), dtype=dtype) if x_bits is None else x_bits
    pc, pa = u.pack_shared(torch.from_numpy(Q).to(DEV), half_dev(A), half_dev(B))
    y = u.gemm_shared_fold(pc, pa, N, K, Ga, x_dev(xb, dtype), out_dtype=out)
    torch.cuda.synchronize()
    return y, (Q, A, B), xb


# ragged M (not a multiple of 16), small M (K split, partial sums), odd group
# counts (half packets), both pair granularities and activation types
@pytest.mark.parametrize("N,K,M", [(16, 128, 1), (64, 384, 5), (64, 256, 33), (80, 640, 64), (128, 1152, 130),
                                   (256, 4096, 7), (96, 512, 300), (64, 6144, 40)])
@pytest.mark.parametrize("per_group", [False, True])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_fold_parity(N, K, M, per_group, dtype):
    Ga = K // 128 if per_group else 1
    y, (Q, A, B), xb = run(N, K, M, Ga, dtype, seed=N + M + 3)
    ref = oracle.matmul_shared(oracle.pack_codes(Q)[0], N, K, A, B, x_f64(xb, dtype))
    assert rel_err(y.cpu().numpy(), ref) <= 5e-4


def test_fold_extreme_token_scales():
    """Tokens far outside the fp16 range (and far below it): x' = A^T x is
    scaled per token before its fp16 rounding, so every token keeps full
    accuracy relative to its own output magnitude."""
    N, K, M = 64, 512, 6
    xb = wl.gen_activations(M, K, seed=33, dtype="bf16")
    x = x_f64(xb, "bf16")
    for t, s in enumerate([1.0, 2.0 ** 40, 2.0 ** -40, 2.0 ** 100, 2.0 ** -100, 3.0e4]):
        x[t] *= s
    xb = wl.f64_to_bf16_bits(x)
    y, (Q, A, B), _ = run(N, K, M, K // 128, "bf16", seed=34, x_bits=xb)
    ref = oracle.matmul_shared(oracle.pack_codes(Q)[0], N, K, A, B, x_f64(xb, "bf16"))
    yy = y.cpu().numpy().astype(np.float64)
    for t in range(M):
        assert np.isfinite(yy[t]).all(), t
        assert np.abs(yy[t] - ref[t]).max() <= 5e-4 * np.abs(ref[t]).max(), t


def test_fold_deterministic_and_close_to_decode_path():
    """Reruns are bit-identical (fixed summation orders, K split included);
    the decode path (unisvq_gemm_shared) agrees within the rounding of both."""
    N, K, M, Ga = 256, 2048, 48, 1
    Q, A, B = wl.gen_shared_weights(N, K, Ga, seed=35)
    xb = wl.gen_activations(M, K, seed=36, dtype="f16")
    pc, pa = u.pack_shared(torch.from_numpy(Q).to(DEV), half_dev(A), half_dev(B))
    x = x_dev(xb, "f16")
    y1 = u.gemm_shared_fold(pc, pa, N, K, Ga, x, out_dtype=torch.float32)
    y2 = u.gemm_shared_fold(pc, pa, N, K, Ga, x, out_dtype=torch.float32)
    yd = u.gemm_shared(pc, pa, N, K, Ga, x, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert rel_err(y1.cpu().numpy(), yd.cpu().numpy().astype(np.float64)) <= 1e-3
