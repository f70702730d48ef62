"""Full-tensor GPU parity at every configured workload shape.

Each test runs the product path the benchmark times for one configured shape
and compares EVERY output element with the fp64 oracle (threaded, row-streamed
C; about 7 GMAC/s on eight host threads, so the largest prefill layer,
2048 x 11008 x 4096, takes 10-15 s).  Distinct shapes only: q/k/v/o share
4096 x 4096 and gate/up share 11008 x 4096 (7B); 8192 x 8192 serves q and o,
1024 x 8192 k and v, 28672 x 8192 gate and up (70B).  Bars: 2e-3 of max|y|
for fp16 outputs (the stated bar); for fp32 outputs 1e-5 on the matrix-vector
kernel (exact products, fp32 sums) and 5e-4 on the tiled kernels (one fp16
rounding of each decoded weight, or of x' in the fold).
"""
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


def shape_id(layer):
    return f"{layer.N}x{layer.K}"


SHAPES_7B = [wl.LLAMA7B[0], wl.LLAMA7B[4], wl.LLAMA7B[6]]          # 4096^2, 11008x4096, 4096x11008
SHAPES_70B = [wl.LLAMA70B[0], wl.LLAMA70B[1], wl.LLAMA70B[4], wl.LLAMA70B[6]]  # 8192^2, 1024x8192, 28672x8192, 8192x28672


def full_format_case(layer, M, dtype, seed, outliers):
    Q, A, B = wl.gen_weights(layer.N, layer.K, seed=seed)
    xb = wl.gen_activations(M, layer.K, seed=wl.activation_seed(seed, M), dtype=dtype, outliers=outliers)
    pk_ref, _ = oracle.pack(Q, A, B)
    pk = u.pack(torch.from_numpy(Q).to(DEV), half_dev(A), half_dev(B))
    ref = oracle.matmul(pk_ref, layer.N, layer.K, x_f64(xb, dtype))
    torch.cuda.synchronize()
    return pk, x_dev(xb, dtype), ref


def check_both_outputs(fn, pk, layer, x, ref, fp32_bar):
    """fp32 outputs at the kernel's own bar, fp16 outputs at the stated 2e-3."""
    y32 = fn(pk, layer.N, layer.K, x, out_dtype=torch.float32)
    y16 = fn(pk, layer.N, layer.K, x, out_dtype=torch.float16)
    torch.cuda.synchronize()
    assert rel_err(y32.cpu().numpy(), ref) <= fp32_bar
    assert rel_err(y16.cpu().numpy(), ref) <= 2e-3
    return y32


# ---------------------------------------------------------------- small batch (7B, M = 4, 16, 64)

@pytest.mark.parametrize("M", [4, 16, 64])
@pytest.mark.parametrize("layer", SHAPES_7B, ids=shape_id)
def test_smallbatch_7b_full_tensor(layer, M):
    """7B shapes at 4, 16 and 64 tokens with 1% of the input channels scaled
    by 20 (outlier channels): 4 tokens through the matrix-vector kernel,
    more through unisvq_gemm (small-batch kernel, or the tiled kernel with a
    K split); every element checked, reruns bit-identical."""
    pk, x, ref = full_format_case(layer, M, "f16", seed=40 + M, outliers=True)
    fn = u.gemv if M <= 4 else u.gemm
    y = check_both_outputs(fn, pk, layer, x, ref, 1e-5 if M <= 4 else 5e-4)
    y2 = fn(pk, layer.N, layer.K, x, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


# ---------------------------------------------------------------- 70B shapes, M = 1 and 16

@pytest.mark.parametrize("M", [1, 16])
@pytest.mark.parametrize("layer", SHAPES_70B, ids=shape_id)
def test_llama70b_full_tensor(layer, M):
    pk, x, ref = full_format_case(layer, M, "f16", seed=10 + M + layer.N % 7, outliers=False)
    fn = u.gemv if M <= 4 else u.gemm
    check_both_outputs(fn, pk, layer, x, ref, 1e-5 if M <= 4 else 5e-4)


# ---------------------------------------------------------------- prefill, M = 2048, bf16

@pytest.mark.parametrize("layer", wl.PREFILL7B, ids=shape_id)
def test_prefill_m2048_full_tensor(layer):
    """Per-(row, group) pairs through the tiled kernel at its real size."""
    pk, x, ref = full_format_case(layer, 2048, "bf16", seed=20, outliers=False)
    check_both_outputs(u.gemm, pk, layer, x, ref, 5e-4)


@pytest.mark.parametrize("layer", wl.PREFILL7B, ids=shape_id)
def test_prefill_m2048_shared_and_fold_full_tensor(layer):
    """One (A, B) pair per matrix (the paper's setting) at the real prefill
    size: the decode path (unisvq_gemm_shared) and the Eq. 9 fold
    (unisvq_gemm_shared_fold) against one oracle result."""
    N, K, M = layer.N, layer.K, 2048
    Q, A, B = wl.gen_shared_weights(N, K, 1, seed=22)
    xb = wl.gen_activations(M, K, seed=wl.activation_seed(22, M), dtype="bf16")
    pc, pa = u.pack_shared(torch.from_numpy(Q).to(DEV), half_dev(A), half_dev(B))
    ref = oracle.matmul_shared(oracle.pack_codes(Q)[0], N, K, A, B, x_f64(xb, "bf16"))
    x = x_dev(xb, "bf16")
    for fn in (u.gemm_shared, u.gemm_shared_fold):
        y32 = fn(pc, pa, N, K, 1, x, out_dtype=torch.float32)
        y16 = fn(pc, pa, N, K, 1, x, out_dtype=torch.float16)
        torch.cuda.synchronize()
        assert rel_err(y32.cpu().numpy(), ref) <= 5e-4, fn.__name__
        assert rel_err(y16.cpu().numpy(), ref) <= 2e-3, fn.__name__
