"""GPU parity of the format variants -- b-bit codes (b = 3, Sec. 5.2.5) and
d-dimensional vectors (d = 8, Sec. 5.2.3), codes-only with row-shared pairs --
against the fp64 oracle.

Bars as for the main formats: packed bytes and unpacked values bit-exact;
matrix-vector products with fp32 outputs within 1e-5 of max|y| (the x.q
products are exact on the matrix cores, only the fp32 accumulation rounds),
fp16 outputs within 2e-3; tiled products within 5e-4 (one fp16 rounding of
every decoded weight); integer-valued inputs bit-exact.
"""
import numpy as np
import pytest

import oracle
from paper_2606_10520_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

u = None
DEV = "cuda:0"
VARIANTS = [(3, 4), (2, 8), (3, 8)]
VID = ["b3d4", "b2d8", "b3d8"]


@pytest.fixture(scope="module", autouse=True)
def lib():
    global u
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_10520_amd.unisvq as mod
    mod.load()  # raises if the library is missing: no fallback
    u = mod
    yield mod


def dev_half(a: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(DEV)


def dev_x(bits: np.ndarray, dtype: str):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.float16 if dtype == "f16" else torch.bfloat16).to(DEV)


def x_as_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    return oracle.half_to_double(bits) if dtype == "f16" else oracle.bf16_to_double(bits)


def rel_err(y: np.ndarray, ref: np.ndarray) -> float:
    return float(np.abs(y.astype(np.float64) - ref).max() / max(np.abs(ref).max(), 1e-300))


def upload(Q, A, B, bits, d):
    pc, pa = u.var_pack(torch.from_numpy(Q).to(DEV), dev_half(A), dev_half(B), bits, d)
    torch.cuda.synchronize()
    return pc, pa


def oracle_y(Q, A, B, bits, d, X, rows=None):
    N, K = Q.shape
    return oracle.var_matmul(oracle.var_pack_codes(Q, bits, d)[0], N, K, bits, A, B, X, rows=rows)


@pytest.mark.parametrize("bits,d", VARIANTS, ids=VID)
@pytest.mark.parametrize("N,K", [(16, 128), (32, 384), (48, 1152), (256, 4096)])
@pytest.mark.parametrize("per_group", [False, True])
def test_var_pack_bit_exact(bits, d, N, K, per_group):
    Ga = K // 128 if per_group else 1
    Q, A, B = wl.gen_var_weights(N, K, bits, d, Ga, seed=N + K + bits + d)
    pc, pa = upload(Q, A, B, bits, d)
    ref, bad = oracle.var_pack_codes(Q, bits, d)
    assert bad == 0
    got = pc.cpu().numpy()[:u.var_codes_bytes(N, K, bits, d)]
    assert got.size == ref.size and np.array_equal(got, ref)
    ref_a = oracle.var_pack_affine(A, B, K)
    assert np.array_equal(pa.cpu().numpy()[:ref_a.size], ref_a)
    q2, a2, b2 = u.var_unpack(pc, pa, N, K, bits, d, Ga)
    torch.cuda.synchronize()
    assert np.array_equal(q2.cpu().numpy(), Q)
    assert np.array_equal(a2.cpu().numpy().view(np.uint16), A.view(np.uint16))
    assert np.array_equal(b2.cpu().numpy().view(np.uint16), B.view(np.uint16))


def test_var_pack_counts_out_of_range_codes():
    N, K = 32, 256
    Q, A, B = wl.gen_var_weights(N, K, 3, 8, 1, seed=3)
    Q[1, 2], Q[30, 255] = 8, 200
    bad = torch.zeros(1, dtype=torch.int32, device=DEV)
    pc, _ = u.var_pack(torch.from_numpy(Q).to(DEV), dev_half(A), dev_half(B), 3, 8, bad_codes=bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == 2
    assert np.array_equal(pc.cpu().numpy(), oracle.var_pack_codes(Q, 3, 8)[0])


def run(fn, N, K, M, bits, d, Ga, dtype="f16", out=torch.float32, seed=0):
    Q, A, B = wl.gen_var_weights(N, K, bits, d, Ga, seed=seed)
    xb = wl.gen_activations(M, K, seed=wl.activation_seed(seed, M), dtype=dtype)
    pc, pa = upload(Q, A, B, bits, d)
    y = getattr(u, fn)(pc, pa, N, K, bits, d, Ga, dev_x(xb, dtype), out_dtype=out)
    torch.cuda.synchronize()
    return y, (Q, A, B), xb


@pytest.mark.parametrize("bits,d", VARIANTS, ids=VID)
@pytest.mark.parametrize("N,K,M", [(16, 128, 1), (32, 384, 1), (64, 1152, 2), (256, 4096, 1), (48, 640, 3),
                                   (64, 512, 4), (1024, 8192, 1)])
@pytest.mark.parametrize("per_group", [False, True])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_var_gemv_parity(bits, d, N, K, M, per_group, dtype):
    Ga = K // 128 if per_group else 1
    y, (Q, A, B), xb = run("var_gemv", N, K, M, bits, d, Ga, dtype, seed=N + M + bits)
    ref = oracle_y(Q, A, B, bits, d, x_as_f64(xb, dtype))
    assert rel_err(y.cpu().numpy(), ref) <= 1e-5


@pytest.mark.parametrize("bits,d", VARIANTS, ids=VID)
@pytest.mark.parametrize("layer", ["gate", "down"])
def test_var_gemv_llama7b_shapes(bits, d, layer):
    """7B shapes, one pair per matrix, fp16 outputs (sampled rows)."""
    L = {l.name: l for l in wl.LLAMA7B}[layer]
    y, (Q, A, B), xb = run("var_gemv", L.N, L.K, 1, bits, d, 1, "f16", out=torch.float16, seed=51)
    rows = np.random.default_rng(2).choice(L.N, 192, replace=False)
    rows[:2] = [0, L.N - 1]
    ref = oracle_y(Q, A, B, bits, d, x_as_f64(xb, "f16"), rows=rows)
    assert rel_err(y.cpu().numpy()[:, rows], ref) <= 2e-3


def integer_inputs(N, K, M, bits, d, Ga, seed):
    """A with entries in {-1, 0, 1}, B and x small integers: every decoded
    weight is an integer of magnitude <= 8*7 + 2 and every partial sum of the
    product an integer below 2^24 (K <= 2048), exact in fp32 in any order."""
    rng = np.random.default_rng(seed)
    Q = rng.integers(0, 1 << bits, size=(N, K), dtype=np.uint8)
    A = rng.integers(-1, 2, size=(Ga, d, d)).astype(np.float16)
    B = rng.integers(-2, 3, size=(Ga, d)).astype(np.float16)
    X = rng.integers(-4, 5, size=(M, K)).astype(np.float16)
    return Q, A, B, X


@pytest.mark.parametrize("bits,d", VARIANTS, ids=VID)
@pytest.mark.parametrize("fn,M", [("var_gemv", 1), ("var_gemv", 3), ("var_gemm", 24), ("var_gemm", 200)])
def test_var_integer_inputs_bit_exact(bits, d, fn, M):
    N, K = 64, 1920  # 15 groups: full packets and a half packet
    Q, A, B, X = integer_inputs(N, K, M, bits, d, K // 128, seed=M + bits + d)
    pc, pa = upload(Q, A, B, bits, d)
    x = torch.from_numpy(X.view(np.int16)).view(torch.float16).to(DEV)
    y32 = getattr(u, fn)(pc, pa, N, K, bits, d, K // 128, x, out_dtype=torch.float32)
    y16 = getattr(u, fn)(pc, pa, N, K, bits, d, K // 128, x, out_dtype=torch.float16)
    torch.cuda.synchronize()
    ref = oracle_y(Q, A, B, bits, d, X.astype(np.float64))
    assert np.array_equal(y32.cpu().numpy().astype(np.float64), ref)
    assert np.array_equal(y16.cpu().numpy(), ref.astype(np.float16))


@pytest.mark.parametrize("fn", ["gemv", "gemm"])
@pytest.mark.parametrize("per_group", [False, True])
def test_var_3bit_small_codes_equal_2bit_path(fn, per_group):
    """3-bit codes below 4 through the variant kernels give bit for bit what
    the 2-bit codes-only path gives (the high-bit steps add exact zeros)."""
    N, K, M = 128, 1408, (3 if fn == "gemv" else 80)
    Ga = K // 128 if per_group else 1
    Q, A, B = wl.gen_shared_weights(N, K, Ga, seed=12)
    x = dev_x(wl.gen_activations(M, K, seed=13, dtype="f16"), "f16")
    pc3, pa3 = upload(Q, A, B, 3, 4)
    y3 = getattr(u, "var_" + fn)(pc3, pa3, N, K, 3, 4, Ga, x, out_dtype=torch.float32)
    pc2, pa2 = u.pack_shared(torch.from_numpy(Q).to(DEV), dev_half(A), dev_half(B))
    y2 = getattr(u, fn + "_shared")(pc2, pa2, N, K, Ga, x, out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(y3, y2)


def test_var_gemv_batched_matches_single_calls():
    for bits, d in VARIANTS:
        probs, singles = [], []
        for i, (N, K, ga) in enumerate([(64, 512, 1), (128, 384, 3), (32, 1024, 8)]):
            Q, A, B = wl.gen_var_weights(N, K, bits, d, ga, seed=60 + i)
            pc, pa = upload(Q, A, B, bits, d)
            x = dev_x(wl.gen_activations(2, K, seed=70 + i, dtype="f16"), "f16")
            probs.append(dict(packed_codes=pc, packed_affine=pa, N=N, K=K, affine_groups=ga, x=x))
            singles.append(u.var_gemv(pc, pa, N, K, bits, d, ga, x, out_dtype=torch.float32))
        outs = u.var_gemv_batched(probs, bits, d, out_dtype=torch.float32)
        torch.cuda.synchronize()
        for a, b in zip(outs, singles):
            assert torch.equal(a, b)


@pytest.mark.parametrize("bits,d", VARIANTS, ids=VID)
@pytest.mark.parametrize("N,K,M", [(16, 128, 5), (64, 384, 20), (80, 640, 64), (128, 1152, 130), (256, 4096, 7)])
@pytest.mark.parametrize("per_group", [False, True])
@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_var_gemm_parity(bits, d, N, K, M, per_group, dtype):
    Ga = K // 128 if per_group else 1
    y, (Q, A, B), xb = run("var_gemm", N, K, M, bits, d, Ga, dtype, seed=N + M + 1 + bits)
    ref = oracle_y(Q, A, B, bits, d, x_as_f64(xb, dtype))
    assert rel_err(y.cpu().numpy(), ref) <= 5e-4


@pytest.mark.parametrize("bits,d", VARIANTS, ids=VID)
def test_var_gemm_prefill_m2048_full_tensor(bits, d):
    """Prefill (2048 tokens, bf16) at 4096 x 4096, every element."""
    L = wl.PREFILL7B[0]
    y, (Q, A, B), xb = run("var_gemm", L.N, L.K, 2048, bits, d, 1, "bf16", seed=21)
    ref = oracle_y(Q, A, B, bits, d, x_as_f64(xb, "bf16"))
    assert rel_err(y.cpu().numpy(), ref) <= 5e-4
