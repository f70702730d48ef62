"""GPU: the decode-phase product with the input-side transform of Eq. 5
fused in (unisvq_gemv_rht_batched).

Bars: bit-exact against the two-launch path it replaces (unisvq_rht mode 0
with the activation dtype as output, then unisvq_gemv_batched on the
result) -- same arithmetic, same single rounding of x' -- and, for one case
per K, the fp64 oracle chain (transform, then the product) within the
2e-3 bar of the fp16 outputs.
"""
import numpy as np
import pytest

import oracle
from paper_2606_10520_amd import workloads as wl

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

u = None
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def lib():
    global u
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_10520_amd.unisvq as mod
    mod.load()  # raises if the library is missing: no fallback
    u = mod
    yield mod


def dev_u16_as_half(a: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(DEV)


def dev_x(bits: np.ndarray, dtype: str):
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.float16 if dtype == "f16" else torch.bfloat16).to(DEV)


def weights(N, K, seed):
    Q, A, B = wl.gen_weights(N, K, seed=seed)
    pk = u.pack(torch.from_numpy(Q).to(DEV), dev_u16_as_half(A), dev_u16_as_half(B))
    return Q, A, B, pk


def signs(K, seed):
    return torch.from_numpy(np.random.default_rng(seed).choice(np.array([-1, 1], np.int8), K)).to(DEV)


@pytest.mark.parametrize("K", [4096, 8192])
@pytest.mark.parametrize("M", [1, 2, 3, 4])
@pytest.mark.parametrize("xdt", ["f16", "bf16"])
@pytest.mark.parametrize("ydt", [torch.float32, torch.float16])
def test_fused_equals_two_launches(K, M, xdt, ydt):
    shapes = [(1024, K), (2048, K), (512, K)]
    probs, ref = [], []
    for i, (N, K_) in enumerate(shapes):
        _, _, _, pk = weights(N, K_, seed=100 + i)
        x = dev_x(wl.gen_activations(M, K_, seed=200 + i, dtype=xdt), xdt)
        s = signs(K_, 300 + i)
        probs.append((pk, N, K_, x, s, None))
        xr = u.rht(x, s, "in")  # x' in the activation dtype
        ref.append(u.gemv_batched([(pk, N, K_, xr, None)], out_dtype=ydt)[0])
    got = u.gemv_rht_batched(probs, out_dtype=ydt)
    torch.cuda.synchronize()
    for g, r in zip(got, ref):
        assert torch.equal(g, r)


@pytest.mark.parametrize("K", [4096, 8192])
def test_fused_matches_oracle_chain(K):
    N, M = 1024, 2
    Q, A, B, pk = weights(N, K, seed=7)
    pk_ref, _ = oracle.pack(Q, A, B)
    xb = wl.gen_activations(M, K, seed=8, dtype="f16")
    s = np.random.default_rng(9).choice(np.array([-1, 1], np.int8), K)
    y = u.gemv_rht_batched([(pk, N, K, dev_x(xb, "f16"), torch.from_numpy(s).to(DEV), None)],
                           out_dtype=torch.float32)[0]
    torch.cuda.synchronize()
    x_rot = oracle.rht(oracle.half_to_double(xb), s, "in")
    ref = oracle.matmul(pk_ref, N, K, x_rot)
    err = float(np.abs(y.cpu().numpy().astype(np.float64) - ref).max() / np.abs(ref).max())
    # x' rounded once to fp16 (2^-11 relative per element) before the product
    assert err <= 2e-3


def test_fused_rejects_unsupported_shapes():
    _, _, _, pk = weights(256, 11008, seed=1)
    x = torch.zeros((1, 11008), dtype=torch.float16, device=DEV)
    s = signs(11008, 2)
    with pytest.raises(u.UniSVQError) as e:
        u.gemv_rht_batched([(pk, 256, 11008, x, s, None)])
    assert e.value.status == -3
    _, _, _, pk4 = weights(256, 4096, seed=3)
    _, _, _, pk8 = weights(256, 8192, seed=4)
    x4 = torch.zeros((1, 4096), dtype=torch.float16, device=DEV)
    x8 = torch.zeros((1, 8192), dtype=torch.float16, device=DEV)
    with pytest.raises(u.UniSVQError) as e:
        u.gemv_rht_batched([(pk4, 256, 4096, x4, signs(4096, 5), None), (pk8, 256, 8192, x8, signs(8192, 6), None)])
    assert e.value.status == -3
