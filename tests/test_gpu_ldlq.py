"""GPU parity of LDLQ (Sec. 3.2.2, Eq. 7) against the fp64 oracle.

The codes are integers decided by fp64 distances to u = W + sum_k E_k U[k][.],
each sum one fma chain in increasing k on both sides, so the GPU codes must
equal the oracle's bit for bit.  The feedback factor U comes from a seeded
synthetic Hessian with strongly coupled columns (X^T X / S of activations that
share a common component, plus mu I with mu = 0.01, Sec. 4.2), factorised
H = U D U^T by the oracle's routine.
"""
import numpy as np
import pytest

import oracle

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


def hessian(rng, K, corr=0.9):
    S = 2 * K
    X = np.sqrt(1 - corr) * rng.standard_normal((S, K)) + np.sqrt(corr) * rng.standard_normal((S, 1)) * rng.standard_normal((1, K))
    return oracle.regularised(X.T @ X / S)


def pairs(rng, N, K, mode):
    s = np.sqrt(12.0 / 15.0)
    n = {"row_group": N * (K // 128), "matrix": 1, "group": K // 128}[mode]
    G = np.linalg.qr(rng.standard_normal((n, 4, 4)))[0]
    A = (s * G).astype(np.float16)
    B = (-1.5 * s * G @ np.ones(4)).astype(np.float16)
    if mode == "row_group":
        A, B = A.reshape(N, K // 128, 4, 4), B.reshape(N, K // 128, 4)
    return A, B, {"row_group": 0, "matrix": 1, "group": K // 128}[mode]


def dev_half(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(DEV)


def run_gpu(W, U, A, B, ga):
    q = u.ldlq(torch.from_numpy(W).to(DEV), torch.from_numpy(U).to(DEV), dev_half(A), dev_half(B), ga)
    torch.cuda.synchronize()
    return q.cpu().numpy()


@pytest.mark.parametrize("N,K", [(16, 128), (32, 384), (64, 1024)])
@pytest.mark.parametrize("mode", ["row_group", "matrix", "group"])
def test_ldlq_bit_exact(N, K, mode):
    rng = np.random.default_rng(N + K + len(mode))
    W = rng.standard_normal((N, K)).astype(np.float32)
    A, B, ga = pairs(rng, N, K, mode)
    U, _ = oracle.ldl_blocks(hessian(rng, K))
    got = run_gpu(W, U, A, B, ga)
    ref, _ = oracle.ldlq(W, U, A, B, shared=(ga != 0))
    assert np.array_equal(got, ref), f"{np.count_nonzero(got != ref)} codes differ"


def test_ldlq_identity_hessian_is_nearest_codeword():
    rng = np.random.default_rng(7)
    N, K = 32, 512
    W = rng.standard_normal((N, K)).astype(np.float32)
    A, B, ga = pairs(rng, N, K, "row_group")
    U = np.eye(K)
    got = run_gpu(W, U, A, B, ga)
    q = u.quantize(torch.from_numpy(W).to(DEV), dev_half(A), dev_half(B), 0)
    torch.cuda.synchronize()
    assert np.array_equal(got, q.cpu().numpy())


def test_ldlq_4096_layer_sampled_rows():
    """A 4096 x 4096 layer (the LLaMA-7B attention shape); rows are
    independent given U, so the oracle evaluates a sample of them."""
    rng = np.random.default_rng(11)
    N, K = 4096, 4096
    W = rng.standard_normal((N, K)).astype(np.float32)
    A, B, ga = pairs(rng, N, K, "matrix")
    U, _ = oracle.ldl_blocks(hessian(rng, K))
    got = run_gpu(W, U, A, B, ga)
    rows = np.array([0, 1, 777, 2048, 4095])
    ref, _ = oracle.ldlq(np.ascontiguousarray(W[rows]), U, A, B, shared=True)
    assert np.array_equal(got[rows], ref)
