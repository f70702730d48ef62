"""GPU block LDL^T factorisation H = U D U^T (Sec. 3.2.2, Eq. 7) against the
fp64 oracle and against what the factorisation must satisfy.

The two sides factorise in different operation orders (the oracle through a
library Cholesky of the reversed matrix, the GPU pivot block by pivot block
over 64-column panels), so the factors agree to rounding: a forward error of
order cond(H) times the fp64 unit roundoff; the bar is 100 cond(H) eps.
Independently of the oracle: U D U^T reproduces H to 1e-12 of max|H| (a
backward-stable factorisation), U has exact identity pivot blocks and exact
zeros below them, and D is symmetric.  Hessians: the coupled synthetic ones
of the LDLQ tests (X^T X / S with a common component, + 0.01 I).
"""
import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

u = None
DEV = "cuda:0"
EPS = np.finfo(np.float64).eps


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


def factor(H, out=None):
    Hd = torch.from_numpy(np.ascontiguousarray(H)).to(DEV)
    U, D, info = u.ldl(Hd, out=Hd if out == "inplace" else None)
    torch.cuda.synchronize()
    return U.cpu().numpy(), D.cpu().numpy(), int(info.item())


def block_diag(D):
    K = 4 * D.shape[0]
    out = np.zeros((K, K))
    for j in range(D.shape[0]):
        out[4 * j:4 * j + 4, 4 * j:4 * j + 4] = D[j]
    return out


@pytest.mark.parametrize("K", [128, 384, 1024, 4096])
def test_ldl_matches_oracle(K):
    rng = np.random.default_rng(K)
    H = hessian(rng, K)
    U, D, info = factor(H)
    assert info == 0
    Uo, Do = oracle.ldl_blocks(H)
    ev = np.linalg.eigvalsh(H)
    tol = 100 * (ev[-1] / ev[0]) * EPS
    assert np.abs(U - Uo).max() <= tol * max(1.0, np.abs(Uo).max())
    assert np.abs(D - Do).max() <= tol * np.abs(Do).max()
    # structure, exactly
    for j in range(K // 4):
        s = slice(4 * j, 4 * j + 4)
        assert np.array_equal(U[s, s], np.eye(4))
        assert not U[4 * j + 4:, s].any()
    assert np.array_equal(D, np.transpose(D, (0, 2, 1)))
    # backward error, without the oracle
    R = U @ block_diag(D) @ U.T
    assert np.abs(R - H).max() <= 1e-12 * np.abs(H).max()


def test_ldl_reads_only_the_upper_triangle_and_runs_in_place():
    rng = np.random.default_rng(5)
    K = 512
    H = hessian(rng, K)
    U0, D0, _ = factor(H)
    Hn = H.copy()
    Hn[np.tril_indices(K, -1)] = np.nan  # never read
    U1, D1, info = factor(Hn)
    assert info == 0
    assert np.array_equal(U0, U1) and np.array_equal(D0, D1)
    U2, D2, info = factor(H, out="inplace")
    assert info == 0
    assert np.array_equal(U0, U2) and np.array_equal(D0, D2)


def test_ldl_diagonal_and_block_diagonal_hessians():
    """H block diagonal: no coupling between pivot blocks, so U = I and D the
    blocks themselves (exactly: nothing is subtracted)."""
    rng = np.random.default_rng(9)
    K = 256
    blocks = []
    for _ in range(K // 4):
        G = rng.standard_normal((4, 4))
        M = G @ G.T + 4 * np.eye(4)
        blocks.append(np.triu(M) + np.triu(M, 1).T)  # exactly symmetric
    H = block_diag(np.array(blocks))
    U, D, info = factor(H)
    assert info == 0
    assert np.array_equal(U, np.eye(K))
    assert np.array_equal(D, np.array(blocks))


def test_ldl_reports_a_pivot_that_is_not_positive_definite():
    K = 256
    H = np.eye(K)
    H[9, 9] = -1.0  # pivot block 2
    _, _, info = factor(H)
    assert info == 3
    _, _, info = factor(-np.eye(K))
    assert info == K // 4  # the last block is taken first


def test_ldl_factor_drives_ldlq():
    """The GPU factor fed to the GPU LDLQ: codes equal the oracle's LDLQ with
    the same factor, bit for bit."""
    rng = np.random.default_rng(13)
    N, K = 32, 512
    U, _, info = factor(hessian(rng, K))
    assert info == 0
    W = rng.standard_normal((N, K)).astype(np.float32)
    s = np.sqrt(12.0 / 15.0)
    G = np.linalg.qr(rng.standard_normal((N * (K // 128), 4, 4)))[0]
    A = (s * G).astype(np.float16).reshape(N, K // 128, 4, 4)
    B = (-1.5 * s * G @ np.ones(4)).astype(np.float16).reshape(N, K // 128, 4)
    dh = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.float16).to(DEV)
    q = u.ldlq(torch.from_numpy(W).to(DEV), torch.from_numpy(U).to(DEV), dh(A), dh(B), 0)
    torch.cuda.synchronize()
    ref, _ = oracle.ldlq(W, U, A, B)
    assert np.array_equal(q.cpu().numpy(), ref)
