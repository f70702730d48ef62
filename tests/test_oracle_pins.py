"""Pins for the fp64 oracle: each test checks it against something other than
itself -- values worked out by hand, closed forms of the paper, special cases
that reduce to a textbook routine, or exact rational arithmetic.

Paper passages: Sec. 2.1 Eq. 1 (Y = X W^T), Sec. 2.2 Eq. 2 (scalar
quantisation), Sec. 3.1 Eq. 4 (affine lattice decode), Sec. 3.2.2 Eq. 6 and
App. A.1 (initialisation and the codebook moments), Sec. 3.2.3 Eq. 8/9
(stacking along the input dimension and the activation-side fold), App. A.2
(the D4 generator matrix).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _rand_params(rng, N, K, a_std=0.02, b_std=0.01):
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    A = (rng.standard_normal((N, K // 128, 4, 4)) * a_std).astype(np.float16)
    B = (rng.standard_normal((N, K // 128, 4)) * b_std).astype(np.float16)
    return Q, A, B


# ---------------------------------------------------------------- conversions

def test_half_to_double_all_bit_patterns():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.half_to_double(bits)
    ref = bits.view(np.float16).astype(np.float64)  # numpy's IEEE binary16
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def test_bf16_to_double_matches_torch():
    torch = pytest.importorskip("torch")
    bits = np.arange(0, 65536, 7, dtype=np.uint32).astype(np.uint16)
    got = oracle.bf16_to_double(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


# ---------------------------------------------------------------- golden decode

def test_golden_d4_generator_decode():
    """Hand-worked decodes with the integer D4 generator of App. A.2.

    A is not symmetric, so applying q^T A instead of A q, or swapping the
    component order of a vector, changes the expected values."""
    g = json.load(open(os.path.join(GOLD, "d4_decode.json")))
    N, K = 1, 128
    Q = np.zeros((N, K), np.uint8)
    for e in g["vectors"]:
        Q[0, 4 * e["v"]:4 * e["v"] + 4] = e["q"]
    A = np.array(g["A"], np.float16).reshape(1, 1, 4, 4)
    B = np.array(g["B"], np.float16).reshape(1, 1, 4)
    W = oracle.decode(Q, A, B)
    for e in g["vectors"]:
        assert W[0, 4 * e["v"]:4 * e["v"] + 4].tolist() == e["w"], e
    # untouched vectors (code 0) decode to B
    untouched = [v for v in range(32) if v not in {e["v"] for e in g["vectors"]}]
    for v in untouched:
        assert W[0, 4 * v:4 * v + 4].tolist() == g["B"]
    # and through the packed path, 16 rows (row 0 carries the fixture)
    Q16 = np.zeros((16, K), np.uint8); Q16[0] = Q[0]
    A16 = np.zeros((16, 1, 4, 4), np.float16); A16[0] = A[0]
    B16 = np.zeros((16, 1, 4), np.float16); B16[0] = B[0]
    packed, bad = oracle.pack(Q16, A16, B16)
    assert bad == 0
    X = np.zeros((1, K)); X[0, 20:24] = 1.0
    Y = oracle.matmul(packed, 16, K, X)
    assert Y[0, 0] == g["x_picks_vector_5"]["y"]


# ---------------------------------------------------------------- special cases

def _nice_scales(rng, shape):
    """fp16 scales with at most 9 significant bits, so s*z (z <= 3) is exact in fp16."""
    m = rng.integers(64, 256, size=shape) | 1
    e = rng.integers(9, 13, size=shape)
    return (m * np.exp2(-e.astype(np.float64))).astype(np.float16)


def test_scalar_quantisation_special_case():
    """A = s I, B = -s z 1 turns the decode into the scalar dequantiser of Eq. 2:
    Phi_SQ(w) = s (clamp(round(w/s) + z, 0, 3) - z), per (row, group)."""
    rng = np.random.default_rng(11)
    N, K = 32, 384
    w = rng.standard_normal((N, K)) * 0.05
    s = _nice_scales(rng, (N, K // 128))
    z = rng.integers(1, 3, size=(N, K // 128))  # integer zero points 1 or 2
    s_col = np.repeat(s.astype(np.float64), 128, axis=1)
    z_col = np.repeat(z, 128, axis=1)
    codes = np.clip(np.round(w / s_col) + z_col, 0, 3)
    phi_sq = s_col * (codes - z_col)  # Eq. 2, computed from w directly
    A = np.zeros((N, K // 128, 4, 4), np.float16)
    for a in range(4):
        A[:, :, a, a] = s
    B = np.repeat((-(s.astype(np.float64)) * z)[..., None], 4, axis=2).astype(np.float16)
    assert np.array_equal(B.astype(np.float64)[..., 0], -(s.astype(np.float64)) * z)  # exact
    W = oracle.decode(codes.astype(np.uint8), A, B)
    assert np.array_equal(W, phi_sq)
    packed, _ = oracle.pack(codes.astype(np.uint8), A, B)
    assert np.array_equal(oracle.decode_packed_rows(packed, N, K, 0, N), phi_sq)


def test_identity_transform_is_plain_integer_matmul():
    """A = I, B = 0: W_hat = Q, so Y = X Q^T (a library matmul on the codes)."""
    rng = np.random.default_rng(5)
    N, K, M = 48, 640, 3  # 5 groups: exercises the half packet
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    A = np.zeros((N, K // 128, 4, 4), np.float16)
    for a in range(4):
        A[:, :, a, a] = 1.0
    B = np.zeros((N, K // 128, 4), np.float16)
    X = rng.integers(-8, 9, size=(M, K)).astype(np.float64)
    packed, _ = oracle.pack(Q, A, B)
    Y = oracle.matmul(packed, N, K, X, threads=3)
    assert np.array_equal(Y, X @ Q.T.astype(np.float64))


# ---------------------------------------------------------------- closed forms

def _all_codes_row(A_g, B_g):
    """One row whose 8 groups enumerate all 256 code tuples, all groups sharing (A_g, B_g)."""
    K = 1024
    c = np.arange(256)
    q = np.stack([(c >> (2 * b)) & 3 for b in range(4)], axis=1)  # tuple of code c
    Q = q.reshape(1, K).astype(np.uint8)
    A = np.broadcast_to(A_g, (1, 8, 4, 4)).astype(np.float16)
    B = np.broadcast_to(B_g, (1, 8, 4)).astype(np.float16)
    return Q, A, B


def test_codebook_moments_closed_form():
    """Over the full code grid: mean = A (1.5 * 1) + B, covariance = 1.25 A A^T,
    since each code is uniform on {0..3} with mean 3/2 and variance 15/12
    (App. A.1).  A A^T differs from A^T A for a general A, so a transposed A
    fails this."""
    rng = np.random.default_rng(3)
    for _ in range(5):
        A_g = (rng.standard_normal((4, 4)) * 0.3).astype(np.float16)
        B_g = (rng.standard_normal(4) * 0.1).astype(np.float16)
        Q, A, B = _all_codes_row(A_g, B_g)
        code_words = oracle.decode(Q, A, B).reshape(256, 4)
        Af, Bf = A_g.astype(np.float64), B_g.astype(np.float64)
        mean = code_words.mean(axis=0)
        cov = (code_words - mean).T @ (code_words - mean) / 256.0
        np.testing.assert_allclose(mean, 1.5 * Af.sum(axis=1) + Bf, rtol=0, atol=1e-12)
        np.testing.assert_allclose(cov, 1.25 * Af @ Af.T, rtol=0, atol=1e-12)


def test_paper_initialisation_gives_centred_unit_grid():
    """Eq. 6 with b = 1.5, s = sqrt(12/15) and G orthogonal: mean 0 and
    covariance I (App. A.1), up to the fp16 rounding of A and B."""
    stats = pytest.importorskip("scipy.stats")
    G = stats.ortho_group.rvs(4, random_state=7)
    s = np.sqrt(12.0 / 15.0)
    A_g = (s * G).astype(np.float16)
    B_g = (-1.5 * s * G @ np.ones(4)).astype(np.float16)
    Q, A, B = _all_codes_row(A_g, B_g)
    cw = oracle.decode(Q, A, B).reshape(256, 4)
    np.testing.assert_allclose(cw.mean(axis=0), 0.0, atol=4e-3)
    cov = np.cov(cw.T, bias=True)
    np.testing.assert_allclose(cov, np.eye(4), atol=4e-3)


def test_fold_identity_for_row_shared_affine():
    """Eq. 9: with (A, B) shared by all rows of a group,
    Y = sum_i (X_i A) W_int,i^T + sum_i (X_i B) 1^T  -- activations folded first."""
    rng = np.random.default_rng(9)
    N, K, M = 32, 512, 4
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    A_grp = (rng.standard_normal((K // 128, 4, 4)) * 0.05).astype(np.float16)
    B_grp = (rng.standard_normal((K // 128, 4)) * 0.02).astype(np.float16)
    A = np.broadcast_to(A_grp, (N,) + A_grp.shape).copy()
    B = np.broadcast_to(B_grp, (N,) + B_grp.shape).copy()
    X = rng.standard_normal((M, K))
    packed, _ = oracle.pack(Q, A, B)
    Y = oracle.matmul(packed, N, K, X)
    Xv = X.reshape(M, K // 4, 4)  # X_i: tokens x d, one per vector i
    g_of_v = np.arange(K // 4) // 32
    XA = np.einsum("tva,vab->tvb", Xv, A_grp.astype(np.float64)[g_of_v])  # X_i A
    XB = np.einsum("tva,va->t", Xv, B_grp.astype(np.float64)[g_of_v])     # sum_i X_i B
    Y_fold = XA.reshape(M, K) @ Q.T.astype(np.float64) + XB[:, None]
    np.testing.assert_allclose(Y, Y_fold, rtol=1e-12, atol=1e-12)


def test_linearity_in_x_and_additivity_in_b():
    rng = np.random.default_rng(21)
    N, K, M = 32, 384, 2
    Q, A, B = _rand_params(rng, N, K)
    X1, X2 = rng.standard_normal((M, K)), rng.standard_normal((M, K))
    pk, _ = oracle.pack(Q, A, B)
    Y1, Y2 = oracle.matmul(pk, N, K, X1), oracle.matmul(pk, N, K, X2)
    Y12 = oracle.matmul(pk, N, K, 2.0 * X1 - 0.5 * X2)
    np.testing.assert_allclose(Y12, 2.0 * Y1 - 0.5 * Y2, rtol=1e-12, atol=1e-12)
    # additivity in B: Y(A, B) = Y(A, 0) + Y(0, B) with Y(0, B)[t][r] = sum_g B[r][g] . Xbar[t][g]
    zA, zB = np.zeros_like(A), np.zeros_like(B)
    Y_A0 = oracle.matmul(oracle.pack(Q, A, zB)[0], N, K, X1)
    Y_0B = oracle.matmul(oracle.pack(Q, zA, B)[0], N, K, X1)
    Xbar = X1.reshape(M, K // 128, 32, 4).sum(axis=2)  # [t][g][a]
    np.testing.assert_allclose(Y_0B, np.einsum("rga,tga->tr", B.astype(np.float64), Xbar),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Y1, Y_A0 + Y_0B, rtol=1e-12, atol=1e-12)
    # linear in A: doubling A (exact in fp16) doubles Y(A, 0)
    Y_2A = oracle.matmul(oracle.pack(Q, (2 * A.astype(np.float32)).astype(np.float16), zB)[0], N, K, X1)
    np.testing.assert_array_equal(Y_2A, 2.0 * Y_A0)


def test_exact_rational_brute_force():
    """Exact rationals on tiny inputs: the fp64 decode is exact (each product is
    an fp16 value times an integer <= 3; 4 of them plus B fit in 53 bits) and Y
    differs from the exact value only by the rounding of one K-term sum."""
    rng = np.random.default_rng(1)
    N, K, M = 16, 256, 2
    Q, A, B = _rand_params(rng, N, K, a_std=0.5, b_std=0.5)
    X = rng.standard_normal((M, K)).astype(np.float16)
    pk, _ = oracle.pack(Q, A, B)
    Y = oracle.matmul(pk, N, K, X.astype(np.float64))
    W = oracle.decode(Q, A, B)
    Af = [[[[Fraction(float(A[r, g, a, b])) for b in range(4)] for a in range(4)]
           for g in range(K // 128)] for r in range(N)]
    for r in range(0, N, 5):
        w_exact = []
        for k in range(K):
            v, a = divmod(k, 4)
            g = 4 * v // 128
            w = Fraction(float(B[r, g, a])) + sum(Af[r][g][a][b] * int(Q[r, 4 * v + b]) for b in range(4))
            w_exact.append(w)
            assert Fraction(W[r, k]) == w  # exact decode
        for t in range(M):
            y = sum(Fraction(float(X[t, k])) * w_exact[k] for k in range(K))
            scale = sum(abs(Fraction(float(X[t, k])) * w_exact[k]) for k in range(K))
            assert abs(Fraction(Y[t, r]) - y) <= scale * Fraction(K, 2 ** 52)


# ---------------------------------------------------------------- packed format

def test_packed_size_is_4p5_bits_per_weight():
    """2-bit codes plus one 40-byte (A, B) set per 128 weights of a row (Sec. 3.1:
    (4*4+4)*2 bytes per set)."""
    for N, K in [(16, 128), (4096, 4096), (11008, 4096), (4096, 11008), (1024, 8192)]:
        assert oracle.packed_bytes(N, K) == N * K // 4 + N * (K // 128) * 40
    for N, K in [(15, 128), (16, 100), (0, 128)]:
        with pytest.raises(oracle.OracleError):
            oracle.packed_bytes(N, K)


def test_packed_byte_positions_worked_by_hand():
    g = json.load(open(os.path.join(GOLD, "pack_positions.json")))
    for c in g["cases"]:
        N, K = c["N"], c["K"]
        Q = np.zeros((N, K), np.uint8)
        A = np.zeros((N, K // 128, 4, 4), np.uint16)
        B = np.zeros((N, K // 128, 4), np.uint16)
        if c["set"] == "Q":
            Q[tuple(c["index"])] = c["value"]
        elif c["set"] == "A":
            A[tuple(c["index"])] = c["bits"]
        else:
            B[tuple(c["index"])] = c["bits"]
        packed, bad = oracle.pack(Q, A, B)
        assert bad == 0
        expect = np.zeros_like(packed)
        for off, val in c["bytes"].items():
            expect[int(off)] = val
        nz = np.nonzero(packed != expect)[0]
        assert nz.size == 0, (c, nz[:8], packed[nz[:8]])


@pytest.mark.parametrize("N,K", [(16, 128), (16, 256), (48, 384), (32, 1152)])
def test_pack_unpack_round_trip(N, K):
    rng = np.random.default_rng(N * 7 + K)
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    A = rng.integers(0, 65536, size=(N, K // 128, 4, 4), dtype=np.uint32).astype(np.uint16)
    B = rng.integers(0, 65536, size=(N, K // 128, 4), dtype=np.uint32).astype(np.uint16)
    packed, bad = oracle.pack(Q, A, B)
    assert bad == 0
    Q2, A2, B2 = oracle.unpack(packed, N, K)
    assert np.array_equal(Q2, Q)
    assert np.array_equal(A2.view(np.uint16), A) and np.array_equal(B2.view(np.uint16), B)
    # every byte is used exactly: distinct inputs give distinct images
    Q[0, 0] ^= 1
    assert not np.array_equal(oracle.pack(Q, A, B)[0], packed)


def test_pack_counts_out_of_range_codes():
    N, K = 16, 256
    Q = np.zeros((N, K), np.uint8)
    Q[3, 7] = 4; Q[15, 200] = 255; Q[0, 0] = 3
    A = np.zeros((N, 2, 4, 4), np.float16); B = np.zeros((N, 2, 4), np.float16)
    _, bad = oracle.pack(Q, A, B)
    assert bad == 2


def test_row_subset_matches_full_product():
    rng = np.random.default_rng(4)
    N, K, M = 64, 384, 3
    Q, A, B = _rand_params(rng, N, K)
    pk, _ = oracle.pack(Q, A, B)
    X = rng.standard_normal((M, K))
    Y = oracle.matmul(pk, N, K, X, threads=4)
    rows = [63, 0, 17, 17, 40]
    Ys = oracle.matmul(pk, N, K, X, rows=rows, threads=2)
    assert np.array_equal(Ys, Y[:, rows])
    # single-threaded and multi-threaded agree bit for bit (each sum is sequential)
    assert np.array_equal(Y, oracle.matmul(pk, N, K, X, threads=1))


# ------------------------------------------- row-shared affine parameters
# (the paper's own setting: one (A, B) per weight matrix, Sec. 3.1 / Sec. 4.2;
# or one pair per 128-column group shared by the rows)

def test_codes_packed_size_is_2_bits_per_weight():
    for N, K in [(16, 128), (4096, 4096), (11008, 4096), (4096, 11008)]:
        assert oracle.codes_packed_bytes(N, K) == N * K // 4
    for N, K in [(15, 128), (16, 100), (0, 128)]:
        with pytest.raises(oracle.OracleError):
            oracle.codes_packed_bytes(N, K)


def test_codes_byte_positions_worked_by_hand():
    g = json.load(open(os.path.join(GOLD, "codes_positions.json")))
    for c in g["cases"]:
        N, K = c["N"], c["K"]
        Q = np.zeros((N, K), np.uint8)
        Q[tuple(c["index"])] = c["value"]
        packed, bad = oracle.pack_codes(Q)
        assert bad == 0
        expect = np.zeros_like(packed)
        for off, val in c["bytes"].items():
            expect[int(off)] = val
        nz = np.nonzero(packed != expect)[0]
        assert nz.size == 0, (c, nz[:8], packed[nz[:8]])


@pytest.mark.parametrize("N,K", [(16, 128), (16, 256), (48, 384), (32, 1152)])
def test_codes_round_trip_and_same_fields_as_full_format(N, K):
    """Codes-only bytes are the code areas of the full format, packet by packet."""
    rng = np.random.default_rng(N * 11 + K)
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    pc, bad = oracle.pack_codes(Q)
    assert bad == 0
    assert np.array_equal(oracle.unpack_codes(pc, N, K), Q)
    A = np.zeros((N, K // 128, 4, 4), np.float16); B = np.zeros((N, K // 128, 4), np.float16)
    pf, _ = oracle.pack(Q, A, B)
    groups = K // 128
    for rb in range(N // 16):
        for p in range((groups + 1) // 2):
            half = groups % 2 == 1 and p == groups // 2
            n = 512 if half else 1024
            full_off = rb * groups * 1152 + p * 2304
            code_off = rb * groups * 512 + p * 1024
            assert np.array_equal(pf[full_off:full_off + n], pc[code_off:code_off + n]), (rb, p)
    Q[N - 1, K - 1] ^= 2
    assert not np.array_equal(oracle.pack_codes(Q)[0], pc)


@pytest.mark.parametrize("Ga_per_group", [False, True])
def test_shared_product_equals_replicated_parameters(Ga_per_group):
    """Row-shared pairs give bit for bit the product of the full format with
    every row holding copies of them."""
    rng = np.random.default_rng(31 + Ga_per_group)
    N, K, M = 32, 384, 3
    Ga = K // 128 if Ga_per_group else 1
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    As = (rng.standard_normal((Ga, 4, 4)) * 0.05).astype(np.float16)
    Bs = (rng.standard_normal((Ga, 4)) * 0.02).astype(np.float16)
    g_src = np.arange(K // 128) if Ga_per_group else np.zeros(K // 128, np.int64)
    A = np.broadcast_to(As[g_src], (N, K // 128, 4, 4)).copy()
    B = np.broadcast_to(Bs[g_src], (N, K // 128, 4)).copy()
    X = rng.standard_normal((M, K))
    Y_full = oracle.matmul(oracle.pack(Q, A, B)[0], N, K, X)
    pc, _ = oracle.pack_codes(Q)
    assert np.array_equal(oracle.matmul_shared(pc, N, K, As, Bs, X), Y_full)
    rows = [31, 0, 7]
    assert np.array_equal(oracle.matmul_shared(pc, N, K, As, Bs, X, rows=rows), Y_full[:, rows])


@pytest.mark.parametrize("Ga_per_group", [False, True])
def test_shared_product_is_the_eq9_fold(Ga_per_group):
    """Eq. 9 of Sec. 3.2.3: with (A, B) shared by the rows, fold A into the
    activations (X_i A per vector i) and B into one column term, then multiply
    by the bare integer codes."""
    rng = np.random.default_rng(77 + Ga_per_group)
    N, K, M = 48, 640, 2
    Ga = K // 128 if Ga_per_group else 1
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    As = (rng.standard_normal((Ga, 4, 4)) * 0.05).astype(np.float16)
    Bs = (rng.standard_normal((Ga, 4)) * 0.02).astype(np.float16)
    X = rng.standard_normal((M, K))
    Y = oracle.matmul_shared(oracle.pack_codes(Q)[0], N, K, As, Bs, X)
    g_of_v = (np.arange(K // 4) // 32) if Ga_per_group else np.zeros(K // 4, np.int64)
    Xv = X.reshape(M, K // 4, 4)
    XA = np.einsum("tva,vab->tvb", Xv, As.astype(np.float64)[g_of_v])
    XB = np.einsum("tva,va->t", Xv, Bs.astype(np.float64)[g_of_v])
    np.testing.assert_allclose(Y, XA.reshape(M, K) @ Q.T.astype(np.float64) + XB[:, None], rtol=1e-12, atol=1e-12)


def test_shared_identity_pair_is_integer_matmul():
    """A = I, B = 0 for the whole matrix: the product of integer activations
    with the codes, exactly."""
    rng = np.random.default_rng(5)
    N, K, M = 16, 256, 2
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    X = rng.integers(-8, 9, size=(M, K)).astype(np.float64)
    As = np.eye(4, dtype=np.float16)[None]
    Bs = np.zeros((1, 4), np.float16)
    Y = oracle.matmul_shared(oracle.pack_codes(Q)[0], N, K, As, Bs, X)
    assert np.array_equal(Y, X @ Q.T.astype(np.float64))


# ------------------------------------------- nearest-codeword quantiser (Sec. 3.2.2)

def test_quantize_recovers_codes_of_on_grid_weights():
    """W built as A q + B (exactly representable): the nearest codeword is q."""
    rng = np.random.default_rng(101)
    N, K = 16, 256
    Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
    # A: multiples of 1/8 in [-2, 2] (exact in fp16), full rank with probability one
    A = (rng.integers(-16, 17, size=(N, K // 128, 4, 4)) / 8).astype(np.float16)
    B = (rng.integers(-16, 17, size=(N, K // 128, 4)) / 8).astype(np.float16)
    W = oracle.decode(Q, A, B).astype(np.float32)
    assert np.array_equal(W.astype(np.float64), oracle.decode(Q, A, B))  # exact on the grid
    Wv = W.reshape(N, K // 4, 4)
    got = oracle.quantize(W, A, B)
    # vectors whose codeword is unique (A of its group nonsingular) must come back exactly
    det = np.linalg.det(A.astype(np.float64))  # [N][G]
    ok_vec = np.abs(det[:, (np.arange(K // 4) * 4) // 128]) > 1e-9
    assert np.array_equal(got.reshape(N, K // 4, 4)[ok_vec], Q.reshape(N, K // 4, 4)[ok_vec])
    assert ok_vec.mean() > 0.9


def test_quantize_scalar_special_case_is_round_to_nearest():
    """A = s I, B = b 1 (Eq. 2, scalar quantisation on a uniform 4-level grid):
    per coordinate clamp(round((w - b) / s), 0, 3)."""
    rng = np.random.default_rng(7)
    N, K = 32, 384
    s, b = 0.75, -1.125
    A = np.zeros((N, K // 128, 4, 4), np.float16)
    A[..., np.arange(4), np.arange(4)] = s
    B = np.full((N, K // 128, 4), b, np.float16)
    W = (rng.standard_normal((N, K)) * 1.5).astype(np.float32)
    ref = np.clip(np.rint((W.astype(np.float64) - b) / s), 0, 3).astype(np.uint8)
    assert np.array_equal(oracle.quantize(W, A, B), ref)


def test_quantize_ties_go_to_the_lowest_index():
    """A = I, B = 0 and w exactly between grid points in three coordinates:
    the codeword with the lowest index q0 + 4 q1 + 16 q2 + 64 q3 wins."""
    N, K = 16, 128
    A = np.zeros((N, 1, 4, 4), np.float16)
    A[..., np.arange(4), np.arange(4)] = 1.0
    B = np.zeros((N, 1, 4), np.float16)
    W = np.zeros((N, K), np.float32)
    W[:, :4] = [0.5, 0.5, 1.5, 2.5]
    W[:, 4:8] = [3.0, 2.5, 0.25, 1.75]
    got = oracle.quantize(W, A, B)
    assert got[0, :4].tolist() == [0, 0, 1, 2]
    assert got[0, 4:8].tolist() == [3, 2, 0, 2]


def test_quantize_no_other_code_is_closer():
    rng = np.random.default_rng(12)
    N, K = 16, 256
    A = (rng.standard_normal((N, K // 128, 4, 4)) * 0.4).astype(np.float16)
    B = (rng.standard_normal((N, K // 128, 4)) * 0.2).astype(np.float16)
    W = rng.standard_normal((N, K)).astype(np.float32)
    Q = oracle.quantize(W, A, B)
    d_best = ((oracle.decode(Q, A, B) - W.astype(np.float64)) ** 2).reshape(N, K // 4, 4).sum(-1)
    for _ in range(64):
        Qo = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
        d_o = ((oracle.decode(Qo, A, B) - W.astype(np.float64)) ** 2).reshape(N, K // 4, 4).sum(-1)
        assert np.all(d_best <= d_o + 1e-12)


@pytest.mark.parametrize("per_group", [False, True])
def test_quantize_shared_pairs_equal_copied_pairs(per_group):
    rng = np.random.default_rng(40 + per_group)
    N, K = 32, 384
    Ga = K // 128 if per_group else 1
    As = (rng.standard_normal((Ga, 4, 4)) * 0.4).astype(np.float16)
    Bs = (rng.standard_normal((Ga, 4)) * 0.2).astype(np.float16)
    src = np.arange(K // 128) if per_group else np.zeros(K // 128, np.int64)
    A = np.broadcast_to(As[src], (N, K // 128, 4, 4)).copy()
    B = np.broadcast_to(Bs[src], (N, K // 128, 4)).copy()
    W = rng.standard_normal((N, K)).astype(np.float32)
    assert np.array_equal(oracle.quantize(W, As, Bs, shared=True), oracle.quantize(W, A, B))


# ------------------------------------------- randomized Hadamard transform (Sec. 3.2.1, Eq. 5)

@pytest.mark.parametrize("n", [1, 2, 4, 12, 20, 28, 44, 112, 344, 688])
def test_hadamard_is_orthogonal(n):
    H = oracle.hadamard(n).astype(np.int64)
    assert set(np.unique(H)) <= {-1, 1}
    assert np.array_equal(H @ H.T, n * np.eye(n, dtype=np.int64))


@pytest.mark.parametrize("n", [12, 28, 44, 344])
def test_paley_part_is_identity_plus_skew(n):
    H = oracle.hadamard(n).astype(np.int64)
    assert oracle.hadamard_factor(n)["m"] == n
    assert np.array_equal(H + H.T, 2 * np.eye(n, dtype=np.int64))


def test_paley_order_12_worked_by_hand():
    g = json.load(open(os.path.join(GOLD, "paley12.json")))
    H = oracle.hadamard(12)
    assert H[0].tolist() == g["row0"]
    assert H[:, 0].tolist() == g["col0"]
    assert H[1].tolist() == g["row1"]


@pytest.mark.parametrize("n", [2, 8, 64, 256])
def test_power_of_two_is_sylvester(n):
    linalg = pytest.importorskip("scipy.linalg")
    assert np.array_equal(oracle.hadamard(n), linalg.hadamard(n).astype(np.int8))


def test_kronecker_layout_of_mixed_orders():
    """n = m * 2^k: H_n = H_m (x) H_{2^k}."""
    linalg = pytest.importorskip("scipy.linalg")
    for n, m, k in [(24, 12, 1), (112, 28, 2), (688, 344, 1)]:
        f = oracle.hadamard_factor(n)
        assert (f["m"], f["k"]) == (m, k)
        assert np.array_equal(oracle.hadamard(n), np.kron(oracle.hadamard(m), linalg.hadamard(2 ** k)).astype(np.int8))


def test_factor_rule_for_the_layer_sizes():
    assert oracle.hadamard_factor(4096) == {"k": 12, "m": 1, "q": 0, "p": 0, "e": 0}
    assert oracle.hadamard_factor(11008) == {"k": 5, "m": 344, "q": 343, "p": 7, "e": 3}
    assert oracle.hadamard_factor(28672) == {"k": 10, "m": 28, "q": 27, "p": 3, "e": 3}
    for n in (100, 86, 43):
        with pytest.raises(oracle.OracleError):
            oracle.hadamard_factor(n)


def test_rht_round_trip_recovers_the_original_product():
    """Eq. 5: W_rot = U S_U W S_V V; at inference y = ((x S_V V) W_rot^T) U S_U
    must equal x W^T.  Built with dense numpy products of the oracle's matrices."""
    rng = np.random.default_rng(55)
    N, K, M = 24, 28, 3
    W = rng.standard_normal((N, K))
    x = rng.standard_normal((M, K))
    sU = rng.choice(np.array([-1, 1], np.int8), N)
    sV = rng.choice(np.array([-1, 1], np.int8), K)
    U = oracle.hadamard(N) / np.sqrt(N)
    V = oracle.hadamard(K) / np.sqrt(K)
    W_rot = U @ np.diag(sU) @ W @ np.diag(sV) @ V
    y_path = oracle.rht(oracle.rht(x, sV, "in") @ W_rot.T, sU, "out")
    np.testing.assert_allclose(y_path, x @ W.T, rtol=1e-12, atol=1e-12)


def test_rht_preserves_norms_and_matches_dense_sylvester():
    linalg = pytest.importorskip("scipy.linalg")
    rng = np.random.default_rng(6)
    n = 256
    x = rng.standard_normal((2, n))
    s = rng.choice(np.array([-1, 1], np.int8), n)
    y = oracle.rht(x, s, "in")
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    np.testing.assert_allclose(y, (x * s) @ linalg.hadamard(n) / np.sqrt(n), rtol=1e-12, atol=1e-12)
    z = oracle.rht(x, s, "out")
    np.testing.assert_allclose(z, (x @ linalg.hadamard(n) / np.sqrt(n)) * s, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- format variants
# b-bit codes, b = 2 or 3 (Sec. 5.2.5: only the integer vectors widen) and
# d-dimensional vectors, d = 4 or 8 (Sec. 5.2.3), with pairs shared by the
# rows (one per matrix, Sec. 4.2, or one per 128-column group).

VARIANTS = [(2, 4), (3, 4), (2, 8), (3, 8)]


def _var_params(rng, N, K, bits, d, Ga, a_std=0.05, b_std=0.02):
    Q = rng.integers(0, 1 << bits, size=(N, K), dtype=np.uint8)
    A = (rng.standard_normal((Ga, d, d)) * a_std).astype(np.float16)
    B = (rng.standard_normal((Ga, d)) * b_std).astype(np.float16)
    return Q, A, B


def test_var_sizes():
    for N, K in [(16, 128), (4096, 4096), (11008, 4096)]:
        assert oracle.var_codes_bytes(N, K, 2) == N * K // 4
        assert oracle.var_codes_bytes(N, K, 3) == N * K * 3 // 8
    assert oracle.var_affine_bytes(4096, 1, 4) == 160
    assert oracle.var_affine_bytes(4096, 1, 8) == 576
    assert oracle.var_affine_bytes(384, 3, 8) == 2 * 576
    with pytest.raises(oracle.OracleError):
        oracle.var_affine_bytes(384, 2, 4)
    with pytest.raises(oracle.OracleError):
        oracle.var_codes_bytes(16, 128, 4)


def test_var_code_positions_worked_by_hand():
    g = json.load(open(os.path.join(GOLD, "var_positions.json")))
    for c in g["codes"]:
        Q = np.zeros((c["N"], c["K"]), np.uint8)
        Q[tuple(c["index"])] = c["value"]
        packed, bad = oracle.var_pack_codes(Q, c["bits"], c["d"])
        assert bad == 0
        expect = np.zeros_like(packed)
        for off, v in c["bytes"].items():
            expect[int(off)] = v
        assert np.array_equal(packed, expect), c["work"]


def test_var_affine_positions_worked_by_hand():
    g = json.load(open(os.path.join(GOLD, "var_positions.json")))
    for c in g["affine"]:
        d, Ga = c["d"], c["Ga"]
        A = np.zeros((Ga, d, d), np.uint16)
        B = np.zeros((Ga, d), np.uint16)
        target = A if c["param"] == "A" else B
        target[(c["pair"],) + tuple(c["index"])] = c["bits16"]
        block = oracle.var_pack_affine(A, B, c["K"])
        expect = np.zeros_like(block)
        for off, v in c["bytes"].items():
            expect[int(off)] = v
        assert np.array_equal(block, expect), c["work"]


@pytest.mark.parametrize("bits,d", VARIANTS)
@pytest.mark.parametrize("N,K", [(16, 128), (32, 384), (48, 1152)])
def test_var_round_trip(bits, d, N, K):
    rng = np.random.default_rng(bits * 100 + d + K)
    for Ga in (1, K // 128):
        Q, A, B = _var_params(rng, N, K, bits, d, Ga)
        packed, bad = oracle.var_pack_codes(Q, bits, d)
        assert bad == 0
        assert np.array_equal(oracle.var_unpack_codes(packed, N, K, bits, d), Q)
        A2, B2 = oracle.var_unpack_affine(oracle.var_pack_affine(A, B, K), K, Ga, d)
        assert np.array_equal(A2.view(np.uint16), A.view(np.uint16))
        assert np.array_equal(B2.view(np.uint16), B.view(np.uint16))


def test_var_2bit_d4_is_the_codes_only_format():
    """The variant layout with b = 2, d = 4 is byte for byte the codes-only
    format (pinned separately by its own hand-worked offsets)."""
    rng = np.random.default_rng(2)
    for N, K in [(16, 128), (32, 640)]:
        Q = rng.integers(0, 4, size=(N, K), dtype=np.uint8)
        assert np.array_equal(oracle.var_pack_codes(Q, 2, 4)[0], oracle.pack_codes(Q)[0])


def test_var_counts_out_of_range_codes():
    Q = np.zeros((16, 256), np.uint8)
    Q[3, 7], Q[9, 200], Q[0, 0] = 8, 9, 7
    _, bad = oracle.var_pack_codes(Q, 3, 8)
    assert bad == 2
    _, bad = oracle.var_pack_codes(Q, 2, 4)
    assert bad == 3


def test_var_unpack_affine_rejects_disagreeing_views():
    A = np.ones((1, 8, 8), np.float16)
    B = np.ones((1, 8), np.float16)
    block = oracle.var_pack_affine(A, B, 256)
    block[300] ^= 1  # one byte of the row view
    with pytest.raises(oracle.OracleError):
        oracle.var_unpack_affine(block, 256, 1, 8)


@pytest.mark.parametrize("d", [4, 8])
def test_var_3bit_with_small_codes_equals_2bit(d):
    """Codes below 4 decode the same whether stored in 2 or 3 bits."""
    rng = np.random.default_rng(31 + d)
    N, K, M = 32, 384, 2
    Q, A, B = _var_params(rng, N, K, 2, d, K // 128)
    X = rng.standard_normal((M, K))
    p2, _ = oracle.var_pack_codes(Q, 2, d)
    p3, _ = oracle.var_pack_codes(Q, 3, d)
    np.testing.assert_array_equal(oracle.var_matmul(p3, N, K, 3, A, B, X), oracle.var_matmul(p2, N, K, 2, A, B, X))


@pytest.mark.parametrize("d", [4, 8])
def test_var_3bit_is_low_part_plus_four_times_high_bit(d):
    """q = (q & 3) + 4 (q >> 2) and the decode is linear in q: decoding the
    3-bit codes equals decoding the low two bits with (A, B) plus the high
    bits with (4A, 0) (4A is exact in fp16)."""
    rng = np.random.default_rng(41 + d)
    N, K, M = 32, 640, 3
    Q, A, B = _var_params(rng, N, K, 3, d, 1)
    X = rng.standard_normal((M, K))
    Y = oracle.var_matmul(oracle.var_pack_codes(Q, 3, d)[0], N, K, 3, A, B, X)
    Y_lo = oracle.var_matmul(oracle.var_pack_codes(Q & 3, 2, d)[0], N, K, 2, A, B, X)
    A4 = (4.0 * A.astype(np.float64)).astype(np.float16)
    assert np.array_equal(A4.astype(np.float64), 4.0 * A.astype(np.float64))
    Y_hi = oracle.var_matmul(oracle.var_pack_codes(Q >> 2, 2, d)[0], N, K, 2, A4, np.zeros_like(B), X)
    np.testing.assert_allclose(Y, Y_lo + Y_hi, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("bits", [2, 3])
def test_var_block_diagonal_d8_equals_d4(bits):
    """An 8-vector whose A is block diagonal diag(A4, A4) with B = (B4, B4) is
    two 4-vectors decoded with (A4, B4): the d = 8 product equals the d = 4
    one (for b = 2 computed by the separately pinned codes-only product)."""
    rng = np.random.default_rng(50 + bits)
    N, K, M = 32, 384, 2
    Ga = K // 128
    Q, A4, B4 = _var_params(rng, N, K, bits, 4, Ga)
    A8 = np.zeros((Ga, 8, 8), np.float16)
    A8[:, :4, :4] = A4
    A8[:, 4:, 4:] = A4
    B8 = np.concatenate([B4, B4], axis=1)
    X = rng.standard_normal((M, K))
    Y8 = oracle.var_matmul(oracle.var_pack_codes(Q, bits, 8)[0], N, K, bits, A8, B8, X)
    Y4 = oracle.var_matmul(oracle.var_pack_codes(Q, bits, 4)[0], N, K, bits, A4, B4, X)
    np.testing.assert_allclose(Y8, Y4, rtol=1e-12, atol=1e-12)
    if bits == 2:
        Yc = oracle.matmul_shared(oracle.pack_codes(Q)[0], N, K, A4, B4, X)
        np.testing.assert_allclose(Y4, Yc, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("bits,d", VARIANTS)
def test_var_identity_and_scalar_special_cases(bits, d):
    """A = I, B = 0 gives W_hat = Q (Y = X Q^T, a library matmul); A = s I,
    B = -s c 1 with c = (2^b - 1)/2 gives the scalar dequantiser of Eq. 2,
    s (Q - c)."""
    rng = np.random.default_rng(60 + 10 * bits + d)
    N, K, M = 32, 384, 2
    Q = rng.integers(0, 1 << bits, size=(N, K), dtype=np.uint8)
    pk, _ = oracle.var_pack_codes(Q, bits, d)
    X = rng.integers(-8, 9, size=(M, K)).astype(np.float64)
    I = np.eye(d, dtype=np.float16)[None]
    Y = oracle.var_matmul(pk, N, K, bits, I, np.zeros((1, d), np.float16), X)
    assert np.array_equal(Y, X @ Q.T.astype(np.float64))
    s, c = 0.0625, ((1 << bits) - 1) / 2.0
    W = oracle.var_decode(Q, (s * np.eye(d))[None].astype(np.float16), np.full((1, d), -s * c, np.float16))
    assert np.array_equal(W, s * (Q.astype(np.float64) - c))


@pytest.mark.parametrize("bits,d", [(2, 4), (3, 4), (2, 8)])
def test_var_codebook_moments_closed_form(bits, d):
    """Over the full grid of 2^(b d) code tuples (App. A.1 for b bits): mean
    = c A 1 + B with c = (2^b - 1)/2 and covariance = ((4^b - 1)/12) A A^T."""
    rng = np.random.default_rng(70 + 10 * bits + d)
    n = 1 << (bits * d)
    idx = np.arange(n)
    q = np.stack([(idx >> (bits * b)) & ((1 << bits) - 1) for b in range(d)], axis=1)
    Q = q.reshape(1, n * d).astype(np.uint8)
    A = (rng.standard_normal((1, d, d)) * 0.3).astype(np.float16)
    B = (rng.standard_normal((1, d)) * 0.1).astype(np.float16)
    cw = oracle.var_decode(Q, A, B).reshape(n, d)
    Af, Bf = A[0].astype(np.float64), B[0].astype(np.float64)
    c, v = ((1 << bits) - 1) / 2.0, ((1 << (2 * bits)) - 1) / 12.0
    mean = cw.mean(axis=0)
    np.testing.assert_allclose(mean, c * Af.sum(axis=1) + Bf, rtol=0, atol=1e-11)
    cov = (cw - mean).T @ (cw - mean) / n
    np.testing.assert_allclose(cov, v * Af @ Af.T, rtol=0, atol=1e-10)


@pytest.mark.parametrize("bits,d", [(3, 4), (2, 8)])
def test_var_paper_initialisation_gives_centred_unit_grid(bits, d):
    """Eq. 6 for b bits: A = s G, B = -s c G 1, s = sqrt(12/(4^b - 1)),
    c = (2^b - 1)/2, G a random orthogonal matrix -> mean 0, covariance I
    (App. A.1), up to the fp16 rounding of A and B."""
    stats = pytest.importorskip("scipy.stats")
    G = stats.ortho_group.rvs(d, random_state=17)
    s, c = np.sqrt(12.0 / ((1 << (2 * bits)) - 1)), ((1 << bits) - 1) / 2.0
    A = (s * G)[None].astype(np.float16)
    B = (-c * s * G @ np.ones(d))[None].astype(np.float16)
    n = 1 << (bits * d)
    idx = np.arange(n)
    q = np.stack([(idx >> (bits * b)) & ((1 << bits) - 1) for b in range(d)], axis=1)
    cw = oracle.var_decode(q.reshape(1, n * d).astype(np.uint8), A, B).reshape(n, d)
    np.testing.assert_allclose(cw.mean(axis=0), 0.0, atol=1e-2)
    np.testing.assert_allclose(np.cov(cw.T, bias=True), np.eye(d), atol=1e-2)


@pytest.mark.parametrize("bits,d", VARIANTS)
def test_var_exact_rational_brute_force(bits, d):
    """Exact rationals: the decode of every weight is exact and Y is within one
    K-term summation rounding of the exact product."""
    rng = np.random.default_rng(80 + 10 * bits + d)
    N, K, M = 16, 256, 2
    Ga = K // 128
    Q, A, B = _var_params(rng, N, K, bits, d, Ga, a_std=0.5, b_std=0.5)
    X = rng.standard_normal((M, K)).astype(np.float16)
    Y = oracle.var_matmul(oracle.var_pack_codes(Q, bits, d)[0], N, K, bits, A, B, X.astype(np.float64))
    Wd = oracle.var_decode(Q, A, B)
    Af = [[[Fraction(float(A[g, a, b])) for b in range(d)] for a in range(d)] for g in range(Ga)]
    for r in range(0, N, 7):
        w_exact = []
        for k in range(K):
            v, a = divmod(k, d)
            g = d * v // 128
            w = Fraction(float(B[g, a])) + sum(Af[g][a][b] * int(Q[r, d * v + b]) for b in range(d))
            w_exact.append(w)
            assert Fraction(Wd[r, k]) == w
        for t in range(M):
            y = sum(Fraction(float(X[t, k])) * w_exact[k] for k in range(K))
            scale = sum(abs(Fraction(float(X[t, k])) * w_exact[k]) for k in range(K))
            assert abs(Fraction(Y[t, r]) - y) <= scale * Fraction(K, 2 ** 52)


# ---------------------------------------------------------------- LDLQ (Eq. 7)
# Reading: the adjustment coefficients of Eq. 7 are the off-diagonal entries of
# U in H = U D U^T (U unit upper block triangular, 4 x 4 identity blocks; D
# block diagonal); H is regularised by mu I, mu = 0.01 (Sec. 4.2).

def _spd(rng, K, rank=None, corr=0.9):
    """A correlated SPD matrix: X^T X / S for activations sharing a common
    component (strong off-diagonal coupling), plus mu I."""
    S = 2 * K if rank is None else rank
    Z = rng.standard_normal((S, K))
    common = rng.standard_normal((S, 1)) * rng.standard_normal((1, K))
    X = np.sqrt(1 - corr) * Z + np.sqrt(corr) * common
    return oracle.regularised(X.T @ X / S)


def test_ldl_blocks_reconstruct_h():
    rng = np.random.default_rng(90)
    K = 256
    H = _spd(rng, K)
    U, D = oracle.ldl_blocks(H)
    Dfull = np.zeros((K, K))
    for j in range(K // 4):
        Dfull[4 * j:4 * j + 4, 4 * j:4 * j + 4] = D[j]
        assert np.allclose(D[j], D[j].T)
        assert np.all(np.linalg.eigvalsh(D[j]) > 0)
        np.testing.assert_array_equal(U[4 * j:4 * j + 4, 4 * j:4 * j + 4], np.eye(4))
        assert np.all(U[4 * j + 4:, 4 * j:4 * j + 4] == 0)  # nothing below the diagonal blocks
    np.testing.assert_allclose(U @ Dfull @ U.T, H, rtol=0, atol=1e-10 * np.abs(H).max())


def _ldlq_case(rng, N, K, shared=False):
    W = rng.standard_normal((N, K)).astype(np.float32)
    s = np.sqrt(12.0 / 15.0)
    if shared:
        G = np.linalg.qr(rng.standard_normal((4, 4)))[0]
        A = (s * G)[None].astype(np.float16)
        B = (-1.5 * s * G @ np.ones(4))[None].astype(np.float16)
    else:
        G = np.linalg.qr(rng.standard_normal((N * (K // 128), 4, 4)))[0]
        A = (s * G).reshape(N, K // 128, 4, 4).astype(np.float16)
        B = (-1.5 * s * G @ np.ones(4)).reshape(N, K // 128, 4).astype(np.float16)
    return W, A, B


@pytest.mark.parametrize("coupling", ["identity", "block_diagonal"])
def test_ldlq_without_cross_vector_coupling_is_nearest_codeword(coupling):
    """No coupling between vectors leaves U = I: no feedback, so LDLQ rounds
    every vector to its nearest codeword."""
    rng = np.random.default_rng(91)
    N, K = 16, 256
    W, A, B = _ldlq_case(rng, N, K)
    H = np.eye(K)
    if coupling == "block_diagonal":
        for j in range(K // 4):
            M = rng.standard_normal((4, 4))
            H[4 * j:4 * j + 4, 4 * j:4 * j + 4] = M @ M.T + np.eye(4)
    U, _ = oracle.ldl_blocks(H)
    Q, E = oracle.ldlq(W, U, A, B)
    assert np.array_equal(Q, oracle.quantize(W, A, B))


@pytest.mark.parametrize("shared", [False, True])
def test_ldlq_decisions_follow_eq7(shared):
    """Every vector's codes are the nearest codeword to its adjusted target
    u = W + E (U - I) (Eq. 7, recomputed here with a library matmul), the
    first vector of a row has no feedback, E = W - W_hat exactly, and the
    proxy loss splits per vector: tr(E H E^T) = sum_j eta_j D_j eta_j^T with
    eta = -E U the rounding errors of the steps."""
    rng = np.random.default_rng(92 + shared)
    N, K = 16, 384
    W, A, B = _ldlq_case(rng, N, K, shared)
    H = _spd(rng, K)
    U, D = oracle.ldl_blocks(H)
    Q, E = oracle.ldlq(W, U, A, B, shared=shared)
    # E is exactly W minus the decoded weights
    What = oracle.var_decode(Q, A, B) if shared else oracle.decode(Q, A, B)
    assert np.array_equal(E, W.astype(np.float64) - What)
    u = W.astype(np.float64) + E @ (U - np.eye(K))
    # the chosen codeword is the nearest to u (fp64 distances; u recomputed with
    # a different summation order, so allow a rounding-level slack)
    cw = What.reshape(N, K // 4, 4)
    d_chosen = ((cw - u.reshape(N, K // 4, 4)) ** 2).sum(axis=2)
    g = np.arange(K // 4) * 4 // 128
    codes = np.arange(256)
    qgrid = np.stack([(codes >> (2 * b)) & 3 for b in range(4)], axis=1).astype(np.float64)  # [256][4]
    Af, Bf = A.astype(np.float64), B.astype(np.float64)
    for r in range(N):
        for v in range(K // 4):
            Ag = Af[0] if shared else Af[r, g[v]]
            Bg = Bf[0] if shared else Bf[r, g[v]]
            all_cw = qgrid @ Ag.T + Bg
            d_all = ((all_cw - u[r, 4 * v:4 * v + 4]) ** 2).sum(axis=1)
            assert d_chosen[r, v] <= d_all.min() + 1e-9
    assert np.array_equal(Q[:, :4], oracle.quantize(W, A, B, shared=shared)[:, :4])  # no feedback yet
    eta = -E @ U
    loss = np.einsum("rk,kl,rl->r", E, H, E)
    split = sum(np.einsum("ra,ab,rb->r", eta[:, 4 * j:4 * j + 4], D[j], eta[:, 4 * j:4 * j + 4]) for j in range(K // 4))
    np.testing.assert_allclose(loss, split, rtol=1e-9)


def test_ldlq_feedback_lowers_the_proxy_loss():
    """With strongly coupled columns the error feedback lowers the Hessian
    proxy loss tr(E H E^T) against plain nearest-codeword rounding (the
    'Hessian compensation' component of Sec. 5.2.1)."""
    rng = np.random.default_rng(93)
    N, K = 32, 512
    W, A, B = _ldlq_case(rng, N, K)
    H = _spd(rng, K, corr=0.95)
    U, _ = oracle.ldl_blocks(H)
    _, E_ldlq = oracle.ldlq(W, U, A, B)
    E_rtn = W.astype(np.float64) - oracle.decode(oracle.quantize(W, A, B), A, B)
    loss = lambda E: float(np.einsum("rk,kl,rl->", E, H, E))
    assert loss(E_ldlq) < 0.8 * loss(E_rtn), (loss(E_ldlq), loss(E_rtn))
