/*
 * UniSVQ reference oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously-correct CPU implementation (fp64) of what the
 * UniSVQ inference path computes.  Only tests/, the smoke check and the
 * CPU-baseline leg of the benchmark may load this code; the product library
 * never does.  It shares no code, header, table or helper with the HIP path:
 * the packed byte format is re-implemented here from its written definition
 * (the format block in include/unisvq.h, restated below).
 *
 * What is computed (paper: "UniSVQ: 2-bit Unified Scalar-Vector
 * Quantization"):
 *   - Each weight vector of d = 4 consecutive input columns of one output row
 *     is rebuilt as an affine image of its integer lattice point,
 *     w_hat = A * q + B, q in {0,1,2,3}^4                      (Sec. 3.1, Eq. 4)
 *   - The dequantised matrix is the stack of those vectors along the input
 *     dimension; vector i covers input columns 4i..4i+3          (Sec. 3.2.3, Eq. 8)
 *   - The layer output is Y = X * W_hat^T                       (Sec. 2.1, Eq. 1)
 *   - Codes are the unsigned integers 0..2^bits-1; the centring constant of
 *     the initialisation lives in B                              (Sec. 3.2.2, Eq. 6; App. A.1)
 *   - One (A, B) pair is held per (output row, 128-column group); the paper's
 *     one-pair-per-matrix setting (Sec. 4.2) is the special case where all
 *     pairs are equal.
 *
 * Packed format (restated from its definition; byte offsets little endian):
 *   N % 16 == 0, K % 128 == 0.  Row block rb (rows 16rb..16rb+15) occupies
 *   (K/128)*1152 consecutive bytes starting at rb*(K/128)*1152.  Inside it the
 *   groups g = 0..K/128-1 are taken in pairs: packet p holds groups 2p, 2p+1
 *   (2304 bytes) and, when K/128 is odd, a final half packet holds the last
 *   group (1152 bytes).  Slot s = 0..63 stands for row r = 16rb + s/4 and
 *   component b = s%4.
 *     full packet at offset P:
 *       P +       16s + 8j : 8-byte code field F(r, 2p+j, b)      j = 0,1
 *       P + 1024 + 16s + 8j : A[r][2p+j][a][b], a = 0..3 (fp16 each)
 *       P + 2048 +  4s + 2j : B[r][2p+j][b] (fp16)
 *     half packet at offset P (group g):
 *       P +        8s : F(r, g, b);  P + 512 + 8s : A[r][g][0..3][b];
 *       P + 1024 + 2s : B[r][g][b]
 *   Code field F(r, g, b) is a 64-bit little-endian word whose bits 2v, 2v+1
 *   hold Q[r][128g + 4v + b], v = 0..31.
 *
 * Codes-only packed format, for affine parameters shared by all rows (the
 * paper's own setting: one (A, B) per weight matrix, Sec. 3.1 and Sec. 4.2;
 * or one per 128-column group, shared by the rows):
 *   Row block rb occupies (K/128)*512 bytes starting at rb*(K/128)*512.
 *   Packet p (groups 2p, 2p+1) is 1024 bytes: P + 16s + 8j holds F(r, 2p+j, b);
 *   a final half packet (last group when K/128 is odd) is 512 bytes: P + 8s
 *   holds F(r, g, b).  Slots and code fields as above.
 *   Shared parameters: As fp16 [Ga][4][4], Bs fp16 [Ga][4] with Ga = 1 (one
 *   pair for the matrix) or K/128 (one pair per group); group g uses pair
 *   (Ga == 1 ? 0 : g).
 *
 * Canonical (unpacked) arrays:
 *   Q uint8  [N][K]           codes, valid values 0..3
 *   A fp16   [N][K/128][4][4] A[r][g][a][b] multiplies q_b into output a
 *   B fp16   [N][K/128][4]
 *   X double [M][K], Y double [M][N]
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_D 4
#define OR_G 128
#define OR_ROWBLOCK 16
#define OR_GROUP_BYTES_PER_BLOCK 1152 /* 16 rows * (32 code bytes + 40 affine bytes) */

enum { OR_OK = 0, OR_EINVAL = -1, OR_ESHAPE = -2 };

/* ---- scalar conversions, written from the IEEE-754 / bfloat16 definitions ---- */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits. */
double oracle_half_to_double(uint16_t h) {
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1f;
    int f = h & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24); /* subnormal: f * 2^-14 * 2^-10 */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25); /* (1 + f/1024) * 2^(e-15) */
    return sign ? -v : v;
}

/* bfloat16: the upper 16 bits of a binary32. */
double oracle_bf16_to_double(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

void oracle_half_array_to_double(const uint16_t* h, double* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_half_to_double(h[i]);
}

void oracle_bf16_array_to_double(const uint16_t* h, double* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = oracle_bf16_to_double(h[i]);
}

/* ---- packed format ---- */

static int shape_ok(int64_t N, int64_t K) {
    return N > 0 && K > 0 && N % OR_ROWBLOCK == 0 && K % OR_G == 0;
}

int64_t oracle_packed_bytes(int64_t N, int64_t K) {
    if (!shape_ok(N, K)) return OR_ESHAPE;
    return (N / OR_ROWBLOCK) * (K / OR_G) * OR_GROUP_BYTES_PER_BLOCK;
}

/* Where the three parts of group g of row block rb live, and at what stride
 * per slot.  Returns byte offsets of slot 0. */
typedef struct {
    int64_t code, a, b;   /* offsets of slot 0 */
    int64_t code_stride;  /* bytes between slots in the code area */
    int64_t a_stride;     /* bytes between slots in the A area */
    int64_t b_stride;     /* bytes between slots in the B area */
} group_place;

static group_place place_group(int64_t K, int64_t rb, int64_t g) {
    int64_t groups = K / OR_G;
    int64_t base = rb * groups * OR_GROUP_BYTES_PER_BLOCK;
    int64_t p = g / 2, j = g % 2;
    int64_t pkt = base + p * 2 * OR_GROUP_BYTES_PER_BLOCK;
    group_place gp;
    int half = (groups % 2 == 1) && (g == groups - 1);
    if (!half) {
        gp.code = pkt + 8 * j;
        gp.a = pkt + 1024 + 8 * j;
        gp.b = pkt + 2048 + 2 * j;
        gp.code_stride = 16;
        gp.a_stride = 16;
        gp.b_stride = 4;
    } else {
        gp.code = pkt;
        gp.a = pkt + 512;
        gp.b = pkt + 1024;
        gp.code_stride = 8;
        gp.a_stride = 8;
        gp.b_stride = 2;
    }
    return gp;
}

static void put_u16(uint8_t* p, uint16_t v) { p[0] = (uint8_t)(v & 0xff); p[1] = (uint8_t)(v >> 8); }
static uint16_t get_u16(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }

/* Pack canonical arrays into the packed byte format.  Returns the number of
 * codes outside 0..3 (their low two bits are stored), or a negative error. */
int64_t oracle_pack(int64_t N, int64_t K, const uint8_t* Q, const uint16_t* A, const uint16_t* B,
                    uint8_t* out) {
    if (!Q || !A || !B || !out) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    int64_t groups = K / OR_G, bad = 0;
    memset(out, 0, (size_t)oracle_packed_bytes(N, K));
    for (int64_t r = 0; r < N; ++r) {
        int64_t rb = r / OR_ROWBLOCK, rl = r % OR_ROWBLOCK;
        for (int64_t g = 0; g < groups; ++g) {
            group_place gp = place_group(K, rb, g);
            for (int b = 0; b < OR_D; ++b) {
                int64_t s = rl * 4 + b;
                uint8_t* field = out + gp.code + s * gp.code_stride;
                for (int v = 0; v < 32; ++v) {
                    uint8_t q = Q[r * K + g * OR_G + 4 * v + b];
                    if (q > 3) ++bad;
                    int bit = 2 * v;
                    field[bit / 8] |= (uint8_t)((q & 3) << (bit % 8));
                }
                uint8_t* acol = out + gp.a + s * gp.a_stride;
                for (int a = 0; a < OR_D; ++a)
                    put_u16(acol + 2 * a, A[((r * groups + g) * OR_D + a) * OR_D + b]);
                put_u16(out + gp.b + s * gp.b_stride, B[(r * groups + g) * OR_D + b]);
            }
        }
    }
    return bad;
}

/* Read back row r's codes and affine parameters from packed bytes. */
static void unpack_row(int64_t K, const uint8_t* packed, int64_t r, uint8_t* q_row,
                       uint16_t* a_row, uint16_t* b_row) {
    int64_t groups = K / OR_G, rb = r / OR_ROWBLOCK, rl = r % OR_ROWBLOCK;
    for (int64_t g = 0; g < groups; ++g) {
        group_place gp = place_group(K, rb, g);
        for (int b = 0; b < OR_D; ++b) {
            int64_t s = rl * 4 + b;
            const uint8_t* field = packed + gp.code + s * gp.code_stride;
            for (int v = 0; v < 32; ++v) {
                int bit = 2 * v;
                q_row[g * OR_G + 4 * v + b] = (uint8_t)((field[bit / 8] >> (bit % 8)) & 3);
            }
            const uint8_t* acol = packed + gp.a + s * gp.a_stride;
            for (int a = 0; a < OR_D; ++a) a_row[(g * OR_D + a) * OR_D + b] = get_u16(acol + 2 * a);
            b_row[g * OR_D + b] = get_u16(packed + gp.b + s * gp.b_stride);
        }
    }
}

int oracle_unpack(int64_t N, int64_t K, const uint8_t* packed, uint8_t* Q, uint16_t* A, uint16_t* B) {
    if (!packed || !Q || !A || !B) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    int64_t groups = K / OR_G;
    for (int64_t r = 0; r < N; ++r)
        unpack_row(K, packed, r, Q + r * K, A + r * groups * 16, B + r * groups * 4);
    return OR_OK;
}

/* ---- codes-only format (row-shared affine parameters) ---- */

#define OR_CODE_BYTES_PER_BLOCK 512 /* 16 rows * 32 code bytes per group */

int64_t oracle_codes_packed_bytes(int64_t N, int64_t K) {
    if (!shape_ok(N, K)) return OR_ESHAPE;
    return (N / OR_ROWBLOCK) * (K / OR_G) * OR_CODE_BYTES_PER_BLOCK;
}

/* Offset of slot 0's code field of group g of row block rb, and the slot stride. */
static void place_codes(int64_t K, int64_t rb, int64_t g, int64_t* off, int64_t* stride) {
    int64_t groups = K / OR_G;
    int64_t pkt = rb * groups * OR_CODE_BYTES_PER_BLOCK + (g / 2) * 2 * OR_CODE_BYTES_PER_BLOCK;
    if ((groups % 2 == 1) && (g == groups - 1)) {
        *off = pkt;
        *stride = 8;
    } else {
        *off = pkt + 8 * (g % 2);
        *stride = 16;
    }
}

int64_t oracle_pack_codes(int64_t N, int64_t K, const uint8_t* Q, uint8_t* out) {
    if (!Q || !out) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    int64_t groups = K / OR_G, bad = 0;
    memset(out, 0, (size_t)oracle_codes_packed_bytes(N, K));
    for (int64_t r = 0; r < N; ++r) {
        int64_t rb = r / OR_ROWBLOCK, rl = r % OR_ROWBLOCK;
        for (int64_t g = 0; g < groups; ++g) {
            int64_t off, stride;
            place_codes(K, rb, g, &off, &stride);
            for (int b = 0; b < OR_D; ++b) {
                uint8_t* field = out + off + (rl * 4 + b) * stride;
                for (int v = 0; v < 32; ++v) {
                    uint8_t q = Q[r * K + g * OR_G + 4 * v + b];
                    if (q > 3) ++bad;
                    field[(2 * v) / 8] |= (uint8_t)((q & 3) << ((2 * v) % 8));
                }
            }
        }
    }
    return bad;
}

static void unpack_codes_row(int64_t K, const uint8_t* packed, int64_t r, uint8_t* q_row) {
    int64_t groups = K / OR_G, rb = r / OR_ROWBLOCK, rl = r % OR_ROWBLOCK;
    for (int64_t g = 0; g < groups; ++g) {
        int64_t off, stride;
        place_codes(K, rb, g, &off, &stride);
        for (int b = 0; b < OR_D; ++b) {
            const uint8_t* field = packed + off + (rl * 4 + b) * stride;
            for (int v = 0; v < 32; ++v)
                q_row[g * OR_G + 4 * v + b] = (uint8_t)((field[(2 * v) / 8] >> ((2 * v) % 8)) & 3);
        }
    }
}

int oracle_unpack_codes(int64_t N, int64_t K, const uint8_t* packed, uint8_t* Q) {
    if (!packed || !Q) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    for (int64_t r = 0; r < N; ++r) unpack_codes_row(K, packed, r, Q + r * K);
    return OR_OK;
}

/* Every row's per-group parameters, replicated from the shared pairs. */
static void expand_shared(int64_t K, int64_t Ga, const uint16_t* As, const uint16_t* Bs, uint16_t* a_row,
                          uint16_t* b_row) {
    int64_t groups = K / OR_G;
    for (int64_t g = 0; g < groups; ++g) {
        int64_t src = Ga == 1 ? 0 : g;
        for (int i = 0; i < 16; ++i) a_row[g * 16 + i] = As[src * 16 + i];
        for (int i = 0; i < 4; ++i) b_row[g * 4 + i] = Bs[src * 4 + i];
    }
}

/* ---- nearest-codeword quantisation (the quantiser of Sec. 3.2.2 without
 *      Hessian feedback: each vector takes the affine-lattice point closest
 *      to it in Euclidean distance) ---- */

/* Squared distance between vector w[0..3] and the codeword A q + B of code
 * index i (q_b = bits 2b, 2b+1 of i), in fp64 with a fixed operation order:
 * c_a = B_a + A_a0 q_0 + A_a1 q_1 + A_a2 q_2 + A_a3 q_3 (left to right; each
 * product of an fp16 value and a small integer is exact), e_a = c_a - w_a,
 * d = fma(e_a, e_a, d) for a = 0..3 starting from d = 0. */
static double codeword_dist(const double* A16, const double* B4, const double* w, int i) {
    double d = 0.0;
    for (int a = 0; a < OR_D; ++a) {
        double c = B4[a];
        for (int b = 0; b < OR_D; ++b) c = c + A16[a * OR_D + b] * (double)((i >> (2 * b)) & 3);
        double e = c - w[a];
        d = fma(e, e, d);
    }
    return d;
}

/* W fp32 [N][K]; pairs per (row, group) when Ga == 0 (A [N][K/128][4][4],
 * B [N][K/128][4]), else row-shared (Ga = 1 or K/128, as the codes-only
 * format).  Q [N][K] receives, per vector, the codes of the nearest codeword;
 * ties go to the lowest index sum_b q_b 4^b. */
int oracle_quantize(int64_t N, int64_t K, const float* W, const uint16_t* A, const uint16_t* B, int64_t Ga,
                    uint8_t* Q) {
    if (!W || !A || !B || !Q) return OR_EINVAL;
    if (N <= 0 || K <= 0 || K % OR_G) return OR_ESHAPE;
    int64_t groups = K / OR_G;
    if (Ga != 0 && Ga != 1 && Ga != groups) return OR_ESHAPE;
    for (int64_t r = 0; r < N; ++r) {
        for (int64_t v = 0; v < K / OR_D; ++v) {
            int64_t g = (OR_D * v) / OR_G;
            int64_t set = Ga == 0 ? r * groups + g : (Ga == 1 ? 0 : g);
            double A16[16], B4[4], w[4];
            for (int i = 0; i < 16; ++i) A16[i] = oracle_half_to_double(A[set * 16 + i]);
            for (int i = 0; i < 4; ++i) B4[i] = oracle_half_to_double(B[set * 4 + i]);
            for (int i = 0; i < 4; ++i) w[i] = (double)W[r * K + OR_D * v + i];
            int best = 0;
            double dbest = codeword_dist(A16, B4, w, 0);
            for (int i = 1; i < 256; ++i) {
                double d = codeword_dist(A16, B4, w, i);
                if (d < dbest) { dbest = d; best = i; }
            }
            for (int b = 0; b < OR_D; ++b) Q[r * K + OR_D * v + b] = (uint8_t)((best >> (2 * b)) & 3);
        }
    }
    return OR_OK;
}

/* ---- randomized Hadamard transform (Sec. 3.2.1, Eq. 5) ----
 *
 * The paper rotates W into U S_U W S_V V with random sign diagonals S_U, S_V
 * and Hadamard matrices U, V; inference undoes it around the product:
 *     y = x W^T = ((x S_V V) W_rot^T) U S_U     (U, V normalised: H / sqrt(n)).
 * Hadamard matrix of order n (the paper names no construction; this is the
 * reading used throughout): n = 2^k * m with the largest k such that m = 1 or
 * m = q + 1 for a prime power q = p^e, e <= 3, q = 3 (mod 4); then
 * H_n = H_m (x) H_{2^k} (Kronecker product, index i = i_m * 2^k + i_2) with
 *   H_{2^k}[i][j] = (-1)^popcount(i & j)          (Sylvester)
 *   H_m = I + [[0, 1^T], [-1, Qj]]                  (Paley's first construction)
 * where Qj[a][b] = chi(a - b) over GF(q): elements are the base-p digit
 * vectors of 0..q-1 read as polynomials over GF(p) modulo the first monic
 * irreducible polynomial of degree e (coefficient vectors in lexicographic
 * order, constant term fastest), and chi is the quadratic character. */

typedef struct {
    int64_t k, m, q, p, e;
    int64_t f[4];        /* monic irreducible f(x) = x^e + f[e-1] x^(e-1) + ... + f[0] */
    signed char* chi;    /* chi of every element index, length q (NULL when m == 1) */
} had_spec;

static int is_prime(int64_t v) {
    if (v < 2) return 0;
    for (int64_t d = 2; d * d <= v; ++d) if (v % d == 0) return 0;
    return 1;
}

/* element index -> digits (constant term first) */
static void gf_digits(int64_t x, int64_t p, int64_t e, int64_t* c) {
    for (int64_t i = 0; i < e; ++i) { c[i] = x % p; x /= p; }
}

static int64_t gf_index(const int64_t* c, int64_t p, int64_t e) {
    int64_t x = 0;
    for (int64_t i = e - 1; i >= 0; --i) x = x * p + c[i];
    return x;
}

/* product of two field elements (digit vectors) modulo f */
static void gf_mul(const int64_t* a, const int64_t* b, const int64_t* f, int64_t p, int64_t e, int64_t* out) {
    int64_t t[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (int64_t i = 0; i < e; ++i)
        for (int64_t j = 0; j < e; ++j) t[i + j] = (t[i + j] + a[i] * b[j]) % p;
    /* reduce degrees 2e-2 .. e using x^e = -(f[e-1] x^(e-1) + ... + f[0]) */
    for (int64_t d = 2 * e - 2; d >= e; --d) {
        int64_t c = t[d];
        if (!c) continue;
        t[d] = 0;
        for (int64_t i = 0; i < e; ++i) t[d - e + i] = ((t[d - e + i] - c * f[i]) % p + p) % p;
    }
    for (int64_t i = 0; i < e; ++i) out[i] = t[i];
}

/* A monic polynomial of degree 2 or 3 is irreducible iff it has no root. */
static int poly_has_root(const int64_t* f, int64_t p, int64_t e) {
    for (int64_t x = 0; x < p; ++x) {
        int64_t v = 1;  /* leading coefficient */
        for (int64_t i = e - 1; i >= 0; --i) v = (v * x + f[i]) % p;
        if (v == 0) return 1;
    }
    return 0;
}

/* Fill spec for order n; returns 0 or OR_ESHAPE when n has no such form. */
static int had_factor(int64_t n, had_spec* hs) {
    memset(hs, 0, sizeof(*hs));
    if (n < 1) return OR_ESHAPE;
    int64_t k = 0;
    while ((n >> (k + 1)) << (k + 1) == n) ++k;  /* largest power of two dividing n */
    for (; k >= 0; --k) {
        int64_t m = n >> k;
        if (m == 1) { hs->k = k; hs->m = 1; return OR_OK; }
        int64_t q = m - 1;
        if (q % 4 != 3) continue;
        for (int64_t p = 2; p <= q; ++p) {
            if (!is_prime(p)) continue;
            int64_t pe = p, e = 1;
            while (pe < q && e < 3) { pe *= p; ++e; }
            if (pe != q) continue;
            hs->k = k; hs->m = m; hs->q = q; hs->p = p; hs->e = e;
            if (e > 1) {  /* first monic irreducible polynomial of degree e */
                int64_t found = 0;
                for (int64_t idx = 0; idx < q && !found; ++idx) {
                    gf_digits(idx, p, e, hs->f);
                    if (!poly_has_root(hs->f, p, e)) found = 1;
                }
                if (!found) return OR_ESHAPE;
            }
            return OR_OK;
        }
    }
    return OR_ESHAPE;
}

static int had_build_chi(had_spec* hs) {
    if (hs->m == 1) return OR_OK;
    int64_t q = hs->q, p = hs->p, e = hs->e;
    hs->chi = calloc((size_t)q, 1);
    if (!hs->chi) return OR_EINVAL;
    for (int64_t x = 1; x < q; ++x) hs->chi[x] = -1;
    for (int64_t y = 1; y < q; ++y) {
        int64_t a[4], sq[4];
        gf_digits(y, p, e, a);
        if (e == 1) sq[0] = (a[0] * a[0]) % p;
        else gf_mul(a, a, hs->f, p, e, sq);
        hs->chi[gf_index(sq, p, e)] = 1;
    }
    return OR_OK;
}

/* Entry (i, j) of the Paley matrix of order q + 1. */
static int paley_entry(const had_spec* hs, int64_t i, int64_t j) {
    if (i == 0) return 1;
    if (j == 0) return -1;
    if (i == j) return 1;
    int64_t a[4], b[4], d[4];
    gf_digits(i - 1, hs->p, hs->e, a);
    gf_digits(j - 1, hs->p, hs->e, b);
    for (int64_t t = 0; t < hs->e; ++t) d[t] = ((a[t] - b[t]) % hs->p + hs->p) % hs->p;
    return hs->chi[gf_index(d, hs->p, hs->e)];
}

static int had_entry(const had_spec* hs, int64_t i, int64_t j) {
    int64_t i2 = i & ((INT64_C(1) << hs->k) - 1), j2 = j & ((INT64_C(1) << hs->k) - 1);
    int sign = (__builtin_popcountll((unsigned long long)(i2 & j2)) & 1) ? -1 : 1;
    if (hs->m == 1) return sign;
    return sign * paley_entry(hs, i >> hs->k, j >> hs->k);
}

/* Order-n factor description: out[0..4] = k, m, q, p, e (m == 1: pure Sylvester). */
int oracle_hadamard_factor(int64_t n, int64_t* out) {
    had_spec hs;
    int st = had_factor(n, &hs);
    if (st != OR_OK) return st;
    out[0] = hs.k; out[1] = hs.m; out[2] = hs.q; out[3] = hs.p; out[4] = hs.e;
    return OR_OK;
}

/* The full +-1 matrix (row-major n x n). */
int oracle_hadamard(int64_t n, signed char* H) {
    if (!H) return OR_EINVAL;
    had_spec hs;
    int st = had_factor(n, &hs);
    if (st != OR_OK) return st;
    if ((st = had_build_chi(&hs)) != OR_OK) return st;
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j) H[i * n + j] = (signed char)had_entry(&hs, i, j);
    free(hs.chi);
    return OR_OK;
}

/* Rows of X [M][n] times the normalised Hadamard matrix, with the sign
 * vector s (+-1) applied before (mode 0: Y = (X diag(s)) H / sqrt(n), the
 * input side x S_V V) or after (mode 1: Y = (X H / sqrt(n)) diag(s), the output
 * side y U S_U).  Plain O(n^2) products, one sequential sum per element. */
int oracle_rht(int64_t n, int64_t M, const double* X, const signed char* s, int mode, double* Y) {
    if (!X || !s || !Y) return OR_EINVAL;
    if (M < 0 || (mode != 0 && mode != 1)) return OR_EINVAL;
    had_spec hs;
    int st = had_factor(n, &hs);
    if (st != OR_OK) return st;
    if ((st = had_build_chi(&hs)) != OR_OK) return st;
    /* the Paley factor as a table (its entries are needed n^2 / m^2 times each) */
    signed char* P = NULL;
    if (hs.m > 1) {
        P = malloc((size_t)(hs.m * hs.m));
        if (!P) { free(hs.chi); return OR_EINVAL; }
        for (int64_t a = 0; a < hs.m; ++a)
            for (int64_t b = 0; b < hs.m; ++b) P[a * hs.m + b] = (signed char)paley_entry(&hs, a, b);
    }
    double norm = 1.0 / sqrt((double)n);
    int64_t mask = (INT64_C(1) << hs.k) - 1;
    for (int64_t t = 0; t < M; ++t) {
        for (int64_t j = 0; j < n; ++j) {
            double acc = 0.0;
            for (int64_t i = 0; i < n; ++i) {
                double xv = X[t * n + i] * (mode == 0 ? (double)s[i] : 1.0);
                int h = (__builtin_popcountll((unsigned long long)(i & j & mask)) & 1) ? -1 : 1;
                if (P) h *= P[(i >> hs.k) * hs.m + (j >> hs.k)];
                acc += xv * (double)h;
            }
            Y[t * n + j] = acc * norm * (mode == 1 ? (double)s[j] : 1.0);
        }
    }
    free(P);
    free(hs.chi);
    return OR_OK;
}

/* ---- decode (Eq. 4 applied along the input dimension as in Eq. 8) ---- */

/* One row: w[k] for k = 4v + a is sum_b A[g][a][b] * q[4v + b] + B[g][a],
 * g = (4v) / 128.  Every product is an fp16 value times a small integer, so the
 * fp64 result is exact. */
static void decode_row(int64_t K, const uint8_t* q_row, const uint16_t* a_row, const uint16_t* b_row,
                       double* w) {
    for (int64_t v = 0; v < K / OR_D; ++v) {
        int64_t g = (OR_D * v) / OR_G;
        for (int a = 0; a < OR_D; ++a) {
            double acc = oracle_half_to_double(b_row[g * OR_D + a]);
            for (int b = 0; b < OR_D; ++b)
                acc += oracle_half_to_double(a_row[(g * OR_D + a) * OR_D + b]) * (double)q_row[OR_D * v + b];
            w[OR_D * v + a] = acc;
        }
    }
}

/* Decode from canonical arrays (no packing involved).  W is [N][K] fp64.
 * Codes are used as given (values above 3 are not masked). */
int oracle_decode(int64_t N, int64_t K, const uint8_t* Q, const uint16_t* A, const uint16_t* B,
                  double* W) {
    if (!Q || !A || !B || !W) return OR_EINVAL;
    if (N <= 0 || K <= 0 || K % OR_G) return OR_ESHAPE;
    int64_t groups = K / OR_G;
    for (int64_t r = 0; r < N; ++r)
        decode_row(K, Q + r * K, A + r * groups * 16, B + r * groups * 4, W + r * K);
    return OR_OK;
}

/* Decode rows [r0, r1) straight from packed bytes into W [(r1-r0)][K]. */
int oracle_decode_packed_rows(int64_t N, int64_t K, const uint8_t* packed, int64_t r0, int64_t r1,
                              double* W) {
    if (!packed || !W) return OR_EINVAL;
    if (!shape_ok(N, K) || r0 < 0 || r1 > N || r0 > r1) return OR_ESHAPE;
    int64_t groups = K / OR_G;
    uint8_t* q = malloc((size_t)K);
    uint16_t* a = malloc((size_t)groups * 16 * sizeof(uint16_t));
    uint16_t* b = malloc((size_t)groups * 4 * sizeof(uint16_t));
    if (!q || !a || !b) { free(q); free(a); free(b); return OR_EINVAL; }
    for (int64_t r = r0; r < r1; ++r) {
        unpack_row(K, packed, r, q, a, b);
        decode_row(K, q, a, b, W + (r - r0) * K);
    }
    free(q); free(a); free(b);
    return OR_OK;
}

/* ---- product Y = X * W_hat^T (Eq. 1), rows of W decoded one at a time ---- */

typedef struct {
    int64_t N, K, M, nrows;
    const uint8_t* packed;
    const double* X;
    const int64_t* rows; /* NULL: all rows in order */
    double* Y;           /* [M][nrows] */
    int64_t first, last; /* index range into the row list for this worker */
    const uint16_t *As, *Bs; /* non-NULL: codes-only bytes with row-shared parameters */
    int64_t Ga;
    int status;
} mm_job;

static void* mm_worker(void* arg) {
    mm_job* j = (mm_job*)arg;
    int64_t K = j->K, groups = K / OR_G;
    uint8_t* q = malloc((size_t)K);
    uint16_t* a = malloc((size_t)groups * 16 * sizeof(uint16_t));
    uint16_t* b = malloc((size_t)groups * 4 * sizeof(uint16_t));
    double* w = malloc((size_t)K * sizeof(double));
    if (!q || !a || !b || !w) { j->status = OR_EINVAL; goto done; }
    if (j->As) expand_shared(K, j->Ga, j->As, j->Bs, a, b);
    for (int64_t i = j->first; i < j->last; ++i) {
        int64_t r = j->rows ? j->rows[i] : i;
        if (j->As)
            unpack_codes_row(K, j->packed, r, q);
        else
            unpack_row(K, j->packed, r, q, a, b);
        decode_row(K, q, a, b, w);
        for (int64_t t = 0; t < j->M; ++t) {
            const double* x = j->X + t * K;
            double acc = 0.0;
            for (int64_t k = 0; k < K; ++k) acc += x[k] * w[k];
            j->Y[t * j->nrows + i] = acc;
        }
    }
    j->status = OR_OK;
done:
    free(q); free(a); free(b); free(w);
    return NULL;
}

/* Y[t][i] = sum_k X[t][k] * W_hat[rows[i]][k] for the listed rows (all rows
 * when rows == NULL, then nrows must equal N).  Work is split over `threads`
 * POSIX threads by output row; each Y element is one plain sequential sum. */
static int matmul_rows(int64_t N, int64_t K, const uint8_t* packed, int64_t Ga, const uint16_t* As,
                       const uint16_t* Bs, int64_t M, const double* X, int64_t nrows, const int64_t* rows,
                       double* Y, int threads) {
    if (!packed || !X || !Y) return OR_EINVAL;
    if (!shape_ok(N, K) || M < 0 || nrows < 0) return OR_ESHAPE;
    if (!rows && nrows != N) return OR_ESHAPE;
    if (rows)
        for (int64_t i = 0; i < nrows; ++i)
            if (rows[i] < 0 || rows[i] >= N) return OR_EINVAL;
    if (M == 0 || nrows == 0) return OR_OK;
    if (threads < 1) threads = 1;
    if (threads > nrows) threads = (int)nrows;
    mm_job* jobs = calloc((size_t)threads, sizeof(mm_job));
    pthread_t* tids = calloc((size_t)threads, sizeof(pthread_t));
    if (!jobs || !tids) { free(jobs); free(tids); return OR_EINVAL; }
    int64_t per = (nrows + threads - 1) / threads;
    int status = OR_OK;
    for (int t = 0; t < threads; ++t) {
        mm_job* j = &jobs[t];
        j->N = N; j->K = K; j->M = M; j->nrows = nrows;
        j->packed = packed; j->X = X; j->rows = rows; j->Y = Y;
        j->As = As; j->Bs = Bs; j->Ga = Ga;
        j->first = t * per;
        j->last = (t + 1) * per < nrows ? (t + 1) * per : nrows;
        if (j->first > j->last) j->first = j->last;
        if (threads == 1) mm_worker(j);
        else if (pthread_create(&tids[t], NULL, mm_worker, j) != 0) { mm_worker(j); tids[t] = 0; }
    }
    if (threads > 1)
        for (int t = 0; t < threads; ++t)
            if (tids[t]) pthread_join(tids[t], NULL);
    for (int t = 0; t < threads; ++t)
        if (jobs[t].status != OR_OK) status = jobs[t].status;
    free(jobs); free(tids);
    return status;
}

int oracle_matmul_rows(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const double* X,
                       int64_t nrows, const int64_t* rows, double* Y, int threads) {
    return matmul_rows(N, K, packed, 0, NULL, NULL, M, X, nrows, rows, Y, threads);
}

int oracle_matmul(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const double* X, double* Y,
                  int threads) {
    return oracle_matmul_rows(N, K, packed, M, X, N, NULL, Y, threads);
}

/* The same product from codes-only bytes and row-shared parameters: every row
 * decodes with pair (Ga == 1 ? 0 : g) of its group g. */
int oracle_matmul_shared_rows(int64_t N, int64_t K, const uint8_t* packed_codes, int64_t Ga,
                              const uint16_t* As, const uint16_t* Bs, int64_t M, const double* X,
                              int64_t nrows, const int64_t* rows, double* Y, int threads) {
    if (!As || !Bs) return OR_EINVAL;
    if (K % OR_G || (Ga != 1 && Ga != K / OR_G)) return OR_ESHAPE;
    return matmul_rows(N, K, packed_codes, Ga, As, Bs, M, X, nrows, rows, Y, threads);
}

/* ======================================================================
 * Format variants: b-bit codes (b = 2 or 3; Sec. 5.2.5, bit-width
 * extensibility: the integer vectors only widen) and d-dimensional vectors
 * (d = 4 or 8; Sec. 5.2.3, vector dimension), with the pairs shared by all
 * rows as the paper keeps them (one (A, B) per weight matrix, Sec. 4.2; or
 * one per 128-column group).  Restated from the definition of the variant
 * codes-only format (include/unisvq.h, variant format block):
 *   One group of one row block takes CB = 512 (b = 2) or 768 (b = 3) bytes;
 *   row block rb starts at rb*(K/128)*CB; packet p (groups 2p, 2p+1) is
 *   2*CB bytes at p*2*CB, a final half packet (odd K/128) CB bytes.
 *   Slot s = 0..63: row r = 16rb + s/4, lane index j = s%4.  The slot's 32
 *   codes of group g are numbered (h, u), h = 0..1, u = 0..15:
 *     d = 4: Q[r][128g + 4(16h + u) + j]  (vector 16h+u, component j)
 *     d = 8: Q[r][128g + 8u + 4h + j]     (vector u, component 4h+j)
 *   Low field (8 bytes): 32-bit word h, bits 2u and 2u+1 = bits 0, 1 of code (h, u).
 *   High field (b = 3, 4 bytes): bit 8n + 4m + 2h + p = bit 2 of code
 *     (h, u = 4n + 2m + p), n = 0..3, m, p = 0..1.
 *   Full packet at P: low field of group 2p+jj at P + 16s + 8jj, high field
 *   at P + 1024 + 8s + 4jj.  Half packet: low at P + 8s, high at P + 512 + 4s.
 *   Shared pairs As fp16 [Ga][d][d] (As[a][b] multiplies q_b into component
 *   a), Bs fp16 [Ga][d], Ga = 1 or K/128; group g uses pair (Ga == 1 ? 0 : g).
 *   Affine block: records of RB = 160 (d = 4) or 576 (d = 8) bytes, one per
 *   pair of groups (a single record when Ga = 1); record R serves groups
 *   2R + jj with pair pi = (Ga == 1 ? 0 : 2R + jj); a group past the last
 *   holds zeros.  Inside a record (fp16 each):
 *     lane view, d = 4: As[pi][a][j] at 16j + 8jj + 2a;  Bs[pi][j] at 64 + 4j + 2jj
 *     lane view, d = 8: As[pi][a][4h+j] at 64j + 32jj + 16h + 2a (a = 0..7);
 *                       Bs[pi][4h+j] at 256 + 8j + 4jj + 2h
 *     row view at V = 80 (d = 4) or 288 (d = 8), E = 2(d*d + d):
 *                       As[pi][a][b] at V + jj*E + 2(d*a + b);  Bs[pi][a] at V + jj*E + 2*d*d + 2a
 * ====================================================================== */

static int var_ok(int bits, int d) { return (bits == 2 || bits == 3) && (d == 4 || d == 8); }

static int64_t var_group_bytes(int bits) { return bits == 3 ? 768 : 512; }

int64_t oracle_var_codes_bytes(int64_t N, int64_t K, int bits) {
    if (bits != 2 && bits != 3) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    return (N / OR_ROWBLOCK) * (K / OR_G) * var_group_bytes(bits);
}

/* Column (within the row) of code (h, u) of lane index j in group g. */
static int64_t var_column(int d, int64_t g, int h, int u, int j) {
    if (d == 4) return g * OR_G + 4 * (16 * h + u) + j;
    return g * OR_G + 8 * u + 4 * h + j;
}

/* Byte offsets of the low and high fields of slot s, group g, row block rb. */
static void var_place(int64_t K, int bits, int64_t rb, int64_t g, int s, int64_t* lo, int64_t* hi) {
    int64_t groups = K / OR_G, cb = var_group_bytes(bits);
    int64_t P = rb * groups * cb + (g / 2) * 2 * cb;
    if ((groups % 2 == 1) && (g == groups - 1)) {
        *lo = P + 8 * s;
        *hi = P + 512 + 4 * s;
    } else {
        *lo = P + 16 * s + 8 * (g % 2);
        *hi = P + 1024 + 8 * s + 4 * (g % 2);
    }
}

/* Bit position of code (h, u) inside the high field. */
static int var_hi_bit(int h, int u) {
    int n = u / 4, m = (u / 2) % 2, p = u % 2;
    return 8 * n + 4 * m + 2 * h + p;
}

static void set_bit(uint8_t* base, int bit) { base[bit / 8] |= (uint8_t)(1u << (bit % 8)); }
static int get_bit(const uint8_t* base, int bit) { return (base[bit / 8] >> (bit % 8)) & 1; }

/* Pack Q [N][K] (codes 0..2^bits-1; larger ones are counted and stored
 * modulo 2^bits).  Returns the count of such codes. */
int64_t oracle_var_pack_codes(int64_t N, int64_t K, int bits, int d, const uint8_t* Q, uint8_t* out) {
    if (!Q || !out || !var_ok(bits, d)) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    int64_t groups = K / OR_G, bad = 0;
    int top = 1 << bits;
    memset(out, 0, (size_t)oracle_var_codes_bytes(N, K, bits));
    for (int64_t r = 0; r < N; ++r) {
        int64_t rb = r / OR_ROWBLOCK, rl = r % OR_ROWBLOCK;
        for (int64_t g = 0; g < groups; ++g)
            for (int j = 0; j < 4; ++j) {
                int s = (int)(rl * 4 + j);
                int64_t lo, hi;
                var_place(K, bits, rb, g, s, &lo, &hi);
                for (int h = 0; h < 2; ++h)
                    for (int u = 0; u < 16; ++u) {
                        int q = Q[r * K + var_column(d, g, h, u, j)];
                        if (q >= top) ++bad;
                        q %= top;
                        /* word h of the low field: bits 32h + 2u, 32h + 2u + 1 */
                        if (q & 1) set_bit(out + lo, 32 * h + 2 * u);
                        if (q & 2) set_bit(out + lo, 32 * h + 2 * u + 1);
                        if (bits == 3 && (q & 4)) set_bit(out + hi, var_hi_bit(h, u));
                    }
            }
    }
    return bad;
}

static void var_unpack_row(int64_t K, int bits, int d, const uint8_t* packed, int64_t r, uint8_t* q_row) {
    int64_t groups = K / OR_G, rb = r / OR_ROWBLOCK, rl = r % OR_ROWBLOCK;
    for (int64_t g = 0; g < groups; ++g)
        for (int j = 0; j < 4; ++j) {
            int s = (int)(rl * 4 + j);
            int64_t lo, hi;
            var_place(K, bits, rb, g, s, &lo, &hi);
            for (int h = 0; h < 2; ++h)
                for (int u = 0; u < 16; ++u) {
                    int q = get_bit(packed + lo, 32 * h + 2 * u) | (get_bit(packed + lo, 32 * h + 2 * u + 1) << 1);
                    if (bits == 3) q |= get_bit(packed + hi, var_hi_bit(h, u)) << 2;
                    q_row[var_column(d, g, h, u, j)] = (uint8_t)q;
                }
        }
}

int oracle_var_unpack_codes(int64_t N, int64_t K, int bits, int d, const uint8_t* packed, uint8_t* Q) {
    if (!packed || !Q || !var_ok(bits, d)) return OR_EINVAL;
    if (!shape_ok(N, K)) return OR_ESHAPE;
    for (int64_t r = 0; r < N; ++r) var_unpack_row(K, bits, d, packed, r, Q + r * K);
    return OR_OK;
}

static int64_t var_record_bytes(int d) { return d == 4 ? 160 : 576; }

int64_t oracle_var_affine_bytes(int64_t K, int64_t Ga, int d) {
    if (d != 4 && d != 8) return OR_EINVAL;
    if (K <= 0 || K % OR_G) return OR_ESHAPE;
    if (Ga != 1 && Ga != K / OR_G) return OR_EINVAL;
    int64_t records = Ga == 1 ? 1 : (K / OR_G + 1) / 2;
    return records * var_record_bytes(d);
}

/* Offsets (inside record R) of As[pi][a][b] and Bs[pi][a] in the lane view
 * and in the row view, for the record's group jj. */
static int64_t var_lane_a(int d, int jj, int a, int b) {
    if (d == 4) return 16 * b + 8 * jj + 2 * a;
    return 64 * (b % 4) + 32 * jj + 16 * (b / 4) + 2 * a;
}
static int64_t var_lane_b(int d, int jj, int a) {
    if (d == 4) return 64 + 4 * a + 2 * jj;
    return 256 + 8 * (a % 4) + 4 * jj + 2 * (a / 4);
}
static int64_t var_row_a(int d, int jj, int a, int b) {
    int64_t V = d == 4 ? 80 : 288, E = 2 * (d * d + d);
    return V + jj * E + 2 * (d * a + b);
}
static int64_t var_row_b(int d, int jj, int a) {
    int64_t V = d == 4 ? 80 : 288, E = 2 * (d * d + d);
    return V + jj * E + 2 * d * d + 2 * a;
}

int oracle_var_pack_affine(int64_t K, int64_t Ga, int d, const uint16_t* As, const uint16_t* Bs, uint8_t* out) {
    if (!As || !Bs || !out) return OR_EINVAL;
    int64_t total = oracle_var_affine_bytes(K, Ga, d);
    if (total < 0) return (int)total;
    int64_t groups = K / OR_G, rb = var_record_bytes(d), records = total / rb;
    memset(out, 0, (size_t)total);
    for (int64_t R = 0; R < records; ++R)
        for (int jj = 0; jj < 2; ++jj) {
            int64_t g = 2 * R + jj;
            if (Ga != 1 && g >= groups) continue; /* past the last group: zeros */
            int64_t pi = Ga == 1 ? 0 : g;
            uint8_t* rec = out + R * rb;
            for (int a = 0; a < d; ++a) {
                for (int b = 0; b < d; ++b) {
                    uint16_t v = As[(pi * d + a) * d + b];
                    put_u16(rec + var_lane_a(d, jj, a, b), v);
                    put_u16(rec + var_row_a(d, jj, a, b), v);
                }
                put_u16(rec + var_lane_b(d, jj, a), Bs[pi * d + a]);
                put_u16(rec + var_row_b(d, jj, a), Bs[pi * d + a]);
            }
        }
    return OR_OK;
}

/* Inverse of oracle_var_pack_affine, read from the lane view; returns
 * OR_EINVAL if the row view disagrees with it anywhere. */
int oracle_var_unpack_affine(int64_t K, int64_t Ga, int d, const uint8_t* rec_block, uint16_t* As, uint16_t* Bs) {
    if (!rec_block || !As || !Bs) return OR_EINVAL;
    int64_t total = oracle_var_affine_bytes(K, Ga, d);
    if (total < 0) return (int)total;
    int64_t rb = var_record_bytes(d);
    for (int64_t pi = 0; pi < Ga; ++pi) {
        int64_t R = Ga == 1 ? 0 : pi / 2;
        int jj = Ga == 1 ? 0 : (int)(pi % 2);
        const uint8_t* rec = rec_block + R * rb;
        for (int a = 0; a < d; ++a) {
            for (int b = 0; b < d; ++b) {
                uint16_t v = get_u16(rec + var_lane_a(d, jj, a, b));
                if (v != get_u16(rec + var_row_a(d, jj, a, b))) return OR_EINVAL;
                As[(pi * d + a) * d + b] = v;
            }
            uint16_t v = get_u16(rec + var_lane_b(d, jj, a));
            if (v != get_u16(rec + var_row_b(d, jj, a))) return OR_EINVAL;
            Bs[pi * d + a] = v;
        }
    }
    return OR_OK;
}

/* One row: vector v covers columns d*v .. d*v+d-1 (Eq. 8); component a is
 * sum_b As[pi][a][b] * q[dv + b] + Bs[pi][a] (Eq. 4), pi the pair of group
 * g = d*v / 128.  Products of fp16 values and integers below 8 are exact in
 * fp64, and so is the sum of at most 8 of them plus B. */
static void var_decode_row(int64_t K, int d, const uint8_t* q_row, int64_t Ga, const uint16_t* As,
                           const uint16_t* Bs, double* w) {
    for (int64_t v = 0; v < K / d; ++v) {
        int64_t g = (d * v) / OR_G, pi = Ga == 1 ? 0 : g;
        for (int a = 0; a < d; ++a) {
            double acc = oracle_half_to_double(Bs[pi * d + a]);
            for (int b = 0; b < d; ++b)
                acc += oracle_half_to_double(As[(pi * d + a) * d + b]) * (double)q_row[d * v + b];
            w[d * v + a] = acc;
        }
    }
}

/* Decode canonical codes (no packing); N may be any positive count. */
int oracle_var_decode(int64_t N, int64_t K, int d, const uint8_t* Q, int64_t Ga, const uint16_t* As,
                      const uint16_t* Bs, double* W) {
    if (!Q || !As || !Bs || !W || (d != 4 && d != 8)) return OR_EINVAL;
    if (N <= 0 || K <= 0 || K % OR_G) return OR_ESHAPE;
    if (Ga != 1 && Ga != K / OR_G) return OR_EINVAL;
    for (int64_t r = 0; r < N; ++r) var_decode_row(K, d, Q + r * K, Ga, As, Bs, W + r * K);
    return OR_OK;
}

typedef struct {
    int64_t N, K, M, nrows, Ga;
    int bits, d;
    const uint8_t* packed;
    const uint16_t *As, *Bs;
    const double* X;
    const int64_t* rows;
    double* Y;
    int64_t first, last;
    int status;
} var_job;

static void* var_worker(void* arg) {
    var_job* j = (var_job*)arg;
    uint8_t* q = malloc((size_t)j->K);
    double* w = malloc((size_t)j->K * sizeof(double));
    if (!q || !w) { j->status = OR_EINVAL; free(q); free(w); return NULL; }
    for (int64_t i = j->first; i < j->last; ++i) {
        int64_t r = j->rows ? j->rows[i] : i;
        var_unpack_row(j->K, j->bits, j->d, j->packed, r, q);
        var_decode_row(j->K, j->d, q, j->Ga, j->As, j->Bs, w);
        for (int64_t t = 0; t < j->M; ++t) {
            const double* x = j->X + t * j->K;
            double acc = 0.0;
            for (int64_t k = 0; k < j->K; ++k) acc += x[k] * w[k];
            j->Y[t * j->nrows + i] = acc;
        }
    }
    j->status = OR_OK;
    free(q); free(w);
    return NULL;
}

/* Y[t][i] = sum_k X[t][k] * W_hat[rows[i]][k] (Eq. 1) from variant codes-only
 * bytes and the canonical shared pairs; rows == NULL means all N rows. */
int oracle_var_matmul_rows(int64_t N, int64_t K, int bits, int d, const uint8_t* packed, int64_t Ga,
                           const uint16_t* As, const uint16_t* Bs, int64_t M, const double* X, int64_t nrows,
                           const int64_t* rows, double* Y, int threads) {
    if (!packed || !As || !Bs || !X || !Y || !var_ok(bits, d)) return OR_EINVAL;
    if (!shape_ok(N, K) || M < 0 || nrows < 0) return OR_ESHAPE;
    if (Ga != 1 && Ga != K / OR_G) return OR_EINVAL;
    if (!rows && nrows != N) return OR_ESHAPE;
    if (rows)
        for (int64_t i = 0; i < nrows; ++i)
            if (rows[i] < 0 || rows[i] >= N) return OR_EINVAL;
    if (M == 0 || nrows == 0) return OR_OK;
    if (threads < 1) threads = 1;
    if (threads > nrows) threads = (int)nrows;
    var_job* jobs = calloc((size_t)threads, sizeof(var_job));
    pthread_t* tids = calloc((size_t)threads, sizeof(pthread_t));
    if (!jobs || !tids) { free(jobs); free(tids); return OR_EINVAL; }
    int64_t per = (nrows + threads - 1) / threads;
    for (int t = 0; t < threads; ++t) {
        var_job* j = &jobs[t];
        j->N = N; j->K = K; j->M = M; j->nrows = nrows; j->Ga = Ga;
        j->bits = bits; j->d = d; j->packed = packed; j->As = As; j->Bs = Bs;
        j->X = X; j->rows = rows; j->Y = Y;
        j->first = t * per;
        j->last = (t + 1) * per < nrows ? (t + 1) * per : nrows;
        if (j->first > j->last) j->first = j->last;
        if (threads == 1) var_worker(j);
        else if (pthread_create(&tids[t], NULL, var_worker, j) != 0) { var_worker(j); tids[t] = 0; }
    }
    int status = OR_OK;
    if (threads > 1)
        for (int t = 0; t < threads; ++t)
            if (tids[t]) pthread_join(tids[t], NULL);
    for (int t = 0; t < threads; ++t)
        if (jobs[t].status != OR_OK) status = jobs[t].status;
    free(jobs); free(tids);
    return status;
}

/* ---- LDLQ: nearest-codeword rounding with Hessian error feedback
 *      (Sec. 3.2.2, Eq. 7; regularisation of Sec. 4.2) ----
 * Vectors of d = 4 consecutive columns are rounded left to right.  Before
 * vector j (columns 4j..4j+3) is rounded, its weights are moved by the errors
 * of all earlier columns (Eq. 7):
 *     u_c = W[r][4j+c] + sum_{k < 4j} E[r][k] * U[k][4j+c],
 *     E[r][k] = W[r][k] - W_hat[r][k],
 * where the adjustment coefficients are the off-diagonal entries of the
 * factor of H = U D U^T with U unit upper block triangular (4 x 4 identity
 * blocks on the diagonal) and D block diagonal -- the orientation for which
 * the proxy loss tr(E H E^T) splits into independent per-vector terms when
 * columns run left to right (checked by a pin).  u is rounded to the nearest
 * codeword with the operation order and tie rule of oracle_quantize.
 * Arithmetic: the sum is one fma chain in increasing k starting from 0, then
 * u = W + sum; codewords and E in fp64 (exact: fp16 times a small integer).
 *   U   fp64 [K][K] row-major; only U[k][c] with k < 4 floor(c / 4) is read
 *   E   nullable fp64 [N][K]: the errors W - W_hat */
typedef struct {
    int64_t N, K, Ga, r0, r1;
    const float* W;
    const double* U;
    const uint16_t *A, *B;
    uint8_t* Q;
    double* E;
    int status;
} ldlq_job;

static void* ldlq_worker(void* arg) {
    ldlq_job* jb = (ldlq_job*)arg;
    int64_t K = jb->K, groups = K / OR_G;
    double* e = malloc((size_t)K * sizeof(double));
    if (!e) { jb->status = OR_EINVAL; return NULL; }
    for (int64_t r = jb->r0; r < jb->r1; ++r) {
        for (int64_t v = 0; v < K / OR_D; ++v) {
            int64_t j0 = OR_D * v, g = j0 / OR_G;
            int64_t set = jb->Ga == 0 ? r * groups + g : (jb->Ga == 1 ? 0 : g);
            double A16[16], B4[4], u[4];
            for (int i = 0; i < 16; ++i) A16[i] = oracle_half_to_double(jb->A[set * 16 + i]);
            for (int i = 0; i < 4; ++i) B4[i] = oracle_half_to_double(jb->B[set * 4 + i]);
            for (int c = 0; c < OR_D; ++c) {
                double s = 0.0;
                for (int64_t k = 0; k < j0; ++k) s = fma(e[k], jb->U[k * K + j0 + c], s);
                u[c] = (double)jb->W[r * K + j0 + c] + s;
            }
            int best = 0;
            double dbest = codeword_dist(A16, B4, u, 0);
            for (int i = 1; i < 256; ++i) {
                double d = codeword_dist(A16, B4, u, i);
                if (d < dbest) { dbest = d; best = i; }
            }
            for (int a = 0; a < OR_D; ++a) {
                double cw = B4[a];
                for (int b = 0; b < OR_D; ++b) cw = cw + A16[a * OR_D + b] * (double)((best >> (2 * b)) & 3);
                e[j0 + a] = (double)jb->W[r * K + j0 + a] - cw;
                jb->Q[r * K + j0 + a] = (uint8_t)((best >> (2 * a)) & 3);
            }
        }
        if (jb->E) memcpy(jb->E + r * K, e, (size_t)K * sizeof(double));
    }
    free(e);
    jb->status = OR_OK;
    return NULL;
}

int oracle_ldlq(int64_t N, int64_t K, const float* W, const double* U, const uint16_t* A, const uint16_t* B,
                int64_t Ga, uint8_t* Q, double* E, int threads) {
    if (!W || !U || !A || !B || !Q) return OR_EINVAL;
    if (N <= 0 || K <= 0 || K % OR_G) return OR_ESHAPE;
    if (Ga != 0 && Ga != 1 && Ga != K / OR_G) return OR_ESHAPE;
    if (threads < 1) threads = 1;
    if (threads > N) threads = (int)N;
    ldlq_job* jobs = calloc((size_t)threads, sizeof(ldlq_job));
    pthread_t* tids = calloc((size_t)threads, sizeof(pthread_t));
    if (!jobs || !tids) { free(jobs); free(tids); return OR_EINVAL; }
    int64_t per = (N + threads - 1) / threads;
    for (int t = 0; t < threads; ++t) {
        ldlq_job* jb = &jobs[t];
        jb->N = N; jb->K = K; jb->Ga = Ga; jb->W = W; jb->U = U; jb->A = A; jb->B = B; jb->Q = Q; jb->E = E;
        jb->r0 = t * per < N ? t * per : N;
        jb->r1 = (t + 1) * per < N ? (t + 1) * per : N;
        if (threads == 1) ldlq_worker(jb);
        else if (pthread_create(&tids[t], NULL, ldlq_worker, jb) != 0) { ldlq_worker(jb); tids[t] = 0; }
    }
    int status = OR_OK;
    if (threads > 1)
        for (int t = 0; t < threads; ++t)
            if (tids[t]) pthread_join(tids[t], NULL);
    for (int t = 0; t < threads; ++t)
        if (jobs[t].status != OR_OK) status = jobs[t].status;
    free(jobs); free(tids);
    return status;
}
