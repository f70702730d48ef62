// Randomized Hadamard transform around the product (Sec. 3.2.1, Eq. 5) on
// gfx950.  The weights are quantised in the rotated basis W_rot = U S_U W S_V V,
// so inference computes  y = ((x S_V V) W_rot^T) U S_U  with the normalised
// Hadamard matrices U = H_N / sqrt(N), V = H_K / sqrt(K):
//   input side  (mode 0):  x' = (x diag(s)) H / sqrt(n)
//   output side (mode 1):  y  = (y' H / sqrt(n)) diag(s)
// Hadamard matrix of order n: n = 2^k * m with the largest k such that m = 1
// or m = q + 1, q = p^e a prime power = 3 (mod 4), e <= 3; H = P (x) S with S
// the Sylvester matrix of order 2^k ((-1)^popcount(i & j)) and P Paley's first
// construction over GF(q) (I + [[0, 1^T], [-1, Qj]], Qj[a][b] = chi(a - b);
// elements are base-p digit vectors of their indices, polynomials modulo the
// first monic irreducible polynomial of degree e, chi the quadratic character).
//
// One workgroup per (row, slice of output blocks).  The row goes to LDS in
// fp32 (signs applied on the input side); the Paley factor, if any, runs as a
// dense product for the workgroup's output blocks -- on the matrix cores in
// fp32 (rht_paley_kernel), or on the vector ALUs when its tables would not fit
// the LDS (rht_kernel) -- with its entries built in LDS from the quadratic
// character, then the Sylvester factor as an in-place fast transform inside
// each of those blocks of 2^k.  fp32 throughout, one rounding to the output
// dtype.
#include <cmath>
#include <type_traits>

#include "common.hpp"
#include "fwht.hpp"

namespace unisvq {

struct HadSpec {
    int k, m, q, p, e;
    int f[3];  // f(x) = x^e + f[e-1] x^(e-1) + ... + f[0]
};

namespace {

constexpr int kRhtThreads = 1024;
constexpr int kRhtMaxN = 32768;  // fp32 row in LDS

// Sign i through a buffer descriptor: reads past the end return zero, so the
// load needs no guarding branch (a branch would make the wait counters drain
// at its join).
__device__ inline float ld_sign(__amdgpu_buffer_rsrc_t r, int i) {
    return static_cast<float>(static_cast<signed char>(__builtin_amdgcn_raw_buffer_load_b8(r, static_cast<uint32_t>(i), 0, 0)));
}

// Eight consecutive elements of a row and their signs: raw bits from one or
// two 16-byte loads and one 8-byte load (wide loads keep the address units'
// work per element low; a row is read by every workgroup of a Paley launch).
template <typename XT>
struct RowChunk {
    uint4 a, b;  // b used for fp32 only
    uint2 s;
};

template <typename XT>
__device__ inline void fetch_chunk(__amdgpu_buffer_rsrc_t rx, __amdgpu_buffer_rsrc_t rs, int i0, RowChunk<XT>& c) {
    const uint32_t off = static_cast<uint32_t>(i0) * sizeof(XT);
    c.a = ld128(rx, off);
    if constexpr (sizeof(XT) == 4) c.b = ld128(rx, off + 16u);
    c.s = ld64(rs, static_cast<uint32_t>(i0));
}

// The chunk's elements as fp32, times their signs on the input side (mode 0),
// into z[i0 .. i0 + 8) where below n.
template <typename XT>
__device__ inline void put_chunk(const RowChunk<XT>& c, int i0, int n, int mode, float* z) {
    float v[8];
    if constexpr (sizeof(XT) == 4) {
        const uint32_t w[8] = {c.a.x, c.a.y, c.a.z, c.a.w, c.b.x, c.b.y, c.b.z, c.b.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = __builtin_bit_cast(float, w[e]);
    } else {
        const uint32_t w[4] = {c.a.x, c.a.y, c.a.z, c.a.w};
#pragma unroll
        for (int e = 0; e < 8; ++e)
            v[e] = static_cast<float>(__builtin_bit_cast(XT, static_cast<uint16_t>(w[e >> 1] >> (16 * (e & 1)))));
    }
    if (mode == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const uint32_t sw = e < 4 ? c.s.x : c.s.y;
            v[e] *= static_cast<float>(static_cast<signed char>((sw >> (8 * (e & 3))) & 0xffu));
        }
    }
    if (i0 + 8 <= n) {
        *reinterpret_cast<f32x4*>(z + i0) = f32x4{v[0], v[1], v[2], v[3]};
        *reinterpret_cast<f32x4*>(z + i0 + 4) = f32x4{v[4], v[5], v[6], v[7]};
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (i0 + e < n) z[i0 + e] = v[e];
    }
}

// The row into LDS as fp32 (signs applied on the input side).
template <typename XT>
__device__ inline void load_row(const XT* __restrict__ xr, const signed char* __restrict__ signs, int mode, int n,
                                float* z, int tid) {
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(xr, static_cast<uint32_t>(n) * sizeof(XT));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(signs, static_cast<uint32_t>(n));
    constexpr int C = kRhtMaxN / (8 * kRhtThreads);
    RowChunk<XT> c[C];
#pragma unroll
    for (int u = 0; u < C; ++u) fetch_chunk<XT>(rx, rs, 8 * (tid + u * kRhtThreads), c[u]);
#pragma unroll
    for (int u = 0; u < C; ++u) put_chunk<XT>(c[u], 8 * (tid + u * kRhtThreads), n, mode, z);
}

// x mod p for |x| < 2^22 through the float reciprocal rp = 1/p: the quotient
// estimate is off by at most one, which one correction either way fixes.
__device__ inline int mod_p(int x, int p, float rp) {
    int r = x - static_cast<int>(floorf(static_cast<float>(x) * rp)) * p;
    r += r < 0 ? p : 0;
    r -= r >= p ? p : 0;
    return r;
}

// digits of field element x (constant term first)
__device__ inline void gf_digits(int x, int p, int e, int* c) {
    const float rp = 1.0f / static_cast<float>(p);
    for (int i = 0; i < 3; ++i) {
        const int r = mod_p(x, p, rp);  // x < q <= 32767
        c[i] = i < e ? r : 0;
        // (x - r) / p is an integer: the float quotient rounds to it exactly
        x = i < e ? static_cast<int>(rintf(static_cast<float>(x - r) * rp)) : x;
    }
}

__device__ inline int gf_index(const int* c, int p, int e) {
    int x = 0;
    for (int i = 2; i >= 0; --i)
        if (i < e) x = x * p + c[i];
    return x;
}

// x^2 in GF(p^e) modulo f (e <= 3), written out per degree so that no array
// is indexed at run time.  For e = 1 the square can reach 2^30 and is reduced
// in 64 bits; for e >= 2, p <= 181 keeps every intermediate below 2^17 in
// magnitude, within mod_p's range.  With f = x^e + f[e-1] x^(e-1) + ... + f[0],
// x^e = -(f[e-1] x^(e-1) + ... + f[0]) removes the top coefficients one by one.
__device__ inline int gf_square(int x, const HadSpec& h) {
    const int p = h.p;
    if (h.e == 1) return static_cast<int>(static_cast<int64_t>(x) * x % p);
    const float rp = 1.0f / static_cast<float>(p);
    int a[3];
    gf_digits(x, p, h.e, a);
    if (h.e == 2) {
        int t0 = mod_p(a[0] * a[0], p, rp), t1 = mod_p(2 * a[0] * a[1], p, rp);
        const int t2 = mod_p(a[1] * a[1], p, rp);
        t0 = mod_p(t0 - t2 * h.f[0], p, rp);
        t1 = mod_p(t1 - t2 * h.f[1], p, rp);
        return t0 + p * t1;
    }
    int t0 = mod_p(a[0] * a[0], p, rp);
    int t1 = mod_p(2 * a[0] * a[1], p, rp);
    int t2 = mod_p(a[1] * a[1] + 2 * a[0] * a[2], p, rp);
    int t3 = mod_p(2 * a[1] * a[2], p, rp);
    const int t4 = mod_p(a[2] * a[2], p, rp);
    // x^4 = x * x^3
    t1 = mod_p(t1 - t4 * h.f[0], p, rp);
    t2 = mod_p(t2 - t4 * h.f[1], p, rp);
    t3 = mod_p(t3 - t4 * h.f[2], p, rp);
    // x^3
    t0 = mod_p(t0 - t3 * h.f[0], p, rp);
    t1 = mod_p(t1 - t3 * h.f[1], p, rp);
    t2 = mod_p(t2 - t3 * h.f[2], p, rp);
    return t0 + p * (t1 + p * t2);
}

__device__ inline int paley_entry(const signed char* chi, const HadSpec& h, int i, int j) {
    if (i == 0) return 1;
    if (j == 0) return -1;
    if (i == j) return 1;
    int a[3], b[3], d[3];
    gf_digits(i - 1, h.p, h.e, a);
    gf_digits(j - 1, h.p, h.e, b);
    for (int t = 0; t < 3; ++t) {
        d[t] = a[t] - b[t];
        d[t] += d[t] < 0 ? h.p : 0;
    }
    return chi[gf_index(d, h.p, h.e)];
}

// In-place fast Sylvester transform of every block of 2^k consecutive
// elements of buf[0 .. len): two stages (index bits st, st+1) per pass.
__device__ inline void sylvester_blocks(float* buf, int len, int k, int tid) {
    int st = 0;
    for (; st + 2 <= k; st += 2) {
        const int l = 1 << st;
        for (int b = tid; b < len / 4; b += kRhtThreads) {
            const int base = ((b >> st) << (st + 2)) | (b & (l - 1));  // bits st, st+1 clear
            const float a0 = buf[base], a1 = buf[base + l], a2 = buf[base + 2 * l], a3 = buf[base + 3 * l];
            const float b0 = a0 + a1, b1 = a0 - a1, b2 = a2 + a3, b3 = a2 - a3;
            buf[base] = b0 + b2;
            buf[base + l] = b1 + b3;
            buf[base + 2 * l] = b0 - b2;
            buf[base + 3 * l] = b1 - b3;
        }
        __syncthreads();
    }
    if (st < k) {  // one stage left
        const int l = 1 << st;
        for (int b = tid; b < len / 2; b += kRhtThreads) {
            const int lo = ((b >> st) << (st + 1)) | (b & (l - 1));  // bit st clear
            const float u = buf[lo], w = buf[lo + l];
            buf[lo] = u + w;
            buf[lo + l] = u - w;
        }
        __syncthreads();
    }
}

// One workgroup per (row, slice of output blocks [jb0, jb0 + blocks_per_wg)).
// H = P (x) S factors as (P (x) I)(I (x) S): the Paley factor first, for this
// workgroup's output blocks only, then the Sylvester transform of just those
// blocks -- no work is repeated across the workgroups of a row.
template <typename XT>
__global__ __launch_bounds__(kRhtThreads) void rht_kernel(const XT* __restrict__ x,
                                                          const signed char* __restrict__ signs, int mode,
                                                          void* __restrict__ y, int y_dtype, int n, HadSpec h,
                                                          int blocks_per_wg, float norm) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    float* z = reinterpret_cast<float*>(smem);  // [n] the row
    const int64_t row = blockIdx.y;
    const int tid = threadIdx.x;
    const int half = 1 << h.k;

    // 1. the row, with the signs on the input side
    load_row<XT>(x + row * n, signs, mode, n, z, tid);
    if (h.m == 1) {  // Sylvester only: one workgroup per row
        __syncthreads();
        sylvester_blocks(z, n, h.k, tid);
        for (int j = tid; j < n; j += kRhtThreads) {
            float v = z[j] * norm;
            if (mode == 1) v *= static_cast<float>(signs[j]);
            store_out(y, row * n + j, v, y_dtype);
        }
        return;
    }
    const int jb0 = blockIdx.x * blocks_per_wg;
    const int cnt = min(h.m, jb0 + blocks_per_wg) - jb0;
    float* pcol = z + n;                                                  // [cnt][m] P[im][jb0 + jl]
    float* w = pcol + blocks_per_wg * h.m;                                // [cnt][half]
    signed char* chi = reinterpret_cast<signed char*>(w + blocks_per_wg * half);  // [q]
    // 2. quadratic character: chi[0] = 0, squares +1, the rest -1
    for (int i = tid; i < h.q; i += kRhtThreads) chi[i] = i == 0 ? 0 : -1;
    __syncthreads();
    for (int v = 1 + tid; v < h.q; v += kRhtThreads) chi[gf_square(v, h)] = 1;
    __syncthreads();
    for (int t = tid; t < cnt * h.m; t += kRhtThreads) {
        const int jl = t / h.m, im = t - jl * h.m;
        pcol[t] = static_cast<float>(paley_entry(chi, h, im, jb0 + jl));
    }
    __syncthreads();
    // 3. Paley factor: w[jl][i2] = sum_im P[im][jb0 + jl] z[im][i2]
    for (int o = tid; o < cnt * half; o += kRhtThreads) {
        const int jl = o >> h.k, i2 = o & (half - 1);
        const float* pc = pcol + jl * h.m;
        float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
        int im = 0;
        for (; im + 4 <= h.m; im += 4) {
            a0 = __builtin_fmaf(pc[im], z[im * half + i2], a0);
            a1 = __builtin_fmaf(pc[im + 1], z[(im + 1) * half + i2], a1);
            a2 = __builtin_fmaf(pc[im + 2], z[(im + 2) * half + i2], a2);
            a3 = __builtin_fmaf(pc[im + 3], z[(im + 3) * half + i2], a3);
        }
        for (; im < h.m; ++im) a0 = __builtin_fmaf(pc[im], z[im * half + i2], a0);
        w[o] = (a0 + a1) + (a2 + a3);
    }
    __syncthreads();
    // 4. Sylvester factor inside each of this workgroup's blocks
    sylvester_blocks(w, cnt * half, h.k, tid);
    for (int o = tid; o < cnt * half; o += kRhtThreads) {
        const int j = jb0 * half + o;
        float v = w[o] * norm;
        if (mode == 1) v *= static_cast<float>(signs[j]);
        store_out(y, row * n + j, v, y_dtype);
    }
}

// ---------------------------------------------------------------------------
// Pure Sylvester orders n = 2^k, 2^10 <= n <= 2^15: one workgroup of
// T = 64 * 2^W threads per row, R = 2^LR elements per thread, k = 6 + W + LR,
// W <= LR.  Index bits 0..5 live in the lanes, bits 6 .. 6+W-1 in the
// wavefront number, the top LR bits in the thread's registers:
//   phase 1: element i = lane | wave << 6 | r << (6 + W); the register bits'
//            butterflies in registers, then the lane bits' across lanes (DPP
//            for distances 1 and 2, bpermute for 4 .. 32);
//   exchange through LDS (written and read in lane order: no bank conflicts);
//   phase 2: element i = lane | (r mod 2^W) << 6 | (r >> W) << (6 + W) |
//            wave << (6 + LR), i.e. the wavefront bits now in registers;
//            their butterflies, then the store straight from registers.
// Every element takes one butterfly per index bit, (a, b) -> (a + b, a - b),
// in fp32.

template <typename XT, int W, int LR>
__global__ __launch_bounds__(64 << W) void fwht_kernel(const XT* __restrict__ x, const signed char* __restrict__ signs,
                                                       int mode, void* __restrict__ y, int y_dtype, float norm) {
    constexpr int R = 1 << LR;
    constexpr int K = 6 + W + LR;
    constexpr int N = 1 << K;
    static_assert(W <= LR && R <= 32, "register and wavefront bits");
    __shared__ float z[N];
    const int64_t row = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const XT* xr = x + row * N;

    // phase-2 element of register r (its sign is fetched early on the output side)
    auto idx2 = [&](int r) { return lane | (r & ((1 << W) - 1)) << 6 | (r >> W) << (6 + W) | wave << (6 + LR); };
    float v[R];
    signed char so[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = lane | wave << 6 | r << (6 + W);
        v[r] = static_cast<float>(xr[i]);
        so[r] = mode == 1 ? signs[idx2(r)] : 1;
    }
    if (mode == 0) {
#pragma unroll
        for (int r = 0; r < R; ++r) v[r] *= static_cast<float>(signs[lane | wave << 6 | r << (6 + W)]);
    }
    reg_stages<R, 0, LR>(v);
    lane_stage<R, 1>(v, lane);
    lane_stage<R, 2>(v, lane);
    lane_stage<R, 4>(v, lane);
    lane_stage<R, 8>(v, lane);
    lane_stage<R, 16>(v, lane);
    lane_stage<R, 32>(v, lane);
    if constexpr (W > 0) {
#pragma unroll
        for (int r = 0; r < R; ++r) z[lane | wave << 6 | r << (6 + W)] = v[r];
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) v[r] = z[idx2(r)];
        reg_stages<R, 0, W>(v);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
        store_out(y, row * N + idx2(r), v[r] * norm * static_cast<float>(so[r]), y_dtype);
}

// ---------------------------------------------------------------------------
// The Paley factor on the matrix cores.  For a workgroup's cnt <= 16 output
// blocks, W[jl][i2] = sum_im P[im][jb0 + jl] z[im][i2] is a (16 x m) by
// (m x 2^k) product, run as v_mfma_f32_16x16x4_f32 steps: A lane (jl, kk) =
// P[4s + kk][jb0 + jl], B lane (kk, c) = z[4s + kk][16 nt + c] -- fp32
// operands (the entries of P are 0 and +-1, so every product is exact) and
// fp32 accumulation.  The 16 wavefronts split the column tiles and, when
// there are fewer than 16 of them, the k range; partial sums meet in LDS and
// are added in a fixed order.  P's entries come from digit tables of the
// field elements and the quadratic character (no division in the entries).

// Packed base-p digits of field element x: for e >= 2 (then p <= 181) one
// byte per digit, constant term in the low byte; for e = 1 x itself.
__device__ inline int gf_packed(int x, int p, int e) {
    if (e == 1) return x;
    int c[3];
    gf_digits(x, p, e, c);
    return c[0] | (c[1] << 8) | (c[2] << 16);
}

// Index of the field element a - b from packed digits.
__device__ inline int gf_sub_index(int a, int b, int p, int e) {
    if (e == 1) {
        const int d = a - b;
        return d < 0 ? d + p : d;
    }
    int idx = 0;
#pragma unroll
    for (int t = 2; t >= 0; --t) {
        int d = ((a >> (8 * t)) & 0xff) - ((b >> (8 * t)) & 0xff);
        d += d < 0 ? p : 0;
        idx = idx * p + d;
    }
    return idx;
}

struct PaleyPlan {
    int cnt;     // output blocks per workgroup (<= 16)
    int ntiles;  // 16-column tiles of a block of 2^k
    int ksplit;  // wavefronts sharing one column tile's k range
};

__host__ __device__ inline size_t paley_lds_bytes(const HadSpec& h, int n, const PaleyPlan& pl) {
    const size_t half = size_t{1} << h.k;
    const size_t hp = pl.ntiles * 16;  // padded block width
    const size_t mp = static_cast<size_t>(h.m + 3) / 4 * 4;  // rows padded to whole k steps
    size_t b = mp * half * 4;                         // z, zero rows past m
    b += mp * 16 * 4;                                 // pcol [mp][16]
    b += static_cast<size_t>(pl.cnt) * half * 4;      // w [cnt][half]
    if (pl.ksplit > 1) b += static_cast<size_t>(pl.ksplit) * pl.cnt * hp * 4;  // partials
    b += static_cast<size_t>(h.q) * 4 + h.q;          // digits, character
    return b;
}

template <typename XT>
__global__ __launch_bounds__(kRhtThreads) void rht_paley_kernel(const XT* __restrict__ x,
                                                                const signed char* __restrict__ signs, int mode,
                                                                void* __restrict__ y, int y_dtype, int n, HadSpec h,
                                                                PaleyPlan pl, float norm) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int half = 1 << h.k;
    const int m = h.m;
    const int hp = pl.ntiles * 16;
    const int mp = (m + 3) & ~3;                                // rows padded to whole k steps
    float* z = reinterpret_cast<float*>(smem);                 // [mp][half], zero rows past m
    float* pcol = z + mp * half;                                // [mp][16], zero rows past m
    float* w = pcol + mp * 16;                                  // [cnt][half]
    float* part = w + pl.cnt * half;                            // [ksplit][cnt][hp]
    int* dig = reinterpret_cast<int*>(part + (pl.ksplit > 1 ? pl.ksplit * pl.cnt * hp : 0));  // [q]
    signed char* chi = reinterpret_cast<signed char*>(dig + h.q);                              // [q]
    const int64_t row = blockIdx.y;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int jb0 = blockIdx.x * pl.cnt;
    const int cnt = min(m, jb0 + pl.cnt) - jb0;

    // 1. the row's loads go out first, raw into registers, and land while the
    //    digit and character tables are built; then the row goes to LDS
    //    (signs applied on the input side)
    constexpr int C = kRhtMaxN / (8 * kRhtThreads);
    RowChunk<XT> rc[C];
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + row * n, static_cast<uint32_t>(n) * sizeof(XT));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(signs, static_cast<uint32_t>(n));
#pragma unroll
    for (int u = 0; u < C; ++u) fetch_chunk<XT>(rx, rs, 8 * (tid + u * kRhtThreads), rc[u]);
    // output-side signs of this thread's (at most two) outputs
    float so[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) so[u] = ld_sign(rs, jb0 * half + tid + u * kRhtThreads);
    for (int i = tid; i < h.q; i += kRhtThreads) {
        chi[i] = i == 0 ? 0 : -1;
        dig[i] = gf_packed(i, h.p, h.e);
    }
    __syncthreads();
    for (int v = 1 + tid; v < h.q; v += kRhtThreads) chi[gf_square(v, h)] = 1;
#pragma unroll
    for (int u = 0; u < C; ++u) put_chunk<XT>(rc[u], 8 * (tid + u * kRhtThreads), n, mode, z);
    __syncthreads();
    // 2. pcol[im][jl] = P[im][jb0 + jl] (0 past the workgroup's blocks and
    //    past row m-1); table reads clamped into range and the cases picked
    //    by selects, so the loop body has no branch
    for (int t = tid; t < mp * 16; t += kRhtThreads) {
        const int im = t >> 4, jl = t & 15;
        const int j = jb0 + jl;
        const int a = dig[min(max(im - 1, 0), h.q - 1)];
        const int b = dig[min(max(j - 1, 0), h.q - 1)];
        const float c = static_cast<float>(chi[gf_sub_index(a, b, h.p, h.e)]);
        float v = im == j ? 1.f : (j == 0 ? -1.f : c);
        v = im == 0 ? 1.f : v;
        pcol[t] = (jl < cnt && im < m) ? v : 0.f;
    }
    // zero rows of z past m
    for (int i = n + tid; i < mp * half; i += kRhtThreads) z[i] = 0.f;
    __syncthreads();
    // 3. the product.  Long blocks (fewer than 8 per workgroup, so at most
    //    256 rows m) on the vector ALUs, one output per thread and pass, four
    //    fma chains over the padded rows; otherwise on the matrix cores, one
    //    work item (column tile nt, k chunk kc) per wavefront and pass.
    const int ksteps = (m + 3) >> 2;
    const int per = (ksteps + pl.ksplit - 1) / pl.ksplit;
    const int r16 = lane & 15, kk = lane >> 4;
    if (pl.cnt < 8) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int o = tid + u * kRhtThreads;
            if (o < pl.cnt * half) {
                const int jl = o >> h.k, i2 = o & (half - 1);
                float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
                for (int im = 0; im < mp; im += 4) {
                    a0 = __builtin_fmaf(pcol[im * 16 + jl], z[im * half + i2], a0);
                    a1 = __builtin_fmaf(pcol[(im + 1) * 16 + jl], z[(im + 1) * half + i2], a1);
                    a2 = __builtin_fmaf(pcol[(im + 2) * 16 + jl], z[(im + 2) * half + i2], a2);
                    a3 = __builtin_fmaf(pcol[(im + 3) * 16 + jl], z[(im + 3) * half + i2], a3);
                }
                w[o] = (a0 + a1) + (a2 + a3);
            }
        }
    }
    for (int it = wave; pl.cnt >= 8 && it < pl.ntiles * pl.ksplit; it += kRhtThreads / 64) {
        const int nt = it % pl.ntiles, kc = it / pl.ntiles;
        const int s0 = kc * per, s1 = min(ksteps, s0 + per);
        const int col = 16 * nt + r16;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        // rows past m are zero in both tables; columns past the block
        // (blocks under 16 wide) read a clamped column and are never stored
        const int colc = min(col, half - 1);
        const float* pa = pcol + (4 * s0 + kk) * 16 + r16;
        const float* pb = z + (4 * s0 + kk) * half + colc;
        int s = s0;
        for (; s + 4 <= s1; s += 4) {
            float a[4], b[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                a[u] = pa[64 * u];
                b[u] = pb[4 * half * u];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u], b[u], acc, 0, 0, 0);
            pa += 256;
            pb += 16 * half;
        }
        for (; s < s1; ++s) {
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(*pa, *pb, acc, 0, 0, 0);
            pa += 64;
            pb += 4 * half;
        }
        // D lane (r16, kk), element e: block 4 kk + e, column col
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int jl = 4 * kk + e;
            if (jl < pl.cnt && col < half) {
                if (pl.ksplit > 1)
                    part[(kc * pl.cnt + jl) * hp + col] = acc[e];
                else
                    w[jl * half + col] = acc[e];
            }
        }
    }
    __syncthreads();
    if (pl.cnt >= 8 && pl.ksplit > 1) {
        for (int o = tid; o < pl.cnt * half; o += kRhtThreads) {
            const int jl = o >> h.k, c = o & (half - 1);
            float s = part[jl * hp + c];
            for (int kc = 1; kc < pl.ksplit; ++kc) s += part[(kc * pl.cnt + jl) * hp + c];
            w[o] = s;
        }
        __syncthreads();
    }
    // 4. Sylvester factor inside each of this workgroup's blocks
    sylvester_blocks(w, cnt * half, h.k, tid);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int o = tid + u * kRhtThreads;
        if (o < cnt * half) {
            const float v = w[o] * norm;
            store_out(y, row * n + jb0 * half + o, mode == 1 ? v * so[u] : v, y_dtype);
        }
    }
}

// The Paley factor for 16-bit rows (fp16, bf16; blocks of 2^k >= 16): a
// row's values times +-1 signs and the +-1 Paley entries are exact in the
// row's own type, so the product runs on v_mfma_f32_16x16x32_{f16,bf16} with
// fp32 sums.  Both operands sit transposed in LDS, k (the Paley index) fastest
// and rows padded by 8 halves, so that each operand is one conflict-free
// 16-byte read per lane: zt[c][im] = z[im][c] (the row, zero past m),
// pt[jl][im] = P[im][jb0 + jl].  The workgroup's Paley columns are built while
// the row is in flight; one wavefront per 16-column tile, the k range in
// steps of 32.  The Sylvester factor and the store are as above.
constexpr int kP16Pad = 8;
// The quadratic character of GF(q), bit i = 1 when element i is a nonzero
// square, computed on the host for q <= kChiBitsMax (it rides in the kernel
// arguments; the workgroups would otherwise each rebuild it).
constexpr int kChiBitsMax = 2048;
struct ChiBits {
    uint64_t w[kChiBitsMax / 64];
    int given;
};

__host__ __device__ inline int paley16_kp(const HadSpec& h) { return (h.m + 31) / 32 * 32; }
__host__ __device__ inline int paley16_pitch(const HadSpec& h) { return paley16_kp(h) + kP16Pad; }
__host__ __device__ inline size_t paley16_lds_bytes(const HadSpec& h, const PaleyPlan& pl) {
    const size_t half = size_t{1} << h.k, pitch = static_cast<size_t>(paley16_pitch(h));
    return half * pitch * 2 + 16 * pitch * 2 + static_cast<size_t>(pl.cnt) * half * 4 + static_cast<size_t>(h.q) * 5;
}

template <typename XT>
__global__ __launch_bounds__(kRhtThreads) void rht_paley16_kernel(const XT* __restrict__ x,
                                                                  const signed char* __restrict__ signs, int mode,
                                                                  void* __restrict__ y, int y_dtype, int n, HadSpec h,
                                                                  PaleyPlan pl, float norm, const ChiBits cb) {
    typedef XT xt8 __attribute__((ext_vector_type(8)));
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int half = 1 << h.k;
    const int m = h.m;
    const int kp = paley16_kp(h), pitch = paley16_pitch(h);
    XT* zt = reinterpret_cast<XT*>(smem);                          // [half][pitch]
    XT* pt = zt + half * pitch;                                     // [16][pitch]
    float* w = reinterpret_cast<float*>(pt + 16 * pitch);          // [cnt][half]
    int* dig = reinterpret_cast<int*>(w + pl.cnt * half);           // [q]
    signed char* chi = reinterpret_cast<signed char*>(dig + h.q);   // [q]
    const int64_t row = blockIdx.y;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int jb0 = blockIdx.x * pl.cnt;
    const int cnt = min(m, jb0 + pl.cnt) - jb0;

    // 1. the row's loads go out first, raw into registers (with the first
    //    word of the character a wavefront needs, see 2.)
    const uint64_t cw0 = cb.given ? cb.w[__builtin_amdgcn_readfirstlane(tid >> 6)] : 0;
    constexpr int C = kRhtMaxN / (8 * kRhtThreads);
    RowChunk<XT> rc[C];
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + row * n, static_cast<uint32_t>(n) * sizeof(XT));
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(signs, static_cast<uint32_t>(n));
#pragma unroll
    for (int u = 0; u < C; ++u) fetch_chunk<XT>(rx, rs, 8 * (tid + u * kRhtThreads), rc[u]);
    float so[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) so[u] = ld_sign(rs, jb0 * half + tid + u * kRhtThreads);
    // 2. digit and character tables (the character from the arguments when
    //    given: wavefront w reads word w of each 512-element stretch), then
    //    this workgroup's Paley columns (pt rows past cnt and columns past m
    //    are zero)
    if (cb.given) {
        for (int i0 = 0; i0 < h.q; i0 += kRhtThreads) {
            const uint64_t word = i0 == 0 ? cw0 : cb.w[__builtin_amdgcn_readfirstlane((i0 + tid) >> 6)];
            const int i = i0 + tid;
            if (i < h.q) {
                chi[i] = i == 0 ? 0 : ((word >> (i & 63)) & 1u ? 1 : -1);
                dig[i] = gf_packed(i, h.p, h.e);
            }
        }
        __syncthreads();
    } else {
        for (int i = tid; i < h.q; i += kRhtThreads) {
            chi[i] = i == 0 ? 0 : -1;
            dig[i] = gf_packed(i, h.p, h.e);
        }
        __syncthreads();
        for (int v = 1 + tid; v < h.q; v += kRhtThreads) chi[gf_square(v, h)] = 1;
        __syncthreads();
    }
    {
        // a thread keeps one column (the stride is a multiple of 16)
        const int jl = tid & 15, j = jb0 + jl;
        const int b = dig[min(max(j - 1, 0), h.q - 1)];
#pragma unroll 4
        for (int t = tid; t < 16 * kp; t += kRhtThreads) {
            const int im = t >> 4;
            const int a = dig[min(max(im - 1, 0), h.q - 1)];
            const float c = static_cast<float>(chi[gf_sub_index(a, b, h.p, h.e)]);
            float v = im == j ? 1.f : (j == 0 ? -1.f : c);
            v = im == 0 ? 1.f : v;
            pt[jl * pitch + im] = static_cast<XT>((jl < cnt && im < m) ? v : 0.f);
        }
    }
    // 3. the row, transposed, and zero Paley rows m .. kp - 1.  A chunk's 8
    //    elements share one Paley index and take 8 consecutive block
    //    positions (8 divides the block, and n is a multiple of 16); the sign
    //    of the input side flips the 16-bit value's sign bit (exact: the
    //    stored value is x times +-1), the byte of -1 having its top bit set.
#pragma unroll
    for (int u = 0; u < C; ++u) {
        const int i0 = 8 * (tid + u * kRhtThreads);
        if (i0 < n) {
            const uint32_t wd[4] = {rc[u].a.x, rc[u].a.y, rc[u].a.z, rc[u].a.w};
            uint16_t* const dst = reinterpret_cast<uint16_t*>(zt + (i0 & (half - 1)) * pitch + (i0 >> h.k));
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                uint32_t bits = (wd[e >> 1] >> (16 * (e & 1))) & 0xffffu;
                if (mode == 0) {
                    const uint32_t sw = e < 4 ? rc[u].s.x : rc[u].s.y;
                    bits ^= ((sw >> (8 * (e & 3) + 7)) & 1u) << 15;
                }
                dst[e * pitch] = static_cast<uint16_t>(bits);
            }
        }
    }
    for (int t = tid; t < (kp - m) * half; t += kRhtThreads) {
        const int c = t & (half - 1), im = m + (t >> h.k);
        zt[c * pitch + im] = static_cast<XT>(0.f);
    }
    __syncthreads();
    // 4. the product: wavefront item nt = one 16-column tile; D lane: column
    //    16 nt + lane % 16, blocks 4 (lane / 16) + e
    const int ntiles = half >> 4;
    for (int nt = wave; nt < ntiles; nt += kRhtThreads / 64) {
        const XT* pa = pt + (lane & 15) * pitch + 8 * (lane >> 4);
        const XT* pb = zt + (16 * nt + (lane & 15)) * pitch + 8 * (lane >> 4);
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        for (int k0 = 0; k0 < kp; k0 += 32) {
            const xt8 av = *reinterpret_cast<const xt8*>(pa + k0);
            const xt8 bv = *reinterpret_cast<const xt8*>(pb + k0);
            if constexpr (sizeof(XT) == 2 && std::is_same<XT, _Float16>::value)
                acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, bv, acc, 0, 0, 0);
            else
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int jl = 4 * (lane >> 4) + e;
            if (jl < cnt) w[jl * half + 16 * nt + (lane & 15)] = acc[e];
        }
    }
    __syncthreads();
    // 5. Sylvester factor inside each of this workgroup's blocks
    sylvester_blocks(w, cnt * half, h.k, tid);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int o = tid + u * kRhtThreads;
        if (o < cnt * half) {
            const float v = w[o] * norm;
            store_out(y, row * n + jb0 * half + o, mode == 1 ? v * so[u] : v, y_dtype);
        }
    }
}

bool is_prime(int v) {
    if (v < 2) return false;
    for (int d = 2; d * d <= v; ++d)
        if (v % d == 0) return false;
    return true;
}

}  // namespace

// Order-n construction, or false when n has none of the supported forms.
bool hadamard_spec(int64_t n, HadSpec* out) {
    if (n < 1 || n > kRhtMaxN) return false;
    int k = 0;
    while (n % (int64_t{2} << k) == 0) ++k;
    for (; k >= 0; --k) {
        const int m = static_cast<int>(n >> k);
        HadSpec h{};
        h.k = k;
        h.m = m;
        if (m == 1) {
            *out = h;
            return true;
        }
        const int q = m - 1;
        if (q % 4 != 3) continue;
        // q = p^e with e <= 3
        for (int p = 2; p <= q; ++p) {
            if (!is_prime(p)) continue;
            int pe = p, e = 1;
            while (pe < q && e < 3) {
                pe *= p;
                ++e;
            }
            if (pe != q) continue;
            h.q = q;
            h.p = p;
            h.e = e;
            if (e > 1) {
                // first monic f of degree e (coefficient vector counted with the
                // constant term fastest) with no root in GF(p): irreducible for e <= 3
                bool found = false;
                for (int idx = 0; idx < q && !found; ++idx) {
                    int c[3] = {idx % p, (idx / p) % p, (idx / p / p) % p};
                    bool root = false;
                    for (int xv = 0; xv < p && !root; ++xv) {
                        int v = 1;
                        for (int i = e - 1; i >= 0; --i) v = (v * xv + c[i]) % p;
                        root = v == 0;
                    }
                    if (!root) {
                        h.f[0] = c[0];
                        h.f[1] = c[1];
                        h.f[2] = c[2];
                        found = true;
                    }
                }
                if (!found) return false;
            }
            *out = h;
            return true;
        }
    }
    return false;
}

constexpr size_t kRhtMaxLds = 160 * 1024;

// Bit i set when field element i (digits base p, constant term first) is a
// nonzero square of GF(p^e) modulo f: x^2 for every x != 0, the product's
// degrees e .. 2e - 2 removed from the top with x^e = -(f[e-1] x^(e-1) + ...
// + f[0]).  Host side of the character the transform kernels build from the
// same definition (q <= kChiBitsMax).
static void square_bits(const HadSpec& h, uint64_t* w) {
    const int p = h.p, e = h.e;
    for (int i = 0; i < kChiBitsMax / 64; ++i) w[i] = 0;
    for (int x = 1; x < h.q; ++x) {
        int a[3] = {0, 0, 0};
        for (int i = 0, v = x; i < e; ++i, v /= p) a[i] = v % p;
        int64_t c[5] = {0, 0, 0, 0, 0};
        for (int i = 0; i < e; ++i)
            for (int j = 0; j < e; ++j) c[i + j] += static_cast<int64_t>(a[i]) * a[j];
        for (int d = 2 * e - 2; d >= e; --d)
            for (int i = 0; i < e; ++i) c[d - e + i] -= c[d] * h.f[i];
        int idx = 0;
        for (int i = e - 1; i >= 0; --i) idx = idx * p + static_cast<int>(((c[i] % p) + p) % p);
        w[idx >> 6] |= uint64_t{1} << (idx & 63);
    }
}

size_t rht_lds_bytes(const HadSpec& h, int n, int per) {
    size_t b = static_cast<size_t>(n) * 4;
    if (h.m > 1)
        b += static_cast<size_t>(per) * h.m * 4 + static_cast<size_t>(per) * (size_t{1} << h.k) * 4 +
             static_cast<size_t>(h.q);
    return b;
}

// Output blocks of the Paley factor per workgroup: at most one output per
// thread, and few enough blocks that a row spreads over about 32 workgroups
// or more (the dense factor is bound by LDS reads); fewer when the slice of
// the Paley matrix would not fit the LDS.
int rht_blocks_per_wg(const HadSpec& h, int n) {
    int per = kRhtThreads >> h.k;
    const int spread = h.m / 32;
    if (spread >= 1 && per > spread) per = spread;
    per = per < 1 ? 1 : (per > h.m ? h.m : per);
    while (per > 1 && rht_lds_bytes(h, n, per) > kRhtMaxLds) per /= 2;
    return per;
}

template <int W, int LR>
static int launch_fwht(const void* x, int x_dtype, const signed char* signs, int mode, void* y, int y_dtype,
                       float norm, dim3 grid, hipStream_t s) {
    const dim3 block(64 << W);
    if (x_dtype == UNISVQ_F16)
        hipLaunchKernelGGL((fwht_kernel<_Float16, W, LR>), grid, block, 0, s, static_cast<const _Float16*>(x), signs,
                           mode, y, y_dtype, norm);
    else if (x_dtype == UNISVQ_BF16)
        hipLaunchKernelGGL((fwht_kernel<__bf16, W, LR>), grid, block, 0, s, static_cast<const __bf16*>(x), signs,
                           mode, y, y_dtype, norm);
    else
        hipLaunchKernelGGL((fwht_kernel<float, W, LR>), grid, block, 0, s, static_cast<const float*>(x), signs, mode,
                           y, y_dtype, norm);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

// Output blocks per workgroup (at most 16, the matrix-core tile height, and
// at most 512 outputs, so that long blocks spread over more workgroups),
// 16-column tiles per block, and the k split that gives the 16 wavefronts
// one (tile, k chunk) item each when there are fewer tiles.  With fewer than
// 8 blocks the matrix-core tile would be mostly idle and the kernel sums on
// the vector ALUs instead.
static PaleyPlan paley_plan(const HadSpec& h) {
    const int half = 1 << h.k;
    PaleyPlan pl;
    pl.ntiles = half >= 16 ? half / 16 : 1;
    int c = 512 / half;
    c = c < 1 ? 1 : (c > 16 ? 16 : c);
    pl.cnt = c < h.m ? c : h.m;
    pl.ksplit = pl.ntiles >= 16 ? 1 : 16 / pl.ntiles;
    return pl;
}

int launch_rht(int64_t n, int64_t M, const void* x, int x_dtype, const signed char* signs, int mode, void* y,
               int y_dtype, hipStream_t s) {
    HadSpec h;
    if (!hadamard_spec(n, &h)) return UNISVQ_EUNSUP;
    const int per = h.m > 1 ? rht_blocks_per_wg(h, static_cast<int>(n)) : 1;
    const size_t lds = rht_lds_bytes(h, static_cast<int>(n), per);
    if (lds > kRhtMaxLds) return UNISVQ_EUNSUP;
    // the dynamic-LDS limits, raised once per kernel and device
    static std::atomic<uint64_t> attr_done[8];
    const void* fns[8] = {reinterpret_cast<const void*>(&rht_kernel<_Float16>),
                          reinterpret_cast<const void*>(&rht_kernel<__bf16>),
                          reinterpret_cast<const void*>(&rht_kernel<float>),
                          reinterpret_cast<const void*>(&rht_paley_kernel<_Float16>),
                          reinterpret_cast<const void*>(&rht_paley_kernel<__bf16>),
                          reinterpret_cast<const void*>(&rht_paley_kernel<float>),
                          reinterpret_cast<const void*>(&rht_paley16_kernel<_Float16>),
                          reinterpret_cast<const void*>(&rht_paley16_kernel<__bf16>)};
    for (int i = 0; i < 8; ++i) {
        const int st = ensure_lds_limit(fns[i], static_cast<int>(kRhtMaxLds), attr_done[i]);
        if (st != UNISVQ_OK) return st;
    }
    const float norm = static_cast<float>(1.0 / std::sqrt(static_cast<double>(n)));
    if (h.m == 1 && h.k >= 10) {  // 2^10 .. 2^15: registers, lanes and one exchange
        const dim3 fgrid(static_cast<unsigned>(M));
        int st = UNISVQ_OK;
        switch (h.k) {
            case 10: st = launch_fwht<2, 2>(x, x_dtype, signs, mode, y, y_dtype, norm, fgrid, s); break;
            case 11: st = launch_fwht<2, 3>(x, x_dtype, signs, mode, y, y_dtype, norm, fgrid, s); break;
            case 12: st = launch_fwht<3, 3>(x, x_dtype, signs, mode, y, y_dtype, norm, fgrid, s); break;
            case 13: st = launch_fwht<3, 4>(x, x_dtype, signs, mode, y, y_dtype, norm, fgrid, s); break;
            case 14: st = launch_fwht<4, 4>(x, x_dtype, signs, mode, y, y_dtype, norm, fgrid, s); break;
            default: st = launch_fwht<4, 5>(x, x_dtype, signs, mode, y, y_dtype, norm, fgrid, s); break;
        }
        return st;
    }
    if (h.m > 1 && h.k >= 4 && (x_dtype == UNISVQ_F16 || x_dtype == UNISVQ_BF16)) {
        // 16-bit rows: the Paley factor on the 16-bit matrix cores
        const PaleyPlan pl = paley_plan(h);
        const size_t plds = paley16_lds_bytes(h, pl);
        if (plds <= kRhtMaxLds && pl.cnt << h.k <= 2 * kRhtThreads) {  // at most two outputs per thread
            const dim3 pgrid(static_cast<unsigned>((h.m + pl.cnt - 1) / pl.cnt), static_cast<unsigned>(M));
            ChiBits cb{};
            if (h.q <= kChiBitsMax) {
                square_bits(h, cb.w);
                cb.given = 1;
            }
            if (x_dtype == UNISVQ_F16)
                hipLaunchKernelGGL(rht_paley16_kernel<_Float16>, pgrid, dim3(kRhtThreads), plds, s,
                                   static_cast<const _Float16*>(x), signs, mode, y, y_dtype, static_cast<int>(n), h,
                                   pl, norm, cb);
            else
                hipLaunchKernelGGL(rht_paley16_kernel<__bf16>, pgrid, dim3(kRhtThreads), plds, s,
                                   static_cast<const __bf16*>(x), signs, mode, y, y_dtype, static_cast<int>(n), h,
                                   pl, norm, cb);
            return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
        }
    }
    if (h.m > 1) {
        // matrix-core Paley factor whenever its tables fit the LDS
        const PaleyPlan pl = paley_plan(h);
        const size_t plds = paley_lds_bytes(h, static_cast<int>(n), pl);
        if (plds <= kRhtMaxLds && pl.cnt << h.k <= 2 * kRhtThreads) {  // at most two outputs per thread
            const dim3 pgrid(static_cast<unsigned>((h.m + pl.cnt - 1) / pl.cnt), static_cast<unsigned>(M));
            if (x_dtype == UNISVQ_F16)
                hipLaunchKernelGGL(rht_paley_kernel<_Float16>, pgrid, dim3(kRhtThreads), plds, s,
                                   static_cast<const _Float16*>(x), signs, mode, y, y_dtype, static_cast<int>(n), h,
                                   pl, norm);
            else if (x_dtype == UNISVQ_BF16)
                hipLaunchKernelGGL(rht_paley_kernel<__bf16>, pgrid, dim3(kRhtThreads), plds, s,
                                   static_cast<const __bf16*>(x), signs, mode, y, y_dtype, static_cast<int>(n), h,
                                   pl, norm);
            else
                hipLaunchKernelGGL(rht_paley_kernel<float>, pgrid, dim3(kRhtThreads), plds, s,
                                   static_cast<const float*>(x), signs, mode, y, y_dtype, static_cast<int>(n), h, pl,
                                   norm);
            return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
        }
    }
    const unsigned gx = h.m > 1 ? static_cast<unsigned>((h.m + per - 1) / per) : 1u;
    const dim3 grid(gx, static_cast<unsigned>(M));
    if (x_dtype == UNISVQ_F16)
        hipLaunchKernelGGL(rht_kernel<_Float16>, grid, dim3(kRhtThreads), lds, s, static_cast<const _Float16*>(x),
                           signs, mode, y, y_dtype, static_cast<int>(n), h, per, norm);
    else if (x_dtype == UNISVQ_BF16)
        hipLaunchKernelGGL(rht_kernel<__bf16>, grid, dim3(kRhtThreads), lds, s, static_cast<const __bf16*>(x), signs,
                           mode, y, y_dtype, static_cast<int>(n), h, per, norm);
    else
        hipLaunchKernelGGL(rht_kernel<float>, grid, dim3(kRhtThreads), lds, s, static_cast<const float*>(x), signs,
                           mode, y, y_dtype, static_cast<int>(n), h, per, norm);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

}  // namespace unisvq
