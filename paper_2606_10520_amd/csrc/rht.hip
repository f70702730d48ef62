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
// dense product for the workgroup's output blocks with its entries built in
// LDS from the quadratic character, then the Sylvester factor as an in-place
// fast transform inside each of those blocks of 2^k.  fp32 throughout, one
// rounding to the output dtype.
#include <cmath>

#include "common.hpp"

namespace unisvq {

struct HadSpec {
    int k, m, q, p, e;
    int f[3];  // f(x) = x^e + f[e-1] x^(e-1) + ... + f[0]
};

namespace {

constexpr int kRhtThreads = 1024;
constexpr int kRhtMaxN = 32768;  // fp32 row in LDS

// The row into LDS as fp32 (signs applied on the input side): eight
// independent loads in flight per thread before their LDS writes.
template <typename XT>
__device__ inline void load_row(const XT* __restrict__ xr, const signed char* __restrict__ signs, int mode, int n,
                                float* z, int tid) {
    constexpr int U = 8;
    for (int i0 = tid; i0 < n; i0 += kRhtThreads * U) {
        float v[U];
        float sg[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kRhtThreads;
            v[u] = i < n ? static_cast<float>(xr[i]) : 0.f;
            sg[u] = (mode == 0 && i < n) ? static_cast<float>(signs[i]) : 1.f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * kRhtThreads;
            if (i < n) z[i] = v[u] * sg[u];
        }
    }
}

// digits of field element x (constant term first)
__device__ inline void gf_digits(int x, int p, int e, int* c) {
    for (int i = 0; i < 3; ++i) {
        c[i] = i < e ? x % p : 0;
        x = i < e ? x / p : x;
    }
}

__device__ inline int gf_index(const int* c, int p, int e) {
    int x = 0;
    for (int i = 2; i >= 0; --i)
        if (i < e) x = x * p + c[i];
    return x;
}

// x^2 in GF(p^e) modulo f (e <= 3)
__device__ inline int gf_square(int x, const HadSpec& h) {
    int a[3], t[5] = {0, 0, 0, 0, 0};
    gf_digits(x, h.p, h.e, a);
    for (int i = 0; i < h.e; ++i)
        for (int j = 0; j < h.e; ++j) t[i + j] = (t[i + j] + a[i] * a[j]) % h.p;
    for (int d = 2 * h.e - 2; d >= h.e; --d) {
        const int c = t[d];
        if (!c) continue;
        t[d] = 0;
        for (int i = 0; i < h.e; ++i) t[d - h.e + i] = ((t[d - h.e + i] - c * h.f[i]) % h.p + h.p) % h.p;
    }
    return gf_index(t, h.p, h.e);
}

__device__ inline int paley_entry(const signed char* chi, const HadSpec& h, int i, int j) {
    if (i == 0) return 1;
    if (j == 0) return -1;
    if (i == j) return 1;
    int a[3], b[3], d[3];
    gf_digits(i - 1, h.p, h.e, a);
    gf_digits(j - 1, h.p, h.e, b);
    for (int t = 0; t < 3; ++t) d[t] = ((a[t] - b[t]) % h.p + h.p) % h.p;
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

int launch_rht(int64_t n, int64_t M, const void* x, int x_dtype, const signed char* signs, int mode, void* y,
               int y_dtype, hipStream_t s) {
    HadSpec h;
    if (!hadamard_spec(n, &h)) return UNISVQ_EUNSUP;
    const int per = h.m > 1 ? rht_blocks_per_wg(h, static_cast<int>(n)) : 1;
    const size_t lds = rht_lds_bytes(h, static_cast<int>(n), per);
    if (lds > kRhtMaxLds) return UNISVQ_EUNSUP;
    static bool attr_done = false;  // idempotent; racing first calls set the same value
    if (!attr_done) {
        const void* fns[3] = {reinterpret_cast<const void*>(&rht_kernel<_Float16>),
                              reinterpret_cast<const void*>(&rht_kernel<__bf16>),
                              reinterpret_cast<const void*>(&rht_kernel<float>)};
        for (const void* f : fns)
            if (hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kRhtMaxLds)) !=
                hipSuccess)
                return UNISVQ_EHIP;
        attr_done = true;
    }
    const unsigned gx = h.m > 1 ? static_cast<unsigned>((h.m + per - 1) / per) : 1u;
    const float norm = static_cast<float>(1.0 / std::sqrt(static_cast<double>(n)));
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
