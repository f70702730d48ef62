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
// fp32 (signs applied on the input side), the Sylvester factor runs as an
// in-place fast transform inside each block of 2^k, and the Paley factor, if
// any, as a dense m x m product for the workgroup's output blocks, with its
// entries built in LDS from the quadratic character.  fp32 throughout, one
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
constexpr int kMaxPaleyBlocks = 8;  // output blocks of the Paley factor per workgroup

template <typename T>
__device__ inline float to_f32(const void* p, int64_t i) {
    return static_cast<float>(static_cast<const T*>(p)[i]);
}

__device__ inline float load_any(const void* p, int64_t i, int dtype) {
    if (dtype == UNISVQ_F32) return static_cast<const float*>(p)[i];
    if (dtype == UNISVQ_F16) return to_f32<_Float16>(p, i);
    return to_f32<__bf16>(p, i);
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

__global__ __launch_bounds__(kRhtThreads) void rht_kernel(const void* __restrict__ x, int x_dtype,
                                                          const signed char* __restrict__ signs, int mode,
                                                          void* __restrict__ y, int y_dtype, int n, HadSpec h,
                                                          int blocks_per_wg, float norm) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    float* z = reinterpret_cast<float*>(smem);                                // [n]
    signed char* chi = reinterpret_cast<signed char*>(smem + 4 * n);          // [q]
    signed char* pcol = chi + (h.q + 15) / 16 * 16;                           // [blocks_per_wg][m]
    const int64_t row = blockIdx.y;
    const int tid = threadIdx.x;
    const int half = 1 << h.k;

    // 1. the row, with the signs on the input side
    for (int i = tid; i < n; i += kRhtThreads) {
        const float v = load_any(x, row * n + i, x_dtype);
        z[i] = mode == 0 ? v * static_cast<float>(signs[i]) : v;
    }
    // quadratic character: chi[0] = 0, squares +1, the rest -1
    if (h.m > 1) {
        for (int i = tid; i < h.q; i += kRhtThreads) chi[i] = i == 0 ? 0 : -1;
    }
    __syncthreads();
    if (h.m > 1) {
        for (int v = 1 + tid; v < h.q; v += kRhtThreads) chi[gf_square(v, h)] = 1;
    }
    // 2. Sylvester factor: in-place fast transform inside every block of 2^k
    for (int len = 1; len < half; len <<= 1) {
        for (int b = tid; b < n / 2; b += kRhtThreads) {
            const int lo = (b / len) * 2 * len + (b % len);  // element with bit `len` clear
            const float u = z[lo], w = z[lo + len];
            z[lo] = u + w;
            z[lo + len] = u - w;
        }
        __syncthreads();
    }
    if (h.m == 1) {
        for (int j = tid; j < n; j += kRhtThreads) {
            float v = z[j] * norm;
            if (mode == 1) v *= static_cast<float>(signs[j]);
            store_out(y, row * n + j, v, y_dtype);
        }
        return;
    }
    // 3. Paley factor for output blocks [jb0, jb1): y[jm][j2] = sum_im P[im][jm] z[im][j2]
    const int jb0 = blockIdx.x * blocks_per_wg;
    const int jb1 = min(h.m, jb0 + blocks_per_wg);
    __syncthreads();  // chi complete
    for (int t = tid; t < (jb1 - jb0) * h.m; t += kRhtThreads) {
        const int jl = t / h.m, im = t % h.m;
        pcol[jl * h.m + im] = static_cast<signed char>(paley_entry(chi, h, im, jb0 + jl));
    }
    __syncthreads();
    for (int o = tid; o < (jb1 - jb0) * half; o += kRhtThreads) {
        const int jl = o / half, j2 = o % half;
        const signed char* pc = pcol + jl * h.m;
        float acc = 0.f;
        for (int im = 0; im < h.m; ++im) acc += static_cast<float>(pc[im]) * z[im * half + j2];
        const int j = (jb0 + jl) * half + j2;
        float v = acc * norm;
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

size_t rht_lds_bytes(const HadSpec& h, int n) {
    size_t b = static_cast<size_t>(n) * 4;
    if (h.m > 1) b += static_cast<size_t>((h.q + 15) / 16 * 16) + static_cast<size_t>(kMaxPaleyBlocks) * h.m;
    return b;
}

int launch_rht(int64_t n, int64_t M, const void* x, int x_dtype, const signed char* signs, int mode, void* y,
               int y_dtype, hipStream_t s) {
    HadSpec h;
    if (!hadamard_spec(n, &h)) return UNISVQ_EUNSUP;
    const size_t lds = rht_lds_bytes(h, static_cast<int>(n));
    if (lds > 160 * 1024) return UNISVQ_EUNSUP;
    static bool attr_done = false;  // idempotent; racing first calls set the same value
    if (!attr_done) {
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&rht_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                                160 * 1024) != hipSuccess)
            return UNISVQ_EHIP;
        attr_done = true;
    }
    const int per = h.m > 1 ? (h.m >= 64 ? kMaxPaleyBlocks : 1) : 1;
    const unsigned gx = h.m > 1 ? static_cast<unsigned>((h.m + per - 1) / per) : 1u;
    const float norm = static_cast<float>(1.0 / std::sqrt(static_cast<double>(n)));
    hipLaunchKernelGGL(rht_kernel, dim3(gx, static_cast<unsigned>(M)), dim3(kRhtThreads), lds, s, x, x_dtype, signs,
                       mode, y, y_dtype, static_cast<int>(n), h, per, norm);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

}  // namespace unisvq
