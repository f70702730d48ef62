// LDLQ on gfx950: nearest-codeword rounding with Hessian error feedback
// (Sec. 3.2.2, Eq. 7).  Vectors of 4 columns are rounded left to right; the
// target of vector j is u = W_j + sum_{k < 4j} E_k U[k][j] (E = W - W_hat,
// U the unit upper block-triangular factor of H = U D U^T).
//
// The running feedback F[r][c] = sum_k E[r][k] U[k][c] lives in the
// workspace (fp64) and is accumulated lazily, 128 columns (one group) at a
// time: the step kernel rounds the 32 vectors of block b row by row, feeding
// each vector's error forward to the later columns of the same block; then the
// update kernel adds the block's errors to every column to its right.  Every
// F element is therefore one fma chain in increasing k, exactly the sum of
// the definition, and the decision on u = W + F is taken in fp64 with the
// nearest-codeword quantiser's operation order and tie rule: the codes equal
// a plain sequential evaluation of Eq. 7 bit for bit.
#include "common.hpp"
#include "fwht.hpp"

namespace unisvq {
namespace {

constexpr int kLdlqBlock = 128;  // columns per lazy block (= one group)

__device__ inline double h2d(uint16_t h) {
    return static_cast<double>(static_cast<float>(__builtin_bit_cast(_Float16, h)));
}

__device__ inline double readlane_f64(double v, int src) {
    const uint2 u = __builtin_bit_cast(uint2, v);
    return __builtin_bit_cast(double, uint2{static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u.x), src)),
                                            static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u.y), src))});
}

// Codeword i (q_b = bits 2b, 2b+1 of i) of the pair (a, b): each component
// summed left to right, in the fixed order of the nearest-codeword quantiser.
__device__ inline void cw_build(const double (&a)[16], const double (&b)[4], int i, double (&c)[4]) {
    const double q0 = static_cast<double>(i & 3), q1 = static_cast<double>((i >> 2) & 3);
    const double q2 = static_cast<double>((i >> 4) & 3), q3 = static_cast<double>((i >> 6) & 3);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        double v = b[k];
        v = v + a[4 * k + 0] * q0;
        v = v + a[4 * k + 1] * q1;
        v = v + a[4 * k + 2] * q2;
        v = v + a[4 * k + 3] * q3;
        c[k] = v;
    }
}

// Squared distance from u to codeword c, accumulated with fmas in component order.
__device__ inline double cw_dist(const double (&c)[4], const double (&u)[4]) {
    double d = 0.0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const double e = c[k] - u[k];
        d = __builtin_fma(e, e, d);
    }
    return d;
}

// One butterfly step of the minimum over the wavefront: the (distance,
// index) pair of lane (lane ^ D) through the vector-ALU lane exchanges (no
// LDS round trip on the rounding's serial path); the lower index wins ties.
template <int D>
__device__ inline void min_step(double& bd, int& bi, int lane) {
    const uint2 w = __builtin_bit_cast(uint2, bd);
    const uint2 o{__builtin_bit_cast(uint32_t, lane_xor<D>(__builtin_bit_cast(float, w.x), lane)),
                  __builtin_bit_cast(uint32_t, lane_xor<D>(__builtin_bit_cast(float, w.y), lane))};
    const double od = __builtin_bit_cast(double, o);
    const int oi = __builtin_bit_cast(int, lane_xor<D>(__builtin_bit_cast(float, bi), lane));
    if (od < bd || (od == bd && oi < bi)) {
        bd = od;
        bi = oi;
    }
}

__global__ __launch_bounds__(256) void ldlq_fill_kernel(double* __restrict__ F, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < n) F[i] = 0.0;
}

// Block b: one wavefront per row; lane l holds columns 128 b + 2l, 2l + 1.
// Candidates i = l, l + 64, l + 128, l + 192 per lane, then a butterfly
// minimum over the wavefront that keeps the lower index on equal distances
// (the sequential scan's first minimum).
__global__ __launch_bounds__(256) void ldlq_block_kernel(int64_t N, int64_t K, int b, const float* __restrict__ W,
                                                         const double* __restrict__ U,
                                                         const uint16_t* __restrict__ A,
                                                         const uint16_t* __restrict__ B, int64_t affine_groups,
                                                         const double* __restrict__ F, double* __restrict__ E,
                                                         uint8_t* __restrict__ codes) {
    const int lane = threadIdx.x & 63;
    const int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (r >= N) return;  // uniform per wavefront
    const int64_t groups = K / kGroup;
    const int64_t set = affine_groups == 0 ? r * groups + b : (affine_groups == 1 ? 0 : b);
    double a[16], bb[4];
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = h2d(A[set * 16 + i]);
#pragma unroll
    for (int i = 0; i < 4; ++i) bb[i] = h2d(B[set * 4 + i]);

    const int64_t c0 = static_cast<int64_t>(b) * kLdlqBlock + 2 * lane;
    const double2 fv = *reinterpret_cast<const double2*>(F + r * K + c0);
    const float2 wv = *reinterpret_cast<const float2*>(W + r * K + c0);
    double f0 = fv.x, f1 = fv.y;
    const double w0 = wv.x, w1 = wv.y;
    double e0 = 0.0, e1 = 0.0;
    uint32_t mycodes = 0;
    // This lane's four candidate codewords i (q_b = bits 2b, 2b+1 of i; the
    // pair is fixed for the block), built once in the quantiser's operation
    // order: components summed left to right (cw_dist then only subtracts
    // and accumulates the squared distance with fmas in component order).
    double cw[4][4];
#pragma unroll
    for (int s = 0; s < 4; ++s) cw_build(a, bb, lane + 64 * s, cw[s]);
    // rows of U for the feedback of vector v, loaded one vector ahead
    const double* Ur = U + static_cast<int64_t>(b) * kLdlqBlock * K + c0;
    double2 un[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) un[k] = *reinterpret_cast<const double2*>(Ur + static_cast<int64_t>(k) * K);
    for (int v = 0; v < kLdlqBlock / 4; ++v) {
        double2 uc[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) uc[k] = un[k];
        const int vn = v + 1 < kLdlqBlock / 4 ? v + 1 : v;  // (the last step reloads its own rows)
#pragma unroll
        for (int k = 0; k < 4; ++k)
            un[k] = *reinterpret_cast<const double2*>(Ur + static_cast<int64_t>(4 * vn + k) * K);
        const double t0 = w0 + f0, t1 = w1 + f1;  // u of this lane's columns
        const double u[4] = {readlane_f64(t0, 2 * v), readlane_f64(t1, 2 * v), readlane_f64(t0, 2 * v + 1),
                             readlane_f64(t1, 2 * v + 1)};
        int bi = lane;
        double bd = cw_dist(cw[0], u);
#pragma unroll
        for (int s = 1; s < 4; ++s) {
            const double d = cw_dist(cw[s], u);
            if (d < bd) {
                bd = d;
                bi = lane + 64 * s;
            }
        }
        min_step<1>(bd, bi, lane);
        min_step<2>(bd, bi, lane);
        min_step<4>(bd, bi, lane);
        min_step<8>(bd, bi, lane);
        min_step<16>(bd, bi, lane);
        min_step<32>(bd, bi, lane);
        const int best = __builtin_amdgcn_readfirstlane(bi);
        // the chosen codeword (exact) and the errors of the vector's columns
        const double q[4] = {static_cast<double>(best & 3), static_cast<double>((best >> 2) & 3),
                             static_cast<double>((best >> 4) & 3), static_cast<double>((best >> 6) & 3)};
        const double wvv[4] = {readlane_f64(w0, 2 * v), readlane_f64(w1, 2 * v), readlane_f64(w0, 2 * v + 1),
                               readlane_f64(w1, 2 * v + 1)};
        double ev[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            double c = bb[k];
            c = c + a[4 * k + 0] * q[0];
            c = c + a[4 * k + 1] * q[1];
            c = c + a[4 * k + 2] * q[2];
            c = c + a[4 * k + 3] * q[3];
            ev[k] = wvv[k] - c;
        }
        if ((lane >> 1) == v) {
            const int h = lane & 1;
            e0 = h ? ev[2] : ev[0];
            e1 = h ? ev[3] : ev[1];
            mycodes = h ? (((best >> 4) & 3) | (((best >> 6) & 3) << 8)) : ((best & 3) | (((best >> 2) & 3) << 8));
        }
        // feed the errors forward, in increasing k, to this block's columns
        // (an earlier column gets U = 0 and the vector's own columns their
        // identity block; neither is read again)
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            f0 = __builtin_fma(ev[k], uc[k].x, f0);
            f1 = __builtin_fma(ev[k], uc[k].y, f1);
        }
    }
    *reinterpret_cast<double2*>(E + r * kLdlqBlock + 2 * lane) = double2{e0, e1};
    *reinterpret_cast<uint16_t*>(codes + r * K + c0) = static_cast<uint16_t>(mycodes);
}

// F[r][c] += sum_k E[r][k] U[128 b + k][c] for the columns right of block b,
// each element one fma chain in increasing k.  128-row x 64-column output
// tiles; thread (ty, tx) owns rows ty + 16 i (i < 8) and columns tx + 16 j
// (j < 4).  k runs in chunks of 16 through two LDS buffers: the global loads
// of chunk c + 1 are issued into registers before the fmas of chunk c and
// land in the other buffer after them, one barrier per chunk.
constexpr int kUpdRows = 128;
constexpr int kUpdCols = 64;
constexpr int kUpdChunk = 16;

__global__ __launch_bounds__(256) void ldlq_update_kernel(int64_t N, int64_t K, int b, const double* __restrict__ E,
                                                          const double* __restrict__ U, double* __restrict__ F) {
    __shared__ double Es[2][kUpdChunk][kUpdRows + 1];
    __shared__ double Us[2][kUpdChunk][kUpdCols + 1];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int64_t row0 = static_cast<int64_t>(blockIdx.x) * kUpdRows;
    const int64_t col0 = static_cast<int64_t>(b + 1) * kLdlqBlock + static_cast<int64_t>(blockIdx.y) * kUpdCols;
    const double* Ub = U + static_cast<int64_t>(b) * kLdlqBlock * K + col0;
    // this thread's share of a chunk: E rows rr = t >> 4 (8 of them), k = t & 15;
    // U k-rows kk = t >> 6 (4 of them), column cc = t & 63
    double pe[8], pu[4];
    auto fetch = [&](int kc) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int t = threadIdx.x + 256 * u;
            const int64_t r = row0 + (t >> 4);
            pe[u] = r < N ? E[r * kLdlqBlock + kc + (t & 15)] : 0.0;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int t = threadIdx.x + 256 * u;
            pu[u] = Ub[static_cast<int64_t>(kc + (t >> 6)) * K + (t & 63)];
        }
    };
    auto park = [&](int buf) {
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int t = threadIdx.x + 256 * u;
            Es[buf][t & 15][t >> 4] = pe[u];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int t = threadIdx.x + 256 * u;
            Us[buf][t >> 6][t & 63] = pu[u];
        }
    };
    fetch(0);
    double acc[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = row0 + ty + 16 * i;
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = r < N ? F[r * K + col0 + tx + 16 * j] : 0.0;
    }
    park(0);
    __syncthreads();
    for (int c = 0; c < kLdlqBlock / kUpdChunk; ++c) {
        const int buf = c & 1;
        const bool more = c + 1 < kLdlqBlock / kUpdChunk;
        if (more) fetch((c + 1) * kUpdChunk);
#pragma unroll 4
        for (int k = 0; k < kUpdChunk; ++k) {
            double ek[8], uk[4];
#pragma unroll
            for (int i = 0; i < 8; ++i) ek[i] = Es[buf][k][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) uk[j] = Us[buf][k][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 8; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fma(ek[i], uk[j], acc[i][j]);
        }
        // the other buffer was last read in chunk c - 1, before the previous barrier
        if (more) park(buf ^ 1);
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int64_t r = row0 + ty + 16 * i;
        if (r < N)
#pragma unroll
            for (int j = 0; j < 4; ++j) F[r * K + col0 + tx + 16 * j] = acc[i][j];
    }
}

}  // namespace

size_t ldlq_workspace_bytes(int64_t N, int64_t K) {
    return static_cast<size_t>(N) * static_cast<size_t>(K) * 8 + static_cast<size_t>(N) * kLdlqBlock * 8;
}

hipError_t launch_ldlq(int64_t N, int64_t K, const float* W, const double* U, const uint16_t* A, const uint16_t* B,
                       int64_t affine_groups, uint8_t* codes, void* workspace, hipStream_t s) {
    double* F = static_cast<double*>(workspace);
    double* E = F + N * K;
    const int64_t n = N * K;
    hipLaunchKernelGGL(ldlq_fill_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, s, F, n);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    const int blocks = static_cast<int>(K / kLdlqBlock);
    for (int b = 0; b < blocks; ++b) {
        hipLaunchKernelGGL(ldlq_block_kernel, dim3(static_cast<unsigned>((N + 3) / 4)), dim3(256), 0, s, N, K, b, W,
                           U, A, B, affine_groups, F, E, codes);
        if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
        if (b + 1 < blocks) {
            const dim3 grid(static_cast<unsigned>((N + kUpdRows - 1) / kUpdRows),
                            static_cast<unsigned>((K - (b + 1) * kLdlqBlock) / kUpdCols));
            hipLaunchKernelGGL(ldlq_update_kernel, grid, dim3(256), 0, s, N, K, b, E, U, F);
            if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
        }
    }
    return hipSuccess;
}

}  // namespace unisvq
