// Block LDL^T factorisation of the layer Hessian on gfx950 (Sec. 3.2.2,
// Eq. 7): H = U D U^T with U unit upper block-triangular (4 x 4 identity
// blocks on the diagonal, zeros below them) and D block diagonal with 4 x 4
// blocks -- the factor whose off-diagonal entries are LDLQ's feedback
// coefficients.  All arithmetic in fp64.
//
// With U unit upper triangular the factorisation runs from the last column
// block to the first (the last pivot is H's own last diagonal block).  With
// S the part of H not yet factorised (its upper triangle held in U's own
// buffer), one 4 x 4 pivot block j gives
//     D_j = S_jj,   U[0:j, j] = S[0:j, j] D_j^-1,
//     S[0:j, 0:j] -= U[0:j, j] D_j U[0:j, j]^T.
// Blocked over panels of 64 columns (16 pivot blocks), right to left:
//  1. diag: one workgroup factorises the panel's 64 x 64 diagonal block
//     in LDS, pivot block by pivot block, and keeps the 16 inverses D_j^-1;
//  2. strip: every row r above the panel solves w U_pp^T = S[r, panel]
//     (U_pp the panel's factor, unit upper: a back substitution over its
//     pivot blocks) and stores w and U[r, panel] = w D_p^-1, one wavefront
//     per row, lane c = panel column c;
//  3. trailing: S[a][b] -= sum_k W[a][k] U[b][k] over the panel's 64
//     columns, for a <= b above the panel (64 x 64 tiles of the upper
//     triangle on the fp64 matrix cores).
// Every pivot block is checked for positive definiteness (its leading
// principal minors); the first failure is reported through `info`.
#include "common.hpp"

namespace unisvq {
namespace {

constexpr int kLdlP = 64;          // panel width (16 pivot blocks of 4)
constexpr int kLdlPitch = kLdlP + 1;  // LDS row pitch (doubles) of the diagonal block

__device__ inline double lane_f64(double v, int src) {
    const uint2 u = __builtin_bit_cast(uint2, v);
    return __builtin_bit_cast(double, uint2{static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u.x), src)),
                                            static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u.y), src))});
}

// U = upper triangle of H (a <= b), zeros below; info = 0.  Two elements per
// thread (K is even).  In place when U == H: each element is read and
// written by the same thread.
__global__ __launch_bounds__(256) void ldl_init_kernel(const double* H, double* U, int64_t K, int32_t* info) {
    const int64_t e = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 2;
    if (e == 0 && info) *info = 0;
    if (e >= K * K) return;
    const int64_t a = e / K, b = e - a * K;
    const double2 h = *reinterpret_cast<const double2*>(H + e);
    *reinterpret_cast<double2*>(U + e) = double2{a <= b ? h.x : 0.0, a <= b + 1 ? h.y : 0.0};
}

// Inverse of a 4 x 4 matrix by Laplace expansion along its first two rows
// (complementary 2 x 2 minors: s_ of rows 0, 1, c_ of rows 2, 3), every
// index fixed at compile time; returns the determinant.
__device__ inline double inverse4(const double (&m)[4][4], double (&b)[4][4]) {
    const double s0 = m[0][0] * m[1][1] - m[1][0] * m[0][1], s1 = m[0][0] * m[1][2] - m[1][0] * m[0][2];
    const double s2 = m[0][0] * m[1][3] - m[1][0] * m[0][3], s3 = m[0][1] * m[1][2] - m[1][1] * m[0][2];
    const double s4 = m[0][1] * m[1][3] - m[1][1] * m[0][3], s5 = m[0][2] * m[1][3] - m[1][2] * m[0][3];
    const double c5 = m[2][2] * m[3][3] - m[3][2] * m[2][3], c4 = m[2][1] * m[3][3] - m[3][1] * m[2][3];
    const double c3 = m[2][1] * m[3][2] - m[3][1] * m[2][2], c2 = m[2][0] * m[3][3] - m[3][0] * m[2][3];
    const double c1 = m[2][0] * m[3][2] - m[3][0] * m[2][2], c0 = m[2][0] * m[3][1] - m[3][0] * m[2][1];
    const double det = s0 * c5 - s1 * c4 + s2 * c3 + s3 * c2 - s4 * c1 + s5 * c0;
    const double r = 1.0 / det;
    b[0][0] = (m[1][1] * c5 - m[1][2] * c4 + m[1][3] * c3) * r;
    b[0][1] = (-m[0][1] * c5 + m[0][2] * c4 - m[0][3] * c3) * r;
    b[0][2] = (m[3][1] * s5 - m[3][2] * s4 + m[3][3] * s3) * r;
    b[0][3] = (-m[2][1] * s5 + m[2][2] * s4 - m[2][3] * s3) * r;
    b[1][0] = (-m[1][0] * c5 + m[1][2] * c2 - m[1][3] * c1) * r;
    b[1][1] = (m[0][0] * c5 - m[0][2] * c2 + m[0][3] * c1) * r;
    b[1][2] = (-m[3][0] * s5 + m[3][2] * s2 - m[3][3] * s1) * r;
    b[1][3] = (m[2][0] * s5 - m[2][2] * s2 + m[2][3] * s1) * r;
    b[2][0] = (m[1][0] * c4 - m[1][1] * c2 + m[1][3] * c0) * r;
    b[2][1] = (-m[0][0] * c4 + m[0][1] * c2 - m[0][3] * c0) * r;
    b[2][2] = (m[3][0] * s4 - m[3][1] * s2 + m[3][3] * s0) * r;
    b[2][3] = (-m[2][0] * s4 + m[2][1] * s2 - m[2][3] * s0) * r;
    b[3][0] = (-m[1][0] * c3 + m[1][1] * c1 - m[1][2] * c0) * r;
    b[3][1] = (m[0][0] * c3 - m[0][1] * c1 + m[0][2] * c0) * r;
    b[3][2] = (-m[3][0] * s3 + m[3][1] * s1 - m[3][2] * s0) * r;
    b[3][3] = (m[2][0] * s3 - m[2][1] * s1 + m[2][2] * s0) * r;
    return det;
}

// Panel [c0, c0 + 64): its diagonal block factorised in LDS, pivot block by
// pivot block (a = 4 jb, the last first).  Per pivot, two phases:
//  A. every thread t < max(1, a) inverts D_j itself (inverse4) and forms
//     row t of u = S[0:a, a:a+4] D_j^-1; thread 0 also writes D_j, D_j^-1 and
//     checks positive definiteness (the leading principal minors);
//  B. S[r][c] -= u[r] . S[c][a:a+4] for r <= c < a (thread: column c = t % 64,
//     rows t / 64 + 4k; computed for the whole block, without branches),
//     and u and the identity pivot block go to U.
// Entries below the pivot blocks keep the zeros written by the set-up, so
// the LDS block is never written back.  The 16 inverses go to dinv.
__global__ __launch_bounds__(256) void ldl_diag_kernel(double* U, int64_t K, int64_t c0, double* D, int32_t* info,
                                                       double* dinv) {
    __shared__ double B[kLdlP * kLdlPitch];
    __shared__ double Di[16 * 16];
    __shared__ double uu[kLdlP * 4];
    const int t = threadIdx.x;
    double* const blk = U + c0 * K + c0;
    const int c = t & 63, rq = t >> 6;
    {
        // all 16 loads of a thread in flight at once (row rq + 4k, column c)
        double v[kLdlP / 4];
#pragma unroll
        for (int k = 0; k < kLdlP / 4; ++k) v[k] = blk[(rq + 4 * k) * K + c];
#pragma unroll
        for (int k = 0; k < kLdlP / 4; ++k) B[(rq + 4 * k) * kLdlPitch + c] = v[k];
    }
    __syncthreads();
    for (int jb = kLdlP / 4 - 1; jb >= 0; --jb) {
        const int a = 4 * jb;
        // A.
        if (t == 0 || t < a) {
            double d[4][4], inv[4][4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) d[i][j] = B[(a + (i < j ? i : j)) * kLdlPitch + a + (i < j ? j : i)];
            const double det = inverse4(d, inv);
            if (t == 0) {
#pragma unroll
                for (int i = 0; i < 16; ++i) Di[jb * 16 + i] = inv[i >> 2][i & 3];
                if (D) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) D[(c0 / 4 + jb) * 16 + i] = d[i >> 2][i & 3];
                }
                const double m2 = d[0][0] * d[1][1] - d[1][0] * d[0][1];
                const double m3 = d[0][0] * (d[1][1] * d[2][2] - d[1][2] * d[2][1]) -
                                  d[0][1] * (d[1][0] * d[2][2] - d[1][2] * d[2][0]) +
                                  d[0][2] * (d[1][0] * d[2][1] - d[1][1] * d[2][0]);
                const bool ok = d[0][0] > 0.0 && m2 > 0.0 && m3 > 0.0 && det > 0.0;  // false on NaN
                if (!ok && info && *info == 0) *info = static_cast<int32_t>(c0 / 4 + jb + 1);
            }
            if (t < a) {
                double x[4];
#pragma unroll
                for (int n = 0; n < 4; ++n) x[n] = B[t * kLdlPitch + a + n];
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    double v = 0.0;
#pragma unroll
                    for (int n = 0; n < 4; ++n) v = fma(x[n], inv[n][m], v);
                    uu[t * 4 + m] = v;
                }
            }
        }
        __syncthreads();
        // B.  Only S[r][c] with r <= c < a is live: the LDS entries below the
        // diagonal and those of columns a and beyond are never read again
        // (the factor goes straight to U), so the whole block is updated
        // without branches; the dead entries take whatever they get.
        {
            double bc[4];
#pragma unroll
            for (int n = 0; n < 4; ++n) bc[n] = B[c * kLdlPitch + a + n];
#pragma unroll
            for (int k = 0; k < kLdlP / 4; ++k) {
                const int r = rq + 4 * k;
                double v = 0.0;
#pragma unroll
                for (int n = 0; n < 4; ++n) v = fma(uu[r * 4 + n], bc[n], v);
                B[r * kLdlPitch + c] -= v;
            }
        }
        if (t < 4 * a) blk[(t >> 2) * K + a + (t & 3)] = uu[t];
        if (t < 16) blk[(a + (t >> 2)) * K + a + (t & 3)] = (t >> 2) == (t & 3) ? 1.0 : 0.0;
        __syncthreads();
    }
    dinv[t] = Di[t];  // 256 threads, 16 x 16 values
}

// Rows r < c0 against the panel [c0, c0 + 64): w U_pp^T = S[r, panel]
// (back substitution, the last pivot block first), W[r] = w,
// U[r, panel] = w D_p^-1.  One wavefront per row, lane c = column c0 + c.
__global__ __launch_bounds__(256) void ldl_strip_kernel(double* U, int64_t K, int64_t c0, const double* dinv,
                                                        double* W) {
    __shared__ double Up[kLdlP * kLdlPitch];
    __shared__ double Di[16 * 16];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const double* const blk = U + c0 * K + c0;
    {
        double v[kLdlP / 4];
#pragma unroll
        for (int k = 0; k < kLdlP / 4; ++k) v[k] = blk[(wave + 4 * k) * K + lane];
        const double di = dinv[t];
#pragma unroll
        for (int k = 0; k < kLdlP / 4; ++k) Up[(wave + 4 * k) * kLdlPitch + lane] = v[k];
        Di[t] = di;
    }
    __syncthreads();
    const int b = lane >> 2;  // the lane's pivot block
    for (int64_t r = static_cast<int64_t>(blockIdx.x) * 4 + wave; r < c0; r += static_cast<int64_t>(gridDim.x) * 4) {
        double s = U[r * K + c0 + lane];
        for (int jb = kLdlP / 4 - 1; jb >= 1; --jb) {
            // block jb is final: remove its part from the lanes of the blocks before it
            const double w0 = lane_f64(s, 4 * jb), w1 = lane_f64(s, 4 * jb + 1);
            const double w2 = lane_f64(s, 4 * jb + 2), w3 = lane_f64(s, 4 * jb + 3);
            if (b < jb) {
                const double* const up = Up + lane * kLdlPitch + 4 * jb;
                double acc = w0 * up[0];
                acc = fma(w1, up[1], acc);
                acc = fma(w2, up[2], acc);
                acc = fma(w3, up[3], acc);
                s -= acc;
            }
        }
        W[r * kLdlP + lane] = s;
        // u = w D^-1 within the lane's pivot block
        double u = 0.0;
#pragma unroll
        for (int n = 0; n < 4; ++n) u = fma(__shfl(s, (lane & ~3) + n, 64), Di[b * 16 + n * 4 + (lane & 3)], u);
        U[r * K + c0 + lane] = u;
    }
}

// S[a][b] -= sum_k W[a][k] U[b][c0 + k] for a <= b < c0: workgroup (tb, ta)
// takes the 64 x 64 tile of rows 64 ta, columns 64 tb (tiles below the
// diagonal return at once) on the fp64 matrix cores.  Both 64 x 64 operands
// are staged row-major in LDS (pitch 68 doubles: an operand read touches
// every bank the minimum number of times); wavefront w computes the 32 x 32
// quarter (rows 32 (w / 2), columns 32 (w % 2)) as 2 x 2 blocks of
// v_mfma_f64_16x16x4f64 over 16 steps of 4 columns of k.  Operand lanes:
// A[i][k] at lane i + 16 k, B[k][j] at lane j + 16 k; result D[i][j] at
// lane j + 16 (i % 4), item i / 4.
constexpr int kLdlMPitch = kLdlP + 4;
typedef double f64x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void ldl_trailing_kernel(double* U, int64_t K, int64_t c0, const double* W) {
    const int ta = blockIdx.y, tb = blockIdx.x;
    if (ta > tb) return;  // uniform
    __shared__ double Ws[kLdlP * kLdlMPitch];  // [row][k]
    __shared__ double Us[kLdlP * kLdlMPitch];  // [column][k]
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int64_t a0 = static_cast<int64_t>(ta) * kLdlP, b0 = static_cast<int64_t>(tb) * kLdlP;
    const int wr = 32 * (wave >> 1), wc = 32 * (wave & 1);
    const int li = lane & 15, lk = lane >> 4;
    // this lane's 16 outputs, read now (every one in bounds: the tile lies
    // above row c0) and written back after the products
    double old[2][2][4];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                old[bi][bj][v] = U[(a0 + wr + 16 * bi + lk + 4 * v) * K + b0 + wc + 16 * bj + li];
    {
        // the operands, 16 + 16 coalesced loads per thread in flight at once
        // (row rq + 4k, column c of each 64 x 64 operand)
        const int c = t & 63, rq = t >> 6;
        double wv[kLdlP / 4], uv[kLdlP / 4];
#pragma unroll
        for (int k = 0; k < kLdlP / 4; ++k) {
            wv[k] = W[(a0 + rq + 4 * k) * kLdlP + c];
            uv[k] = U[(b0 + rq + 4 * k) * K + c0 + c];
        }
#pragma unroll
        for (int k = 0; k < kLdlP / 4; ++k) {
            Ws[(rq + 4 * k) * kLdlMPitch + c] = wv[k];
            Us[(rq + 4 * k) * kLdlMPitch + c] = uv[k];
        }
    }
    __syncthreads();
    f64x4 acc[2][2];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) acc[bi][bj] = f64x4{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int s = 0; s < kLdlP / 4; ++s) {
        double av[2], bv[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            av[q] = Ws[(wr + 16 * q + li) * kLdlMPitch + 4 * s + lk];
            bv[q] = Us[(wc + 16 * q + li) * kLdlMPitch + 4 * s + lk];
        }
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int bj = 0; bj < 2; ++bj)
                acc[bi][bj] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[bi], bv[bj], acc[bi][bj], 0, 0, 0);
    }
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t a = a0 + wr + 16 * bi + lk + 4 * v;
                const int64_t bcol = b0 + wc + 16 * bj + li;
                if (a <= bcol) U[a * K + bcol] = old[bi][bj][v] - acc[bi][bj][v];
            }
}

}  // namespace

size_t ldl_workspace_bytes(int64_t K) {
    return static_cast<size_t>(K) * kLdlP * 8 + 16 * 16 * 8;
}

hipError_t launch_ldl(int64_t K, const double* H, double* U, double* D, int32_t* info, void* workspace,
                      hipStream_t s) {
    double* const W = static_cast<double*>(workspace);
    double* const dinv = W + K * kLdlP;
    const int64_t pairs = K * K / 2;
    hipLaunchKernelGGL(ldl_init_kernel, dim3(static_cast<unsigned>((pairs + 255) / 256)), dim3(256), 0, s, H, U, K,
                       info);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    for (int64_t c0 = K - kLdlP; c0 >= 0; c0 -= kLdlP) {
        hipLaunchKernelGGL(ldl_diag_kernel, dim3(1), dim3(256), 0, s, U, K, c0, D, info, dinv);
        if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
        if (c0 == 0) break;
        const int64_t rows4 = c0 / 4;
        hipLaunchKernelGGL(ldl_strip_kernel, dim3(static_cast<unsigned>(rows4 < 1024 ? rows4 : 1024)), dim3(256), 0,
                           s, U, K, c0, dinv, W);
        if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
        const unsigned nt = static_cast<unsigned>(c0 / kLdlP);
        hipLaunchKernelGGL(ldl_trailing_kernel, dim3(nt, nt), dim3(256), 0, s, U, K, c0, W);
        if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    }
    return hipSuccess;
}

}  // namespace unisvq
