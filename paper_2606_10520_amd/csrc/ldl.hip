// Block LDL^T factorisation of the layer Hessian on gfx950 (Sec. 3.2.2,
// Eq. 7): H = U D U^T with U unit upper block-triangular (4 x 4 identity
// blocks on the diagonal, zeros below them) and D block diagonal with 4 x 4
// blocks -- the factor whose off-diagonal entries are LDLQ's feedback
// coefficients.  All arithmetic in fp64.
//
// The factorisation runs from the last column block to the first, the way
// the feedback runs from the later columns' point of view.  With S the part
// of H not yet factorised (its upper triangle held in U's own buffer), one
// 4 x 4 pivot block j gives
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
//     triangle, 4 x 4 outputs per thread).
// Every pivot block is checked for positive definiteness (its 4 x 4
// Cholesky factor); the first failure is reported through `info`.
#include "common.hpp"

namespace unisvq {
namespace {

constexpr int kLdlP = 64;          // panel width (16 pivot blocks of 4)
constexpr int kLdlPitch = kLdlP + 1;  // LDS row pitch (doubles) of the diagonal block
constexpr int kLdlTPitch = kLdlP + 2;  // LDS pitch of the transposed trailing operands

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

// Panel [c0, c0 + 64): its diagonal block factorised in LDS.  Writes the
// block's U (identity pivot blocks, zeros below them), D (when given) and
// the 16 inverses D_j^-1 to dinv[16][4][4].
__global__ __launch_bounds__(256) void ldl_diag_kernel(double* U, int64_t K, int64_t c0, double* D, int32_t* info,
                                                       double* dinv) {
    __shared__ double B[kLdlP * kLdlPitch];
    __shared__ double Di[16 * 16];
    __shared__ double uu[kLdlP * 4];
    const int t = threadIdx.x;
    double* const blk = U + c0 * K + c0;
    for (int i = t; i < kLdlP * kLdlP; i += 256) {
        const int r = i / kLdlP, c = i % kLdlP;
        B[r * kLdlPitch + c] = r <= c ? blk[r * K + c] : 0.0;
    }
    __syncthreads();
    for (int jb = kLdlP / 4 - 1; jb >= 0; --jb) {
        const int a = 4 * jb;
        if (t == 0) {
            // D_j from the upper triangle, its Cholesky factor L, then
            // D_j^-1 = L^-T L^-1
            double d[4][4], L[4][4] = {}, Li[4][4] = {};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) d[i][j] = B[(a + (i < j ? i : j)) * kLdlPitch + a + (i < j ? j : i)];
            if (D) {
#pragma unroll
                for (int i = 0; i < 16; ++i) D[(c0 / 4 + jb) * 16 + i] = d[i >> 2][i & 3];
            }
            bool ok = true;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                double s = d[j][j];
#pragma unroll
                for (int k = 0; k < j; ++k) s -= L[j][k] * L[j][k];
                if (!(s > 0.0)) ok = false;  // also NaN
                L[j][j] = sqrt(s);
#pragma unroll
                for (int i = j + 1; i < 4; ++i) {
                    double v = d[i][j];
#pragma unroll
                    for (int k = 0; k < j; ++k) v -= L[i][k] * L[j][k];
                    L[i][j] = v / L[j][j];
                }
            }
            if (!ok && info && *info == 0) *info = static_cast<int32_t>(c0 / 4 + jb + 1);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                Li[i][i] = 1.0 / L[i][i];
#pragma unroll
                for (int j = 0; j < i; ++j) {
                    double s = 0.0;
#pragma unroll
                    for (int k = j; k < i; ++k) s += L[i][k] * Li[k][j];
                    Li[i][j] = -s / L[i][i];
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    double s = 0.0;
#pragma unroll
                    for (int k = (i > j ? i : j); k < 4; ++k) s += Li[k][i] * Li[k][j];
                    Di[jb * 16 + i * 4 + j] = s;
                }
        }
        __syncthreads();
        // the rows above the pivot: u = S[0:a, a:a+4] D_j^-1
        if (t < 4 * a) {
            const int r = t >> 2, m = t & 3;
            double s = 0.0;
#pragma unroll
            for (int n = 0; n < 4; ++n) s = fma(B[r * kLdlPitch + a + n], Di[jb * 16 + n * 4 + m], s);
            uu[r * 4 + m] = s;
        }
        __syncthreads();
        // S[r][c] -= u[r] . S[c][a:a+4] for r <= c < a
        for (int i = t; i < a * a; i += 256) {
            const int r = i / a, c = i - r * a;
            if (r <= c) {
                double s = 0.0;
#pragma unroll
                for (int m = 0; m < 4; ++m) s = fma(uu[r * 4 + m], B[c * kLdlPitch + a + m], s);
                B[r * kLdlPitch + c] -= s;
            }
        }
        __syncthreads();
        if (t < 4 * a) B[(t >> 2) * kLdlPitch + a + (t & 3)] = uu[t];
        if (t < 16) B[(a + (t >> 2)) * kLdlPitch + a + (t & 3)] = (t >> 2) == (t & 3) ? 1.0 : 0.0;
        __syncthreads();
    }
    for (int i = t; i < kLdlP * kLdlP; i += 256) {
        const int r = i / kLdlP, c = i % kLdlP;
        blk[r * K + c] = B[r * kLdlPitch + c];
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
    for (int i = t; i < kLdlP * kLdlP; i += 256) {
        const int r = i / kLdlP, c = i % kLdlP;
        Up[r * kLdlPitch + c] = blk[r * K + c];
    }
    Di[t] = dinv[t];
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
// diagonal return at once); thread (ty, tx) 4 x 4 outputs.
__global__ __launch_bounds__(256) void ldl_trailing_kernel(double* U, int64_t K, int64_t c0, const double* W) {
    const int ta = blockIdx.y, tb = blockIdx.x;
    if (ta > tb) return;  // uniform
    __shared__ double Wt[kLdlP * kLdlTPitch];  // [k][row]
    __shared__ double Ut[kLdlP * kLdlTPitch];  // [k][column]
    const int t = threadIdx.x;
    const int64_t a0 = static_cast<int64_t>(ta) * kLdlP, b0 = static_cast<int64_t>(tb) * kLdlP;
    for (int e = t; e < kLdlP * kLdlP; e += 256) {
        const int i = e >> 6, k = e & 63;
        Wt[k * kLdlTPitch + i] = W[(a0 + i) * kLdlP + k];
        Ut[k * kLdlTPitch + i] = U[(b0 + i) * K + c0 + k];
    }
    __syncthreads();
    const int ty = t >> 4, tx = t & 15;
    double acc[4][4] = {};
    for (int k = 0; k < kLdlP; ++k) {
        double wv[4], uv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            wv[i] = Wt[k * kLdlTPitch + 4 * ty + i];
            uv[i] = Ut[k * kLdlTPitch + 4 * tx + i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = fma(wv[i], uv[j], acc[i][j]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t a = a0 + 4 * ty + i;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t bcol = b0 + 4 * tx + j;
            if (a <= bcol) U[a * K + bcol] -= acc[i][j];
        }
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
