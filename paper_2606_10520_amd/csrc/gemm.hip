// Prefill product y = x * W_hat^T for any M on gfx950.
//
// For large M the dense product dominates, so each weight vector is decoded
// once per output tile as w_hat = A q + B (Sec. 3.1, Eq. 4; vectors along K
// as in Eq. 8) in fp32 and staged in LDS next to a tile of activations; the
// tile product runs on v_mfma_f32_16x16x32_{f16,bf16} with fp32 accumulation.
// Decoded weights exist only in LDS, never in global memory.
//   fp16 activations: w_hat is rounded once to fp16 (relative error 2^-11).
//   bf16 activations: a single bf16 rounding of w_hat (2^-9) would cost as
//   much as the whole output tolerance, so w_hat is carried as hi + lo, two
//   bf16 values (hi = bf16(w), lo = bf16(w - hi), relative error ~2^-17), and
//   the tile takes two matrix-core products.
//
// Tile: BM = 64 tokens x BN = 64 output rows per workgroup of 4 wavefronts
// (each 32 x 32 = 2 x 2 matrix-core tiles); the K loop steps one 128-column
// group at a time, the granularity of the affine parameters.
#include "common.hpp"

namespace unisvq {
namespace {

constexpr int BM = 64, BN = 64, BK = 128;
constexpr int LDS_STRIDE = BK + 8;  // elements; 16-byte pad against bank conflicts

template <typename XT>
struct GemmOps;
template <>
struct GemmOps<_Float16> {
    typedef f16x8 vec8;
    static constexpr bool kSplit = false;
    __device__ static inline f32x4 mfma(vec8 a, vec8 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <>
struct GemmOps<__bf16> {
    typedef bf16x8 vec8;
    static constexpr bool kSplit = true;
    __device__ static inline f32x4 mfma(vec8 a, vec8 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};

__device__ inline float bits_to_f32(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

template <typename XT>
__global__ __launch_bounds__(256) void gemm_kernel(const uint8_t* __restrict__ packed,
                                                   const XT* __restrict__ x, void* __restrict__ y,
                                                   int N, int K, int M, int y_dtype) {
    typedef typename GemmOps<XT>::vec8 vec8;
    __shared__ __attribute__((aligned(16))) XT xt[BM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) XT wt[BN * LDS_STRIDE];
    constexpr bool kSplit = GemmOps<XT>::kSplit;
    __shared__ __attribute__((aligned(16))) XT wlo[kSplit ? BN * LDS_STRIDE : 8];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int m0 = blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int groups = K >> 7;

    // decode assignment: row rho of the tile, vectors 8*part .. 8*part+7
    const int rho = tid >> 2, part = tid & 3;
    const int row = n0 + rho;
    const bool row_ok = row < N;
    const int rb = row >> 4, beta = row & 15;
    const uint8_t* blk = packed + static_cast<size_t>(rb) * groups * kGroupBlockBytes;

    const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
    f32x4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int g = 0; g < groups; ++g) {
        // activations: 64 tokens x 128 columns, 16 bytes per load
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 256 * i;
            const int tr = c >> 4, c16 = c & 15;
            uint4 v = {0u, 0u, 0u, 0u};
            if (m0 + tr < M)
                v = *reinterpret_cast<const uint4*>(x + static_cast<size_t>(m0 + tr) * K + g * BK + c16 * 8);
            *reinterpret_cast<uint4*>(xt + tr * LDS_STRIDE + c16 * 8) = v;
        }
        // weights: decode 8 vectors (32 weights) of one row
        XT wv[32], wl[32];
        if (row_ok) {
            const int p = g >> 1, j = g & 1;
            const bool half = (groups & 1) && g == groups - 1;
            const uint8_t* pk = blk + static_cast<size_t>(p) * kPacketBytes;
            uint32_t c16[4];
            float Am[4][4], Bv[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const int s = 4 * beta + b;
                const uint8_t* cf = half ? pk + 8 * s : pk + 16 * s + 8 * j;
                const uint8_t* af = half ? pk + kHalfAffineOff + 8 * s : pk + kPacketAffineOff + 16 * s + 8 * j;
                const uint8_t* bf = half ? pk + kHalfBiasOff + 2 * s : pk + kPacketBiasOff + 4 * s + 2 * j;
                c16[b] = *reinterpret_cast<const uint16_t*>(cf + 2 * part);
                const uint2 acol = *reinterpret_cast<const uint2*>(af);
                Am[0][b] = bits_to_f32(acol.x & 0xffffu);
                Am[1][b] = bits_to_f32(acol.x >> 16);
                Am[2][b] = bits_to_f32(acol.y & 0xffffu);
                Am[3][b] = bits_to_f32(acol.y >> 16);
                Bv[b] = bits_to_f32(*reinterpret_cast<const uint16_t*>(bf));
            }
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                float q[4];
#pragma unroll
                for (int b = 0; b < 4; ++b) q[b] = static_cast<float>((c16[b] >> (2 * v)) & 3u);
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    float w = Bv[a];
#pragma unroll
                    for (int b = 0; b < 4; ++b) w = __builtin_fmaf(Am[a][b], q[b], w);
                    const XT hi = static_cast<XT>(w);
                    wv[4 * v + a] = hi;
                    if (kSplit) wl[4 * v + a] = static_cast<XT>(w - static_cast<float>(hi));
                }
            }
        } else {
#pragma unroll
            for (int e = 0; e < 32; ++e) wv[e] = wl[e] = static_cast<XT>(0.f);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            *reinterpret_cast<uint4*>(wt + rho * LDS_STRIDE + part * 32 + 8 * e) =
                *reinterpret_cast<const uint4*>(wv + 8 * e);
            if (kSplit)
                *reinterpret_cast<uint4*>(wlo + rho * LDS_STRIDE + part * 32 + 8 * e) =
                    *reinterpret_cast<const uint4*>(wl + 8 * e);
        }
        __syncthreads();

#pragma unroll
        for (int kk = 0; kk < BK / 32; ++kk) {
            const int kof = kk * 32 + 8 * (lane >> 4);
            vec8 aop[2], bop[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                aop[i] = *reinterpret_cast<const vec8*>(xt + (wm + 16 * i + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bop[j] = *reinterpret_cast<const vec8*>(wt + (wn + 16 * j + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = GemmOps<XT>::mfma(aop[i], bop[j], acc[i][j]);
            if (kSplit) {
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bop[j] = *reinterpret_cast<const vec8*>(wlo + (wn + 16 * j + (lane & 15)) * LDS_STRIDE + kof);
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) acc[i][j] = GemmOps<XT>::mfma(aop[i], bop[j], acc[i][j]);
            }
        }
        __syncthreads();
    }

    // D lane layout: column (output row) = lane%16, rows (tokens) 4*(lane/16) + reg
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int r = n0 + wn + 16 * j + (lane & 15);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int t = m0 + wm + 16 * i + 4 * (lane >> 4) + e;
                if (t < M && r < N) store_out(y, static_cast<int64_t>(t) * N + r, acc[i][j][e], y_dtype);
            }
        }
}

}  // namespace

int launch_gemm(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>((M + BM - 1) / BM), static_cast<unsigned>((N + BN - 1) / BN));
    if (x_dtype == UNISVQ_F16)
        hipLaunchKernelGGL(gemm_kernel<_Float16>, grid, dim3(256), 0, s, packed,
                           static_cast<const _Float16*>(x), y, static_cast<int>(N), static_cast<int>(K),
                           static_cast<int>(M), y_dtype);
    else
        hipLaunchKernelGGL(gemm_kernel<__bf16>, grid, dim3(256), 0, s, packed,
                           static_cast<const __bf16*>(x), y, static_cast<int>(N), static_cast<int>(K),
                           static_cast<int>(M), y_dtype);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

}  // namespace unisvq
