// Decode-phase product y = x * W_hat^T for M <= 4 tokens on gfx950.
//
// The affine decode commutes with the product (Sec. 3.1; Eq. 9 of Sec.
// 3.2.3), so instead of rebuilding every weight (A q + B: four multiply-adds
// per weight) the kernel forms, per (row r, group g, token t), the 4x4 matrix
//     T[a][b] = sum_{v in g} x[t][128g + 4v + a] * q[r][128g + 4v + b]
// on the matrix cores, and then applies the group's parameters once:
//     y[t][r] += sum_{a,b} A[a][b] T[a][b] + sum_a B[a] * xbar[t][g][a],
// with xbar[t][g][a] = sum_v x[t][128g + 4v + a].  This is exactly
// sum_k x[t][k] * W_hat[r][k] (distributivity), accumulated in fp32.
//
// Matrix-core mapping (v_mfma_f32_4x4x4_16b, 16 independent 4x4x4 blocks):
//   block beta = lane/4 <-> row 16*rb + beta, column j = lane%4 <-> component b,
//   k (4 per instruction, 8 instructions per group) <-> vectors of the group.
//   SrcA = activations x[v][a] -- identical for all 16 blocks, so it is held
//   only by lanes 0..3 and broadcast to every block (CBSZ = 4, ABID = 0).
//   SrcB = codes q[v][b]: lane s of a packet slot already holds component b of
//   all 32 vectors of its row (packed format v1), converted to exact small
//   integers with the fp4 (e2m1) converter: a 2-bit code c in the low bits of
//   a nibble is the e2m1 value c/2, scaled by 2.
//   D lane (beta, b) holds T[a = 0..3][b]; it needs A[r][g][0..3][b] and
//   B[r][g][b], which is exactly that lane's affine slot.
// The dequantised weights never leave registers (they are never formed).
//
// Work split: one workgroup per 16-row block; its WAVES wavefronts split the
// packets along K; partial sums meet in LDS.  Activations for the whole K
// range are staged in LDS once per workgroup in matrix-core operand order.
#include <atomic>

#include "common.hpp"

namespace unisvq {
namespace {

template <typename XT>
struct XOps;

template <>
struct XOps<_Float16> {
    typedef f16x4 vec4;
    template <int SEL>
    __device__ static inline f16x2 cvt2(uint32_t w) {
        return __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 2.0f, SEL);
    }
    __device__ static inline f32x4 mfma(vec4 a, vec4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_4x4x4f16(a, b, c, 4, 0, 0);
    }
};

template <>
struct XOps<__bf16> {
    typedef bf16x4 vec4;
    template <int SEL>
    __device__ static inline bf16x2 cvt2(uint32_t w) {
        return __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 2.0f, SEL);
    }
    __device__ static inline f32x4 mfma(vec4 a, vec4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(a, b, c, 4, 0, 0);
    }
};

// 16 codes of one 32-bit word (vectors 16h .. 16h+15 of one component) ->
// four SrcB operands.  Operand n holds vectors 4n+0, 4n+2, 4n+1, 4n+3 (the
// nibble order the e2m1 converter produces); the activation operand uses the
// same slot order.
template <typename XT, int N>
__device__ inline typename XOps<XT>::vec4 code_operand(uint32_t e, uint32_t o) {
    auto lo = XOps<XT>::template cvt2<N>(e);
    auto hi = XOps<XT>::template cvt2<N>(o);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
}

template <typename XT>
__device__ inline void word_operands(uint32_t w, typename XOps<XT>::vec4* ops) {
    const uint32_t e = w & 0x33333333u;
    const uint32_t o = (w >> 2) & 0x33333333u;
    ops[0] = code_operand<XT, 0>(e, o);
    ops[1] = code_operand<XT, 1>(e, o);
    ops[2] = code_operand<XT, 2>(e, o);
    ops[3] = code_operand<XT, 3>(e, o);
}

// Position of vector v (0..31 in its group) inside the 32-slot operand
// order of one (token, group, component) line of the staged activations.
__device__ inline int operand_slot(int v) {
    const int j = v & 3;
    return (v & ~3) | ((j & 1) << 1) | (j >> 1);
}

__device__ inline float h2f(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

// Contract one group: codes (two words = the lane's 64-bit field), A column,
// B value; adds the group's contribution for every token into acc.
template <typename XT, int MT>
__device__ inline void group_step(uint32_t w0, uint32_t w1, uint32_t a01, uint32_t a23, uint32_t bbits,
                                  const XT* __restrict__ xs_g, const float* __restrict__ xbar_g,
                                  int xs_tok_stride, int xbar_tok_stride, int M, int lane,
                                  typename XOps<XT>::vec4 (&xop)[8], float (&acc)[MT]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop[8];
    word_operands<XT>(w0, cop);
    word_operands<XT>(w1, cop + 4);
    const float A0 = h2f(a01 & 0xffffu), A1 = h2f(a01 >> 16);
    const float A2 = h2f(a23 & 0xffffu), A3 = h2f(a23 >> 16);
    const float Bv = h2f(bbits);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        if (t < M) {
            if (lane < 4) {
                const vec4* src = reinterpret_cast<const vec4*>(xs_g + t * xs_tok_stride + lane * 32);
#pragma unroll
                for (int s = 0; s < 8; ++s) xop[s] = src[s];
            }
            f32x4 d = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < 8; ++s) d = XOps<XT>::mfma(xop[s], cop[s], d);
            const float xb = xbar_g[t * xbar_tok_stride + (lane & 3)];
            float r = acc[t];
            r = __builtin_fmaf(A0, d[0], r);
            r = __builtin_fmaf(A1, d[1], r);
            r = __builtin_fmaf(A2, d[2], r);
            r = __builtin_fmaf(A3, d[3], r);
            acc[t] = __builtin_fmaf(Bv, xb, r);
        }
    }
}

template <typename XT, int WAVES, int MT, int PF>
__global__ __launch_bounds__(WAVES * 64) void gemv_kernel(const uint8_t* __restrict__ packed,
                                                          const XT* __restrict__ x,
                                                          void* __restrict__ y, int N, int K, int M,
                                                          int y_dtype) {
    typedef typename XOps<XT>::vec4 vec4;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int groups = K >> 7;
    const int nfull = groups >> 1;
    const bool has_half = (groups & 1) != 0;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int rb = blockIdx.x;

    XT* xs = reinterpret_cast<XT*>(smem);                                     // [M][groups][4][32]
    float* xbar = reinterpret_cast<float*>(smem + static_cast<size_t>(M) * groups * 256);  // [M][groups][4]
    float* red = xbar + M * groups * 4;                                       // [WAVES][MT][16]

    const uint8_t* blk = packed + static_cast<size_t>(rb) * groups * kGroupBlockBytes;
    const int per = (nfull + WAVES - 1) / WAVES;
    const int p0 = min(nfull, wave * per);
    const int np = min(nfull, p0 + per) - p0;

    // 1. Issue this wave's first PF packet loads; they do not depend on x.
    uint4 cbuf[PF], abuf[PF];
    uint32_t bbuf[PF];
    if (np > 0) {
#pragma unroll
        for (int i = 0; i < PF; ++i) {
            const uint8_t* pk = blk + static_cast<size_t>(p0 + min(i, np - 1)) * kPacketBytes;
            cbuf[i] = *reinterpret_cast<const uint4*>(pk + 16 * lane);
            abuf[i] = *reinterpret_cast<const uint4*>(pk + kPacketAffineOff + 16 * lane);
            bbuf[i] = *reinterpret_cast<const uint32_t*>(pk + kPacketBiasOff + 4 * lane);
        }
    }
    const bool do_half = has_half && wave == WAVES - 1;
    uint2 hc = {0u, 0u}, ha = {0u, 0u};
    uint32_t hb = 0;
    if (do_half) {
        const uint8_t* pk = blk + static_cast<size_t>(nfull) * kPacketBytes;
        hc = *reinterpret_cast<const uint2*>(pk + 8 * lane);
        ha = *reinterpret_cast<const uint2*>(pk + kHalfAffineOff + 8 * lane);
        hb = *reinterpret_cast<const uint16_t*>(pk + kHalfBiasOff + 2 * lane);
    }

    // 2. Stage activations in operand order and their per-(group, component) sums.
    const int chunks_per_tok = K >> 3;
    for (int c = threadIdx.x; c < M * chunks_per_tok; c += WAVES * 64) {
        const int t = c / chunks_per_tok;
        const int k0 = (c - t * chunks_per_tok) << 3;
        const uint4 raw = *reinterpret_cast<const uint4*>(x + static_cast<size_t>(t) * K + k0);
        const uint16_t* v16 = reinterpret_cast<const uint16_t*>(&raw);
        const int g = k0 >> 7;
        const int vbase = (k0 & 127) >> 2;
        uint16_t* line = reinterpret_cast<uint16_t*>(xs) + (static_cast<size_t>(t) * groups + g) * 128;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int v = vbase + (e >> 2), a = e & 3;
            line[a * 32 + operand_slot(v)] = v16[e];
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < M * groups * 4; i += WAVES * 64) {
        const XT* src = xs + static_cast<size_t>(i) * 32;
        float s = 0.f;
#pragma unroll
        for (int v = 0; v < 32; ++v) s += static_cast<float>(src[v]);
        xbar[i] = s;
    }
    __syncthreads();

    // 3. Main loop over this wave's full packets, PF loads in flight.
    float acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = 0.f;
    vec4 xop[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) xop[s] = vec4{};
    const int xs_tok = groups * 128;  // elements per token in xs
    const int xb_tok = groups * 4;
    for (int i = 0; i < np; i += PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j) {
            if (i + j < np) {
                const uint4 c = cbuf[j], a = abuf[j];
                const uint32_t bw = bbuf[j];
                const int nxt = min(i + j + PF, np - 1);
                const uint8_t* pk = blk + static_cast<size_t>(p0 + nxt) * kPacketBytes;
                cbuf[j] = *reinterpret_cast<const uint4*>(pk + 16 * lane);
                abuf[j] = *reinterpret_cast<const uint4*>(pk + kPacketAffineOff + 16 * lane);
                bbuf[j] = *reinterpret_cast<const uint32_t*>(pk + kPacketBiasOff + 4 * lane);
                const int g = 2 * (p0 + i + j);
                group_step<XT, MT>(c.x, c.y, a.x, a.y, bw & 0xffffu, xs + g * 128, xbar + g * 4,
                                   xs_tok, xb_tok, M, lane, xop, acc);
                group_step<XT, MT>(c.z, c.w, a.z, a.w, bw >> 16, xs + (g + 1) * 128,
                                   xbar + (g + 1) * 4, xs_tok, xb_tok, M, lane, xop, acc);
            }
        }
    }
    if (do_half) {
        const int g = groups - 1;
        group_step<XT, MT>(hc.x, hc.y, ha.x, ha.y, hb, xs + g * 128, xbar + g * 4, xs_tok, xb_tok, M,
                           lane, xop, acc);
    }

    // 4. Sum the four component lanes of each row, then the waves.
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        float v = acc[t];
        v += __shfl_xor(v, 1);
        v += __shfl_xor(v, 2);
        if ((lane & 3) == 0) red[(wave * MT + t) * 16 + (lane >> 2)] = v;
    }
    __syncthreads();
    if (threadIdx.x < M * 16) {
        const int t = threadIdx.x >> 4, r = threadIdx.x & 15;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += red[(w * MT + t) * 16 + r];
        store_out(y, static_cast<int64_t>(t) * N + static_cast<int64_t>(rb) * kRowBlock + r, s, y_dtype);
    }
}

template <typename XT, int WAVES, int MT>
size_t gemv_lds_bytes(int K, int M) {
    const size_t groups = K / kGroup;
    return static_cast<size_t>(M) * groups * (256 + 16) + static_cast<size_t>(WAVES) * MT * 16 * 4;
}

constexpr int kPrefetch = 4;
constexpr size_t kMaxLds = 160 * 1024;

template <typename XT, int WAVES, int MT>
int launch_cfg(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, void* y,
               int y_dtype, hipStream_t s) {
    const size_t lds = gemv_lds_bytes<XT, WAVES, MT>(static_cast<int>(K), static_cast<int>(M));
    if (lds > kMaxLds) return UNISVQ_EUNSUP;
    // Raising the dynamic-LDS limit is idempotent; do it once per instantiation.
    static std::atomic<int> attr_done{0};
    if (!attr_done.load(std::memory_order_acquire)) {
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<XT, WAVES, MT, kPrefetch>),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(kMaxLds)) != hipSuccess)
            return UNISVQ_EHIP;
        attr_done.store(1, std::memory_order_release);
    }
    hipLaunchKernelGGL((gemv_kernel<XT, WAVES, MT, kPrefetch>), dim3(static_cast<unsigned>(N / kRowBlock)), dim3(WAVES * 64), lds, s,
                       packed, static_cast<const XT*>(x), y, static_cast<int>(N), static_cast<int>(K),
                       static_cast<int>(M), y_dtype);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

template <typename XT, int MT>
int launch_waves(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, void* y,
                 int y_dtype, hipStream_t s) {
    // Enough wavefronts to cover 256 CUs several times over, while keeping
    // at least two packets per wavefront.
    const int64_t blocks = N / kRowBlock;
    const int64_t packets = (K / kGroup) / 2;
    int waves = 4;
    while (waves < 16 && blocks * waves < 2048 && packets >= 2 * (waves * 2)) waves *= 2;
    if (waves == 4) return launch_cfg<XT, 4, MT>(N, K, packed, M, x, y, y_dtype, s);
    if (waves == 8) return launch_cfg<XT, 8, MT>(N, K, packed, M, x, y, y_dtype, s);
    return launch_cfg<XT, 16, MT>(N, K, packed, M, x, y, y_dtype, s);
}

template <typename XT>
int launch_tokens(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, void* y,
                  int y_dtype, hipStream_t s) {
    if (M == 1) return launch_waves<XT, 1>(N, K, packed, M, x, y, y_dtype, s);
    if (M == 2) return launch_waves<XT, 2>(N, K, packed, M, x, y, y_dtype, s);
    return launch_waves<XT, 4>(N, K, packed, M, x, y, y_dtype, s);
}

}  // namespace

int launch_gemv(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, hipStream_t s) {
    if (M > 4) return UNISVQ_EUNSUP;
    if (x_dtype == UNISVQ_F16) return launch_tokens<_Float16>(N, K, packed, M, x, y, y_dtype, s);
    return launch_tokens<__bf16>(N, K, packed, M, x, y, y_dtype, s);
}

}  // namespace unisvq
