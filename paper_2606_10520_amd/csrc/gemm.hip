// Prefill product y = x * W_hat^T for any M on gfx950.
//
// For large M the dense product dominates.  Each workgroup owns a tile of
// BM tokens x 128 output rows and walks K one 128-column group (one affine
// parameter set per row, Sec. 3.1) at a time:
//   * the group's weights are decoded once per workgroup, w_hat = A q + B
//     (Eq. 4, vectors along K as in Eq. 8), in fp32 (the fp16 parameters
//     times the exact small-integer codes), rounded once to fp16 and written
//     to LDS -- decoded weights never reach global memory;
//   * every wavefront owns 16*MI tokens and multiplies them with all 128
//     decoded rows on v_mfma_f32_16x16x32_f16 (fp32 accumulation); its
//     activation operands come straight from global memory in the matrix-
//     core layout, the weight operands from LDS.
// The decode of group g+1 (into the second LDS buffer, from packet data
// loaded one group earlier still) is interleaved with the products of group
// g, so the vector ALUs work under the matrix cores.
//
// bf16 activations are multiplied in fp16 as well: a pre-pass scales each
// token's row by a power of two 2^s_t so that its largest magnitude lies in
// [2^14, 2^15) and rounds it to fp16 -- exact for every element not more
// than 2^-28 below that maximum (fp16 keeps 11 significant bits, bf16 has
// 8) -- and the epilogue multiplies by 2^-s_t.  The product therefore
// carries the same single rounding of w_hat to fp16 (2^-11 relative) as the
// fp16 path, where bf16 operands would need w_hat split into two bf16 terms
// and twice the matrix-core work.
#include "common.hpp"

namespace unisvq {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kNI = 8;                // 16-row output tiles per wavefront
constexpr int kBN = 16 * kNI;         // output rows per workgroup
constexpr int kLdsRow = kGroup + 8;   // halves per decoded row in LDS (16-byte pad)
constexpr int kWBuf = kBN * kLdsRow;  // halves per decoded-weight buffer

__device__ inline float h2f(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

// The packet data one thread decodes for one group: row r of the tile,
// vectors 16*hv .. 16*hv+15 of the group, all four components b.
struct Piece {
    uint32_t code[4];  // F(r, g, b) bits 32*hv .. 32*hv+31: 16 codes of component b
    uint2 acol[4];     // A[r][g][0..3][b]
    uint4 bias;        // the B values of the row's four slots (layout depends on `half`)
    bool half;         // group stored in a half packet
};

// g >= groups loads nothing (offsets past the end of the buffer).
__device__ inline void load_piece(__amdgpu_buffer_rsrc_t rw, uint32_t rowblk, int g, int groups, int beta,
                                  int hv, Piece& pc) {
    const int p = g >> 1, j = g & 1;
    const bool half = (groups & 1) && g == groups - 1;
    const uint32_t P = g < groups ? rowblk + static_cast<uint32_t>(p) * kPacketBytes : kOutOfRange;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        const uint32_t s = 4 * beta + b;
        const uint32_t co = half ? P + 8 * s + 4 * hv : P + 16 * s + 8 * j + 4 * hv;
        const uint32_t ao = half ? P + kHalfAffineOff + 8 * s : P + kPacketAffineOff + 16 * s + 8 * j;
        pc.code[b] = ld32(rw, co);
        pc.acol[b] = ld64(rw, ao);
    }
    // Full packet: 4 bytes per slot (groups 2p, 2p+1); half packet: 2 bytes
    // per slot (the 16 bytes read cover this row's four slots and whatever
    // follows them, which is not used).
    pc.bias = ld128(rw, half ? P + kHalfBiasOff + 8 * beta : P + kPacketBiasOff + 16 * beta);
    pc.half = half;
}

// B[r][g][a] from the piece.
__device__ inline uint32_t piece_bias(const Piece& pc, int a, int j) {
    const uint32_t w[4] = {pc.bias.x, pc.bias.y, pc.bias.z, pc.bias.w};
    if (pc.half) return (a & 1) ? w[a >> 1] >> 16 : w[a >> 1] & 0xffffu;
    return j ? w[a] >> 16 : w[a] & 0xffffu;
}

// Decode vectors 4*SEL .. 4*SEL+3 of the piece (16 weights) and store them,
// in K order, at dst (16 halves).
template <int SEL>
__device__ inline void decode4(const Piece& pc, int j, _Float16* dst) {
    f16x2 qe[4], qo[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
        // nibble n of e holds vector 2n, nibble n of o vector 2n+1; the fp4
        // converter turns byte SEL into exact halves (code / 2, scaled by 2)
        const uint32_t e = pc.code[b] & 0x33333333u;
        const uint32_t o = (pc.code[b] >> 2) & 0x33333333u;
        qe[b] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(e, 2.0f, SEL);  // vectors 4SEL, 4SEL+2
        qo[b] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(o, 2.0f, SEL);  // vectors 4SEL+1, 4SEL+3
    }
    f16x8 out[2];
#pragma unroll
    for (int vi = 0; vi < 4; ++vi) {
        float q[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const f16x2 src = (vi & 1) ? qo[b] : qe[b];
            q[b] = static_cast<float>(vi < 2 ? src.x : src.y);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            float w = h2f(piece_bias(pc, a, j));
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                const uint32_t word = a < 2 ? pc.acol[b].x : pc.acol[b].y;
                w = __builtin_fmaf(h2f((a & 1) ? word >> 16 : word & 0xffffu), q[b], w);
            }
            out[vi >> 1][4 * (vi & 1) + a] = static_cast<_Float16>(w);
        }
    }
    *reinterpret_cast<f16x8*>(dst) = out[0];
    *reinterpret_cast<f16x8*>(dst + 8) = out[1];
}

// One 32-column step of the tile product: MI x kNI matrix-core tiles.
template <int MI>
__device__ inline void mma_step(const f16x8 (&xa)[MI], const _Float16* wsrc, f32x4 (&acc)[MI][kNI]) {
    f16x8 wb[kNI];
#pragma unroll
    for (int n = 0; n < kNI; ++n) wb[n] = *reinterpret_cast<const f16x8*>(wsrc + 16 * n * kLdsRow);
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int n = 0; n < kNI; ++n) acc[i][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[i], wb[n], acc[i][n], 0, 0, 0);
}

template <int MI>
__device__ inline void load_x(__amdgpu_buffer_rsrc_t rx, uint32_t off, uint32_t row_step, f16x8 (&xa)[MI]) {
#pragma unroll
    for (int i = 0; i < MI; ++i) {
        const uint4 v = ld128(rx, off + i * row_step);
        xa[i] = __builtin_bit_cast(f16x8, v);
    }
}

// One K step (group g): products of the four 32-column slices of buffer
// `cur`, with the next group's decode (if any) written to the other buffer.
template <int MI, int S>
__device__ inline void group_slice(__amdgpu_buffer_rsrc_t rx, uint32_t xoff, uint32_t row_step, uint32_t next_off,
                                   f16x8 (&xa)[MI], const _Float16* wsrc, bool decode_next, const Piece& nxt, int jn,
                                   _Float16* wdst, f32x4 (&acc)[MI][kNI]) {
    f16x8 xn[MI];
    load_x<MI>(rx, S < 3 ? xoff + 64 * (S + 1) : next_off, row_step, xn);  // prefetch the next slice
    mma_step<MI>(xa, wsrc + 32 * S, acc);
    if (decode_next) decode4<S>(nxt, jn, wdst + 16 * S);
#pragma unroll
    for (int i = 0; i < MI; ++i) xa[i] = xn[i];
}

template <int MI>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const uint8_t* __restrict__ packed,
                                                        const _Float16* __restrict__ x,
                                                        const float* __restrict__ inv_scale, void* y, int N,
                                                        int K, int M, int y_dtype, int m_tiles, int n_tiles) {
    __shared__ __attribute__((aligned(16))) _Float16 wsh[2 * kWBuf];
    constexpr int BM = kWaves * 16 * MI;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    // Tile of this workgroup.  Workgroups are dealt to the 8 XCDs round-robin;
    // renumbering them so that each XCD gets a contiguous run of tiles makes
    // the tiles that share activation rows share that XCD's L2.
    const int T = m_tiles * n_tiles;
    int L = blockIdx.x;
    if ((T & 7) == 0) L = (L & 7) * (T >> 3) + (L >> 3);
    const int mt = L / n_tiles, nt = L - mt * n_tiles;
    const int n0 = nt * kBN;
    const int tok0 = mt * BM + wave * 16 * MI;
    const int groups = K >> 7;

    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(M) * K * 2u);
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(packed, static_cast<uint32_t>(N / kRowBlock) * groups * kGroupBlockBytes);

    // Decode role: row rr of the tile, vectors 16*hv .. of each group.
    const int rr = threadIdx.x >> 1, hv = threadIdx.x & 1;
    const int r = n0 + rr;
    const uint32_t rowblk = r < N ? static_cast<uint32_t>(r >> 4) * groups * kGroupBlockBytes : kOutOfRange;
    const int beta = r & 15;
    _Float16* wdst = wsh + rr * kLdsRow + 64 * hv;

    // Activation operand of tile i, 32-column slice s of group g, lane
    // (m = lane % 16, kb = lane / 16): 8 halves of token tok0 + 16 i + m at
    // column 128 g + 32 s + 8 kb.  Tokens past M read zeros.
    const uint32_t row_step = 16u * K * 2u;
    const uint32_t xbase = (static_cast<uint32_t>(tok0 + (lane & 15)) * K + 8 * (lane >> 4)) * 2u;
    // Weight operand of tile n: row 16 n + lane % 16, same columns.
    const _Float16* wlane = wsh + (lane & 15) * kLdsRow + 8 * (lane >> 4);

    f32x4 acc[MI][kNI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int n = 0; n < kNI; ++n) acc[i][n] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Prologue: decode group 0 into buffer 0; packet data of group 1 in flight.
    Piece cur, nxt;
    load_piece(rw, rowblk, 0, groups, beta, hv, cur);
    load_piece(rw, rowblk, 1, groups, beta, hv, nxt);
    decode4<0>(cur, 0, wdst);
    decode4<1>(cur, 0, wdst + 16);
    decode4<2>(cur, 0, wdst + 32);
    decode4<3>(cur, 0, wdst + 48);
    f16x8 xa[MI];
    load_x<MI>(rx, xbase, row_step, xa);
    __syncthreads();

    for (int g = 0; g < groups; ++g) {
        const _Float16* wsrc = wlane + (g & 1) * kWBuf;
        _Float16* wnext = wdst + ((g + 1) & 1) * kWBuf;
        const bool decode_next = g + 1 < groups;
        // packet data two groups ahead
        Piece far;
        load_piece(rw, rowblk, g + 2, groups, beta, hv, far);
        const int jn = (g + 1) & 1;
        const uint32_t xoff = xbase + static_cast<uint32_t>(g) * 256u;
        const uint32_t next_off = decode_next ? xoff + 256u : kOutOfRange;
        group_slice<MI, 0>(rx, xoff, row_step, next_off, xa, wsrc, decode_next, nxt, jn, wnext, acc);
        group_slice<MI, 1>(rx, xoff, row_step, next_off, xa, wsrc, decode_next, nxt, jn, wnext, acc);
        group_slice<MI, 2>(rx, xoff, row_step, next_off, xa, wsrc, decode_next, nxt, jn, wnext, acc);
        group_slice<MI, 3>(rx, xoff, row_step, next_off, xa, wsrc, decode_next, nxt, jn, wnext, acc);
        nxt = far;
        __syncthreads();
    }

    // Epilogue.  D lane layout: output row 16 n + lane % 16, tokens
    // 16 i + 4 (lane / 16) + e.
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = tok0 + 16 * i + 4 * (lane >> 4) + e;
            if (t >= M) continue;
            const float sc = inv_scale ? inv_scale[t] : 1.0f;
#pragma unroll
            for (int n = 0; n < kNI; ++n) {
                const int row = n0 + 16 * n + (lane & 15);
                if (row < N) store_out(y, static_cast<int64_t>(t) * N + row, acc[i][n][e] * sc, y_dtype);
            }
        }
    }
}

// bf16 activations -> fp16 with a power-of-two scale per token (see the top
// of the file).  One workgroup per token row.
__global__ __launch_bounds__(256) void scale_rows_kernel(const uint16_t* __restrict__ xb, int K,
                                                         _Float16* __restrict__ xh, float* __restrict__ inv_scale) {
    __shared__ float wmax[4];
    const int t = blockIdx.x;
    const uint16_t* row = xb + static_cast<size_t>(t) * K;
    _Float16* out = xh + static_cast<size_t>(t) * K;
    const int chunks = K >> 3;  // 8 values per 16-byte chunk
    auto val = [](uint32_t bits16) { return __builtin_bit_cast(float, bits16 << 16); };
    float mx = 0.f;
    for (int c = threadIdx.x; c < chunks; c += 256) {
        const uint4 v = *reinterpret_cast<const uint4*>(row + 8 * c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            mx = fmaxf(mx, fabsf(val(w[h] & 0xffffu)));
            mx = fmaxf(mx, fabsf(val(w[h] >> 16)));
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = mx;
    __syncthreads();
    mx = fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]));
    int s = 0;
    if (mx > 0.f && mx <= 3.4e38f) {
        int e;
        frexpf(mx, &e);  // mx in [2^(e-1), 2^e)
        s = min(max(15 - e, -126), 126);
    }
    for (int c = threadIdx.x; c < chunks; c += 256) {
        const uint4 v = *reinterpret_cast<const uint4*>(row + 8 * c);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
        f16x8 o;
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            o[2 * h] = static_cast<_Float16>(ldexpf(val(w[h] & 0xffffu), s));
            o[2 * h + 1] = static_cast<_Float16>(ldexpf(val(w[h] >> 16), s));
        }
        *reinterpret_cast<f16x8*>(out + 8 * c) = o;
    }
    if (threadIdx.x == 0) inv_scale[t] = ldexpf(1.0f, -s);
}

template <int MI>
hipError_t launch_tiles(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const _Float16* x,
                        const float* inv_scale, void* y, int y_dtype, hipStream_t s) {
    constexpr int BM = kWaves * 16 * MI;
    const int m_tiles = static_cast<int>((M + BM - 1) / BM);
    const int n_tiles = static_cast<int>((N + kBN - 1) / kBN);
    hipLaunchKernelGGL(gemm_kernel<MI>, dim3(static_cast<unsigned>(m_tiles) * n_tiles), dim3(kThreads), 0, s,
                       packed, x, inv_scale, y, static_cast<int>(N), static_cast<int>(K), static_cast<int>(M),
                       y_dtype, m_tiles, n_tiles);
    return hipGetLastError();
}

}  // namespace

size_t gemm_workspace_bytes(int64_t K, int64_t M) {
    const size_t xh = (static_cast<size_t>(M) * K * 2 + 255) & ~size_t{255};
    return xh + static_cast<size_t>(M) * 4;
}

int launch_gemm(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, void* workspace, hipStream_t s) {
    const _Float16* xh = static_cast<const _Float16*>(x);
    const float* inv = nullptr;
    if (x_dtype == UNISVQ_BF16) {
        _Float16* wxh = static_cast<_Float16*>(workspace);
        float* winv = reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                               ((static_cast<size_t>(M) * K * 2 + 255) & ~size_t{255}));
        hipLaunchKernelGGL(scale_rows_kernel, dim3(static_cast<unsigned>(M)), dim3(256), 0, s,
                           static_cast<const uint16_t*>(x), static_cast<int>(K), wxh, winv);
        if (hipGetLastError() != hipSuccess) return UNISVQ_EHIP;
        xh = wxh;
        inv = winv;
    }
    // The activation buffer is addressed with 32-bit offsets: slice M.
    const int64_t max_rows = kMaxBufferBytes / (2 * K) / 256 * 256;
    for (int64_t m0 = 0; m0 < M; m0 += max_rows) {
        const int64_t mc = M - m0 < max_rows ? M - m0 : max_rows;
        const _Float16* xs = xh + m0 * K;
        const float* is = inv ? inv + m0 : nullptr;
        void* ys = static_cast<uint8_t*>(y) + m0 * N * (y_dtype == UNISVQ_F32 ? 4 : 2);
        const hipError_t e = mc > 128 ? launch_tiles<4>(N, K, packed, mc, xs, is, ys, y_dtype, s)
                                      : launch_tiles<1>(N, K, packed, mc, xs, is, ys, y_dtype, s);
        if (e != hipSuccess) return UNISVQ_EHIP;
    }
    return UNISVQ_OK;
}

}  // namespace unisvq
