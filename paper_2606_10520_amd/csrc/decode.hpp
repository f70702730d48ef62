// Matrix-core weight decode shared by the prefill GEMM and the small-batch
// kernel (gfx950 only).  Internal header; see common.hpp for the format.
#pragma once

#include "common.hpp"

namespace unisvq {
namespace {

__device__ inline float h2f(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

// ---------------------------------------------------------------------------
// Weight decode on the matrix cores.  For one 16-row block and one group,
// v_mfma_f32_4x4x4_16b computes, per row (one of the 16 blocks) and per
// 4 consecutive vectors v = 4n .. 4n+3:
//     D[a][v] = sum_b A[a][b] q[v][b] + B[a]          (Eq. 4)
// with SrcA lane (row, i) = row i of A, SrcB lane (row, j) = the four codes
// of vector 4n+j, C = B; the products of fp16 parameters and exact integer
// codes are exact in fp32.  D lane (row, j) then holds the four weights of
// vector 4n+j -- four consecutive columns -- which go to LDS as fp16 (one
// rounding).  Eight instructions decode a 16 x 128 tile.

// Packet data of one row block for lane (beta, j) = packet slot 4 beta + j:
// exactly what the slot holds, so the loads are fully coalesced.  A full
// packet covers two groups (jj = 0, 1); a trailing half packet one (jj = 0).
struct Piece {
    uint4 c;      // F(r, 2p + jj, j): .x/.y for jj = 0, .z/.w for jj = 1
    uint4 a;      // A[r][2p + jj][0..3][j]: .x/.y for jj = 0, .z/.w for jj = 1
    uint32_t b;   // B[r][2p + jj][j]: low half jj = 0, high half jj = 1
};

// Packet p of a row block: full, half (the last group of an odd count), or
// nothing at or past group `gend` (the end of the range being decoded; a
// range ends at a packet boundary or at the last group).  STREAM selects the
// non-temporal loads for weights read exactly once.
template <bool STREAM = false>
__device__ inline void load_packet(__amdgpu_buffer_rsrc_t rw, uint32_t rowblk, int p, int gend, int lane,
                                   Piece& pc) {
    const bool full = 2 * p + 1 < gend;
    const bool half = 2 * p + 1 == gend;
    const uint32_t P = full || half ? rowblk + static_cast<uint32_t>(p) * kPacketBytes : kOutOfRange;
    if (half) {
        const uint2 c = STREAM ? ld64_stream(rw, P + 8 * lane) : ld64(rw, P + 8 * lane);
        const uint2 a = STREAM ? ld64_stream(rw, P + kHalfAffineOff + 8 * lane) : ld64(rw, P + kHalfAffineOff + 8 * lane);
        pc.c = uint4{c.x, c.y, 0u, 0u};
        pc.a = uint4{a.x, a.y, 0u, 0u};
        pc.b = STREAM ? ld16_stream(rw, P + kHalfBiasOff + 2 * lane) : ld16(rw, P + kHalfBiasOff + 2 * lane);
    } else {
        pc.c = STREAM ? ld128_stream(rw, P + 16 * lane) : ld128(rw, P + 16 * lane);
        pc.a = STREAM ? ld128_stream(rw, P + kPacketAffineOff + 16 * lane) : ld128(rw, P + kPacketAffineOff + 16 * lane);
        pc.b = STREAM ? ld32_stream(rw, P + kPacketBiasOff + 4 * lane) : ld32(rw, P + kPacketBiasOff + 4 * lane);
    }
}

// The same piece from codes-only bytes (row block at `rowblk`, 512 bytes
// per group) and the shared affine block: lane (beta, j) takes its A column
// and B values from record p (record 0 for a single pair).  A half packet
// keeps only its group's parameters.
template <bool STREAM = false>
__device__ inline void load_packet_shared(__amdgpu_buffer_rsrc_t rc, __amdgpu_buffer_rsrc_t ra, uint32_t rowblk,
                                          int p, int gend, int affine_one, int lane, Piece& pc) {
    const bool full = 2 * p + 1 < gend;
    const bool half = 2 * p + 1 == gend;
    const uint32_t P = full || half ? rowblk + static_cast<uint32_t>(p) * kCodePacketBytes : kOutOfRange;
    const uint32_t R = full || half ? static_cast<uint32_t>(affine_one ? 0 : p) * kAffineRecordBytes : kOutOfRange;
    const int j = lane & 3;
    if (half) {
        const uint2 c = STREAM ? ld64_stream(rc, P + 8 * lane) : ld64(rc, P + 8 * lane);
        const uint2 a = ld64(ra, R + 16 * j);
        pc.c = uint4{c.x, c.y, 0u, 0u};
        pc.a = uint4{a.x, a.y, 0u, 0u};
        pc.b = ld16(ra, R + kRecordBiasOff + 4 * j);
    } else {
        pc.c = STREAM ? ld128_stream(rc, P + 16 * lane) : ld128(rc, P + 16 * lane);
        pc.a = ld128(ra, R + 16 * j);
        pc.b = ld32(ra, R + kRecordBiasOff + 4 * j);
    }
}

// Value of lane b of this lane's quad.
template <int B>
__device__ inline uint32_t quad_lane(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), B * 0x55, 0xf, 0xf, false));
}

// Decode operands prepared from a piece.
struct DecOps {
    uint32_t p01[2], p23[2];  // byte n of word h: nibbles (q_0, q_1) / (q_2, q_3) of vector 4(4h+n)+j
    f16x4 arow;               // A[j][0..3]
    f32x4 bvec;               // B[0..3]
};

// Gather, for group 2p + jj, the codes of vectors 4n+j, row j of A and all
// of B from the four slots of the quad.
__device__ inline void prepare(const Piece& pc, int j, int jj, DecOps& d) {
    const uint32_t cl = jj ? pc.c.z : pc.c.x, ch = jj ? pc.c.w : pc.c.y;
    const uint32_t al = jj ? pc.a.z : pc.a.x, ah = jj ? pc.a.w : pc.a.y;
    const uint32_t bv = jj ? pc.b >> 16 : pc.b & 0xffffu;
    const uint32_t cw[2][4] = {{quad_lane<0>(cl), quad_lane<1>(cl), quad_lane<2>(cl), quad_lane<3>(cl)},
                               {quad_lane<0>(ch), quad_lane<1>(ch), quad_lane<2>(ch), quad_lane<3>(ch)}};
    const int sh = 2 * j;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        uint32_t m[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) m[b] = (cw[h][b] >> sh) & 0x03030303u;
        d.p01[h] = m[0] | (m[1] << 4);
        d.p23[h] = m[2] | (m[3] << 4);
    }
    // row j of A: half (j & 1) of word (j >> 1) of every column b
    const uint32_t lo[4] = {quad_lane<0>(al), quad_lane<1>(al), quad_lane<2>(al), quad_lane<3>(al)};
    const uint32_t hi[4] = {quad_lane<0>(ah), quad_lane<1>(ah), quad_lane<2>(ah), quad_lane<3>(ah)};
    uint32_t w[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) w[b] = j < 2 ? lo[b] : hi[b];
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
    const uint32_t a01 = __builtin_amdgcn_perm(w[1], w[0], sel);
    const uint32_t a23 = __builtin_amdgcn_perm(w[3], w[2], sel);
    d.arow = __builtin_bit_cast(f16x4, uint2{a01, a23});
    d.bvec[0] = h2f(quad_lane<0>(bv));
    d.bvec[1] = h2f(quad_lane<1>(bv));
    d.bvec[2] = h2f(quad_lane<2>(bv));
    d.bvec[3] = h2f(quad_lane<3>(bv));
}

// Vectors 4N .. 4N+3 of the row block: one matrix-core instruction; lane
// (beta, j) stores vector 4N+j at dst + 16N + 4j (dst = the lane's row).
template <int N>
__device__ inline void decode_vecs(const DecOps& d, _Float16* dst, int j) {
    const f16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(d.p01[N >> 2], 2.0f, N & 3);
    const f16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(d.p23[N >> 2], 2.0f, N & 3);
    const f16x4 q = __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
    const f32x4 w = __builtin_amdgcn_mfma_f32_4x4x4f16(d.arow, q, d.bvec, 0, 0, 0);
    f16x4 o;
#pragma unroll
    for (int a = 0; a < 4; ++a) o[a] = static_cast<_Float16>(w[a]);
    *reinterpret_cast<f16x4*>(dst + 16 * N + 4 * j) = o;
}

}  // namespace
}  // namespace unisvq
