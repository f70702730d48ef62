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

// load_packet without branches: both shapes issue the same three loads, so
// the compiler's wait counts for the code that follows stay exact.  A half
// packet's 8-byte slots are read 16 bytes at a time and the upper halves
// dropped; its 2-byte B values come from the aligned word that holds them.
// (The tiled GEMM keeps the branching form: this one costs it registers.)
template <bool STREAM = false>
__device__ inline void load_packet_flat(__amdgpu_buffer_rsrc_t rw, uint32_t rowblk, int p, int gend, int lane,
                                   Piece& pc) {
    const bool full = 2 * p + 1 < gend;
    const bool half = 2 * p + 1 == gend;
    const uint32_t P = full || half ? rowblk + static_cast<uint32_t>(p) * kPacketBytes : kOutOfRange;
    const uint32_t slot = (half ? 8u : 16u) * static_cast<uint32_t>(lane);
    const uint32_t aoff = P + (half ? kHalfAffineOff : kPacketAffineOff) + slot;
    const uint32_t boff = P + (half ? kHalfBiasOff + 4 * (lane >> 1) : kPacketBiasOff + 4 * lane);
    const uint4 c = STREAM ? ld128_stream(rw, P + slot) : ld128(rw, P + slot);
    const uint4 a = STREAM ? ld128_stream(rw, aoff) : ld128(rw, aoff);
    const uint32_t b = STREAM ? ld32_stream(rw, boff) : ld32(rw, boff);
    pc.c = half ? uint4{c.x, c.y, 0u, 0u} : c;
    pc.a = half ? uint4{a.x, a.y, 0u, 0u} : a;
    pc.b = half ? (lane & 1 ? b >> 16 : b & 0xffffu) : b;
}

// load_packet_shared without branches (same three loads for both shapes).
template <bool STREAM = false>
__device__ inline void load_packet_shared_flat(__amdgpu_buffer_rsrc_t rc, __amdgpu_buffer_rsrc_t ra, uint32_t rowblk,
                                          int p, int gend, int affine_one, int lane, Piece& pc) {
    const bool full = 2 * p + 1 < gend;
    const bool half = 2 * p + 1 == gend;
    const uint32_t P = full || half ? rowblk + static_cast<uint32_t>(p) * kCodePacketBytes : kOutOfRange;
    const uint32_t R = full || half ? static_cast<uint32_t>(affine_one ? 0 : p) * kAffineRecordBytes : kOutOfRange;
    const int j = lane & 3;
    const uint32_t slot = (half ? 8u : 16u) * static_cast<uint32_t>(lane);
    const uint4 c = STREAM ? ld128_stream(rc, P + slot) : ld128(rc, P + slot);
    const uint4 a = ld128(ra, R + 16 * j);
    const uint32_t b = ld32(ra, R + kRecordBiasOff + 4 * j);
    pc.c = half ? uint4{c.x, c.y, 0u, 0u} : c;
    pc.a = half ? uint4{a.x, a.y, 0u, 0u} : a;
    pc.b = half ? b & 0xffffu : b;
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

// Lane permutation within each quad (DPP quad_perm): dest lane i reads lane
// ((CTRL >> 2i) & 3).
template <int CTRL>
__device__ inline uint32_t quad_perm(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), CTRL, 0xf, 0xf, false));
}

// Gather, for group 2p + jj, the codes of vectors 4n+j, row j of A and all
// of B from the four slots of the quad.
//   Codes: lane b's word holds component b's 2-bit codes, field k of each
//   byte for vector 4(byte) + k; lane j needs field j of every lane's word,
//   as nibbles for the e2m1 converter: component 0 in the low nibble, 1 in
//   the high one (p01), likewise 2 and 3 (p23).  The high nibble comes from a
//   rotation of the other word by 2j - 4, which lands field j at bits 4-5 of
//   each byte (bits that wrap around fall outside the mask).
//   A: lane b holds column b (rows 0, 1 in word al, rows 2, 3 in ah); lane j
//   needs row j.  A 4 x 4 transpose of 16-bit elements in two butterfly
//   stages: the word pair across lanes j ^ 2, then the halves across j ^ 1.
//   B: the word holds B[b] of both groups; each lane needs all four.
// CODES_ONLY (the Eq. 9 fold, where A and B act on the activations): the
// codes alone.
template <bool CODES_ONLY = false>
__device__ inline void prepare(const Piece& pc, int j, int jj, DecOps& d) {
    const uint32_t cl = jj ? pc.c.z : pc.c.x, ch = jj ? pc.c.w : pc.c.y;
    const uint32_t al = jj ? pc.a.z : pc.a.x, ah = jj ? pc.a.w : pc.a.y;
    const uint32_t cw[2][4] = {{quad_lane<0>(cl), quad_lane<1>(cl), quad_lane<2>(cl), quad_lane<3>(cl)},
                               {quad_lane<0>(ch), quad_lane<1>(ch), quad_lane<2>(ch), quad_lane<3>(ch)}};
    const int sh = 2 * j;
    const int rot = (sh - 4) & 31;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        d.p01[h] = ((cw[h][0] >> sh) & 0x03030303u) | (__builtin_amdgcn_alignbit(cw[h][1], cw[h][1], rot) & 0x30303030u);
        d.p23[h] = ((cw[h][2] >> sh) & 0x03030303u) | (__builtin_amdgcn_alignbit(cw[h][3], cw[h][3], rot) & 0x30303030u);
    }
    if constexpr (CODES_ONLY) return;
    const bool low = j < 2, odd = (j & 1) != 0;
    // stage 1: lanes j < 2 keep rows 0, 1 of column j and receive those of
    // column j + 2; lanes j >= 2 keep rows 2, 3 of column j, receive column j - 2
    const uint32_t recv = quad_perm<0x4e>(low ? ah : al);  // [2, 3, 0, 1]
    const uint32_t lowc = low ? al : recv;                 // column j & 1
    const uint32_t highc = low ? recv : ah;                // column (j & 1) + 2
    // stage 2: even lanes send their odd rows' halves, odd lanes their even
    // rows'; each keeps its own row's halves
    const uint32_t send2 = __builtin_amdgcn_perm(highc, lowc, odd ? 0x05040100u : 0x07060302u);
    const uint32_t recv2 = quad_perm<0xb1>(send2);  // [1, 0, 3, 2]
    const uint32_t a01 = __builtin_amdgcn_perm(recv2, lowc, odd ? 0x03020504u : 0x05040100u);
    const uint32_t a23 = __builtin_amdgcn_perm(recv2, highc, odd ? 0x03020706u : 0x07060100u);
    d.arow = __builtin_bit_cast(f16x4, uint2{a01, a23});
    // B of both groups per lane (the same four moves for either group)
    const uint32_t bw[4] = {quad_lane<0>(pc.b), quad_lane<1>(pc.b), quad_lane<2>(pc.b), quad_lane<3>(pc.b)};
#pragma unroll
    for (int b = 0; b < 4; ++b) d.bvec[b] = h2f(jj ? bw[b] >> 16 : bw[b] & 0xffffu);
}

// Vectors 4N .. 4N+3 of the row block: one matrix-core instruction; lane
// (beta, j) stores vector 4N+j at dst + 16N + 4j (dst = the lane's row).
// CODES_ONLY: the four codes themselves (exact small integers in fp16) are
// stored as the vector's weights.
template <int N, bool CODES_ONLY = false>
__device__ inline void decode_vecs(const DecOps& d, _Float16* dst, int j) {
    const f16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(d.p01[N >> 2], 2.0f, N & 3);
    const f16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(d.p23[N >> 2], 2.0f, N & 3);
    const f16x4 q = __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
    if constexpr (CODES_ONLY) {
        *reinterpret_cast<f16x4*>(dst + 16 * N + 4 * j) = q;
        return;
    }
    const f32x4 w = __builtin_amdgcn_mfma_f32_4x4x4f16(d.arow, q, d.bvec, 0, 0, 0);
    f16x4 o;
#pragma unroll
    for (int a = 0; a < 4; ++a) o[a] = static_cast<_Float16>(w[a]);
    *reinterpret_cast<f16x4*>(dst + 16 * N + 4 * j) = o;
}

}  // namespace
}  // namespace unisvq

namespace unisvq {
namespace {

// ---------------------------------------------------------------------------
// Weight decode for the format variants: b-bit codes (b = 2, 3; Sec. 5.2.5)
// and d-dimensional vectors (d = 4, 8; Sec. 5.2.3), codes-only with row-shared
// pairs.  Codes are gathered from the quad exactly as above (for d = 8 code
// word h of a slot holds component 4h + j, so byte n of the gathered word h
// holds vector 4n + j, components 4h .. 4h+3); the high bits of 3-bit codes
// are gathered the same way from the high field, whose layout puts the bit
// of (word h, vector index 4n + j) at 8n + 4(j >> 1) + 2h + (j & 1).  A and B
// come from the row view of the group's shared record.
//   d = 4: one v_mfma_f32_4x4x4_16b per 4 vectors, as above;
//   d = 8: per 4 vectors and half ah of the output components, two chained
//          instructions (code components 0..3, then 4..7):
//          D[a][v] = sum_b A[4 ah + a][b] q[v][b] + B[4 ah + a];
//   b = 3: q = lo + 4 hi, so each instruction is followed by one with the high
//          bits (the e2m1 converter with scale 8 gives 0 or 4) into the same
//          accumulator.
// All products are exact in fp32; the weight is rounded once to fp16.

// Low and high fields of one slot of a variant packet.
struct VarPiece {
    uint4 c;  // low fields: .x/.y group 2p, .z/.w group 2p+1
    uint2 h;  // high fields (b = 3): .x group 2p, .y group 2p+1
};

template <int BITS>
__device__ inline void load_packet_var(__amdgpu_buffer_rsrc_t rc, uint32_t rowblk, int p, int gend, int lane,
                                       VarPiece& pc) {
    const bool full = 2 * p + 1 < gend;
    const bool half = 2 * p + 1 == gend;
    const uint32_t P =
        full || half ? rowblk + static_cast<uint32_t>(p) * 2u * var_group_bytes(BITS) : kOutOfRange;
    if (half) {
        const uint2 c = ld64(rc, P + 8 * lane);
        pc.c = uint4{c.x, c.y, 0u, 0u};
        pc.h = uint2{BITS == 3 ? ld32(rc, P + kVarHalfHiOff + 4 * lane) : 0u, 0u};
    } else {
        pc.c = ld128(rc, P + 16 * lane);
        pc.h = BITS == 3 ? ld64(rc, P + kVarHiOff + 8 * lane) : uint2{0u, 0u};
    }
}

// A rows and B of one group, from the row view of its record.
template <int D>
struct VarAffine {
    f16x4 arow[D / 4][D / 4];  // [ah][kb] = A[4 ah + j][4 kb .. 4 kb + 3]
    f32x4 bvec[D / 4];         // [ah] = B[4 ah .. 4 ah + 3]
};

// Group gd of the product: record (one pair: 0; else gd / 2), its group gd % 2.
template <int D>
__device__ inline void load_var_affine(__amdgpu_buffer_rsrc_t ra, int affine_one, int gd, int j, VarAffine<D>& af) {
    const uint32_t base = static_cast<uint32_t>(affine_one ? 0 : gd >> 1) * var_record_bytes(D) +
                          var_row_view_off(D) + static_cast<uint32_t>(gd & 1) * var_row_view_group_bytes(D);
#pragma unroll
    for (int ah = 0; ah < D / 4; ++ah) {
#pragma unroll
        for (int kb = 0; kb < D / 4; ++kb)
            af.arow[ah][kb] = __builtin_bit_cast(f16x4, ld64(ra, base + 2u * (D * (4 * ah + j) + 4 * kb)));
        const uint2 bv = ld64(ra, base + 2u * D * D + 8u * ah);
        af.bvec[ah] = f32x4{h2f(bv.x & 0xffffu), h2f(bv.x >> 16), h2f(bv.y & 0xffffu), h2f(bv.y >> 16)};
    }
}

template <int BITS>
struct VarDecOps {
    uint32_t p01[2], p23[2];  // low bits: byte n of word h, nibbles of components (0, 1) / (2, 3) of the word's four
    uint32_t h01[2], h23[2];  // high bits, same places (b = 3)
};

template <int BITS>
__device__ inline void prepare_var(const VarPiece& pc, int j, int jj, VarDecOps<BITS>& d) {
    const uint32_t cl = jj ? pc.c.z : pc.c.x, ch = jj ? pc.c.w : pc.c.y;
    const uint32_t cw[2][4] = {{quad_lane<0>(cl), quad_lane<1>(cl), quad_lane<2>(cl), quad_lane<3>(cl)},
                               {quad_lane<0>(ch), quad_lane<1>(ch), quad_lane<2>(ch), quad_lane<3>(ch)}};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        uint32_t m[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) m[b] = (cw[h][b] >> (2 * j)) & 0x03030303u;
        d.p01[h] = m[0] | (m[1] << 4);
        d.p23[h] = m[2] | (m[3] << 4);
    }
    if constexpr (BITS == 3) {
        const uint32_t H = jj ? pc.h.y : pc.h.x;
        const uint32_t hw[4] = {quad_lane<0>(H), quad_lane<1>(H), quad_lane<2>(H), quad_lane<3>(H)};
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int sh = 4 * (j >> 1) + (j & 1) + 2 * h;
            uint32_t m[4];
#pragma unroll
            for (int b = 0; b < 4; ++b) m[b] = (hw[b] >> sh) & 0x01010101u;
            d.h01[h] = m[0] | (m[1] << 4);
            d.h23[h] = m[2] | (m[3] << 4);
        }
    }
}

// Codes of word h, byte n as an operand (low part, or the high part times 4).
template <int H, int NB>
__device__ inline f16x4 var_codes(const uint32_t (&p01)[2], const uint32_t (&p23)[2], float scale) {
    const f16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(p01[H], scale, NB);
    const f16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(p23[H], scale, NB);
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3);
}

__device__ inline void store_w4(const f32x4& w, _Float16* dst) {
    f16x4 o;
#pragma unroll
    for (int a = 0; a < 4; ++a) o[a] = static_cast<_Float16>(w[a]);
    *reinterpret_cast<f16x4*>(dst) = o;
}

// d = 4: vectors 4N .. 4N+3; lane (beta, j) stores vector 4N+j at dst + 16N + 4j.
template <int BITS, int N>
__device__ inline void decode_var4(const VarDecOps<BITS>& d, const VarAffine<4>& af, _Float16* dst, int j) {
    f32x4 w = __builtin_amdgcn_mfma_f32_4x4x4f16(af.arow[0][0], var_codes<N / 4, N % 4>(d.p01, d.p23, 2.0f),
                                                 af.bvec[0], 0, 0, 0);
    if constexpr (BITS == 3)
        w = __builtin_amdgcn_mfma_f32_4x4x4f16(af.arow[0][0], var_codes<N / 4, N % 4>(d.h01, d.h23, 8.0f), w, 0, 0,
                                               0);
    store_w4(w, dst + 16 * N + 4 * j);
}

// d = 8: vectors 4n .. 4n+3, output components 4 AH .. 4 AH + 3; lane
// (beta, j) stores them at dst + 8 (4n + j) + 4 AH.
template <int BITS, int NV, int AH>
__device__ inline void decode_var8(const VarDecOps<BITS>& d, const VarAffine<8>& af, _Float16* dst, int j) {
    f32x4 w = __builtin_amdgcn_mfma_f32_4x4x4f16(af.arow[AH][0], var_codes<0, NV>(d.p01, d.p23, 2.0f), af.bvec[AH],
                                                 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_4x4x4f16(af.arow[AH][1], var_codes<1, NV>(d.p01, d.p23, 2.0f), w, 0, 0, 0);
    if constexpr (BITS == 3) {
        w = __builtin_amdgcn_mfma_f32_4x4x4f16(af.arow[AH][0], var_codes<0, NV>(d.h01, d.h23, 8.0f), w, 0, 0, 0);
        w = __builtin_amdgcn_mfma_f32_4x4x4f16(af.arow[AH][1], var_codes<1, NV>(d.h01, d.h23, 8.0f), w, 0, 0, 0);
    }
    store_w4(w, dst + 8 * (4 * NV + j) + 4 * AH);
}

// Half S (0: first half of the vectors, 1: second) of one row block's group.
template <int BITS, int D, int S>
__device__ inline void decode_var_half(const VarDecOps<BITS>& d, const VarAffine<D>& af, _Float16* dst, int j) {
    if constexpr (D == 4) {
        decode_var4<BITS, 4 * S + 0>(d, af, dst, j);
        decode_var4<BITS, 4 * S + 1>(d, af, dst, j);
        decode_var4<BITS, 4 * S + 2>(d, af, dst, j);
        decode_var4<BITS, 4 * S + 3>(d, af, dst, j);
    } else {
        decode_var8<BITS, 2 * S, 0>(d, af, dst, j);
        decode_var8<BITS, 2 * S, 1>(d, af, dst, j);
        decode_var8<BITS, 2 * S + 1, 0>(d, af, dst, j);
        decode_var8<BITS, 2 * S + 1, 1>(d, af, dst, j);
    }
}

}  // namespace
}  // namespace unisvq
