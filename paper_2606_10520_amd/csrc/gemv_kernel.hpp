// Decode-phase product y = x * W_hat^T for M <= 4 tokens on gfx950: the
// kernel template and its launch helper (internal header, included by
// gemv.hip and gemv_var.hip).
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
//   SrcA = activations x[v][a] -- identical for all 16 blocks, so one block's
//   lanes supply it and the broadcast (CBSZ = 4) hands it to every block;
//   ABID picks the supplying block.  All 16 instructions of a packet (two
//   groups x 8 steps) therefore take their activation operands from ONE
//   register pair: lane 4*(8 gi + s) + a holds component a of the four
//   vectors of step s of group gi, and instruction (gi, s) uses ABID 8 gi + s.
//   SrcB = codes q[v][b]: lane s of a packet slot already holds component b of
//   all 32 vectors of its row (packed format v1), converted to exact small
//   integers with the fp4 (e2m1) converter: a 2-bit code c in the low bits of
//   a nibble is the e2m1 value c/2, scaled by 2.
//   D lane (beta, b) holds T[a = 0..3][b]; it needs A[r][g][0..3][b] and
//   B[r][g][b], which is exactly that lane's affine slot.
// The dequantised weights never leave registers (they are never formed).
//
// Schedule.  One workgroup per 16-row block of one problem (several
// independent problems may share a launch); its WAVES wavefronts split the
// block's packets along K into contiguous runs.  Each wavefront first loads
// its activations (8 bytes per lane per packet and token: four consecutive
// vectors per quad), then issues its packet loads, and while those are in
// flight turns the activations into operand order with a 4x4 transpose
// inside each quad (DPP), forms the per-group sums xbar with DPP row sums,
// and parks both in LDS (one 8-byte write per lane per packet).  The main
// loop consumes packets as they arrive (PF loads in flight per wavefront),
// one 8-byte LDS read of activations per packet and token, four independent
// matrix-core chains per packet.  Partial row sums meet in LDS at the end.
#pragma once

#include "common.hpp"
#include "fwht.hpp"

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
    // a lone nibble bit 0 (e2m1 0.5) becomes 4: the high bit of a 3-bit code
    template <int SEL>
    __device__ static inline f16x2 cvt2x8(uint32_t w) {
        return __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w, 8.0f, SEL);
    }
    template <int ABID>
    __device__ static inline f32x4 mfma(vec4 a, vec4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_4x4x4f16(a, b, c, 4, ABID, 0);
    }
    // sum of the four activations of one operand lane, in fp32
    __device__ static inline float sum4(uint2 w) {
        const f16x2 one = {static_cast<_Float16>(1.0f), static_cast<_Float16>(1.0f)};
        const float s = __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, w.x), one, 0.0f, false);
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, w.y), one, s, false);
    }
};

template <>
struct XOps<__bf16> {
    typedef bf16x4 vec4;
    template <int SEL>
    __device__ static inline bf16x2 cvt2(uint32_t w) {
        return __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 2.0f, SEL);
    }
    template <int SEL>
    __device__ static inline bf16x2 cvt2x8(uint32_t w) {
        return __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, 8.0f, SEL);
    }
    template <int ABID>
    __device__ static inline f32x4 mfma(vec4 a, vec4 b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(a, b, c, 4, ABID, 0);
    }
    // sum of the four activations of one operand lane, in fp32 (a bf16 value
    // is the upper half of its fp32 value)
    __device__ static inline float sum4(uint2 w) {
        return (__builtin_bit_cast(float, w.x << 16) + __builtin_bit_cast(float, w.x & 0xffff0000u)) +
               (__builtin_bit_cast(float, w.y << 16) + __builtin_bit_cast(float, w.y & 0xffff0000u));
    }
};

// 16 codes of one 32-bit word (vectors 16h .. 16h+15 of one component) ->
// four SrcB operands.  Operand n holds vectors 4n+0, 4n+2, 4n+1, 4n+3 (the
// nibble order the e2m1 converter produces); the activation operand uses the
// same slot order.
template <typename XT, int SEL>
__device__ inline typename XOps<XT>::vec4 code_operand(uint32_t e, uint32_t o) {
    auto lo = XOps<XT>::template cvt2<SEL>(e);
    auto hi = XOps<XT>::template cvt2<SEL>(o);
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

__device__ inline float h2f(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

template <int CTRL>
__device__ inline float dpp(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 0xf, 0xf, true));
}

// Sum over the 4 lanes of a quad, result in every lane of the quad.
__device__ inline float quad_sum(float v) {
    v += dpp<0xB1>(v);  // quad_perm [1,0,3,2]
    v += dpp<0x4E>(v);  // quad_perm [2,3,0,1]
    return v;
}

template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_mov_dpp(static_cast<int>(v), CTRL, 0xf, 0xf, false));
}

// 4 x 4 transpose of 16-bit elements inside each quad: lane i holds row i
// (elements 0, 1 in w.x, 2, 3 in w.y); afterwards lane a holds column a
// (rows 0, 1 in .x, rows 2, 3 in .y).  Two steps: swap the off-diagonal
// 2 x 2 blocks between lanes i and i ^ 2, then transpose each 2 x 2 block
// between lanes i and i ^ 1.
__device__ inline uint2 quad_transpose16(uint2 w, int i) {
    const bool upper = (i & 2) == 0;
    const uint32_t t = dpp_u32<0x4E>(upper ? w.y : w.x);  // quad_perm [2,3,0,1]
    const uint32_t f0 = upper ? w.x : t;
    const uint32_t f1 = upper ? t : w.y;
    const uint32_t u0 = dpp_u32<0xB1>(f0);  // quad_perm [1,0,3,2]
    const uint32_t u1 = dpp_u32<0xB1>(f1);
    // even lane: (own low half, partner's low half); odd lane: (partner's
    // high half, own high half)
    const uint32_t sel = (i & 1) ? 0x03020706u : 0x05040100u;
    return uint2{__builtin_amdgcn_perm(u0, f0, sel), __builtin_amdgcn_perm(u1, f1, sel)};
}

// Lane l of a wavefront loads the 4 activations of vector swz(l) of a packet
// (swz swaps the two low bits: the e2m1 converter delivers a word's codes in
// the vector order 0, 2, 1, 3 of each step).
__device__ inline uint32_t operand_vector(int lane) {
    return static_cast<uint32_t>((lane & ~3) | ((lane & 1) << 1) | ((lane >> 1) & 1));
}

// The four activations lane l loads, in units of 4 elements within a packet:
// d = 4, vector operand_vector(l); d = 8, half ia of vector 16 gi + 4 s +
// swz(l % 4), where block l / 4 = 8 gi + 4 ia + s.
template <int D>
__device__ inline uint32_t operand_unit(int lane) {
    if constexpr (D == 4) {
        return operand_vector(lane);
    } else {
        const int q = lane >> 2;
        const int gi = q >> 3, ia = (q >> 2) & 1, st = q & 3;
        const int v = 16 * gi + 4 * st + ((lane & 1) << 1) + ((lane >> 1) & 1);
        return static_cast<uint32_t>(2 * v + ia);
    }
}

}  // namespace

struct GemvBatch {
    GemvProblem p[kMaxBatch];
    int count;
    int M;
    int y_dtype;
    // fused input transform (RHT launches only): the signs S_V of each
    // problem and 1/sqrt(K)
    const signed char* signs[kMaxBatch];
    float rht_norm;
};

namespace {

// Activation operands of one (token, packet) in LDS: 64 lanes x 8 bytes, in
// the operand order of the broadcast A operand.  The per-group sums xbar are
// kept as the four DPP row sums of the packet, [component][row]: rows 0, 1
// belong to group 2P, rows 2, 3 to group 2P + 1.
constexpr int kXsPacketBytes = 64 * 8;
constexpr int kXbarPacketBytes = 16 * 4;

// One loaded activation word (lane's vector of packet P, token t) -> operand
// order in LDS, plus the per-group sums.  Packet-major layout: entry
// P * MT + t, so a packet's tokens sit at constant offsets from each other.
template <typename XT, int MT>
__device__ inline void stage_packet(uint2 raw, int t, int P, int lane, uint2* xs, float* xbar) {
    const uint2 op = quad_transpose16(raw, lane & 3);
    const size_t tp = static_cast<size_t>(P) * MT + t;
    xs[tp * 64 + lane] = op;
    // lane 4*(8 gi + s) + a holds component a of the 4 vectors of step s;
    // the 4 steps of one DPP row sum up in its lanes 12..15
    float v = XOps<XT>::sum4(op);
    v += dpp<0x114>(v);  // row_shr:4
    v += dpp<0x118>(v);  // row_shr:8
    if ((lane & 15) >= 12) xbar[tp * 16 + (lane & 3) * 4 + (lane >> 4)] = v;
}

template <typename XT>
__device__ inline void epilogue(const f32x4& d, uint32_t a01, uint32_t a23, uint32_t bbits, float xb,
                                float& acc) {
    float r = acc;
    r = __builtin_fmaf(h2f(a01 & 0xffffu), d[0], r);
    r = __builtin_fmaf(h2f(a01 >> 16), d[1], r);
    r = __builtin_fmaf(h2f(a23 & 0xffffu), d[2], r);
    r = __builtin_fmaf(h2f(a23 >> 16), d[3], r);
    acc = __builtin_fmaf(h2f(bbits), xb, r);
}

// Step S of both groups of a packet: two independent chains (one per
// group; a dependent matrix-core instruction takes its accumulator straight
// from the previous one).
template <typename XT, int S>
__device__ inline void chain_step(typename XOps<XT>::vec4 xo, const typename XOps<XT>::vec4 (&c0)[8],
                                  const typename XOps<XT>::vec4 (&c1)[8], f32x4& d0, f32x4& d1) {
    d0 = XOps<XT>::template mfma<S>(xo, c0[S], d0);
    d1 = XOps<XT>::template mfma<8 + S>(xo, c1[S], d1);
}

template <typename XT, int S>
__device__ inline void chain_step_half(typename XOps<XT>::vec4 xo, const typename XOps<XT>::vec4 (&c0)[8], f32x4& d) {
    d = XOps<XT>::template mfma<S>(xo, c0[S], d);
}

// One full packet P: groups 2P and 2P+1 of the row block.
template <typename XT, int MT>
__device__ inline void packet_step(const uint4& c, const uint4& a, uint32_t bw, int P, const uint2* xs,
                                   const float* xbar, int lane, float (&acc)[MT]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop0[8], cop1[8];
    word_operands<XT>(c.x, cop0);
    word_operands<XT>(c.y, cop0 + 4);
    word_operands<XT>(c.z, cop1);
    word_operands<XT>(c.w, cop1 + 4);
    const uint2* xp = xs + static_cast<size_t>(P) * MT * 64 + lane;
    const float* bp = xbar + static_cast<size_t>(P) * MT * 16 + (lane & 3) * 4;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        {
            const vec4 xo = __builtin_bit_cast(vec4, xp[t * 64]);
            const f32x4 xb = *reinterpret_cast<const f32x4*>(bp + t * 16);
            f32x4 d0 = {0.f, 0.f, 0.f, 0.f}, d1 = d0;
            chain_step<XT, 0>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 1>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 2>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 3>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 4>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 5>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 6>(xo, cop0, cop1, d0, d1);
            chain_step<XT, 7>(xo, cop0, cop1, d0, d1);
            epilogue<XT>(d0, a.x, a.y, bw & 0xffffu, xb[0] + xb[1], acc[t]);
            epilogue<XT>(d1, a.z, a.w, bw >> 16, xb[2] + xb[3], acc[t]);
        }
    }
}

// The last group of a row block when the group count is odd (packet P,
// first group only).
template <typename XT, int MT>
__device__ inline void half_step(const uint2& c, const uint2& a, uint32_t bbits, int P, const uint2* xs,
                                 const float* xbar, int lane, float (&acc)[MT]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop[8];
    word_operands<XT>(c.x, cop);
    word_operands<XT>(c.y, cop + 4);
    const uint2* xp = xs + static_cast<size_t>(P) * MT * 64 + lane;
    const float* bp = xbar + static_cast<size_t>(P) * MT * 16 + (lane & 3) * 4;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        {
            const vec4 xo = __builtin_bit_cast(vec4, xp[t * 64]);
            const f32x4 xb = *reinterpret_cast<const f32x4*>(bp + t * 16);
            f32x4 d = {0.f, 0.f, 0.f, 0.f};
            chain_step_half<XT, 0>(xo, cop, d);
            chain_step_half<XT, 1>(xo, cop, d);
            chain_step_half<XT, 2>(xo, cop, d);
            chain_step_half<XT, 3>(xo, cop, d);
            chain_step_half<XT, 4>(xo, cop, d);
            chain_step_half<XT, 5>(xo, cop, d);
            chain_step_half<XT, 6>(xo, cop, d);
            chain_step_half<XT, 7>(xo, cop, d);
            epilogue<XT>(d, a.x, a.y, bbits, xb[0] + xb[1], acc[t]);
        }
    }
}

// ---------------------------------------------------------------------------
// Format variants: b-bit codes (b = 2, 3) and d-dimensional vectors (d = 4,
// 8) with the pairs shared by the rows (variant format block in unisvq.h).
//
// d = 8: T is 8 x 8 per (row, group, token), taken as four 4 x 4 quadrants
//   T_(ia, jb)[a][b] = sum_v x[v][4 ia + a] q[v][4 jb + b]
// (v over the group's 16 vectors), each a chain of four matrix-core steps
// with the same operand mapping as d = 4: the activation operand of block
// 8 gi + 4 ia + n holds half ia of vectors 4n .. 4n+3 of group gi, and code
// word jb of a slot holds component 4 jb + j of the 16 vectors.  Lane
// (beta, j) then needs A[0..7][j] and A[0..7][4 + j] (lane view of the
// record).
// b = 3: q = lo + 4 hi (Sec. 5.2.5: only the integer vectors widen); the
// high bits become a second operand per step (the e2m1 converter with scale
// 8 turns a lone low nibble bit into 0 or 4) accumulated into the same
// chain, so T comes out whole.

// Packet data of one lane as loaded.
template <int BITS, int D>
struct LanePacket {
    uint4 c;                     // low fields: .x/.y group 0, .z/.w group 1
    uint2 h;                     // high fields (b = 3): .x group 0, .y group 1
    uint4 a[D == 8 ? 4 : 1];     // d = 4: A[0..3][j] (.x/.y group 0, .z/.w group 1);
                                 // d = 8: a[2 gi + jb] = A[0..7][4 jb + j] of group gi
    uint32_t b[D == 8 ? 2 : 1];  // d = 4: B[j] of groups 0 | 1 << 16; d = 8: b[gi] = B[j] | B[4+j] << 16
};

// High-bit operands of one high field H: operand 4h + n pairs with low
// operand 4h + n (same vector order 4n, 4n+2, 4n+1, 4n+3).
template <typename XT>
__device__ inline void high_operands(uint32_t H, typename XOps<XT>::vec4* ops) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const uint32_t e = (H >> (2 * h)) & 0x11111111u;
        const uint32_t o = (H >> (2 * h + 1)) & 0x11111111u;
        ops[4 * h + 0] = __builtin_shufflevector(XOps<XT>::template cvt2x8<0>(e), XOps<XT>::template cvt2x8<0>(o), 0, 1, 2, 3);
        ops[4 * h + 1] = __builtin_shufflevector(XOps<XT>::template cvt2x8<1>(e), XOps<XT>::template cvt2x8<1>(o), 0, 1, 2, 3);
        ops[4 * h + 2] = __builtin_shufflevector(XOps<XT>::template cvt2x8<2>(e), XOps<XT>::template cvt2x8<2>(o), 0, 1, 2, 3);
        ops[4 * h + 3] = __builtin_shufflevector(XOps<XT>::template cvt2x8<3>(e), XOps<XT>::template cvt2x8<3>(o), 0, 1, 2, 3);
    }
}

// One step of a chain: activation operand block ABID times code operand
// index I (low part, then high part for b = 3).
template <typename XT, int BITS, int ABID, int I>
__device__ inline void var_step(typename XOps<XT>::vec4 xo, const typename XOps<XT>::vec4 (&lo)[8],
                                const typename XOps<XT>::vec4 (&hi)[8], f32x4& d) {
    d = XOps<XT>::template mfma<ABID>(xo, lo[I], d);
    if constexpr (BITS == 3) d = XOps<XT>::template mfma<ABID>(xo, hi[I], d);
}

// acc += sum_a A[4 ia + a][col] * d[a] for the 4 fp16 values in w01, w23.
__device__ inline void quad_apply(const f32x4& d, uint32_t w01, uint32_t w23, float& acc) {
    float r = acc;
    r = __builtin_fmaf(h2f(w01 & 0xffffu), d[0], r);
    r = __builtin_fmaf(h2f(w01 >> 16), d[1], r);
    r = __builtin_fmaf(h2f(w23 & 0xffffu), d[2], r);
    acc = __builtin_fmaf(h2f(w23 >> 16), d[3], r);
}

// Group gi (0 or 1) of a variant packet for one token.
template <typename XT, int BITS, int D, int GI>
__device__ inline void var_group(typename XOps<XT>::vec4 xo, const f32x4& xb, const typename XOps<XT>::vec4 (&lo)[8],
                                 const typename XOps<XT>::vec4 (&hi)[8], const LanePacket<BITS, D>& pk, float& acc) {
    constexpr int B0 = 8 * GI;
    if constexpr (D == 4) {
        f32x4 d = {0.f, 0.f, 0.f, 0.f};
        var_step<XT, BITS, B0 + 0, 0>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 1, 1>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 2, 2>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 3, 3>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 4, 4>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 5, 5>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 6, 6>(xo, lo, hi, d);
        var_step<XT, BITS, B0 + 7, 7>(xo, lo, hi, d);
        const uint4& a = pk.a[0];
        epilogue<XT>(d, GI ? a.z : a.x, GI ? a.w : a.y, GI ? pk.b[0] >> 16 : pk.b[0] & 0xffffu,
                     xb[2 * GI] + xb[2 * GI + 1], acc);
    } else {
        // quadrant (ia, jb): activation blocks B0 + 4 ia + n, code operands 4 jb + n
        f32x4 d00 = {0.f, 0.f, 0.f, 0.f}, d01 = d00, d10 = d00, d11 = d00;
        var_step<XT, BITS, B0 + 0, 0>(xo, lo, hi, d00);
        var_step<XT, BITS, B0 + 0, 4>(xo, lo, hi, d01);
        var_step<XT, BITS, B0 + 4, 0>(xo, lo, hi, d10);
        var_step<XT, BITS, B0 + 4, 4>(xo, lo, hi, d11);
        var_step<XT, BITS, B0 + 1, 1>(xo, lo, hi, d00);
        var_step<XT, BITS, B0 + 1, 5>(xo, lo, hi, d01);
        var_step<XT, BITS, B0 + 5, 1>(xo, lo, hi, d10);
        var_step<XT, BITS, B0 + 5, 5>(xo, lo, hi, d11);
        var_step<XT, BITS, B0 + 2, 2>(xo, lo, hi, d00);
        var_step<XT, BITS, B0 + 2, 6>(xo, lo, hi, d01);
        var_step<XT, BITS, B0 + 6, 2>(xo, lo, hi, d10);
        var_step<XT, BITS, B0 + 6, 6>(xo, lo, hi, d11);
        var_step<XT, BITS, B0 + 3, 3>(xo, lo, hi, d00);
        var_step<XT, BITS, B0 + 3, 7>(xo, lo, hi, d01);
        var_step<XT, BITS, B0 + 7, 3>(xo, lo, hi, d10);
        var_step<XT, BITS, B0 + 7, 7>(xo, lo, hi, d11);
        const uint4& c0 = pk.a[2 * GI];      // A[0..7][j]
        const uint4& c1 = pk.a[2 * GI + 1];  // A[0..7][4 + j]
        float r = acc;
        quad_apply(d00, c0.x, c0.y, r);
        quad_apply(d10, c0.z, c0.w, r);
        quad_apply(d01, c1.x, c1.y, r);
        quad_apply(d11, c1.z, c1.w, r);
        const uint32_t bw = pk.b[GI];
        r = __builtin_fmaf(h2f(bw & 0xffffu), xb[2 * GI], r);
        acc = __builtin_fmaf(h2f(bw >> 16), xb[2 * GI + 1], r);
    }
}

// A variant packet P: both groups (NG = 2) or the trailing half packet (NG = 1).
template <typename XT, int MT, int BITS, int D, int NG>
__device__ inline void var_packet_step(const LanePacket<BITS, D>& pk, int P, const uint2* xs, const float* xbar,
                                       int lane, float (&acc)[MT]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 lo0[8], lo1[8], hi0[8], hi1[8];
    word_operands<XT>(pk.c.x, lo0);
    word_operands<XT>(pk.c.y, lo0 + 4);
    if constexpr (NG == 2) {
        word_operands<XT>(pk.c.z, lo1);
        word_operands<XT>(pk.c.w, lo1 + 4);
    }
    if constexpr (BITS == 3) {
        high_operands<XT>(pk.h.x, hi0);
        if constexpr (NG == 2) high_operands<XT>(pk.h.y, hi1);
    }
    const uint2* xp = xs + static_cast<size_t>(P) * MT * 64 + lane;
    const float* bp = xbar + static_cast<size_t>(P) * MT * 16 + (lane & 3) * 4;
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        {
            const vec4 xo = __builtin_bit_cast(vec4, xp[t * 64]);
            const f32x4 xb = *reinterpret_cast<const f32x4*>(bp + t * 16);
            var_group<XT, BITS, D, 0>(xo, xb, lo0, hi0, pk, acc[t]);
            if constexpr (NG == 2) var_group<XT, BITS, D, 1>(xo, xb, lo1, hi1, pk, acc[t]);
        }
    }
}

// LDS of the matrix-vector kernel (M tokens): staged operands xs
// [packets][M][64], per-group sums xbar [packets][M][16], the
// cross-wavefront sums red [waves][M][16]; with the fused transform also the
// transformed rows xt [M][K] (activation type) and the transform's exchange
// buffer z [K] (fp32), which starts at offset 0 over xs (dead until the
// staging writes it) and, for a single row, xt too.
__host__ __device__ inline size_t gemv_lds_bytes(int K, int M, int waves) {
    const size_t packets = (K / kGroup + 1) / 2;
    return static_cast<size_t>(M) * packets * (kXsPacketBytes + kXbarPacketBytes) +
           static_cast<size_t>(waves) * M * 16 * 4;
}
__host__ __device__ inline size_t gemv_rht_xt_offset(int K, int M, int waves) {
    return (gemv_lds_bytes(K, M, waves) + 15) / 16 * 16;
}
__host__ __device__ inline size_t gemv_rht_z_offset(int K, int M, int waves) {
    // one row: z may overlap xt as well (the row's x' is written after the
    // last read of z); several rows: the next row's z must not overwrite x'
    if (M == 1) return 0;
    const size_t base = gemv_lds_bytes(K, M, waves);
    return static_cast<size_t>(K) * 4 <= base ? 0 : gemv_rht_xt_offset(K, M, waves) + static_cast<size_t>(M) * K * 2;
}
__host__ __device__ inline size_t gemv_rht_lds_bytes(int K, int M, int waves) {
    const size_t zo = gemv_rht_z_offset(K, M, waves);
    const size_t end_xt = gemv_rht_xt_offset(K, M, waves) + static_cast<size_t>(M) * K * 2;
    const size_t end_z = zo + static_cast<size_t>(K) * 4;
    return end_xt > end_z ? end_xt : end_z;
}

// The input-side transform of MT rows of K = 2^KLOG elements on eight
// wavefronts (512 threads; in a sixteen-wavefront workgroup the other eight
// wait at the barriers), with the thread layout and the butterfly order of
// the standalone transform for the same K (W = 3 wavefront bits, KLOG - 9
// register bits), so x' is the same to the bit: registers hold elements
// lane | wave << 6 | r << 9, their register and lane bits are done there,
// one exchange through z puts the wavefront bits into registers, and x' * norm
// rounded to XT goes to xt[t][..].  xraw: the raw 16-bit activations, sraw:
// the signs, both loaded by the caller.
template <typename XT, int KLOG, int MT>
__device__ inline void rht_prologue(const uint32_t (&xraw)[MT][1 << (KLOG - 9)], const float (&sraw)[1 << (KLOG - 9)],
                                    int lane, int wave, float norm, float* z, XT* xt) {
    constexpr int LR = KLOG - 9, R = 1 << LR, K = 1 << KLOG;
    const bool tw = wave < 8;  // a sixteen-wavefront workgroup's upper half only passes the barriers
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        {
            float v[R];
#pragma unroll
            for (int r = 0; r < R; ++r)
                v[r] = static_cast<float>(__builtin_bit_cast(XT, static_cast<uint16_t>(xraw[t][r]))) * sraw[r];
            reg_stages<R, 0, LR>(v);
            lane_stage<R, 1>(v, lane);
            lane_stage<R, 2>(v, lane);
            lane_stage<R, 4>(v, lane);
            lane_stage<R, 8>(v, lane);
            lane_stage<R, 16>(v, lane);
            lane_stage<R, 32>(v, lane);
            if (t > 0) __syncthreads();  // z of the previous row fully read
            if (tw) {
#pragma unroll
                for (int r = 0; r < R; ++r) z[lane | wave << 6 | r << 9] = v[r];
            }
            __syncthreads();
            if (tw) {
#pragma unroll
                for (int r = 0; r < R; ++r) v[r] = z[lane | (r & 7) << 6 | (r >> 3) << 9 | wave << (6 + LR)];
                reg_stages<R, 0, 3>(v);
            }
            __syncthreads();  // every read of z done: x' may overwrite it
            if (tw) {
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    // x' * norm rounded to fp32 first, as the standalone
                    // transform does: the empty asm keeps the compiler from
                    // fusing product and conversion into one mixed-precision
                    // instruction that would round only once
                    float p = v[r] * norm;
                    asm volatile("" : "+v"(p));
                    xt[t * K + (lane | (r & 7) << 6 | (r >> 3) << 9 | wave << (6 + LR))] = static_cast<XT>(p);
                }
            }
        }
    }
    __syncthreads();  // xt complete; z dead
}

// Template parameters: WAVES wavefronts per workgroup, MT the token count
// (exactly; 1 to 4), PF packets in flight per wavefront, QX the packets per
// wavefront whose activations (all MT tokens) are loaded ahead of the packet
// loads (the rest are staged after them), OCC the minimum
// wavefronts per SIMD the register allocation must allow; SHARED: codes-only
// weights with row-shared pairs; BITS, D: the code width and vector
// dimension (anything but 2, 4 is a variant, always SHARED).
// RHTK > 0: the activations enter in the original basis and the workgroup
// first applies the input-side transform x' = (x diag(s)) H / sqrt(K) of
// Eq. 5 itself, K = 2^RHTK (see rht_prologue).
template <typename XT, int WAVES, int MT, int PF, int QX, int OCC, bool SHARED, int BITS = 2, int D = 4, int RHTK = 0>
__global__ __launch_bounds__(WAVES * 64, OCC) void gemv_kernel(const GemvBatch batch) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    constexpr bool kVar = BITS != 2 || D != 4;
    static_assert(!kVar || SHARED, "format variants keep their pairs in a shared block");
    static_assert(RHTK == 0 || ((WAVES == 8 || WAVES == 16) && !kVar), "the fused transform runs on eight wavefronts");

    // problem of this workgroup (uniform scalar selection)
    const int bid = blockIdx.x;
    const uint8_t* packed = batch.p[0].packed;
    const XT* x = static_cast<const XT*>(batch.p[0].x);
    void* y = batch.p[0].y;
    const uint8_t* affine = batch.p[0].affine;
    int N = batch.p[0].N, K = batch.p[0].K, rb0 = 0, affine_one = batch.p[0].affine_one;
    const signed char* sgn = RHTK > 0 ? batch.signs[0] : nullptr;
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i) {
        if (i < batch.count && bid >= batch.p[i].rb_begin) {
            packed = batch.p[i].packed;
            x = static_cast<const XT*>(batch.p[i].x);
            y = batch.p[i].y;
            N = batch.p[i].N;
            K = batch.p[i].K;
            rb0 = batch.p[i].rb_begin;
            affine = batch.p[i].affine;
            affine_one = batch.p[i].affine_one;
            if constexpr (RHTK > 0) sgn = batch.signs[i];
        }
    }
    const int rb = bid - rb0;
    const int groups = K >> 7;
    const int nfull = groups >> 1;
    const bool has_half = (groups & 1) != 0;
    const int packets = nfull + (has_half ? 1 : 0);  // the half packet counts as one
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    uint2* xs = reinterpret_cast<uint2*>(smem);                                                     // [packets][MT][64]
    float* xbar = reinterpret_cast<float*>(smem + static_cast<size_t>(MT) * packets * kXsPacketBytes);  // [packets][MT][4][4]
    float* red = xbar + static_cast<size_t>(MT) * packets * 16;                                     // [WAVES][MT][16]

    // This wavefront's run: full packets [p0, p0 + np), plus the trailing
    // half packet (packet nfull) for the last wavefront.
    const int per = (nfull + WAVES - 1) / WAVES;
    const int p0 = min(nfull, wave * per);
    const int np = min(nfull, p0 + per) - p0;
    const bool do_half = has_half && wave == WAVES - 1;
    const int npw = np + (do_half ? 1 : 0);  // packets whose activations this wavefront stages
    const int pbeg = do_half && np == 0 ? nfull : p0;

    // 1. Activation loads for exactly this wavefront's packets, before the
    //    packet loads so that staging them waits for nothing else: for each
    //    token t and each of the first QX packets pbeg + q of the run, lane l
    //    reads the four activations operand_unit<D>(l) of the packet.  Loads
    //    stay outside any branch (a branch around a load makes the wait
    //    counters drain completely at the join); a load past the run, and the
    //    second group of the half packet, get an offset past the end of the
    //    buffer and return zeros without touching memory.
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(MT) * K * 2u);
    const uint32_t vlane = operand_unit<D>(lane);
    auto x_off = [&](int t, int q) -> uint32_t {
        const uint32_t k = static_cast<uint32_t>(pbeg + q) * 256u + 4u * vlane;
        return q < npw && k < static_cast<uint32_t>(K) ? (static_cast<uint32_t>(t) * K + k) * 2u : kOutOfRange;
    };
    uint2 xr[MT][QX];
    constexpr int kRR = RHTK > 0 ? 1 << (RHTK - 9) : 1;  // transform elements per thread and token
    uint32_t xraw[RHTK > 0 ? MT : 1][kRR];
    float sraw[kRR];
    if constexpr (RHTK > 0) {
        // the whole rows, for the transform (element lane | wave << 6 | r << 9)
        const __amdgpu_buffer_rsrc_t rsg = make_rsrc(sgn, static_cast<uint32_t>(K));
#pragma unroll
        for (int r = 0; r < kRR; ++r) {
            const int i = lane | wave << 6 | r << 9;
            const bool tw = wave < 8;  // the transform's wavefronts
#pragma unroll
            for (int t = 0; t < MT; ++t)
                xraw[t][r] = ld16(rx, tw ? (static_cast<uint32_t>(t) * K + i) * 2u : kOutOfRange);
            sraw[r] = static_cast<float>(static_cast<signed char>(
                __builtin_amdgcn_raw_buffer_load_b8(rsg, tw ? static_cast<uint32_t>(i) : kOutOfRange, 0, 0)));
        }
    } else {
#pragma unroll
        for (int t = 0; t < MT; ++t)
#pragma unroll
            for (int q = 0; q < QX; ++q) xr[t][q] = ld64(rx, x_off(t, q));
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the activation loads ahead of the packet loads

    // 2. The first PF packets of this wavefront's run.  With row-shared pairs
    //    (SHARED) the weights are bare codes and each lane reads its A column
    //    and B values from the small shared block (cached, the same for every
    //    row block) instead of the packet.
    constexpr uint32_t kBlockBytes =
        kVar ? var_group_bytes(BITS) : (SHARED ? kCodeGroupBlockBytes : kGroupBlockBytes);
    constexpr uint32_t kPktBytes = kVar ? 2 * var_group_bytes(BITS) : (SHARED ? kCodePacketBytes : kPacketBytes);
    constexpr uint32_t kRecBytes = kVar ? var_record_bytes(D) : kAffineRecordBytes;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(packed, static_cast<uint32_t>(N / kRowBlock) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra =
        make_rsrc(affine, SHARED ? static_cast<uint32_t>(affine_one ? 1 : packets) * kRecBytes : 0u);
    const uint32_t blk = static_cast<uint32_t>(rb) * groups * kBlockBytes;
    const uint32_t jcol = static_cast<uint32_t>(lane & 3);
    // packet p of the row block (or nothing when !valid)
    auto load_pkt = [&](int p, bool valid, uint4& c, uint4& a, uint32_t& b) {
        const uint32_t off = valid ? blk + static_cast<uint32_t>(p) * kPktBytes : kOutOfRange;
        c = ld128_stream(rw, off + 16 * lane);
        if constexpr (SHARED) {
            const uint32_t R = valid ? static_cast<uint32_t>(affine_one ? 0 : p) * kAffineRecordBytes : kOutOfRange;
            a = ld128(ra, R + 16 * jcol);
            b = ld32(ra, R + kRecordBiasOff + 4 * jcol);
        } else {
            a = ld128_stream(rw, off + kPacketAffineOff + 16 * lane);
            b = ld32_stream(rw, off + kPacketBiasOff + 4 * lane);
        }
    };
    // the same for a variant packet (codes-only, pairs from the shared block)
    auto load_var = [&](int p, bool valid, LanePacket<BITS, D>& pk) {
        const uint32_t off = valid ? blk + static_cast<uint32_t>(p) * kPktBytes : kOutOfRange;
        pk.c = ld128_stream(rw, off + 16 * lane);
        if constexpr (BITS == 3) pk.h = ld64_stream(rw, off + kVarHiOff + 8 * lane);
        const uint32_t R = valid ? static_cast<uint32_t>(affine_one ? 0 : p) * kRecBytes : kOutOfRange;
        if constexpr (D == 8) {
#pragma unroll
            for (int i = 0; i < 4; ++i) pk.a[i] = ld128(ra, R + 64 * jcol + 16 * i);
            const uint2 b2 = ld64(ra, R + kVarBiasOff8 + 8 * jcol);
            pk.b[0] = b2.x;
            pk.b[1] = b2.y;
        } else {
            pk.a[0] = ld128(ra, R + 16 * jcol);
            pk.b[0] = ld32(ra, R + kRecordBiasOff + 4 * jcol);
        }
    };
    uint4 cbuf[kVar ? 1 : PF], abuf[kVar ? 1 : PF];
    uint32_t bbuf[kVar ? 1 : PF];
    LanePacket<BITS, D> vbuf[kVar ? PF : 1];
    if constexpr (kVar) {
#pragma unroll
        for (int i = 0; i < PF; ++i) load_var(p0 + i, i < np, vbuf[i]);
    } else {
#pragma unroll
        for (int i = 0; i < PF; ++i) load_pkt(p0 + i, i < np, cbuf[i], abuf[i], bbuf[i]);
    }
    __builtin_amdgcn_sched_barrier(0);

    // 3. Stage this wavefront's activations in operand order, with the
    //    per-group sums.  Only this wavefront reads them, so no workgroup
    //    barrier is needed -- LDS accesses of one wavefront complete in order.
    if constexpr (RHTK > 0) {
        // the transformed rows x' (rounded to the activation type, as a
        // standalone transform writing XT would) into LDS, then staged from there
        XT* xt = reinterpret_cast<XT*>(smem + gemv_rht_xt_offset(K, MT, WAVES));
        float* z = reinterpret_cast<float*>(smem + gemv_rht_z_offset(K, MT, WAVES));
        rht_prologue<XT, RHTK, MT>(xraw, sraw, lane, wave, batch.rht_norm, z, xt);
        for (int q = 0; q < npw; ++q) {
#pragma unroll
            for (int t = 0; t < MT; ++t) {
                const uint32_t off = x_off(t, q);
                const uint2 raw = off < kOutOfRange ? *reinterpret_cast<const uint2*>(
                                                          reinterpret_cast<const unsigned char*>(xt) + off)
                                                    : uint2{0u, 0u};
                stage_packet<XT, MT>(raw, t, pbeg + q, lane, xs, xbar);
            }
        }
    } else {
#pragma unroll
        for (int q = 0; q < QX; ++q) {
            if (q < npw) {
#pragma unroll
                for (int t = 0; t < MT; ++t) stage_packet<XT, MT>(xr[t][q], t, pbeg + q, lane, xs, xbar);
            }
        }
        for (int q = QX; q < npw; ++q) {  // more than QX packets: not overlapped with the packet loads
#pragma unroll
            for (int t = 0; t < MT; ++t) stage_packet<XT, MT>(ld64(rx, x_off(t, q)), t, pbeg + q, lane, xs, xbar);
        }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // 4. Packets.  When the whole run fits the prefetch buffers (np <= PF) it is
    //    consumed straight from them; otherwise each buffer slot is refilled PF
    //    packets ahead right after it is consumed.
    float acc[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[t] = 0.f;
    if constexpr (kVar) {
        if (np <= PF) {
#pragma unroll
            for (int j = 0; j < PF; ++j)
                if (j < np) var_packet_step<XT, MT, BITS, D, 2>(vbuf[j], p0 + j, xs, xbar, lane, acc);
        } else {
            for (int i = 0; i < np; i += PF) {
#pragma unroll
                for (int j = 0; j < PF; ++j) {
                    if (i + j < np)
                        var_packet_step<XT, MT, BITS, D, 2>(vbuf[j], p0 + i + j, xs, xbar, lane, acc);
                    const int nxt = i + j + PF;
                    load_var(p0 + nxt, nxt < np, vbuf[j]);
                }
            }
        }
    } else {
        if (np <= PF) {
#pragma unroll
            for (int j = 0; j < PF; ++j)
                if (j < np)
                    packet_step<XT, MT>(cbuf[j], abuf[j], bbuf[j], p0 + j, xs, xbar, lane, acc);
        } else {
            for (int i = 0; i < np; i += PF) {
#pragma unroll
                for (int j = 0; j < PF; ++j) {
                    if (i + j < np)
                        packet_step<XT, MT>(cbuf[j], abuf[j], bbuf[j], p0 + i + j, xs, xbar, lane, acc);
                    const int nxt = i + j + PF;
                    load_pkt(p0 + nxt, nxt < np, cbuf[j], abuf[j], bbuf[j]);
                }
            }
        }
    }
    // The trailing half packet (odd group count) of the last wavefront: loaded
    // and used here, outside the pipelined part.
    if (do_half) {
        const uint32_t hoff = blk + static_cast<uint32_t>(nfull) * kPktBytes;
        if constexpr (kVar) {
            LanePacket<BITS, D> hp;
            const uint2 c = ld64_stream(rw, hoff + 8 * lane);
            hp.c = uint4{c.x, c.y, 0u, 0u};
            if constexpr (BITS == 3) hp.h = uint2{ld32_stream(rw, hoff + kVarHalfHiOff + 4 * lane), 0u};
            const uint32_t R = static_cast<uint32_t>(affine_one ? 0 : nfull) * kRecBytes;
            if constexpr (D == 8) {
                hp.a[0] = ld128(ra, R + 64 * jcol);
                hp.a[1] = ld128(ra, R + 64 * jcol + 16);
                hp.b[0] = ld32(ra, R + kVarBiasOff8 + 8 * jcol);
            } else {
                const uint2 a = ld64(ra, R + 16 * jcol);
                hp.a[0] = uint4{a.x, a.y, 0u, 0u};
                hp.b[0] = ld16(ra, R + kRecordBiasOff + 4 * jcol);
            }
            var_packet_step<XT, MT, BITS, D, 1>(hp, nfull, xs, xbar, lane, acc);
        } else {
            const uint2 hc = ld64_stream(rw, hoff + 8 * lane);
            uint2 ha;
            uint32_t hb;
            if constexpr (SHARED) {
                const uint32_t R = static_cast<uint32_t>(affine_one ? 0 : nfull) * kAffineRecordBytes;
                ha = ld64(ra, R + 16 * jcol);
                hb = ld16(ra, R + kRecordBiasOff + 4 * jcol);
            } else {
                ha = ld64_stream(rw, hoff + kHalfAffineOff + 8 * lane);
                hb = ld16_stream(rw, hoff + kHalfBiasOff + 2 * lane);
            }
            half_step<XT, MT>(hc, ha, hb, nfull, xs, xbar, lane, acc);
        }
    }

    // 5. Sum the four component lanes of each row, then the wavefronts.
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const float v = quad_sum(acc[t]);
        if ((lane & 3) == 0) red[(wave * MT + t) * 16 + (lane >> 2)] = v;
    }
    __syncthreads();
    if (threadIdx.x < MT * 16) {
        const int t = threadIdx.x >> 4, r = threadIdx.x & 15;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += red[(w * MT + t) * 16 + r];
        store_out(y, static_cast<int64_t>(t) * N + static_cast<int64_t>(rb) * kRowBlock + r, s,
                  batch.y_dtype);
    }
}

constexpr size_t kMaxLds = 160 * 1024;


template <typename XT, bool SHARED, int WAVES, int MT, int PF, int QX, int BITS = 2, int D = 4>
int launch_cfg(const GemvBatch& b, int blocks, int maxK, hipStream_t s) {
    const size_t lds = gemv_lds_bytes(maxK, MT, WAVES);
    if (lds > kMaxLds) return UNISVQ_EUNSUP;
    // the dynamic-LDS limit, raised once per instantiation and device
    static std::atomic<uint64_t> attr_done{0};
    const int st = ensure_lds_limit(reinterpret_cast<const void*>(&gemv_kernel<XT, WAVES, MT, PF, QX, 1, SHARED, BITS, D>),
                                    static_cast<int>(kMaxLds), attr_done);
    if (st != UNISVQ_OK) return st;
    hipLaunchKernelGGL((gemv_kernel<XT, WAVES, MT, PF, QX, 1, SHARED, BITS, D>), dim3(static_cast<unsigned>(blocks)),
                       dim3(WAVES * 64), lds, s, b);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

// Launch geometry for a batch: WAVES wavefronts per 16-row block, PF packets
// in flight per wavefront, QX packets per wavefront whose activations are
// loaded up front.
struct GemvPlan {
    int waves, pf, qx;
};

// Packets per wavefront whose activations load up front: the whole run (the
// half packet included), as a power of two, at most 8 loads for all tokens.
inline int plan_qx(int per_wave, int M) {
    const int cap = M == 1 ? 8 : (M == 2 ? 4 : 2);
    int q = 1;
    while (q < per_wave && q < cap) q *= 2;
    return q;
}

GemvPlan plan_gemv(int64_t blocks, int min_groups, int max_groups, int M) {
    (void)blocks;
    const int packets = max_groups / 2;
    // 8 wavefronts per 16-row block; 16 for one token when every problem of
    // the launch has the same, long K (more than 16 packets per row block: a
    // mix of K sizes leaves the short problems with LDS sized for the long
    // one).  Two packets in flight per wavefront; four for one token when
    // the runs are three or four packets long.  Swept per shape on MI355X:
    // e.g. 4 tokens x 4096 x 4096 6.0 us with 8 wavefronts and 2 in flight,
    // 8.5 us with 4 and 2; one token x 8192 x 28672 22.2 us with 16 and 2,
    // 24.6 us with 8 and 4; one token x 4096 x 11008 6.6 us with 16 and 4,
    // 7.0 us with 16 and 2; the seven 70B-shaped products in one launch
    // 72.8 us with 8 and 4, 93.8 us with 16 and 2.
    GemvPlan p;
    p.waves = M == 1 && min_groups == max_groups && packets > 16 ? 16 : 8;
    const int per = (packets + p.waves - 1) / p.waves;
    const int per_min = (min_groups / 2 + p.waves - 1) / p.waves;
    p.pf = M == 1 && per_min > 2 && per_min <= 4 ? 4 : 2;
    p.qx = plan_qx(per + (max_groups & 1), M);
    return p;
}

}  // namespace
}  // namespace unisvq
