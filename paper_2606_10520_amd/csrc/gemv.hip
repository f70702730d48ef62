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

}  // namespace

struct GemvBatch {
    GemvProblem p[kMaxBatch];
    int count;
    int M;
    int y_dtype;
};

namespace {

// Activation operands of one (token, packet) in LDS: 64 lanes x 8 bytes, in
// the operand order of the broadcast A operand.  The per-group sums xbar are
// kept as the four DPP row sums of the packet, [component][row]: rows 0, 1
// belong to group 2P, rows 2, 3 to group 2P + 1.
constexpr int kXsPacketBytes = 64 * 8;
constexpr int kXbarPacketBytes = 16 * 4;

// One loaded activation word (lane's vector of packet P, token t) -> operand
// order in LDS, plus the per-group sums.
template <typename XT>
__device__ inline void stage_packet(uint2 raw, int t, int P, int packets, int lane, uint2* xs, float* xbar) {
    const uint2 op = quad_transpose16(raw, lane & 3);
    const size_t tp = static_cast<size_t>(t) * packets + P;
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
                                   const float* xbar, int packets, int M, int lane, float (&acc)[MT]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop0[8], cop1[8];
    word_operands<XT>(c.x, cop0);
    word_operands<XT>(c.y, cop0 + 4);
    word_operands<XT>(c.z, cop1);
    word_operands<XT>(c.w, cop1 + 4);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        if (t < M) {
            const size_t tp = static_cast<size_t>(t) * packets + P;
            const vec4 xo = __builtin_bit_cast(vec4, xs[tp * 64 + lane]);
            const f32x4 xb = *reinterpret_cast<const f32x4*>(xbar + tp * 16 + (lane & 3) * 4);
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
                                 const float* xbar, int packets, int M, int lane, float (&acc)[MT]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop[8];
    word_operands<XT>(c.x, cop);
    word_operands<XT>(c.y, cop + 4);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        if (t < M) {
            const size_t tp = static_cast<size_t>(t) * packets + P;
            const vec4 xo = __builtin_bit_cast(vec4, xs[tp * 64 + lane]);
            const f32x4 xb = *reinterpret_cast<const f32x4*>(xbar + tp * 16 + (lane & 3) * 4);
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

// Template parameters: WAVES wavefronts per workgroup, MT the largest token
// count, PF packets in flight per wavefront, NX activation load instructions
// per wavefront (issued ahead of the packet loads), OCC the minimum
// wavefronts per SIMD the register allocation must allow.
template <typename XT, int WAVES, int MT, int PF, int NX, int OCC, bool SHARED>
__global__ __launch_bounds__(WAVES * 64, OCC) void gemv_kernel(const GemvBatch batch) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];

    // problem of this workgroup (uniform scalar selection)
    const int bid = blockIdx.x;
    const uint8_t* packed = batch.p[0].packed;
    const XT* x = static_cast<const XT*>(batch.p[0].x);
    void* y = batch.p[0].y;
    const uint8_t* affine = batch.p[0].affine;
    int N = batch.p[0].N, K = batch.p[0].K, rb0 = 0, affine_one = batch.p[0].affine_one;
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
        }
    }
    const int M = batch.M;
    const int rb = bid - rb0;
    const int groups = K >> 7;
    const int nfull = groups >> 1;
    const bool has_half = (groups & 1) != 0;
    const int packets = nfull + (has_half ? 1 : 0);  // the half packet counts as one
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    uint2* xs = reinterpret_cast<uint2*>(smem);                                                    // [M][packets][64]
    float* xbar = reinterpret_cast<float*>(smem + static_cast<size_t>(M) * packets * kXsPacketBytes);  // [M][packets][4][4]
    float* red = xbar + static_cast<size_t>(M) * packets * 16;                                     // [WAVES][MT][16]

    // This wavefront's run: full packets [p0, p0 + np), plus the trailing
    // half packet (packet nfull) for the last wavefront.
    const int per = (nfull + WAVES - 1) / WAVES;
    const int p0 = min(nfull, wave * per);
    const int np = min(nfull, p0 + per) - p0;
    const bool do_half = has_half && wave == WAVES - 1;
    const int npw = np + (do_half ? 1 : 0);  // packets whose activations this wavefront stages
    const int pbeg = do_half && np == 0 ? nfull : p0;

    // 1. Activation loads for exactly this wavefront's packets, before the
    //    packet loads so that staging them waits for nothing else.  Load c
    //    covers token c / npw, packet pbeg + c % npw; lane l reads vector
    //    operand_vector(l) of the packet.  Loads stay outside any branch (a
    //    branch around a load makes the wait counters drain completely at the
    //    join); an unneeded load, and the second group of the half packet, get
    //    an offset past the end of the buffer and return zeros without
    //    touching memory.
    const int loads_w = M * npw;
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(M) * K * 2u);
    const uint32_t vlane = operand_vector(lane);
    auto x_off = [&](int c) -> uint32_t {
        const int t = MT == 1 || npw == 0 ? 0 : c / npw;
        const int P = pbeg + (c - t * npw);
        const uint32_t k = static_cast<uint32_t>(P) * 256u + 4u * vlane;
        return c < loads_w && k < static_cast<uint32_t>(K) ? (static_cast<uint32_t>(t) * K + k) * 2u
                                                           : kOutOfRange;
    };
    uint2 xr[NX];
#pragma unroll
    for (int i = 0; i < NX; ++i) xr[i] = ld64(rx, x_off(i));
    __builtin_amdgcn_sched_barrier(0);  // keep the activation loads ahead of the packet loads

    // 2. The first PF packets of this wavefront's run.  With row-shared pairs
    //    (SHARED) the weights are bare codes and each lane reads its A column
    //    and B values from the small shared block (cached, the same for every
    //    row block) instead of the packet.
    constexpr uint32_t kBlockBytes = SHARED ? kCodeGroupBlockBytes : kGroupBlockBytes;
    constexpr uint32_t kPktBytes = SHARED ? kCodePacketBytes : kPacketBytes;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(packed, static_cast<uint32_t>(N / kRowBlock) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra =
        make_rsrc(affine, SHARED ? static_cast<uint32_t>(affine_one ? 1 : packets) * kAffineRecordBytes : 0u);
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
    uint4 cbuf[PF], abuf[PF];
    uint32_t bbuf[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i) load_pkt(p0 + i, i < np, cbuf[i], abuf[i], bbuf[i]);
    __builtin_amdgcn_sched_barrier(0);

    // 3. Stage this wavefront's activations in operand order, with the
    //    per-group sums.  Only this wavefront reads them, so no workgroup
    //    barrier is needed -- LDS accesses of one wavefront complete in order.
#pragma unroll
    for (int i = 0; i < NX; ++i) {
        if (i < loads_w) {
            const int t = MT == 1 ? 0 : i / npw;
            stage_packet<XT>(xr[i], t, pbeg + (i - t * npw), packets, lane, xs, xbar);
        }
    }
    for (int i = NX; i < loads_w; ++i) {  // more than NX loads: not overlapped with the packets
        const int t = MT == 1 ? 0 : i / npw;
        stage_packet<XT>(ld64(rx, x_off(i)), t, pbeg + (i - t * npw), packets, lane, xs, xbar);
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
    if (np <= PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j)
            if (j < np)
                packet_step<XT, MT>(cbuf[j], abuf[j], bbuf[j], p0 + j, xs, xbar, packets, M, lane, acc);
    } else {
        for (int i = 0; i < np; i += PF) {
#pragma unroll
            for (int j = 0; j < PF; ++j) {
                if (i + j < np)
                    packet_step<XT, MT>(cbuf[j], abuf[j], bbuf[j], p0 + i + j, xs, xbar, packets, M, lane, acc);
                const int nxt = i + j + PF;
                load_pkt(p0 + nxt, nxt < np, cbuf[j], abuf[j], bbuf[j]);
            }
        }
    }
    // The trailing half packet (odd group count) of the last wavefront: loaded
    // and used here, outside the pipelined part.
    if (do_half) {
        const uint32_t hoff = blk + static_cast<uint32_t>(nfull) * kPktBytes;
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
        half_step<XT, MT>(hc, ha, hb, nfull, xs, xbar, packets, M, lane, acc);
    }

    // 5. Sum the four component lanes of each row, then the wavefronts.
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        const float v = quad_sum(acc[t]);
        if ((lane & 3) == 0) red[(wave * MT + t) * 16 + (lane >> 2)] = v;
    }
    __syncthreads();
    if (threadIdx.x < M * 16) {
        const int t = threadIdx.x >> 4, r = threadIdx.x & 15;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += red[(w * MT + t) * 16 + r];
        store_out(y, static_cast<int64_t>(t) * N + static_cast<int64_t>(rb) * kRowBlock + r, s,
                  batch.y_dtype);
    }
}

constexpr size_t kMaxLds = 160 * 1024;

size_t gemv_lds_bytes(int K, int M, int waves, int mt) {
    const size_t packets = (K / kGroup + 1) / 2;
    return static_cast<size_t>(M) * packets * (kXsPacketBytes + kXbarPacketBytes) +
           static_cast<size_t>(waves) * mt * 16 * 4;
}

template <typename XT, bool SHARED, int WAVES, int MT, int PF, int NX>
int launch_cfg(const GemvBatch& b, int blocks, int maxK, hipStream_t s) {
    const size_t lds = gemv_lds_bytes(maxK, b.M, WAVES, MT);
    if (lds > kMaxLds) return UNISVQ_EUNSUP;
    // Raising the dynamic-LDS limit is idempotent; do it once per instantiation.
    static std::atomic<int> attr_done{0};
    if (!attr_done.load(std::memory_order_acquire)) {
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<XT, WAVES, MT, PF, NX, 1, SHARED>),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(kMaxLds)) != hipSuccess)
            return UNISVQ_EHIP;
        attr_done.store(1, std::memory_order_release);
    }
    hipLaunchKernelGGL((gemv_kernel<XT, WAVES, MT, PF, NX, 1, SHARED>), dim3(static_cast<unsigned>(blocks)),
                       dim3(WAVES * 64), lds, s, b);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

// Launch geometry for a batch: WAVES wavefronts per 16-row block, PF packets
// in flight per wavefront, NX activation loads per wavefront issued up front.
struct GemvPlan {
    int waves, pf, nx;
};

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
    // one activation load per packet and token (the half packet included)
    const int loads = M * (per + (max_groups & 1));
    p.nx = loads <= 1 ? 1 : (loads <= 2 ? 2 : (loads <= 4 ? 4 : 8));
    return p;
}

template <typename XT, bool SHARED, int WAVES, int MT, int PF>
int launch_nx(const GemvBatch& b, int blocks, int maxK, int nx, hipStream_t s) {
    if (nx == 1) return launch_cfg<XT, SHARED, WAVES, MT, PF, 1>(b, blocks, maxK, s);
    if (nx == 2) return launch_cfg<XT, SHARED, WAVES, MT, PF, 2>(b, blocks, maxK, s);
    if (nx == 4) return launch_cfg<XT, SHARED, WAVES, MT, PF, 4>(b, blocks, maxK, s);
    return launch_cfg<XT, SHARED, WAVES, MT, PF, 8>(b, blocks, maxK, s);
}

template <typename XT, bool SHARED, int WAVES, int MT>
int launch_pf(const GemvBatch& b, int blocks, int maxK, const GemvPlan& p, hipStream_t s) {
    if (p.pf == 2) return launch_nx<XT, SHARED, WAVES, MT, 2>(b, blocks, maxK, p.nx, s);
    return launch_nx<XT, SHARED, WAVES, MT, 4>(b, blocks, maxK, p.nx, s);
}

template <typename XT, bool SHARED, int MT>
int launch_waves(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    const GemvPlan p = plan_gemv(blocks, minK / kGroup, maxK / kGroup, b.M);
    if (MT == 1 && p.waves == 16) return launch_pf<XT, SHARED, 16, 1>(b, blocks, maxK, p, s);
    return launch_pf<XT, SHARED, 8, MT>(b, blocks, maxK, p, s);
}

template <typename XT, bool SHARED>
int launch_tokens(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    if (b.M == 1) return launch_waves<XT, SHARED, 1>(b, blocks, minK, maxK, s);
    if (b.M == 2) return launch_waves<XT, SHARED, 2>(b, blocks, minK, maxK, s);
    return launch_waves<XT, SHARED, 4>(b, blocks, minK, maxK, s);
}

}  // namespace

int launch_gemv_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype,
                      hipStream_t s) {
    if (M > 4 || count < 1 || count > kMaxBatch) return UNISVQ_EUNSUP;
    GemvBatch b{};
    int blocks = 0, maxK = 0, minK = 1 << 30;
    for (int i = 0; i < count; ++i) {
        b.p[i] = probs[i];
        b.p[i].rb_begin = blocks;
        blocks += probs[i].N / kRowBlock;
        maxK = probs[i].K > maxK ? probs[i].K : maxK;
        minK = probs[i].K < minK ? probs[i].K : minK;
    }
    b.count = count;
    b.M = static_cast<int>(M);
    b.y_dtype = y_dtype;
    // every problem of a batch has the same weight format (checked by the caller)
    const bool shared = probs[0].affine != nullptr;
    if (x_dtype == UNISVQ_F16)
        return shared ? launch_tokens<_Float16, true>(b, blocks, minK, maxK, s)
                      : launch_tokens<_Float16, false>(b, blocks, minK, maxK, s);
    return shared ? launch_tokens<__bf16, true>(b, blocks, minK, maxK, s)
                  : launch_tokens<__bf16, false>(b, blocks, minK, maxK, s);
}

int launch_gemv(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, hipStream_t s) {
    GemvProblem p{packed, x, y, static_cast<int>(N), static_cast<int>(K), 0, nullptr, 0};
    return launch_gemv_batch(&p, 1, M, x_dtype, y_dtype, s);
}

}  // namespace unisvq
