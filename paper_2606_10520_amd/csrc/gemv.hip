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
// Schedule.  One workgroup per 16-row block of one problem (several
// independent problems may share a launch); its WAVES wavefronts split the
// block's packets along K into contiguous runs.  Each workgroup first loads
// its activations, then issues the wavefronts' packet loads, and stages the
// activations into LDS in operand order -- with the per-group sums xbar
// formed by DPP row reductions -- while the packet data is still in flight.
// The main loop consumes packets as they arrive (PF loads in flight per
// wavefront), running four independent matrix-core chains per packet.
// Partial row sums meet in LDS at the end.
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

// Position of vector v (0..31 in its group) inside the 32-slot operand
// order of one (token, group, component) line of the staged activations.
__device__ inline int operand_slot(int v) {
    const int j = v & 3;
    return (v & ~3) | ((j & 1) << 1) | (j >> 1);
}

__device__ inline float h2f(uint32_t bits16) {
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

template <int CTRL>
__device__ inline float dpp(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                 0xf, 0xf, true));
}

// Inclusive sum over the 16 lanes of a DPP row; lane 15 of the row ends
// with the row total.
__device__ inline float row16_sum_to_last(float v) {
    v += dpp<0x111>(v);  // row_shr:1
    v += dpp<0x112>(v);  // row_shr:2
    v += dpp<0x114>(v);  // row_shr:4
    v += dpp<0x118>(v);  // row_shr:8
    return v;
}

// Sum over the 4 lanes of a quad, result in every lane of the quad.
__device__ inline float quad_sum(float v) {
    v += dpp<0xB1>(v);  // quad_perm [1,0,3,2]
    v += dpp<0x4E>(v);  // quad_perm [2,3,0,1]
    return v;
}

}  // namespace

struct GemvBatch {
    GemvProblem p[kMaxBatch];
    int count;
    int M;
    int y_dtype;
};

namespace {


// One 16-byte activation chunk: vectors 2*q16 and 2*q16+1 of group g, token t.
template <typename XT>
__device__ inline void stage_chunk(const uint4& raw, int t, int g, int q16, int groups, XT* xs, float* xbar) {
    const int vbase = 2 * q16;
    uint16_t* line = reinterpret_cast<uint16_t*>(xs) + (static_cast<size_t>(t) * groups + g) * 128;
    const uint16_t* v16 = reinterpret_cast<const uint16_t*>(&raw);
    float part[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) {
        line[a * 32 + operand_slot(vbase)] = v16[a];
        line[a * 32 + operand_slot(vbase + 1)] = v16[4 + a];
        part[a] = static_cast<float>(__builtin_bit_cast(XT, v16[a])) +
                  static_cast<float>(__builtin_bit_cast(XT, v16[4 + a]));
    }
    // The 16 lanes of a DPP row hold the 16 chunks of one group.
#pragma unroll
    for (int a = 0; a < 4; ++a) part[a] = row16_sum_to_last(part[a]);
    if (q16 == 15) {
        float* xb = xbar + (static_cast<size_t>(t) * groups + g) * 4;
#pragma unroll
        for (int a = 0; a < 4; ++a) xb[a] = part[a];
    }
}

template <typename XT, int MT>
__device__ inline void epilogue(const f32x4& d, uint32_t a01, uint32_t a23, uint32_t bbits, float xb,
                                float& acc) {
    float r = acc;
    r = __builtin_fmaf(h2f(a01 & 0xffffu), d[0], r);
    r = __builtin_fmaf(h2f(a01 >> 16), d[1], r);
    r = __builtin_fmaf(h2f(a23 & 0xffffu), d[2], r);
    r = __builtin_fmaf(h2f(a23 >> 16), d[3], r);
    acc = __builtin_fmaf(h2f(bbits), xb, r);
}

// One full packet: groups g and g+1 of the row block, both contracted with
// interleaved, independent matrix-core chains.
// x0 / x1 hold the activation operand; only lanes 0..3 are ever written
// (the other lanes keep zeros -- the broadcast ignores them).
template <typename XT, int MT>
__device__ inline void packet_step(const uint4& c, const uint4& a, uint32_t bw, int g, const XT* xs,
                                   const float* xbar, int groups, int M, int lane, float (&acc)[MT],
                                   typename XOps<XT>::vec4 (&x0)[8], typename XOps<XT>::vec4 (&x1)[8]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop0[8], cop1[8];
    word_operands<XT>(c.x, cop0);
    word_operands<XT>(c.y, cop0 + 4);
    word_operands<XT>(c.z, cop1);
    word_operands<XT>(c.w, cop1 + 4);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        if (t < M) {
            if (lane < 4) {
                const vec4* s0 = reinterpret_cast<const vec4*>(xs + ((static_cast<size_t>(t) * groups + g) * 4 + lane) * 32);
                const vec4* s1 = s0 + 32;  // next group: 128 elements further
#pragma unroll
                for (int s = 0; s < 8; ++s) { x0[s] = s0[s]; x1[s] = s1[s]; }
            }
            f32x4 d0a = {0.f, 0.f, 0.f, 0.f}, d0b = d0a, d1a = d0a, d1b = d0a;
#pragma unroll
            for (int s = 0; s < 8; s += 2) {
                d0a = XOps<XT>::mfma(x0[s], cop0[s], d0a);
                d1a = XOps<XT>::mfma(x1[s], cop1[s], d1a);
                d0b = XOps<XT>::mfma(x0[s + 1], cop0[s + 1], d0b);
                d1b = XOps<XT>::mfma(x1[s + 1], cop1[s + 1], d1b);
            }
            const float* xb = xbar + (static_cast<size_t>(t) * groups + g) * 4 + (lane & 3);
            epilogue<XT, MT>(d0a + d0b, a.x, a.y, bw & 0xffffu, xb[0], acc[t]);
            epilogue<XT, MT>(d1a + d1b, a.z, a.w, bw >> 16, xb[4], acc[t]);
        }
    }
}

// The last group of a row block when the group count is odd.
template <typename XT, int MT>
__device__ inline void half_step(const uint2& c, const uint2& a, uint32_t bbits, int g, const XT* xs,
                                 const float* xbar, int groups, int M, int lane, float (&acc)[MT],
                                 typename XOps<XT>::vec4 (&x0)[8]) {
    typedef typename XOps<XT>::vec4 vec4;
    vec4 cop[8];
    word_operands<XT>(c.x, cop);
    word_operands<XT>(c.y, cop + 4);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        if (t < M) {
            if (lane < 4) {
                const vec4* s0 = reinterpret_cast<const vec4*>(xs + ((static_cast<size_t>(t) * groups + g) * 4 + lane) * 32);
#pragma unroll
                for (int s = 0; s < 8; ++s) x0[s] = s0[s];
            }
            f32x4 da = {0.f, 0.f, 0.f, 0.f}, db = da;
#pragma unroll
            for (int s = 0; s < 8; s += 2) {
                da = XOps<XT>::mfma(x0[s], cop[s], da);
                db = XOps<XT>::mfma(x0[s + 1], cop[s + 1], db);
            }
            const float xb = xbar[(static_cast<size_t>(t) * groups + g) * 4 + (lane & 3)];
            epilogue<XT, MT>(da + db, a.x, a.y, bbits, xb, acc[t]);
        }
    }
}

// Template parameters: WAVES wavefronts per workgroup, MT the largest token
// count, PF packets in flight per wavefront, NX activation load instructions
// per wavefront (issued ahead of the packet loads), OCC the minimum
// wavefronts per SIMD the register allocation must allow.
template <typename XT, int WAVES, int MT, int PF, int NX, int OCC>
__global__ __launch_bounds__(WAVES * 64, OCC) void gemv_kernel(const GemvBatch batch) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    constexpr int kThreads = WAVES * 64;

    // problem of this workgroup (uniform scalar selection)
    const int bid = blockIdx.x;
    const uint8_t* packed = batch.p[0].packed;
    const XT* x = static_cast<const XT*>(batch.p[0].x);
    void* y = batch.p[0].y;
    int N = batch.p[0].N, K = batch.p[0].K, rb0 = 0;
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i) {
        if (i < batch.count && bid >= batch.p[i].rb_begin) {
            packed = batch.p[i].packed;
            x = static_cast<const XT*>(batch.p[i].x);
            y = batch.p[i].y;
            N = batch.p[i].N;
            K = batch.p[i].K;
            rb0 = batch.p[i].rb_begin;
        }
    }
    const int M = batch.M;
    const int rb = bid - rb0;
    (void)kThreads;
    const int groups = K >> 7;
    const int nfull = groups >> 1;
    const bool has_half = (groups & 1) != 0;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    XT* xs = reinterpret_cast<XT*>(smem);                                                   // [M][groups][4][32]
    float* xbar = reinterpret_cast<float*>(smem + static_cast<size_t>(M) * groups * 256);  // [M][groups][4]
    float* red = xbar + M * groups * 4;                                                     // [WAVES][MT][16]

    // This wavefront's run: full packets [p0, p0 + np), i.e. groups
    // [2 p0, 2 (p0 + np)), plus the trailing half packet for the last wavefront.
    const int per = (nfull + WAVES - 1) / WAVES;
    const int p0 = min(nfull, wave * per);
    const int np = min(nfull, p0 + per) - p0;
    const bool do_half = has_half && wave == WAVES - 1;
    const int g0 = 2 * p0;
    const int ngw = 2 * np + (do_half ? 1 : 0);  // groups this wavefront reads
    const int gbeg = do_half && np == 0 ? groups - 1 : g0;

    // 1. Activation loads for exactly this wavefront's groups, before the
    //    packet loads so that staging them waits for nothing else.  Each
    //    16-byte chunk holds two vectors; 16 consecutive lanes (a DPP row)
    //    hold one group of one token.  Loads stay outside any branch (a branch
    //    around a load makes the wait counters drain completely at the join);
    //    an unneeded load gets an offset past the end of the buffer and returns
    //    zeros without touching memory.
    const int chunks_w = M * 16 * ngw;
    const int nxi = (chunks_w + 63) >> 6;  // load instructions needed (wave-uniform)
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(M) * K * 2u);
    auto chunk_off = [&](int c) -> uint32_t {  // byte offset of local chunk c in x
        const int t = MT == 1 ? 0 : c / (16 * ngw);
        const int lc = c - t * 16 * ngw;
        return (static_cast<uint32_t>(t) * K + static_cast<uint32_t>(gbeg) * 128 + lc * 8) * 2u;
    };
    uint4 xr[NX];
#pragma unroll
    for (int i = 0; i < NX; ++i) {
        const int c = 64 * i + lane;
        xr[i] = ld128(rx, c < chunks_w ? chunk_off(c) : kOutOfRange);
    }
    __builtin_amdgcn_sched_barrier(0);  // keep the activation loads ahead of the packet loads

    // 2. The first PF packets of this wavefront's run.
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(packed, static_cast<uint32_t>(N / kRowBlock) * groups * kGroupBlockBytes);
    const uint32_t blk = static_cast<uint32_t>(rb) * groups * kGroupBlockBytes;
    uint4 cbuf[PF], abuf[PF];
    uint32_t bbuf[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i) {
        const uint32_t off = i < np ? blk + static_cast<uint32_t>(p0 + i) * kPacketBytes : kOutOfRange;
        cbuf[i] = ld128_stream(rw, off + 16 * lane);
        abuf[i] = ld128_stream(rw, off + kPacketAffineOff + 16 * lane);
        bbuf[i] = ld32_stream(rw, off + kPacketBiasOff + 4 * lane);
    }
    __builtin_amdgcn_sched_barrier(0);

    // 3. Stage this wavefront's activations in operand order, with the
    //    per-(token, group, component) sums.  Only this wavefront reads them,
    //    so no workgroup barrier is needed -- LDS accesses of one wavefront
    //    complete in order.
#pragma unroll
    for (int i = 0; i < NX; ++i) {
        const int c = 64 * i + lane;
        if (c < chunks_w) {
            const int t = MT == 1 ? 0 : c / (16 * ngw);
            const int lc = c - t * 16 * ngw;
            stage_chunk<XT>(xr[i], t, gbeg + (lc >> 4), lc & 15, groups, xs, xbar);
        }
    }
    for (int i = NX; i < nxi; ++i) {  // more than NX instructions: not overlapped with the packets
        const int c = 64 * i + lane;
        const uint4 raw = ld128(rx, c < chunks_w ? chunk_off(c) : kOutOfRange);
        if (c < chunks_w) {
            const int t = MT == 1 ? 0 : c / (16 * ngw);
            const int lc = c - t * 16 * ngw;
            stage_chunk<XT>(raw, t, gbeg + (lc >> 4), lc & 15, groups, xs, xbar);
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
    typename XOps<XT>::vec4 x0[8], x1[8];
#pragma unroll
    for (int s = 0; s < 8; ++s) x0[s] = x1[s] = typename XOps<XT>::vec4{};
    if (np <= PF) {
#pragma unroll
        for (int j = 0; j < PF; ++j)
            if (j < np)
                packet_step<XT, MT>(cbuf[j], abuf[j], bbuf[j], 2 * (p0 + j), xs, xbar, groups, M, lane, acc,
                                    x0, x1);
    } else {
        for (int i = 0; i < np; i += PF) {
#pragma unroll
            for (int j = 0; j < PF; ++j) {
                if (i + j < np)
                    packet_step<XT, MT>(cbuf[j], abuf[j], bbuf[j], 2 * (p0 + i + j), xs, xbar, groups, M,
                                        lane, acc, x0, x1);
                const int nxt = i + j + PF;
                const uint32_t off =
                    nxt < np ? blk + static_cast<uint32_t>(p0 + nxt) * kPacketBytes : kOutOfRange;
                cbuf[j] = ld128_stream(rw, off + 16 * lane);
                abuf[j] = ld128_stream(rw, off + kPacketAffineOff + 16 * lane);
                bbuf[j] = ld32_stream(rw, off + kPacketBiasOff + 4 * lane);
            }
        }
    }
    // The trailing half packet (odd group count) of the last wavefront: loaded
    // and used here, outside the pipelined part.
    if (do_half) {
        const uint32_t hoff = blk + static_cast<uint32_t>(nfull) * kPacketBytes;
        const uint2 hc = ld64_stream(rw, hoff + 8 * lane);
        const uint2 ha = ld64_stream(rw, hoff + kHalfAffineOff + 8 * lane);
        const uint32_t hb = ld16_stream(rw, hoff + kHalfBiasOff + 2 * lane);
        half_step<XT, MT>(hc, ha, hb, groups - 1, xs, xbar, groups, M, lane, acc, x0);
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
    const size_t groups = K / kGroup;
    return static_cast<size_t>(M) * groups * (256 + 16) + static_cast<size_t>(waves) * mt * 16 * 4;
}

template <typename XT, int WAVES, int MT, int PF, int NX>
int launch_cfg(const GemvBatch& b, int blocks, int maxK, hipStream_t s) {
    const size_t lds = gemv_lds_bytes(maxK, b.M, WAVES, MT);
    if (lds > kMaxLds) return UNISVQ_EUNSUP;
    // Raising the dynamic-LDS limit is idempotent; do it once per instantiation.
    static std::atomic<int> attr_done{0};
    if (!attr_done.load(std::memory_order_acquire)) {
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_kernel<XT, WAVES, MT, PF, NX, 1>),
                                hipFuncAttributeMaxDynamicSharedMemorySize,
                                static_cast<int>(kMaxLds)) != hipSuccess)
            return UNISVQ_EHIP;
        attr_done.store(1, std::memory_order_release);
    }
    hipLaunchKernelGGL((gemv_kernel<XT, WAVES, MT, PF, NX, 1>), dim3(static_cast<unsigned>(blocks)),
                       dim3(WAVES * 64), lds, s, b);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

// Launch geometry for a batch: WAVES wavefronts per 16-row block, PF packets
// in flight per wavefront, NX activation loads per wavefront issued up front.
struct GemvPlan {
    int waves, pf, nx;
};

GemvPlan plan_gemv(int64_t blocks, int min_groups, int max_groups, int M) {
    const int packets = max_groups / 2;
    // Short K (in every problem of the batch): 4 wavefronts, whole run
    // prefetched.  Longer K: 8 wavefronts, or 16 when there are at most 256
    // workgroups (one per CU), so that the CU still holds enough loads in
    // flight.  (Measured per shape on MI355X; 16 is slower once there are
    // several workgroups per CU.)
    GemvPlan p;
    p.waves = min_groups / 2 <= 16 ? 4 : (blocks <= 256 ? 16 : 8);
    if (M > 1 && p.waves > 8) p.waves = 8;  // register budget of 1024-thread groups
    while (p.waves > 4 && blocks * p.waves > 16384) p.waves /= 2;
    const int per = (packets + p.waves - 1) / p.waves;
    p.pf = per <= 2 ? 2 : 4;
    const int chunks = M * 16 * (2 * per + (max_groups & 1));
    const int nxi = (chunks + 63) / 64;
    p.nx = nxi <= 1 ? 1 : (nxi <= 2 ? 2 : 4);
    return p;
}

template <typename XT, int WAVES, int MT, int PF>
int launch_nx(const GemvBatch& b, int blocks, int maxK, int nx, hipStream_t s) {
    if (nx == 1) return launch_cfg<XT, WAVES, MT, PF, 1>(b, blocks, maxK, s);
    if (nx == 2) return launch_cfg<XT, WAVES, MT, PF, 2>(b, blocks, maxK, s);
    return launch_cfg<XT, WAVES, MT, PF, 4>(b, blocks, maxK, s);
}

template <typename XT, int WAVES, int MT>
int launch_pf(const GemvBatch& b, int blocks, int maxK, const GemvPlan& p, hipStream_t s) {
    if (p.pf == 2) return launch_nx<XT, WAVES, MT, 2>(b, blocks, maxK, p.nx, s);
    return launch_nx<XT, WAVES, MT, 4>(b, blocks, maxK, p.nx, s);
}

template <typename XT, int MT>
int launch_waves(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    const GemvPlan p = plan_gemv(blocks, minK / kGroup, maxK / kGroup, b.M);
    if (p.waves == 4) return launch_pf<XT, 4, MT>(b, blocks, maxK, p, s);
    if (MT == 1 && p.waves == 16) return launch_pf<XT, 16, 1>(b, blocks, maxK, p, s);
    return launch_pf<XT, 8, MT>(b, blocks, maxK, p, s);
}

template <typename XT>
int launch_tokens(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    if (b.M == 1) return launch_waves<XT, 1>(b, blocks, minK, maxK, s);
    if (b.M == 2) return launch_waves<XT, 2>(b, blocks, minK, maxK, s);
    return launch_waves<XT, 4>(b, blocks, minK, maxK, s);
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
    if (x_dtype == UNISVQ_F16) return launch_tokens<_Float16>(b, blocks, minK, maxK, s);
    return launch_tokens<__bf16>(b, blocks, minK, maxK, s);
}

int launch_gemv(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, hipStream_t s) {
    GemvProblem p{packed, x, y, static_cast<int>(N), static_cast<int>(K), 0};
    return launch_gemv_batch(&p, 1, M, x_dtype, y_dtype, s);
}

}  // namespace unisvq
