// Small-batch product for batches with many rows (4 < M <= 32 tokens): each
// workgroup covers 64 rows -- four 16-row blocks -- and walks K in steps of
// two packets (512 columns).  The activations of a step are staged once in
// LDS and shared by the four row blocks, so activation traffic is a quarter
// of the 16-row kernel's (which re-reads all of x for every 16 rows: 3.5x the
// weight bytes at 16 tokens).
//
// Eight wavefronts: wavefront w decodes and multiplies row block w % 4 of
// packet w / 4 of the step (both groups), so every packet load is the
// coalesced 16-byte-per-lane read of one packet slot per lane.  Per group the
// 16 x 128 weight tile is decoded on the matrix cores (A q + B exactly in fp32
// from the integer codes, Eq. 4; one rounding to fp16) into the wavefront's
// LDS tile and read back as the B operand of v_mfma_f32_16x16x32_f16; the
// activation operands come from the staged step.  Activations and packets
// are loaded three steps ahead into registers (the activations then staged
// into LDS the step before their use, one barrier per step).  The two
// wavefronts of a row block meet in LDS at the end.
#include "common.hpp"
#include "decode.hpp"

namespace unisvq {
namespace {

constexpr int kWaves64 = 8;
constexpr int kRowBlocks64 = 4;                      // row blocks per workgroup
constexpr int kStepPackets = kWaves64 / kRowBlocks64;  // packets per step (per row block)
constexpr int kStepCols = kStepPackets * 256;        // columns per step
constexpr int kXRow = kStepCols + 8;                 // halves per staged token row (16-byte pad)
constexpr int kTRow = kGroup + 16;                   // halves per decoded row of a wavefront tile
constexpr int kTile = 16 * kTRow;

struct Sb64Problem {
    const uint8_t* packed;
    const uint8_t* affine;
    const _Float16* x;
    const float* inv_scale;
    void* y;
    int N, K, wg_begin, affine_one;
};

struct Sb64Batch {
    Sb64Problem p[kMaxBatch];
    int count, M, y_dtype;
};

template <int MT>
__device__ inline void tile_product(const Piece& pc, int jj, int j, _Float16* wrow, const _Float16* wlane,
                                    const _Float16* xlane, f32x4 (&acc)[MT]) {
    DecOps ops;
    prepare(pc, j, jj, ops);
    decode_vecs<0>(ops, wrow, j);
    decode_vecs<1>(ops, wrow, j);
    decode_vecs<2>(ops, wrow, j);
    decode_vecs<3>(ops, wrow, j);
    decode_vecs<4>(ops, wrow, j);
    decode_vecs<5>(ops, wrow, j);
    decode_vecs<6>(ops, wrow, j);
    decode_vecs<7>(ops, wrow, j);
    f16x8 wb[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) wb[c] = *reinterpret_cast<const f16x8*>(wlane + 32 * c);
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int i = 0; i < MT; ++i) {
            const f16x8 xa = *reinterpret_cast<const f16x8*>(xlane + (16 * i) * kXRow + 128 * jj + 32 * c);
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa, wb[c], acc[i], 0, 0, 0);
        }
}

// MT token tiles of 16 (M <= 16 MT); SHARED: codes-only weights with the
// shared affine block.
template <int MT, bool SHARED>
__global__ __launch_bounds__(kWaves64 * 64, 2) void skinny64_kernel(const Sb64Batch batch) {
    constexpr int kXChunks = 16 * MT * kStepCols / 8;  // 16-byte pieces of a staged step
    constexpr int kXPer = kXChunks / (kWaves64 * 64);  // per thread
    __shared__ __attribute__((aligned(16))) _Float16 xbuf[2][16 * MT * kXRow];
    __shared__ __attribute__((aligned(16))) _Float16 wtile[kWaves64 * kTile];
    static_assert(kXChunks % (kWaves64 * 64) == 0, "whole pieces per thread");
    static_assert(kWaves64 * 16 * MT * 16 * 4 <= kWaves64 * kTile * 2, "partial sums reuse the decode tiles");

    const int bid = blockIdx.x;
    Sb64Problem pb = batch.p[0];
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i)
        if (i < batch.count && bid >= batch.p[i].wg_begin) pb = batch.p[i];
    const int M = batch.M;
    const int N = pb.N, K = pb.K;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int rbl = wave % kRowBlocks64;     // row block within the tile
    const int pk = wave / kRowBlocks64;      // packet within the step
    const int rb = (bid - pb.wg_begin) * kRowBlocks64 + rbl;
    const bool row_ok = rb * kRowBlock < N;  // the last tile of a problem may be partial
    const int groups = K >> 7;
    const int packets = (groups + 1) >> 1;
    const int steps = (packets + kStepPackets - 1) / kStepPackets;

    constexpr uint32_t kBlockBytes = SHARED ? kCodeGroupBlockBytes : kGroupBlockBytes;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(pb.packed, static_cast<uint32_t>(N / kRowBlock) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(
        pb.affine, SHARED ? static_cast<uint32_t>(pb.affine_one ? 1 : (groups + 1) / 2) * kAffineRecordBytes : 0u);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(pb.x, static_cast<uint32_t>(M) * K * 2u);
    const uint32_t rowblk = static_cast<uint32_t>(rb) * groups * kBlockBytes;
    const int gend = row_ok ? groups : 0;  // a row block past N reads nothing
    auto load = [&](int step, Piece& pc) {
        const int p = step * kStepPackets + pk;
        if constexpr (SHARED)
            load_packet_shared<true>(rw, ra, rowblk, p, gend, pb.affine_one, lane, pc);
        else
            load_packet<true>(rw, rowblk, p, gend, lane, pc);
    };
    // staging: piece e of a step is token e / (kStepCols / 8), columns
    // 8 (e % (kStepCols / 8)) of the step; past M or K it reads zeros
    auto load_x = [&](int step, uint4 (&v)[kXPer]) {
#pragma unroll
        for (int u = 0; u < kXPer; ++u) {
            const int e = threadIdx.x + u * kWaves64 * 64;
            const int t = e / (kStepCols / 8);
            const int col = step * kStepCols + 8 * (e % (kStepCols / 8));
            const uint32_t off = step < steps && col < K ? (static_cast<uint32_t>(t) * K + col) * 2u : kOutOfRange;
            v[u] = ld128(rx, off);
        }
    };
    auto store_x = [&](int buf, const uint4 (&v)[kXPer]) {
#pragma unroll
        for (int u = 0; u < kXPer; ++u) {
            const int e = threadIdx.x + u * kWaves64 * 64;
            const int t = e / (kStepCols / 8);
            *reinterpret_cast<uint4*>(&xbuf[buf][t * kXRow + 8 * (e % (kStepCols / 8))]) = v[u];
        }
    };

    const int j = lane & 3;
    _Float16* wrow = wtile + wave * kTile + (lane >> 2) * kTRow;
    const _Float16* wlane = wtile + wave * kTile + (lane & 15) * kTRow + 8 * (lane >> 4);
    // activation operand of this lane: token lane % 16 (+ 16 i), columns
    // 8 (lane / 16) + 32 c of group jj of this wavefront's packet
    const int xoff = (lane & 15) * kXRow + 256 * pk + 8 * (lane >> 4);

    f32x4 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Three slots: step s uses slot s % 3.  Loads are issued in the order they
    // are consumed -- the activations of step d, then its packet -- three
    // steps ahead, so an in-order wait never waits on anything later: the
    // packet of step s is needed when step s starts, the activations of step
    // s + 1 when step s ends (staged into the other LDS buffer).
    constexpr int kSlots = 3;
    Piece rg[kSlots];
    uint4 xr[kSlots][kXPer];
#pragma unroll
    for (int d = 0; d < kSlots; ++d) {
        load_x(d, xr[d]);
        load(d, rg[d]);
    }
    store_x(0, xr[0]);
    __syncthreads();
    for (int s0 = 0; s0 < steps; s0 += kSlots) {
#pragma unroll
        for (int k = 0; k < kSlots; ++k) {
            const int s = s0 + k;
            if (s < steps) {  // uniform
                tile_product<MT>(rg[k], 0, j, wrow, wlane, &xbuf[s & 1][xoff], acc);
                tile_product<MT>(rg[k], 1, j, wrow, wlane, &xbuf[s & 1][xoff], acc);
                store_x((s + 1) & 1, xr[(k + 1) % kSlots]);
                load_x(s + kSlots, xr[k]);
                load(s + kSlots, rg[k]);
                __syncthreads();
            }
        }
    }

    // The two wavefronts of each row block meet in LDS (over the tiles).  D
    // lane layout: row lane % 16, tokens 16 i + 4 (lane / 16) + e.
    float* red = reinterpret_cast<float*>(wtile);  // [pk][rbl][16 MT][16]
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
            red[((pk * kRowBlocks64 + rbl) * 16 * MT + 16 * i + 4 * (lane >> 4) + e) * 16 + (lane & 15)] = acc[i][e];
    __syncthreads();
    const int rows = kRowBlocks64 * 16;
    for (int o = threadIdx.x; o < M * rows; o += kWaves64 * 64) {
        const int t = o / rows, rr = o % rows, b = rr >> 4, r = rr & 15;
        const int row = ((bid - pb.wg_begin) * kRowBlocks64 + b) * kRowBlock + r;
        if (row >= N) continue;
        float sum = 0.f;
#pragma unroll
        for (int q = 0; q < kStepPackets; ++q) sum += red[((q * kRowBlocks64 + b) * 16 * MT + t) * 16 + r];
        if (pb.inv_scale) sum *= pb.inv_scale[t];
        store_out(pb.y, static_cast<int64_t>(t) * N + row, sum, batch.y_dtype);
    }
}

template <int MT, bool SHARED>
hipError_t launch64(const Sb64Batch& b, int blocks, hipStream_t s) {
    hipLaunchKernelGGL((skinny64_kernel<MT, SHARED>), dim3(static_cast<unsigned>(blocks)), dim3(kWaves64 * 64), 0, s,
                       b);
    return hipGetLastError();
}

}  // namespace

int64_t skinny64_workgroups(const SkinnyProblem* probs, int count) {
    int64_t wgs = 0;
    for (int i = 0; i < count; ++i) wgs += (probs[i].N / kRowBlock + kRowBlocks64 - 1) / kRowBlocks64;
    return wgs;
}

hipError_t launch_skinny64_batch(const SkinnyProblem* probs, int count, int64_t M, int y_dtype, hipStream_t s) {
    if (count < 1 || count > kMaxBatch || M < 1 || M > kSkinnyMaxM) return hipErrorInvalidValue;
    Sb64Batch b{};
    int blocks = 0;
    for (int i = 0; i < count; ++i) {
        const SkinnyProblem& q = probs[i];
        b.p[i] = Sb64Problem{q.packed, q.affine, q.x, q.inv_scale, q.y, static_cast<int>(q.N), static_cast<int>(q.K),
                             blocks, q.affine_one};
        blocks += static_cast<int>((q.N / kRowBlock + kRowBlocks64 - 1) / kRowBlocks64);
    }
    b.count = count;
    b.M = static_cast<int>(M);
    b.y_dtype = y_dtype;
    const bool shared = probs[0].affine != nullptr;
    if (M <= 16) return shared ? launch64<1, true>(b, blocks, s) : launch64<1, false>(b, blocks, s);
    return shared ? launch64<2, true>(b, blocks, s) : launch64<2, false>(b, blocks, s);
}

}  // namespace unisvq
