// Small-batch product y = x * W_hat^T for up to 32 tokens on gfx950 (the
// product routes 1 to 3 tokens to the matrix-vector kernel where its LDS
// allows).
//
// A workgroup owns RB 16-row blocks (RB = 1, 2, 3, 4, 6 or 7; 1 above 16
// tokens) of one problem over all
// of K; several independent problems may share a launch (a decoder's query,
// key and value projections).  Its sixteen wavefronts split the packets (two
// 128-column groups each) round robin -- wavefront w takes packets w, w + 16,
// ... -- so a 4096-column row is a single round: every wavefront requests all
// it needs at once and no wavefront waits for another until they meet in LDS
// at the end.  Per packet a wavefront loads the activations of the two groups
// first (tokens in tiles of 16, fp16; reused from registers by the RB row
// blocks), then the RB packets, each a coalesced 16-byte-per-lane read of the
// packet slots, and computes row block by row block as the packets arrive.
// With one token tile the activations travel through LDS: each load
// instruction reads four whole token rows of a group (256 contiguous bytes
// each) straight into the wavefront's LDS area, laid out so that the
// operand reads that follow are free of bank conflicts.  Loading the operand
// layout directly from memory would touch sixteen token rows, 64 bytes each,
// per instruction, and every workgroup reads all of the activations.  Per row block and group it decodes the 16 x 128 weight tile on the
// matrix cores (A q + B exactly in fp32 from the integer codes, Eq. 4; one
// rounding to fp16) into its own LDS tile, reads it back as the B operand and
// multiplies it with the activations on v_mfma_f32_16x16x32_f16.  One kernel,
// no workspace, a fixed summation order; decoded weights never leave LDS.
//
// RB trades activation reuse against parallelism: a taller workgroup re-reads
// the activations less but gives fewer workgroups, and every workgroup starts
// by waiting for its first loads.  The launcher picks RB per batch from the
// number of rounds of workgroups over the CUs (pick_rb).
#include "common.hpp"
#include "decode.hpp"

namespace unisvq {
namespace {

constexpr int kWavesS = 16;         // wavefronts per workgroup
constexpr int kTRow = kGroup + 16;  // halves per decoded row of a wavefront tile (32-byte pad)
constexpr int kTile = 16 * kTRow;
// Staged activations of one group (16 tokens x 128 columns, fp16): four
// load instructions of four token rows each, 1 KB per instruction plus a
// 64-byte pad.  Lane l of instruction q reads token 4q + r (r = l / 16),
// 16-byte chunk k = (l % 16) ^ r of the group's row, and the load puts it at
// q * kXInst + 16 l.  The operand read of lane L (token t = L % 16, chunk
// 4c + L / 16) then finds it at kXInst (t / 4) + 256 (t % 4) + 16 ((L / 16) ^
// (t % 4)) + 64 c: sixteen lanes of one read hit sixteen distinct 16-byte
// bank groups.
constexpr int kXInst = 1024 + 64;
// Workgroups of up to this many row blocks may run across two problems.
constexpr int kSkinnySpanMax = 3;
constexpr int kXStage = 4 * kXInst;
static_assert(kXStage <= kTile * 2, "a group's activations fit in a decode tile");

// Row blocks of a batch are numbered globally: problem i's start at
// rb_begin; workgroup w owns global row blocks w RB .. w RB + RB - 1.  When
// the problems share their activations (and K), the numbering is packed and a
// workgroup may run on into the next problem (at most one more: every problem
// then has at least RB row blocks); otherwise each problem starts on a
// multiple of RB and the row blocks in between exist in no problem.
struct SkProblem {
    const uint8_t* packed;   // full format, or codes only when `affine` is set
    const uint8_t* affine;   // shared affine block (codes-only format), else null
    const _Float16* x;       // [M][K] fp16 (bf16 activations arrive as their scaled fp16 copy)
    const float* inv_scale;  // per token (scaled bf16 copies), else null
    void* y;                 // [M][N]
    int N, K, rb_begin, affine_one;
};

struct SkBatch {
    SkProblem p[kMaxBatch];
    int count, M, y_dtype;
};

// Group jj of a piece: decode into the wavefront's tile (lane (beta, j)
// writes row beta), read it back as the B operand (row lane % 16, columns
// 8 (lane / 16) + 32 c) and multiply with the activation operands (token
// lane % 16 + 16 i at the same columns).
template <int MT>
__device__ inline void tile_product(const Piece& pc, int jj, int j, _Float16* wrow, const _Float16* wlane,
                                    const f16x8 (&xa)[MT][4], f32x4 (&acc)[MT]) {
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
        for (int i = 0; i < MT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[i][c], wb[c], acc[i], 0, 0, 0);
}

// Per wavefront: its decode tile, and with one token tile an activation
// area (group 2p; group 2p + 1 is staged in the tile, which is free until
// the first decode of the packet).
template <int MT>
constexpr int skinny_area_bytes() {
    return kTile * 2 + (MT == 1 ? kXStage : 0);
}

template <int MT, int RB>
constexpr int skinny_lds_bytes() {
    constexpr int tiles = kWavesS * skinny_area_bytes<MT>();
    constexpr int red = kWavesS * RB * MT * 64 * 16;
    return tiles > red ? tiles : red;
}

// MT token tiles of 16 (M <= 16 MT), RB row blocks per workgroup; SHARED:
// codes-only weights with the shared affine block.
template <int MT, int RB, bool SHARED>
__global__ __launch_bounds__(kWavesS * 64, (RB * MT <= 1 ? 8 : 4)) void skinny_kernel(const SkBatch batch) {
    __shared__ __attribute__((aligned(16))) unsigned char lds[skinny_lds_bytes<MT, RB>()];
    constexpr bool kStage = MT == 1;  // activations through LDS
    constexpr int kArea = skinny_area_bytes<MT>();

    // problems of this workgroup (uniform scalar selection): `pb` holds its
    // first row block, `pn` the next problem; row blocks b >= bsplit are pn's
    const int bid = blockIdx.x;
    const int g0 = bid * RB;
    int ia = 0;
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i)
        if (i < batch.count && g0 >= batch.p[i].rb_begin) ia = i;
    SkProblem pb = batch.p[0], pn = batch.p[0];
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i) {
        if (i == ia) pb = batch.p[i];
        if (i == ia + 1) pn = batch.p[i];
    }
    // (taller workgroups never span: their scalar registers would spill)
    const int bsplit = kSkinnySpanMax >= RB && ia + 1 < batch.count ? min(max(pn.rb_begin - g0, 0), RB) : RB;
    const int M = batch.M;
    const int K = pb.K;  // (pn, if reached, has the same K and activations)
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int groups = K >> 7;
    const int packets = (groups + 1) >> 1;
    const int rb0 = g0 - pb.rb_begin;  // pb's local row block of b = 0
    const int rbn = g0 - pn.rb_begin;  // pn's local row block of b = 0 (used for b >= bsplit)
    const int nrb = pb.N / kRowBlock, nrbn = pn.N / kRowBlock;
    // row block b: its problem's local index, or -1 where no problem has it
    auto local_rb = [&](int b) {
        const int r = b < bsplit ? rb0 + b : rbn + b;
        return r < (b < bsplit ? nrb : nrbn) ? r : -1;
    };

    constexpr uint32_t kBlockBytes = SHARED ? kCodeGroupBlockBytes : kGroupBlockBytes;
    auto affine_bytes = [&](const SkProblem& q) {
        return SHARED ? static_cast<uint32_t>(q.affine_one ? 1 : (groups + 1) / 2) * kAffineRecordBytes : 0u;
    };
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(pb.packed, static_cast<uint32_t>(nrb) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(pb.affine, affine_bytes(pb));
    const __amdgpu_buffer_rsrc_t rwn = make_rsrc(pn.packed, static_cast<uint32_t>(nrbn) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ran = make_rsrc(pn.affine, affine_bytes(pn));
    // tokens at or past M lie past the end of the buffer: they read zeros
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(pb.x, static_cast<uint32_t>(M) * K * 2u);
    // activation operand of this lane: token lane % 16 + 16 i, columns
    // 8 (lane / 16) + 32 c of a group
    const uint32_t xlane = (static_cast<uint32_t>(lane & 15) * K + 8 * (lane >> 4)) * 2u;
    // staged: the lane's load offset (token lane / 16 of each instruction,
    // swizzled chunk) and its operand read offset within a staging area
    const int xr = lane >> 4, xt = lane & 15;
    const uint32_t xload = static_cast<uint32_t>(xr) * K * 2u + 16u * static_cast<uint32_t>((lane & 15) ^ xr);
    const int xread = kXInst * (xt >> 2) + 256 * (xt & 3) + 16 * ((lane >> 4) ^ (xt & 3));
    // the wavefront's LDS area (a wave-uniform address: the loads' LDS base)
    const int wu = __builtin_amdgcn_readfirstlane(wave);
    unsigned char* const uarea = lds + wu * kArea;
    unsigned char* const warea = lds + wave * kArea;

    auto load_x = [&](int g, f16x8 (&xa)[MT][4]) {
        const uint32_t base = g < groups ? xlane + static_cast<uint32_t>(g) * 256u : kOutOfRange;
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int c = 0; c < 4; ++c)
                xa[i][c] = __builtin_bit_cast(f16x8, ld128(rx, base + static_cast<uint32_t>(i) * (16u * K * 2u) + 64u * c));
    };
    // group g's activations into the staging area at byte `at` of the
    // wavefront's area (past the last group or token: zeros).  Token
    // quads at or past M are not loaded: their rows hold stale values, which
    // reach only the discarded outputs of those tokens.
    auto stage_x = [&](int g, int at) {
        const uint32_t base = g < groups ? xload + static_cast<uint32_t>(g) * 256u : kOutOfRange;
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (4 * q < M)  // uniform
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rx, (__attribute__((address_space(3))) void*)(uarea + at + q * kXInst), 16,
                    base + static_cast<uint32_t>(q) * (4u * K * 2u), 0, 0, 0);
    };
    auto read_x = [&](int at, f16x8 (&xa)[MT][4]) {
#pragma unroll
        for (int c = 0; c < 4; ++c) xa[0][c] = *reinterpret_cast<const f16x8*>(warea + at + xread + 64 * c);
    };
    auto load = [&](int p, int b, Piece& pc) {
        const int rb = local_rb(b);
        const uint32_t rowblk = static_cast<uint32_t>(rb < 0 ? 0 : rb) * groups * kBlockBytes;
        const int gend = rb >= 0 ? groups : 0;
        const bool first = b < bsplit;
        if constexpr (SHARED)
            load_packet_shared_flat<true>(first ? rw : rwn, first ? ra : ran, rowblk, p, gend,
                                          first ? pb.affine_one : pn.affine_one, lane, pc);
        else
            load_packet_flat<true>(first ? rw : rwn, rowblk, p, gend, lane, pc);
    };

    const int j = lane & 3;
    _Float16* const wtile = reinterpret_cast<_Float16*>(warea);
    _Float16* wrow = wtile + (lane >> 2) * kTRow;
    const _Float16* wlane = wtile + (lane & 15) * kTRow + 8 * (lane >> 4);
    f32x4 acc[RB][MT];
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[b][i] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Packets wave, wave + 16, ...: a 4096-column row is one round.  Requests
    // go out in the order they are used: the activations of group 2p, the
    // first row block's piece, the activations of group 2p + 1, the other
    // pieces (past the last group, or N, everything reads zeros without
    // memory traffic).
    // At most three pieces are in flight per wavefront (registers): row
    // block b's piece is requested once row block b - 3 is done.
    constexpr int kRing = RB < 3 ? RB : 3;
    for (int p = wave; p < packets; p += kWavesS) {  // uniform
        Piece pc[kRing];
        f16x8 x0[MT][4], x1[MT][4];
        if constexpr (kStage) {
            // Every read of the previous packet's tile is complete (its
            // products consumed the values), so the tile may be loaded into.
            // The compiler does not order these LDS-bound loads against the
            // LDS reads below: the piece loads stay behind them (memory
            // clobbers) and an explicit count waits for them -- the loads
            // retire in order and exactly 3 per piece follow.
            stage_x(2 * p, kTile * 2);
            stage_x(2 * p + 1, 0);
            asm volatile("" ::: "memory");
#pragma unroll
            for (int b = 0; b < kRing; ++b) load(p, b, pc[b]);
            asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * kRing) : "memory");
            read_x(kTile * 2, x0);
            read_x(0, x1);
        } else {
            load_x(2 * p, x0);
            load(p, 0, pc[0]);
            load_x(2 * p + 1, x1);
#pragma unroll
            for (int b = 1; b < kRing; ++b) load(p, b, pc[b]);
        }
#pragma unroll
        for (int b = 0; b < RB; ++b) {
            if (local_rb(b) >= 0) {  // uniform
                tile_product<MT>(pc[b % kRing], 0, j, wrow, wlane, x0, acc[b]);
                tile_product<MT>(pc[b % kRing], 1, j, wrow, wlane, x1, acc[b]);
            }
            if (b + kRing < RB) load(p, b + kRing, pc[b % kRing]);
        }
    }

    // The sixteen wavefronts meet in LDS (over the decode tiles and staging
    // areas): each stores its accumulators as they are (lane order, 16
    // bytes per lane), and one thread per (row block, token tile, lane) sums
    // the sixteen in wavefront order.  D lane layout: row lane % 16, tokens
    // 16 i + 4 (lane / 16) + e.
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(lds);  // [wave][row block][token tile][lane]
#pragma unroll
    for (int b = 0; b < RB; ++b)
#pragma unroll
        for (int i = 0; i < MT; ++i) red[((wave * RB + b) * MT + i) * 64 + lane] = acc[b][i];
    __syncthreads();
    for (int q = threadIdx.x; q < RB * MT * 64; q += kWavesS * 64) {
        f32x4 v = red[q];
#pragma unroll
        for (int w = 1; w < kWavesS; ++w) v += red[w * RB * MT * 64 + q];
        const int ln = q & 63, bi = q >> 6, b = bi / MT, i = bi % MT;
        const int rb = local_rb(b);
        if (rb < 0) continue;
        const bool first = b < bsplit;
        void* const y = first ? pb.y : pn.y;
        const int N = first ? pb.N : pn.N;
        const int row = rb * kRowBlock + (ln & 15);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = 16 * i + 4 * (ln >> 4) + e;
            if (t < M)
                store_out(y, static_cast<int64_t>(t) * N + row, pb.inv_scale ? v[e] * pb.inv_scale[t] : v[e],
                          batch.y_dtype);
        }
    }
}

template <int MT, int RB, bool SHARED>
hipError_t launch_k(const SkBatch& b, int blocks, hipStream_t s) {
    hipLaunchKernelGGL((skinny_kernel<MT, RB, SHARED>), dim3(static_cast<unsigned>(blocks)), dim3(kWavesS * 64), 0,
                       s, b);
    return hipGetLastError();
}

template <int MT, int RB>
hipError_t launch_rb(const SkBatch& b, int blocks, bool shared, hipStream_t s) {
    return shared ? launch_k<MT, RB, true>(b, blocks, s) : launch_k<MT, RB, false>(b, blocks, s);
}

// Workgroups of height rb for a batch (row blocks packed across problems when
// `span` and rb allows it).
int64_t skinny_wgs(const SkinnyProblem* probs, int count, int rb, bool span) {
    span = span && rb <= kSkinnySpanMax;
    int64_t wgs = 0, rbs = 0;
    for (int i = 0; i < count; ++i) {
        rbs += probs[i].N / kRowBlock;
        wgs += (probs[i].N / kRowBlock + rb - 1) / rb;
    }
    return span ? (rbs + rb - 1) / rb : wgs;
}

// Row blocks per workgroup for a batch: the fewest rounds of workgroups
// over the 256 CUs (one resident workgroup each) times the time of one, taken
// as 3 + RB * (packets per wavefront) in units of one packet's work -- the
// fixed part is the wait for the first loads and the final reduction.  Ties go
// to the taller workgroup (activation operands reused more).
int pick_rb(const SkinnyProblem* probs, int count, int max_rb, bool span) {
    int64_t ppw = 1;
    for (int i = 0; i < count; ++i) {
        const int64_t packets = (probs[i].K / kGroup + 1) / 2;
        const int64_t w = (packets + kWavesS - 1) / kWavesS;
        ppw = w > ppw ? w : ppw;
    }
    constexpr int kHeights[] = {7, 6, 4, 3, 2, 1};
    int best = 1;
    int64_t best_cost = -1;
    for (const int rb : kHeights) {
        if (rb > max_rb) continue;
        const int64_t wgs = skinny_wgs(probs, count, rb, span);
        const int64_t cost = (wgs + 255) / 256 * (3 + rb * ppw);
        if (best_cost < 0 || cost < best_cost) {
            best = rb;
            best_cost = cost;
        }
    }
    return best;
}

}  // namespace

hipError_t launch_skinny_batch(const SkinnyProblem* probs, int count, int64_t M, int y_dtype, hipStream_t s) {
    if (count < 1 || count > kMaxBatch || M < 1 || M > kSkinnyMaxM) return hipErrorInvalidValue;
    // two token tiles: one row block per workgroup (registers)
    const int max_rb = M > 16 ? 1 : 7;
    // workgroups may run across problems that share activations and K, when
    // every problem has at least max_rb row blocks (so at most two meet)
    bool span = count > 1;
    for (int i = 0; i < count && span; ++i)
        span = probs[i].x == probs[0].x && probs[i].inv_scale == probs[0].inv_scale && probs[i].K == probs[0].K &&
               probs[i].N / kRowBlock >= max_rb;
    const int rb = pick_rb(probs, count, max_rb, span);
    SkBatch b{};
    int64_t start = 0;
    for (int i = 0; i < count; ++i) {
        const SkinnyProblem& q = probs[i];
        b.p[i] = SkProblem{q.packed, q.affine, q.x, q.inv_scale, q.y, static_cast<int>(q.N), static_cast<int>(q.K),
                           static_cast<int>(start), q.affine_one};
        const int64_t nrb = q.N / kRowBlock;
        start += span && rb <= kSkinnySpanMax ? nrb : (nrb + rb - 1) / rb * rb;
    }
    const int blocks = static_cast<int>((start + rb - 1) / rb);
    b.count = count;
    b.M = static_cast<int>(M);
    b.y_dtype = y_dtype;
    const bool shared = probs[0].affine != nullptr;
    if (M > 16) return launch_rb<2, 1>(b, blocks, shared, s);
    switch (rb) {
        case 7: return launch_rb<1, 7>(b, blocks, shared, s);
        case 6: return launch_rb<1, 6>(b, blocks, shared, s);
        case 4: return launch_rb<1, 4>(b, blocks, shared, s);
        case 3: return launch_rb<1, 3>(b, blocks, shared, s);
        case 2: return launch_rb<1, 2>(b, blocks, shared, s);
        default: return launch_rb<1, 1>(b, blocks, shared, s);
    }
}

hipError_t launch_skinny(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one,
                         int64_t M, const _Float16* x, const float* inv_scale, void* y, int y_dtype, hipStream_t s) {
    const SkinnyProblem p{packed, affine, affine_one, x, inv_scale, y, N, K};
    return launch_skinny_batch(&p, 1, M, y_dtype, s);
}

}  // namespace unisvq
