// Small-batch product y = x * W_hat^T for 4 < M <= 32 tokens on gfx950.
//
// Laid out like the matrix-vector kernel: one workgroup per 16-row block (of
// one problem of a batch: independent products sharing a launch, e.g. a
// decoder's query, key and value projections), its wavefronts splitting the
// block's packets along K in contiguous runs, every packet load a coalesced
// 16-byte-per-lane read, and partial sums meeting once in LDS -- one kernel,
// no workspace.  Per group a wavefront decodes its 16 x 128 weight tile on
// the matrix cores (A q + B exactly in fp32 from the integer codes, Eq. 4; one
// rounding to fp16) into its LDS tile, reads it back as the B operand and
// multiplies it with the tokens (tiles of 16) on v_mfma_f32_16x16x32_f16,
// activation operands in registers.
//
// Latency: each wavefront keeps two slots in flight, a slot being one packet
// and the activation operands of its two groups, issued in that order (the
// HBM requests first); the in-order wait for a slot never waits on the loads
// of a later one.  One decode tile per wavefront (the read-back of a group
// completes before the next group's decode writes it: LDS accesses of one
// wavefront complete in order) keeps the LDS at 4.6 KB per wavefront, so two
// 8-wavefront workgroups fit a CU; the final partial sums reuse the tiles.
// Decoded weights never leave LDS.
#include <type_traits>

#include "common.hpp"
#include "decode.hpp"

namespace unisvq {
namespace {

constexpr int kSRow = kGroup + 16;  // halves per decoded row of a wavefront's tile (32-byte pad)
constexpr int kSTile = 16 * kSRow;  // halves per wavefront tile (16 rows, one group)

// One problem of a (possibly batched) small-batch launch.
struct SkProblem {
    const uint8_t* packed;     // full format, or codes only when `affine` is set
    const uint8_t* affine;     // shared affine block (codes-only format), else null
    const _Float16* x;         // [M][K] fp16 (bf16 activations arrive as their scaled fp16 copy)
    const float* inv_scale;    // per token (scaled bf16 copies), else null
    void* y;                   // [M][N]
    int N, K, rb_begin, affine_one;
};

struct SkBatch {
    SkProblem p[kMaxBatch];
    int count, M, y_dtype;
};

// Activation operands of one packet: [group][token tile][32-column chunk].
template <int MT>
struct XOperands {
    f16x8 v[2][MT][4];
};

// Weight tile of one group as the B operand: rows lane % 16, columns
// 8 (lane / 16) + 32 c.
__device__ inline void read_tile(const _Float16* wlane, f16x8 (&wb)[4]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) wb[c] = *reinterpret_cast<const f16x8*>(wlane + 32 * c);
}

// Decode group jj of a piece into the wavefront's tile (lane (beta, j) writes
// row beta), read it back as operands and multiply with the tokens.
template <int MT>
__device__ inline void group_product(const Piece& pc, int jj, int j, _Float16* wrow, const _Float16* wlane,
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
    read_tile(wlane, wb);
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[i][c], wb[c], acc[i], 0, 0, 0);
}

// Template parameters: MT token tiles of 16 (M <= 16 MT), WAVES wavefronts
// per workgroup; SHARED: codes-only weights, A and B from the shared affine
// block.
template <int MT, int WAVES, bool SHARED>
__global__ __launch_bounds__(WAVES * 64, 2) void skinny_kernel(const SkBatch batch) {
    __shared__ __attribute__((aligned(16))) _Float16 wtile[WAVES * kSTile];
    static_assert(WAVES * 16 * MT * 16 * 4 <= WAVES * kSTile * 2, "partial sums reuse the decode tiles");

    // problem of this workgroup (uniform scalar selection)
    const int bid = blockIdx.x;
    SkProblem pb = batch.p[0];
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i)
        if (i < batch.count && bid >= batch.p[i].rb_begin) pb = batch.p[i];
    const int M = batch.M;
    const int N = pb.N, K = pb.K;
    const int rb = bid - pb.rb_begin;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int groups = K >> 7;
    const int nfull = groups >> 1;
    const bool has_half = (groups & 1) != 0;

    // This wavefront's run of full packets [p0, p0 + np); the last wavefront
    // also takes the trailing half packet.
    const int per = (nfull + WAVES - 1) / WAVES;
    const int p0 = min(nfull, wave * per);
    const int np = min(nfull, p0 + per) - p0;
    const bool do_half = has_half && wave == WAVES - 1;

    constexpr uint32_t kBlockBytes = SHARED ? kCodeGroupBlockBytes : kGroupBlockBytes;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(pb.packed, static_cast<uint32_t>(N / kRowBlock) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(
        pb.affine, SHARED ? static_cast<uint32_t>(pb.affine_one ? 1 : (groups + 1) / 2) * kAffineRecordBytes : 0u);
    // tokens at or past M lie past the end of the buffer: they read zeros
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(pb.x, static_cast<uint32_t>(M) * K * 2u);
    const uint32_t rowblk = static_cast<uint32_t>(rb) * groups * kBlockBytes;
    const int gend = 2 * (p0 + np);  // packets at or past this group read nothing
    auto load = [&](int p, int end, Piece& pc) {
        if constexpr (SHARED)
            load_packet_shared<true>(rw, ra, rowblk, p, end, pb.affine_one, lane, pc);
        else
            load_packet<true>(rw, rowblk, p, end, lane, pc);
    };
    // activation operands: token 16 i + lane % 16, columns 8 (lane / 16) + 32 c
    // of the group
    const uint32_t xlane = (static_cast<uint32_t>(lane & 15) * K + 8 * (lane >> 4)) * 2u;
    const uint32_t tile_step = 16u * K * 2u;
    // the first NG groups of packet p, or zeros when it is not part of the run
    auto load_x = [&](int p, bool valid, XOperands<MT>& xo, auto ng) {
        const uint32_t base = valid ? xlane + static_cast<uint32_t>(p) * 512u : kOutOfRange;
#pragma unroll
        for (int jj = 0; jj < decltype(ng)::value; ++jj)
#pragma unroll
            for (int i = 0; i < MT; ++i)
#pragma unroll
                for (int c = 0; c < 4; ++c)
                    xo.v[jj][i][c] = __builtin_bit_cast(
                        f16x8, ld128(rx, base + static_cast<uint32_t>(i) * tile_step + 256u * jj + 64u * c));
    };

    // Decode role: lane = packet slot (row beta = lane / 4, component j = lane % 4).
    const int j = lane & 3;
    _Float16* wrow = wtile + wave * kSTile + (lane >> 2) * kSRow;
    // Operand role: weight operand row lane % 16 at columns 8 (lane / 16) + 32 c.
    const _Float16* wlane = wtile + wave * kSTile + (lane & 15) * kSRow + 8 * (lane >> 4);

    f32x4 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Two slots: packet p0 + q lives in slot q % 2.  Loads past the run read
    // zeros (no memory traffic) and are never used.
    Piece ring0, ring1;
    XOperands<MT> xs0, xs1;
    using Both = std::integral_constant<int, 2>;
    load(p0, gend, ring0);
    load_x(p0, 0 < np, xs0, Both{});
    load(p0 + 1, gend, ring1);
    load_x(p0 + 1, 1 < np, xs1, Both{});
    for (int q = 0; q < np; q += 2) {
        group_product<MT>(ring0, 0, j, wrow, wlane, xs0.v[0], acc);
        group_product<MT>(ring0, 1, j, wrow, wlane, xs0.v[1], acc);
        load(p0 + q + 2, gend, ring0);
        load_x(p0 + q + 2, q + 2 < np, xs0, Both{});
        if (q + 1 < np) {
            group_product<MT>(ring1, 0, j, wrow, wlane, xs1.v[0], acc);
            group_product<MT>(ring1, 1, j, wrow, wlane, xs1.v[1], acc);
        }
        load(p0 + q + 3, gend, ring1);
        load_x(p0 + q + 3, q + 3 < np, xs1, Both{});
    }
    if (do_half) {
        Piece h;
        XOperands<MT> xh;
        load(nfull, groups, h);
        load_x(nfull, true, xh, std::integral_constant<int, 1>{});
        group_product<MT>(h, 0, j, wrow, wlane, xh.v[0], acc);
    }

    // Partial sums of the wavefronts meet in LDS (over the decode tiles).  D
    // lane layout: row lane % 16, tokens 16 i + 4 (lane / 16) + e.
    __syncthreads();
    float* red = reinterpret_cast<float*>(wtile);  // [WAVES][16 MT][16]
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) red[(wave * 16 * MT + 16 * i + 4 * (lane >> 4) + e) * 16 + (lane & 15)] = acc[i][e];
    __syncthreads();
    for (int o = threadIdx.x; o < M * 16; o += WAVES * 64) {
        const int t = o >> 4, r = o & 15;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += red[(w * 16 * MT + t) * 16 + r];
        if (pb.inv_scale) s *= pb.inv_scale[t];
        store_out(pb.y, static_cast<int64_t>(t) * N + static_cast<int64_t>(rb) * kRowBlock + r, s, batch.y_dtype);
    }
}

template <int MT, bool SHARED>
hipError_t launch_mt(const SkBatch& b, int blocks, hipStream_t s) {
    hipLaunchKernelGGL((skinny_kernel<MT, 8, SHARED>), dim3(static_cast<unsigned>(blocks)), dim3(8 * 64), 0, s, b);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_skinny_batch(const SkinnyProblem* probs, int count, int64_t M, int y_dtype, hipStream_t s) {
    if (count < 1 || count > kMaxBatch || M < 1 || M > kSkinnyMaxM) return hipErrorInvalidValue;
    // 64-row workgroups when they still give at least 160 of them (the
    // 16-row kernel re-reads all of x for every 16 rows)
    if (skinny64_workgroups(probs, count) >= 160) return launch_skinny64_batch(probs, count, M, y_dtype, s);
    SkBatch b{};
    int blocks = 0;
    for (int i = 0; i < count; ++i) {
        const SkinnyProblem& q = probs[i];
        b.p[i] = SkProblem{q.packed, q.affine, q.x, q.inv_scale, q.y, static_cast<int>(q.N), static_cast<int>(q.K),
                           blocks, q.affine_one};
        blocks += static_cast<int>(q.N / kRowBlock);
    }
    b.count = count;
    b.M = static_cast<int>(M);
    b.y_dtype = y_dtype;
    const bool shared = probs[0].affine != nullptr;
    if (M <= 16) return shared ? launch_mt<1, true>(b, blocks, s) : launch_mt<1, false>(b, blocks, s);
    return shared ? launch_mt<2, true>(b, blocks, s) : launch_mt<2, false>(b, blocks, s);
}

hipError_t launch_skinny(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one,
                         int64_t M, const _Float16* x, const float* inv_scale, void* y, int y_dtype,
                         hipStream_t s) {
    const SkinnyProblem p{packed, affine, affine_one, x, inv_scale, y, N, K};
    return launch_skinny_batch(&p, 1, M, y_dtype, s);
}

}  // namespace unisvq
