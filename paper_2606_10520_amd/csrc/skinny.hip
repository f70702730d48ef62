// Small-batch product y = x * W_hat^T for 4 < M <= 64 tokens on gfx950.
//
// Decode dominates nothing here -- the weight stream does -- so the kernel
// is laid out like the matrix-vector kernel: one workgroup per 16-row block,
// its wavefronts splitting the block's packets along K in contiguous runs,
// every packet load a coalesced 16-byte-per-lane read issued well ahead of
// use, and partial sums meeting once in LDS.  Per group each wavefront
// decodes its 16 x 128 weight tile on the matrix cores (A q + B exactly in
// fp32 from the integer codes, Eq. 4; one rounding to fp16) into one of its
// two LDS tiles and multiplies it with up to 64 tokens on
// v_mfma_f32_16x16x32_f16 (token tiles of 16; activation operands read
// straight from global memory in the matrix-core layout).  The products of
// each group run one decode behind, so a group's decode overlaps the
// previous group's LDS reads and matrix-core work.  Decoded weights never
// leave LDS.
#include "common.hpp"
#include "decode.hpp"

namespace unisvq {
namespace {

constexpr int kSRow = kGroup + 16;      // halves per decoded row of a wavefront's tile (32-byte pad)
constexpr int kSTile = 16 * kSRow;      // halves per wavefront tile (16 rows, one group)

// One group (jj of the piece's packet) of this wavefront's run: decode, read
// the weight operand back, multiply with the MT token tiles.  xo is the
// lane's activation offset of the group's first column (or out of range).
// The three stages of one group, for the pipelined loop below: decode the
// wavefront's 16 x 128 tile into LDS, load the activation operands, multiply.
template <int MT>
__device__ inline void sk_decode(const Piece& pc, int jj, int j, _Float16* wrow) {
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
}
template <int MT>
__device__ inline void sk_load_x(__amdgpu_buffer_rsrc_t rx, uint32_t xo, uint32_t row_step, f16x8 (&xa)[MT][4]) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int s = 0; s < 4; ++s) xa[i][s] = __builtin_bit_cast(f16x8, ld128(rx, xo + i * row_step + 64 * s));
}
template <int MT>
__device__ inline void sk_mma(const _Float16* wlane, const f16x8 (&xa)[MT][4], f32x4 (&acc)[MT]) {
    f16x8 wb[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) wb[s] = *reinterpret_cast<const f16x8*>(wlane + 32 * s);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[i][s], wb[s], acc[i], 0, 0, 0);
}
template <int MT>
__device__ inline void skinny_group(__amdgpu_buffer_rsrc_t rx, uint32_t xo, uint32_t row_step, const Piece& pc,
                                    int jj, int j, _Float16* wrow, const _Float16* wlane, f32x4 (&acc)[MT]) {
    f16x8 xa[MT][4];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int s = 0; s < 4; ++s) xa[i][s] = __builtin_bit_cast(f16x8, ld128(rx, xo + i * row_step + 64 * s));
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
    for (int s = 0; s < 4; ++s) wb[s] = *reinterpret_cast<const f16x8*>(wlane + 32 * s);
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int i = 0; i < MT; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[i][s], wb[s], acc[i], 0, 0, 0);
}

// Template parameters: MT token tiles of 16 (M <= 16 MT), WAVES wavefronts
// per workgroup, PF packets in flight per wavefront.
// SHARED: codes-only weights, A and B from the shared affine block.
template <int MT, int WAVES, int PF, bool SHARED>
__global__ __launch_bounds__(WAVES * 64) void skinny_kernel(const uint8_t* __restrict__ packed,
                                                           const uint8_t* __restrict__ affine, int affine_one,
                                                           const _Float16* __restrict__ x,
                                                           const float* __restrict__ inv_scale, void* y, int N,
                                                           int K, int M, int y_dtype) {
    __shared__ __attribute__((aligned(16))) _Float16 wtile[2 * WAVES * kSTile];
    __shared__ float red[WAVES][MT * 16][16];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int rb = blockIdx.x;
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
        make_rsrc(packed, static_cast<uint32_t>(N / kRowBlock) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(
        affine, SHARED ? static_cast<uint32_t>(affine_one ? 1 : (groups + 1) / 2) * kAffineRecordBytes : 0u);
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(M) * K * 2u);
    const uint32_t rowblk = static_cast<uint32_t>(rb) * groups * kBlockBytes;
    const int gend = 2 * (p0 + np);  // packets at or past this group read nothing
    auto load = [&](int p, int end, Piece& pc) {
        if constexpr (SHARED)
            load_packet_shared<true>(rw, ra, rowblk, p, end, affine_one, lane, pc);
        else
            load_packet<true>(rw, rowblk, p, end, lane, pc);
    };

    // Decode role: lane = packet slot (row beta = lane / 4, component j = lane % 4).
    const int j = lane & 3;
    _Float16* wrow = wtile + wave * kSTile + (lane >> 2) * kSRow;
    // Operand roles: weight operand row lane % 16, activation operand token
    // 16 i + lane % 16, both at columns 8 (lane / 16) + 32 s of the group.
    const _Float16* wlane = wtile + wave * kSTile + (lane & 15) * kSRow + 8 * (lane >> 4);
    const uint32_t row_step = 16u * K * 2u;
    const uint32_t xlane = (static_cast<uint32_t>(lane & 15) * K + 8 * (lane >> 4)) * 2u;

    f32x4 acc[MT];
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Packet ring: packet p0 + q lives in ring[q % PF].  Rounds of PF packets
    // run unconditionally; a packet past the run reads zeros and adds zero.
    Piece ring[PF];
#pragma unroll
    for (int i = 0; i < PF; ++i) load(p0 + i, gend, ring[i]);
    // two tiles per wavefront: group (q, 0) in tile 0, (q, 1) in tile 1; the
    // products of each group run one decode behind
    _Float16* wrow1 = wrow + WAVES * kSTile;
    const _Float16* wlane1 = wlane + WAVES * kSTile;
    f16x8 xp[MT][4];
    for (int q0 = 0; q0 < np; q0 += PF) {
#pragma unroll
        for (int i = 0; i < PF; ++i) {
            const int q = q0 + i;
            const uint32_t xo = q < np ? xlane + static_cast<uint32_t>(p0 + q) * 512u : kOutOfRange;
            f16x8 x0[MT][4];
            sk_load_x<MT>(rx, xo, row_step, x0);
            sk_decode<MT>(ring[i], 0, j, wrow);
            if (q > 0) sk_mma<MT>(wlane1, xp, acc);
            sk_load_x<MT>(rx, q < np ? xo + 256u : kOutOfRange, row_step, xp);
            sk_decode<MT>(ring[i], 1, j, wrow1);
            sk_mma<MT>(wlane, x0, acc);
            load(p0 + q + PF, gend, ring[i]);
        }
    }
    if (np > 0) sk_mma<MT>(wlane1, xp, acc);
    if (do_half) {
        Piece h;
        load(nfull, groups, h);
        skinny_group<MT>(rx, xlane + static_cast<uint32_t>(nfull) * 512u, row_step, h, 0, j, wrow, wlane, acc);
    }

    // Partial sums of the wavefronts meet in LDS.  D lane layout: row
    // lane % 16, tokens 16 i + 4 (lane / 16) + e.
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) red[wave][16 * i + 4 * (lane >> 4) + e][lane & 15] = acc[i][e];
    __syncthreads();
    for (int o = threadIdx.x; o < M * 16; o += WAVES * 64) {
        const int t = o >> 4, r = o & 15;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) s += red[w][t][r];
        if (inv_scale) s *= inv_scale[t];
        store_out(y, static_cast<int64_t>(t) * N + static_cast<int64_t>(rb) * kRowBlock + r, s, y_dtype);
    }
}

template <int MT, int WAVES, int PF, bool SHARED>
hipError_t launch_cfg(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one,
                      int64_t M, const _Float16* x, const float* inv_scale, void* y, int y_dtype, hipStream_t s) {
    hipLaunchKernelGGL((skinny_kernel<MT, WAVES, PF, SHARED>), dim3(static_cast<unsigned>(N / kRowBlock)),
                       dim3(WAVES * 64), 0, s, packed, affine, affine_one, x, inv_scale, y, static_cast<int>(N),
                       static_cast<int>(K), static_cast<int>(M), y_dtype);
    return hipGetLastError();
}

// 8 wavefronts per 16-row block with 2 packets in flight each, for every
// shape: swept on MI355X (16 tokens: 4096 x 4096 7.0 us, 4 wavefronts and 4
// in flight 7.4 us; 4096 x 11008 14.1 us, 8 and 8 18.2 us; deeper prefetch
// is slower because each activation load then waits behind more packet
// loads -- the vector-memory counter retires in order).  Two row blocks per
// workgroup (half the activation reads from L2) gained nothing at 16 tokens.
template <int MT>
hipError_t launch_mt(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one,
                     int64_t M, const _Float16* x, const float* inv_scale, void* y, int y_dtype, hipStream_t s) {
    if (affine) return launch_cfg<MT, 8, 2, true>(N, K, packed, affine, affine_one, M, x, inv_scale, y, y_dtype, s);
    return launch_cfg<MT, 8, 2, false>(N, K, packed, nullptr, 0, M, x, inv_scale, y, y_dtype, s);
}

}  // namespace

hipError_t launch_skinny(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one,
                         int64_t M, const _Float16* x, const float* inv_scale, void* y, int y_dtype,
                         hipStream_t s) {
    if (M <= 16) return launch_mt<1>(N, K, packed, affine, affine_one, M, x, inv_scale, y, y_dtype, s);
    return launch_mt<2>(N, K, packed, affine, affine_one, M, x, inv_scale, y, y_dtype, s);
}

}  // namespace unisvq
