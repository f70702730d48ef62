// Prefill product y = x * W_hat^T for any M on gfx950.
//
// For large M the dense product dominates.  Each workgroup owns a tile of
// BM tokens x 128 output rows and walks K one 128-column group (one affine
// parameter set per row, Sec. 3.1) at a time:
//   * the group's weights are decoded once per workgroup, w_hat = A q + B
//     (Eq. 4, vectors along K as in Eq. 8), on the matrix cores in fp32 (the
//     fp16 parameters times the exact small-integer codes), rounded once to
//     fp16 and written to LDS -- decoded weights never reach global memory;
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
#include <type_traits>

#include "common.hpp"
#include "decode.hpp"

namespace unisvq {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kNI = 8;                // 16-row output tiles per wavefront
constexpr int kBN = 16 * kNI;         // output rows per workgroup
constexpr int kLdsRow = kGroup + 16;  // halves per decoded row in LDS (32-byte pad: no bank conflicts)
constexpr int kWBuf = kBN * kLdsRow;  // halves per decoded-weight buffer
// LDS bytes per token row when a wavefront's outputs are staged for the
// stores (kBN values and 16 bytes of pad; multiples of 16 for 16-byte reads)
constexpr int kStagePitch16 = kBN * 2 + 16;
constexpr int kStagePitch32 = kBN * 4 + 16;
static_assert(kWaves * 32 * kStagePitch32 <= 2 * kWBuf * 2, "the staged outputs fit the decode buffers");

// One product of a (possibly batched) tiled launch; the products of a batch
// share M, the token tiling and the output dtype.
struct TileProb {
    const uint8_t* packed;
    const uint8_t* affine;
    const _Float16* x;
    const float* inv_scale;  // per token, or null
    const float* bias;       // per token (fold), or null
    float* partial;          // [splits][M][N] fp32 when splits > 1, else null
    void* y;
    int affine_one, N, K, n_tiles, splits, gps, wg_begin;
};

struct TileBatch {
    TileProb p[kMaxBatch];
    int count, M, m_tiles, y_dtype;
};

// The K-split products of a batch: their partial sums and outputs.
struct ReduceBatch {
    const float* partial[kMaxBatch];
    const float* inv_scale[kMaxBatch];
    const float* bias[kMaxBatch];
    void* y[kMaxBatch];
    int N[kMaxBatch], splits[kMaxBatch], wg_begin[kMaxBatch];
    int count, M, y_dtype;
};

// One 32-column step of the tile product: MI x kNI matrix-core tiles.
template <int MI>
__device__ inline void mma(const f16x8 (&xa)[MI], const f16x8 (&wb)[kNI], f32x4 (&acc)[MI][kNI]) {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int n = 0; n < kNI; ++n)
            acc[i][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(xa[i], wb[n], acc[i][n], 0, 0, 0);
}

__device__ inline void read_w(const _Float16* src, f16x8 (&wb)[kNI]) {
#pragma unroll
    for (int n = 0; n < kNI; ++n) wb[n] = *reinterpret_cast<const f16x8*>(src + 16 * n * kLdsRow);
}

template <int MI>
__device__ inline void load_x(__amdgpu_buffer_rsrc_t rx, uint32_t off, uint32_t row_step, f16x8 (&xa)[MI]) {
#pragma unroll
    for (int i = 0; i < MI; ++i) xa[i] = __builtin_bit_cast(f16x8, ld128(rx, off + i * row_step));
}

// One 32-column slice S of group g: prefetch activations two slices ahead
// and weights one slice ahead, decode a quarter of the next group (from
// pieces src, group jj of their packet), multiply.
template <int MI, int S, bool FOLD = false>
__device__ inline void slice(__amdgpu_buffer_rsrc_t rx, uint32_t xnext, uint32_t row_step, f16x8 (&xq)[4][MI],
                             f16x8 (&wb)[2][kNI], const _Float16* wsrc, bool decode_next, const Piece (&src)[2],
                             int jj, DecOps (&ops)[2], int j, _Float16* const (&wdst)[2], f32x4 (&acc)[MI][kNI]) {
    load_x<MI>(rx, xnext, row_step, xq[(S + 2) & 3]);
    if (S < 3) read_w(wsrc + 32 * (S + 1), wb[(S + 1) & 1]);
    // (After the last group this decodes zeros into the idle buffer: no
    // branch in the loop body.)
    (void)decode_next;
    {
        constexpr int r = S >> 1;  // local row block of this wavefront
        if ((S & 1) == 0) prepare<FOLD>(src[r], j, jj, ops[r]);
        constexpr int n0 = 4 * (S & 1);
        decode_vecs<n0 + 0, FOLD>(ops[r], wdst[r], j);
        decode_vecs<n0 + 1, FOLD>(ops[r], wdst[r], j);
        decode_vecs<n0 + 2, FOLD>(ops[r], wdst[r], j);
        decode_vecs<n0 + 3, FOLD>(ops[r], wdst[r], j);
    }
    mma<MI>(xq[S & 3], wb[S & 1], acc);
}

// The same for a format variant: the group's A rows and B (af) were loaded
// at the start of the group step.
template <int MI, int S, int BITS, int D>
__device__ inline void slice_var(__amdgpu_buffer_rsrc_t rx, uint32_t xnext, uint32_t row_step, f16x8 (&xq)[4][MI],
                                 f16x8 (&wb)[2][kNI], const _Float16* wsrc, const VarPiece (&src)[2], int jj,
                                 VarDecOps<BITS> (&ops)[2], const VarAffine<D>& af, int j,
                                 _Float16* const (&wdst)[2], f32x4 (&acc)[MI][kNI]) {
    load_x<MI>(rx, xnext, row_step, xq[(S + 2) & 3]);
    if (S < 3) read_w(wsrc + 32 * (S + 1), wb[(S + 1) & 1]);
    {
        constexpr int r = S >> 1;
        if ((S & 1) == 0) prepare_var<BITS>(src[r], j, jj, ops[r]);
        decode_var_half<BITS, D, S & 1>(ops[r], af, wdst[r], j);
    }
    mma<MI>(xq[S & 3], wb[S & 1], acc);
}

// Everything a group step needs besides its pieces.
template <int MI>
struct GemmState {
    __amdgpu_buffer_rsrc_t rx;
    uint32_t xbase, row_step;
    const _Float16* wlane;
    _Float16* wrow[2];
    int gend, j;  // end of this workgroup's group range
    __amdgpu_buffer_rsrc_t ra;  // shared affine block (format variants)
    int affine_one;
};

// Byte strides of the activation operands between 32-column slices: 64 in
// the row-major [M][K] layout, 1024 in the tiled layout (TX) of the bf16
// pre-pass, whose 1 KB tiles hold 16 tokens x 32 columns in the operand's
// lane order; a group is four slices.
template <bool TX>
constexpr uint32_t kSliceBytes = TX ? 1024u : 64u;

// Group g: products of buffer g & 1 (slices 0..3) while group g+1 is decoded
// from `src` (its group jj) into the other buffer.
template <int MI, bool TX = false, bool FOLD = false>
__device__ inline void group_step(const GemmState<MI>& st, int g, const Piece (&src)[2], int jj, f16x8 (&xq)[4][MI],
                                  f32x4 (&acc)[MI][kNI]) {
    constexpr uint32_t SL = kSliceBytes<TX>;
    const _Float16* wsrc = st.wlane + (g & 1) * kWBuf;
    _Float16* const wdst[2] = {st.wrow[0] + ((g + 1) & 1) * kWBuf, st.wrow[1] + ((g + 1) & 1) * kWBuf};
    const bool decode_next = g + 1 < st.gend;
    DecOps ops[2];
    f16x8 wb[2][kNI];
    read_w(wsrc, wb[0]);
    // activation slices 2, 3 of this group, 0, 1 of the next (or nothing)
    const uint32_t xoff = st.xbase + static_cast<uint32_t>(g) * (4 * SL);
    const uint32_t xn = decode_next ? xoff + 4 * SL : kOutOfRange;
    slice<MI, 0, FOLD>(st.rx, xoff + 2 * SL, st.row_step, xq, wb, wsrc, decode_next, src, jj, ops, st.j, wdst, acc);
    slice<MI, 1, FOLD>(st.rx, xoff + 3 * SL, st.row_step, xq, wb, wsrc, decode_next, src, jj, ops, st.j, wdst, acc);
    slice<MI, 2, FOLD>(st.rx, xn, st.row_step, xq, wb, wsrc, decode_next, src, jj, ops, st.j, wdst, acc);
    slice<MI, 3, FOLD>(st.rx, xn + SL, st.row_step, xq, wb, wsrc, decode_next, src, jj, ops, st.j, wdst, acc);
    __syncthreads();
}

// group_step for a format variant.
template <int MI, int BITS, int D>
__device__ inline void group_step_var(const GemmState<MI>& st, int g, const VarPiece (&src)[2], int jj,
                                      f16x8 (&xq)[4][MI], f32x4 (&acc)[MI][kNI]) {
    const _Float16* wsrc = st.wlane + (g & 1) * kWBuf;
    _Float16* const wdst[2] = {st.wrow[0] + ((g + 1) & 1) * kWBuf, st.wrow[1] + ((g + 1) & 1) * kWBuf};
    const bool decode_next = g + 1 < st.gend;
    VarAffine<D> af;
    load_var_affine<D>(st.ra, st.affine_one, g + 1, st.j, af);
    VarDecOps<BITS> ops[2];
    f16x8 wb[2][kNI];
    read_w(wsrc, wb[0]);
    const uint32_t xoff = st.xbase + static_cast<uint32_t>(g) * 256u;
    const uint32_t xn = decode_next ? xoff + 256u : kOutOfRange;
    slice_var<MI, 0, BITS, D>(st.rx, xoff + 128u, st.row_step, xq, wb, wsrc, src, jj, ops, af, st.j, wdst, acc);
    slice_var<MI, 1, BITS, D>(st.rx, xoff + 192u, st.row_step, xq, wb, wsrc, src, jj, ops, af, st.j, wdst, acc);
    slice_var<MI, 2, BITS, D>(st.rx, xn, st.row_step, xq, wb, wsrc, src, jj, ops, af, st.j, wdst, acc);
    slice_var<MI, 3, BITS, D>(st.rx, xn + 64u, st.row_step, xq, wb, wsrc, src, jj, ops, af, st.j, wdst, acc);
    __syncthreads();
}

// SHARED: codes-only weights, A and B from the shared affine block (one pair
// for the matrix when affine_one, else one per group); the decode is the same.
// BITS, D: code width and vector dimension; anything but 2, 4 is a format
// variant (always SHARED, variant layout and records).
// TX: activations in the tiled layout of the bf16 pre-pass (2-bit d = 4 formats).
// FOLD (with SHARED and TX): the Eq. 9 fold -- the activations were already
// multiplied by A (fold pre-pass), so the weights are the bare codes, and
// the per-token bias term sum_v x_v . B is added in the epilogue.
template <int MI, bool SHARED, int BITS = 2, int D = 4, bool TX = false, bool FOLD = false>
__global__ __launch_bounds__(kThreads) void gemm_kernel(const TileBatch tb) {
    __shared__ __attribute__((aligned(16))) _Float16 wsh[2 * kWBuf];
    // problem of this workgroup (uniform scalar selection)
    TileProb prob = tb.p[0];
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i)
        if (i < tb.count && static_cast<int>(blockIdx.x) >= tb.p[i].wg_begin) prob = tb.p[i];
    const uint8_t* packed = prob.packed;
    const uint8_t* affine = prob.affine;
    const _Float16* x = prob.x;
    const float* inv_scale = prob.inv_scale;
    const float* bias = prob.bias;
    float* partial = prob.partial;
    void* y = prob.y;
    const int affine_one = prob.affine_one, N = prob.N, K = prob.K, n_tiles = prob.n_tiles, splits = prob.splits,
              gps = prob.gps;
    const int M = tb.M, y_dtype = tb.y_dtype, m_tiles = tb.m_tiles;
    static_assert(!FOLD || (SHARED && TX && BITS == 2 && D == 4), "the fold runs on the tiled shared-pair kernel");
    constexpr int BM = kWaves * 16 * MI;
    constexpr bool kVar = BITS != 2 || D != 4;
    static_assert(!kVar || SHARED, "format variants keep their pairs in a shared block");
    typedef typename std::conditional<kVar, VarPiece, Piece>::type PieceT;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    // Tile of this workgroup: (K split, token tile, row tile), row tile
    // fastest.  Workgroups are dealt to the 8 XCDs round-robin; renumbering
    // them so that each XCD gets a contiguous run of tiles makes the tiles
    // that share activation rows share that XCD's L2.
    const int T = m_tiles * n_tiles * splits;
    int L = static_cast<int>(blockIdx.x) - prob.wg_begin;
    if ((T & 7) == 0) L = (L & 7) * (T >> 3) + (L >> 3);
    const int nt = L % n_tiles;
    const int mt = (L / n_tiles) % m_tiles;
    const int sp = L / (n_tiles * m_tiles);
    const int n0 = nt * kBN;
    const int tok0 = mt * BM + wave * 16 * MI;
    const int groups = K >> 7;
    // groups [gb, gend) of this split; gb is even (a packet boundary)
    const int gb = sp * gps;
    const int gend = min(groups, gb + gps);

    static_assert(!TX || !kVar, "the tiled activation layout serves the 2-bit d = 4 formats");
    constexpr uint32_t SL = kSliceBytes<TX>;
    // (the tiled layout pads the tokens to whole 16-token tiles with zeros)
    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(x, static_cast<uint32_t>(TX ? (M + 15) / 16 * 16 : M) * K * 2u);
    constexpr uint32_t kBlockBytes =
        kVar ? var_group_bytes(BITS) : (SHARED ? kCodeGroupBlockBytes : kGroupBlockBytes);
    constexpr uint32_t kRecBytes = kVar ? var_record_bytes(D) : kAffineRecordBytes;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(packed, static_cast<uint32_t>(N / kRowBlock) * groups * kBlockBytes);
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(
        affine, SHARED && !FOLD ? static_cast<uint32_t>(affine_one ? 1 : (groups + 1) / 2) * kRecBytes : 0u);
    // (FOLD: no pair is read -- the record loads fall outside the empty range)
    auto load = [&](uint32_t rowblk, int p, PieceT& pc) {
        if constexpr (kVar)
            load_packet_var<BITS>(rw, rowblk, p, gend, lane, pc);
        else if constexpr (SHARED)
            load_packet_shared(rw, ra, rowblk, p, gend, affine_one, lane, pc);
        else
            load_packet(rw, rowblk, p, gend, lane, pc);
    };

    // Decode role: this wavefront decodes local row blocks 2*wave and
    // 2*wave+1; lane (beta = lane / 4, j = lane % 4) = packet slot `lane`.
    GemmState<MI> st;
    const int beta = lane >> 2;
    st.j = lane & 3;
    st.gend = gend;
    if constexpr (kVar) {
        st.ra = ra;
        st.affine_one = affine_one;
    }
    uint32_t rowblk[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const int rb = (n0 >> 4) + 2 * wave + r;
        rowblk[r] = rb < (N >> 4) ? static_cast<uint32_t>(rb) * groups * kBlockBytes : kOutOfRange;
        st.wrow[r] = wsh + (16 * (2 * wave + r) + beta) * kLdsRow;
    }

    // Activation operand of tile i, 32-column slice s of group g, lane
    // (m = lane % 16, kb = lane / 16): 8 halves of token tok0 + 16 i + m at
    // column 128 g + 32 s + 8 kb.  Tokens past M read zeros.
    st.rx = rx;
    st.row_step = 16u * K * 2u;
    // (tiled: tile (tok0 / 16, slice) at ((tok0 / 16) * (K / 32) + slice) * 1 KB,
    // lane l's 16 bytes at 16 l; the next token tile is 16 * K * 2 bytes on,
    // as in the row-major layout)
    st.xbase = TX ? static_cast<uint32_t>(tok0 / 16) * static_cast<uint32_t>(K / 32) * 1024u + 16u * lane
                  : (static_cast<uint32_t>(tok0 + (lane & 15)) * K + 8 * (lane >> 4)) * 2u;
    // Weight operand of tile n: row 16 n + lane % 16, same columns.
    st.wlane = wsh + (lane & 15) * kLdsRow + 8 * (lane >> 4);

    f32x4 acc[MI][kNI];
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int n = 0; n < kNI; ++n) acc[i][n] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Packets two groups ahead of their decode: pa = packet q (groups 2q,
    // 2q+1), pb = packet q+1, pc = packet q+2 (loaded during group 2q+1).
    PieceT pa[2], pb[2], pc[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        load(rowblk[r], gb >> 1, pa[r]);
        load(rowblk[r], (gb >> 1) + 1, pb[r]);
    }
    // Prologue: group gb into buffer gb & 1 (= 0).
    if constexpr (kVar) {
        VarAffine<D> af;
        load_var_affine<D>(ra, affine_one, gb, st.j, af);
        VarDecOps<BITS> ops;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            prepare_var<BITS>(pa[r], st.j, 0, ops);
            decode_var_half<BITS, D, 0>(ops, af, st.wrow[r], st.j);
            decode_var_half<BITS, D, 1>(ops, af, st.wrow[r], st.j);
        }
    } else {
        DecOps ops;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            prepare<FOLD>(pa[r], st.j, 0, ops);
            decode_vecs<0, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<1, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<2, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<3, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<4, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<5, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<6, FOLD>(ops, st.wrow[r], st.j);
            decode_vecs<7, FOLD>(ops, st.wrow[r], st.j);
        }
    }
    f16x8 xq[4][MI];
    load_x<MI>(rx, st.xbase + static_cast<uint32_t>(gb) * (4 * SL), st.row_step, xq[0]);
    load_x<MI>(rx, st.xbase + static_cast<uint32_t>(gb) * (4 * SL) + SL, st.row_step, xq[1]);
    __syncthreads();

    int g = gb;
    if constexpr (kVar) {
        for (; g + 1 < gend; g += 2) {
            const int q = g >> 1;
            group_step_var<MI, BITS, D>(st, g, pa, 1, xq, acc);
#pragma unroll
            for (int r = 0; r < 2; ++r) load(rowblk[r], q + 2, pc[r]);
            group_step_var<MI, BITS, D>(st, g + 1, pb, 0, xq, acc);
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                pa[r] = pb[r];
                pb[r] = pc[r];
            }
        }
        if (g < gend) group_step_var<MI, BITS, D>(st, g, pa, 1, xq, acc);
    } else {
        for (; g + 1 < gend; g += 2) {
            const int q = g >> 1;
            group_step<MI, TX, FOLD>(st, g, pa, 1, xq, acc);  // decodes group 2q+1 (packet q)
#pragma unroll
            for (int r = 0; r < 2; ++r) load(rowblk[r], q + 2, pc[r]);
            group_step<MI, TX, FOLD>(st, g + 1, pb, 0, xq, acc);  // decodes group 2q+2 (packet q+1)
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                pa[r] = pb[r];
                pb[r] = pc[r];
            }
        }
        if (g < gend) group_step<MI, TX, FOLD>(st, g, pa, 1, xq, acc);  // last group (nothing left to decode)
    }

    // Epilogue.  D lane layout: output row 16 n + lane % 16, tokens
    // 16 i + 4 (lane / 16) + e.  With a K split the fp32 partial sums go to
    // partial[split][M][N] and a second kernel adds them up.  Two- and
    // four-byte stores of that layout scatter a token's rows over four
    // segments per instruction; so the outputs (not the partial sums: staging
    // their sixteen-lane runs of 64 bytes measured slower) go through LDS: each
    // wavefront puts its 16 MI tokens x 128 rows there, converted (the
    // buffers are free after the last group's barrier), and writes them back
    // as 16-byte pieces of token rows.  An output not 16-byte aligned takes
    // the element stores.
    if (partial == nullptr && (reinterpret_cast<uintptr_t>(y) & 15) == 0) {  // uniform
        const int esz = y_dtype == UNISVQ_F32 ? 4 : 2;
        unsigned char* const dst = static_cast<unsigned char*>(y);
        const int pitch = esz == 2 ? kStagePitch16 : kStagePitch32;  // bytes per token row in LDS
        unsigned char* const stage = reinterpret_cast<unsigned char*>(wsh) + wave * 16 * MI * pitch;
#pragma unroll
        for (int i = 0; i < MI; ++i) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int tl = 16 * i + 4 * (lane >> 4) + e;  // token of the wavefront's tile
                const int t = tok0 + tl;
                const float sc = inv_scale && t < M ? inv_scale[t] : 1.0f;
                const float bt = bias && t < M ? bias[t] : 0.0f;
#pragma unroll
                for (int n = 0; n < kNI; ++n) {
                    unsigned char* const at = stage + tl * pitch + (16 * n + (lane & 15)) * esz;
                    const float v = bias ? acc[i][n][e] * sc + bt : acc[i][n][e] * sc;
                    if (y_dtype == UNISVQ_F32)
                        *reinterpret_cast<float*>(at) = v;
                    else if (y_dtype == UNISVQ_F16)
                        *reinterpret_cast<_Float16*>(at) = static_cast<_Float16>(v);
                    else
                        *reinterpret_cast<__bf16*>(at) = static_cast<__bf16>(v);
                }
            }
        }
        __syncthreads();
        // 16-byte pieces: kBN * esz / 16 per token row; rows come in whole
        // pieces (N and the row tiles are multiples of 16)
        const int per = kBN * esz / 16;
        for (int k = lane; k < 16 * MI * per; k += 64) {
            const int tl = k / per, c = k - tl * per;
            const int t = tok0 + tl;
            const int row = n0 + c * (16 / esz);
            if (t < M && row < N)
                *reinterpret_cast<uint4*>(dst + (static_cast<int64_t>(t) * N + row) * esz) =
                    *reinterpret_cast<const uint4*>(stage + tl * pitch + 16 * c);
        }
        return;
    }
#pragma unroll
    for (int i = 0; i < MI; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int t = tok0 + 16 * i + 4 * (lane >> 4) + e;
            if (t >= M) continue;
            const float sc = inv_scale ? inv_scale[t] : 1.0f;
            const float bt = bias ? bias[t] : 0.0f;
#pragma unroll
            for (int n = 0; n < kNI; ++n) {
                const int row = n0 + 16 * n + (lane & 15);
                if (row >= N) continue;
                if (partial)
                    partial[(static_cast<int64_t>(sp) * M + t) * N + row] = acc[i][n][e];
                else
                    store_out(y, static_cast<int64_t>(t) * N + row,
                              bias ? acc[i][n][e] * sc + bt : acc[i][n][e] * sc, y_dtype);
            }
        }
    }
}

// y = (sum over the K splits of the partial sums, in split order) *
// per-token scale (+ bias), four outputs per thread (N is a multiple of 16),
// for every split product of a batch; the loads of eight splits are in
// flight at once.
constexpr int kReduceChunk = 8;

__global__ __launch_bounds__(256) void reduce_splits_kernel(const ReduceBatch r) {
    const int bid = blockIdx.x;
    int pi = 0;
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i)
        if (i < r.count && bid >= r.wg_begin[i]) pi = i;
    const int N = r.N[pi], splits = r.splits[pi];
    const int64_t total4 = static_cast<int64_t>(r.M) * N / 4;
    const int64_t i4 = static_cast<int64_t>(bid - r.wg_begin[pi]) * 256 + threadIdx.x;
    if (i4 >= total4) return;
    const f32x4* p = reinterpret_cast<const f32x4*>(r.partial[pi]) + i4;
    f32x4 s = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < splits; k0 += kReduceChunk) {
        f32x4 q[kReduceChunk];
#pragma unroll
        for (int k = 0; k < kReduceChunk; ++k) q[k] = k0 + k < splits ? p[(k0 + k) * total4] : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < kReduceChunk; ++k)
            if (k0 + k < splits) s += q[k];
    }
    const int64_t e0 = 4 * i4;
    const int t = static_cast<int>(e0 / N);
    const float sc = r.inv_scale[pi] ? r.inv_scale[pi][t] : 1.0f;
    void* y = r.y[pi];
    if (r.bias[pi]) {
        const float bt = r.bias[pi][t];
#pragma unroll
        for (int c = 0; c < 4; ++c) store_out(y, e0 + c, s[c] * sc + bt, r.y_dtype);
        return;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) store_out(y, e0 + c, s[c] * sc, r.y_dtype);
}

// bf16 activations -> fp16 with a power-of-two scale per token (see the top
// of the file).  One workgroup per token row; the row is read once and held
// in registers (CH chunks of 8 values per thread, CH * 2048 >= K).
template <int CH>
__global__ __launch_bounds__(256) void scale_rows_kernel(const uint16_t* __restrict__ xb, int K,
                                                         _Float16* __restrict__ xh, float* __restrict__ inv_scale) {
    __shared__ float wmax[4];
    const int t = blockIdx.x;
    const uint16_t* row = xb + static_cast<size_t>(t) * K;
    _Float16* out = xh + static_cast<size_t>(t) * K;
    const int chunks = K >> 3;  // 8 values per 16-byte chunk
    auto val = [](uint32_t bits16) { return __builtin_bit_cast(float, bits16 << 16); };
    uint4 v[CH];
    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = threadIdx.x + 256 * i;
        v[i] = c < chunks ? *reinterpret_cast<const uint4*>(row + 8 * c) : uint4{0u, 0u, 0u, 0u};
        const uint32_t w[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
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
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int c = threadIdx.x + 256 * i;
        if (c >= chunks) break;
        const uint32_t w[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
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

// The same pre-pass writing the tiled layout of the prefill kernel: 1 KB
// tiles of 16 tokens x 32 columns in the operand's lane order (chunk c of
// token t at tile (t / 16, c / 4), lane t % 16 + 16 (c % 4)), tokens padded
// to whole tiles with zero rows.  Tokens 0-7 of a tile fill its 128-byte
// lines 0, 2, 4, 6 and tokens 8-15 lines 1, 3, 5, 7, so one workgroup (16
// wavefronts) per half tile still stores whole lines: lane l handles token
// l % 8 of the half, chunk (l / 8) % 4 of slice 2 (w + 16 i) + l / 32.  The
// half tile's rows are read twice: once for the token maxima (over the eight
// lanes that share a row by lane shuffles, then over the wavefronts in LDS),
// then again, from the L2, for the conversion; nothing is held in
// registers, so any K.
__global__ __launch_bounds__(1024) void scale_tiles_kernel(const uint16_t* __restrict__ xb, int K, int M,
                                                           _Float16* __restrict__ xh, float* __restrict__ inv_scale) {
    __shared__ float wmax[16][8];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int r = lane & 7, q = (lane >> 3) & 3, ps = lane >> 5;
    const int tile = blockIdx.x >> 1, h = blockIdx.x & 1;
    const int t = 16 * tile + 8 * h + r;
    const bool real = t < M;
    const int slices = K >> 5;
    const uint16_t* row = xb + static_cast<size_t>(real ? t : 0) * K + 8 * q;
    auto val = [](uint32_t bits16) { return __builtin_bit_cast(float, bits16 << 16); };
    float mx = 0.f;
    if (real) {
#pragma unroll 4
        for (int sl = 2 * w + ps; sl < slices; sl += 32) {
            const uint4 v = *reinterpret_cast<const uint4*>(row + 32 * sl);
            const uint32_t wd[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) mx = fmaxf(mx, fmaxf(fabsf(val(wd[e] & 0xffffu)), fabsf(val(wd[e] >> 16))));
        }
    }
    mx = fmaxf(mx, __shfl_xor(mx, 8));
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    if (lane < 8) wmax[w][r] = mx;
    __syncthreads();
    mx = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) mx = fmaxf(mx, wmax[j][r]);
    int s = 0;
    if (mx > 0.f && mx <= 3.4e38f) {
        int e;
        frexpf(mx, &e);  // mx in [2^(e-1), 2^e)
        s = min(max(15 - e, -126), 126);
    }
    _Float16* out = xh + static_cast<size_t>(tile) * slices * 512 + 8 * (8 * h + r + 16 * q);
#pragma unroll 4
    for (int sl = 2 * w + ps; sl < slices; sl += 32) {
        const uint4 v = real ? *reinterpret_cast<const uint4*>(row + 32 * sl) : uint4{0u, 0u, 0u, 0u};
        const uint32_t wd[4] = {v.x, v.y, v.z, v.w};
        f16x8 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            o[2 * e] = static_cast<_Float16>(ldexpf(val(wd[e] & 0xffffu), s));
            o[2 * e + 1] = static_cast<_Float16>(ldexpf(val(wd[e] >> 16), s));
        }
        *reinterpret_cast<f16x8*>(out + static_cast<size_t>(sl) * 512) = o;
    }
    if (w == 0 && lane < 8 && real) inv_scale[t] = ldexpf(1.0f, -s);
}

// The Eq. 9 fold for row-shared pairs, as a pre-pass of the tiled product:
// for every vector v (four consecutive columns) of group g the activations
// become x'_v = A_g^T x_v (x'_b = sum_a A[a][b] x_a, fp32 from the fp16
// pair), scaled per token by a power of two 2^s so that the token's largest
// |x'| lies in [2^14, 2^15), rounded to fp16 and written in the tiled layout;
// the token's bias term c_t = sum_v x_v . B_g is summed in fp32 (in a fixed
// order: per lane along its slices, lane shuffles, then the wavefronts).
// The product then multiplies x' by the bare codes:
//     y = 2^-s (x' Q^T) + c.
// Same half-tile organisation and two reads of the rows as
// scale_tiles_kernel; the pair of group g is read from its record (A column
// b at 16 b + 8 (g % 2), B[a] at 64 + 4 a + 2 (g % 2); record 0 for one pair
// per matrix).  BF16: x holds bf16 bits, else fp16.
template <bool BF16>
__global__ __launch_bounds__(1024) void fold_tiles_kernel(const uint16_t* __restrict__ xb, int K, int M,
                                                          const uint8_t* __restrict__ affine, int affine_one,
                                                          _Float16* __restrict__ xh, float* __restrict__ inv_scale,
                                                          float* __restrict__ bias) {
    __shared__ float wmax[16][8], wsum[16][8];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int r = lane & 7, q = (lane >> 3) & 3, ps = lane >> 5;
    const int tile = blockIdx.x >> 1, h = blockIdx.x & 1;
    const int t = 16 * tile + 8 * h + r;
    const bool real = t < M;
    const int slices = K >> 5;
    const uint16_t* row = xb + static_cast<size_t>(real ? t : 0) * K + 8 * q;
    auto val = [](uint32_t bits16) -> float {
        if constexpr (BF16) return __builtin_bit_cast(float, bits16 << 16);
        else return h2f(bits16);
    };
    // the lane's two vectors of slice sl: x' (8 values) and their part of c_t
    auto fold = [&](int sl, float (&xp)[8], float& cs) {
        const int g = sl >> 2;  // the same for both slices of a wavefront step
        const uint8_t* rec = affine + static_cast<size_t>(affine_one ? 0 : g >> 1) * kAffineRecordBytes;
        const int jj = g & 1;
        float A[4][4], Bv[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const uint2 col = *reinterpret_cast<const uint2*>(rec + 16 * b + 8 * jj);
            A[0][b] = h2f(col.x & 0xffffu);
            A[1][b] = h2f(col.x >> 16);
            A[2][b] = h2f(col.y & 0xffffu);
            A[3][b] = h2f(col.y >> 16);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a) Bv[a] = h2f(*reinterpret_cast<const uint16_t*>(rec + kRecordBiasOff + 4 * a + 2 * jj));
        const uint4 v = real ? *reinterpret_cast<const uint4*>(row + 32 * sl) : uint4{0u, 0u, 0u, 0u};
        const uint32_t wd[4] = {v.x, v.y, v.z, v.w};
        float xv[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            xv[2 * e] = val(wd[e] & 0xffffu);
            xv[2 * e + 1] = val(wd[e] >> 16);
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                float acc = 0.f;
#pragma unroll
                for (int a = 0; a < 4; ++a) acc = fmaf(A[a][b], xv[4 * u + a], acc);
                xp[4 * u + b] = acc;
            }
#pragma unroll
            for (int a = 0; a < 4; ++a) cs = fmaf(Bv[a], xv[4 * u + a], cs);
        }
    };
    float mx = 0.f, cs = 0.f;
    for (int sl = 2 * w + ps; sl < slices; sl += 32) {
        float xp[8];
        fold(sl, xp, cs);
#pragma unroll
        for (int e = 0; e < 8; ++e) mx = fmaxf(mx, fabsf(xp[e]));
    }
#pragma unroll
    for (int off = 8; off < 64; off <<= 1) {
        mx = fmaxf(mx, __shfl_xor(mx, off));
        cs += __shfl_xor(cs, off);
    }
    if (lane < 8) {
        wmax[w][r] = mx;
        wsum[w][r] = cs;
    }
    __syncthreads();
    mx = 0.f;
    cs = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        mx = fmaxf(mx, wmax[j][r]);
        cs += wsum[j][r];
    }
    int s = 0;
    if (mx > 0.f && mx <= 3.4e38f) {
        int e;
        frexpf(mx, &e);  // mx in [2^(e-1), 2^e)
        s = min(max(15 - e, -126), 126);
    }
    _Float16* out = xh + static_cast<size_t>(tile) * slices * 512 + 8 * (8 * h + r + 16 * q);
    for (int sl = 2 * w + ps; sl < slices; sl += 32) {
        float xp[8], unused = 0.f;
        fold(sl, xp, unused);
        f16x8 o;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[e] = static_cast<_Float16>(ldexpf(xp[e], s));
        *reinterpret_cast<f16x8*>(out + static_cast<size_t>(sl) * 512) = o;
    }
    if (w == 0 && lane < 8 && real) {
        inv_scale[t] = ldexpf(1.0f, -s);
        bias[t] = cs;
    }
}

template <bool TILED>
hipError_t launch_scale(int64_t K, int64_t M, const uint16_t* x, _Float16* xh, float* inv, hipStream_t s) {
    if (K > 65536) return hipErrorInvalidValue;  // not supported for bf16 activations
    const int k = static_cast<int>(K);
    if (TILED) {
        hipLaunchKernelGGL(scale_tiles_kernel, dim3(static_cast<unsigned>((M + 15) / 16 * 2)), dim3(1024), 0, s, x, k,
                           static_cast<int>(M), xh, inv);
        return hipGetLastError();
    }
    const int64_t per = (K / 8 + 255) / 256;  // chunks per thread
    const dim3 grid(static_cast<unsigned>(M)), block(256);
    if (per <= 1) hipLaunchKernelGGL(scale_rows_kernel<1>, grid, block, 0, s, x, k, xh, inv);
    else if (per <= 2) hipLaunchKernelGGL(scale_rows_kernel<2>, grid, block, 0, s, x, k, xh, inv);
    else if (per <= 4) hipLaunchKernelGGL(scale_rows_kernel<4>, grid, block, 0, s, x, k, xh, inv);
    else if (per <= 8) hipLaunchKernelGGL(scale_rows_kernel<8>, grid, block, 0, s, x, k, xh, inv);
    else if (per <= 16) hipLaunchKernelGGL(scale_rows_kernel<16>, grid, block, 0, s, x, k, xh, inv);
    else hipLaunchKernelGGL(scale_rows_kernel<32>, grid, block, 0, s, x, k, xh, inv);
    return hipGetLastError();
}

// Tiling of one product: token tiles of 64 (M <= 64) or 128 tokens, row
// tiles of 128; when that leaves fewer than 256 workgroups the K range is
// split (at packet boundaries) until there are about 256, and into runs of
// at most 4 packets (swept at 64 tokens: 11008 x 4096 26.0 us with 4 splits,
// 27.5 with 3; 4096 x 11008 24.7 us with 15 splits, 26.3 with 8).
struct GemmPlan {
    int mi, m_tiles, n_tiles, splits, gps;
};

GemmPlan plan_gemm(int64_t N, int64_t K, int64_t M) {
    GemmPlan p;
    p.mi = M > 64 ? 2 : 1;
    const int64_t bm = kWaves * 16 * p.mi;
    p.m_tiles = static_cast<int>((M + bm - 1) / bm);
    p.n_tiles = static_cast<int>((N + kBN - 1) / kBN);
    const int groups = static_cast<int>(K / kGroup);
    p.splits = 1;
    p.gps = groups;
    const int64_t tiles = static_cast<int64_t>(p.m_tiles) * p.n_tiles;
    if (tiles < 256 && groups >= 4) {
        const int packets = (groups + 1) / 2;
        const int fill = static_cast<int>((256 + tiles - 1) / tiles);
        const int want = fill > (packets + 3) / 4 ? fill : (packets + 3) / 4;
        const int s = want < packets ? want : packets;
        p.gps = 2 * ((packets + s - 1) / s);
        p.splits = (groups + p.gps - 1) / p.gps;
    }
    return p;
}

size_t align256(size_t b) { return (b + 255) & ~size_t{255}; }

// Above 16 tokens the small-batch kernel takes two token tiles and one row
// block per workgroup, and beats the tiled product only on narrow batches:
// 7B decoder step at 20 / 24 / 32 tokens, per launch, small-batch against
// tiled: o (4096 rows) 10.0 / 10.6 / 11.9 against 15.3 / 15.5 / 16.1 us, down
// (4096 rows) 21.6 / 22.8 / 26.3 against 24.8 / 25.3 / 25.7, q+k+v (12288)
// 25.2 / 27.2 / 31.1 against 24.3 / 24.5 / 24.8, gate+up (22016) 47.9 / 51.9 /
// 59.9 against 37.2 / 38.7 / 39.0.  So from 17 to 32 tokens a batch goes to
// the small-batch kernel only when it has fewer than this many 128-row tiles.
constexpr int64_t kSkinnyWideMaxTiles = 64;
// The small-batch kernel for M tokens over a batch of `rows` output rows in all.
inline bool use_skinny(int64_t M, int64_t rows) {
    return M <= 16 || (M <= kSkinnyMaxM && (rows + 127) / 128 < kSkinnyWideMaxTiles);
}

size_t partial_bytes(int64_t N, int64_t K, int64_t M) {
    if (M <= 16) return 0;  // the small-batch kernel needs no partials (above: either kernel, see use_skinny)
    const GemmPlan p = plan_gemm(N, K, M);
    return p.splits > 1 ? static_cast<size_t>(p.splits) * M * N * 4 : 0;
}

// Launch a batch of products (one kernel, plus one reduction kernel for
// those split along K).
template <int MI, bool SHARED, int BITS = 2, int D = 4, bool TX = false, bool FOLD = false>
hipError_t launch_tile_batch(TileBatch& b, hipStream_t s) {
    ReduceBatch r{};
    int blocks = 0, rblocks = 0, nred = 0;
    for (int i = 0; i < b.count; ++i) {
        TileProb& q = b.p[i];
        if (q.splits > 1 && q.partial == nullptr) return hipErrorInvalidValue;  // never launch without the partials
        if (q.splits <= 1) q.partial = nullptr;
        q.wg_begin = blocks;
        blocks += b.m_tiles * q.n_tiles * q.splits;
        if (q.splits > 1) {
            r.partial[nred] = q.partial;
            r.inv_scale[nred] = q.inv_scale;
            r.bias[nred] = q.bias;
            r.y[nred] = q.y;
            r.N[nred] = q.N;
            r.splits[nred] = q.splits;
            r.wg_begin[nred] = rblocks;
            rblocks += static_cast<int>((static_cast<int64_t>(b.M) * q.N / 4 + 255) / 256);
            ++nred;
        }
    }
    hipLaunchKernelGGL((gemm_kernel<MI, SHARED, BITS, D, TX, FOLD>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kThreads), 0, s, b);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    if (nred > 0) {
        r.count = nred;
        r.M = b.M;
        r.y_dtype = b.y_dtype;
        hipLaunchKernelGGL(reduce_splits_kernel, dim3(static_cast<unsigned>(rblocks)), dim3(256), 0, s, r);
    }
    return hipGetLastError();
}

template <int MI, bool SHARED, int BITS = 2, int D = 4, bool TX = false, bool FOLD = false>
hipError_t launch_tiles(const GemmPlan& p, int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine,
                        int affine_one, int64_t M, const _Float16* x, const float* inv_scale, void* y,
                        int y_dtype, float* partial, hipStream_t s, const float* bias = nullptr) {
    TileBatch b{};
    b.p[0] = TileProb{packed, affine, x, inv_scale, bias, partial, y, affine_one, static_cast<int>(N),
                      static_cast<int>(K), p.n_tiles, p.splits, p.gps, 0};
    b.count = 1;
    b.M = static_cast<int>(M);
    b.m_tiles = p.m_tiles;
    b.y_dtype = y_dtype;
    return launch_tile_batch<MI, SHARED, BITS, D, TX, FOLD>(b, s);
}

}  // namespace

size_t gemm_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype) {
    size_t b = 0;
    // (above 16 tokens the fp16 copy may be the tiled one: tokens padded to 16)
    const int64_t mx = M > 16 ? (M + 15) / 16 * 16 : M;
    if (x_dtype == UNISVQ_BF16) b += align256(static_cast<size_t>(mx) * K * 2) + align256(static_cast<size_t>(M) * 4);
    return b + partial_bytes(N, K, M);
}

size_t gemm_var_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype) {
    size_t b = 0;
    if (x_dtype == UNISVQ_BF16) b += align256(static_cast<size_t>(M) * K * 2) + align256(static_cast<size_t>(M) * 4);
    const GemmPlan p = plan_gemm(N, K, M);
    return b + (p.splits > 1 ? static_cast<size_t>(p.splits) * M * N * 4 : 0);
}

namespace {

// Tiles of one (sliced) product for a format variant.
template <int BITS, int D>
hipError_t launch_tiles_var(const GemmPlan& p, int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine,
                            int affine_one, int64_t M, const _Float16* x, const float* inv_scale, void* y,
                            int y_dtype, float* partial, hipStream_t s) {
    return p.mi == 2 ? launch_tiles<2, true, BITS, D>(p, N, K, packed, affine, affine_one, M, x, inv_scale, y,
                                                      y_dtype, partial, s)
                     : launch_tiles<1, true, BITS, D>(p, N, K, packed, affine, affine_one, M, x, inv_scale, y,
                                                      y_dtype, partial, s);
}

// bits, d: 2, 4 for the main formats; a format variant otherwise (every M
// goes to the tiled kernel).
int gemm_common(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one, int64_t M,
                const void* x, int x_dtype, void* y, int y_dtype, void* workspace, hipStream_t s, int bits = 2,
                int d = 4) {
    const bool var = bits != 2 || d != 4;
    if (!var && M <= kGemvMaxM) {
        GemvProblem g{packed, x, y, static_cast<int>(N), static_cast<int>(K), 0, affine, affine_one};
        const int st = launch_gemv_batch(&g, 1, M, x_dtype, y_dtype, s);
        if (st != UNISVQ_EUNSUP) return st;  // else K too long for its LDS: the small-batch kernel
    }
    const _Float16* xh = static_cast<const _Float16*>(x);
    const float* inv = nullptr;
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    // bf16 activations for the tiled kernel (2-bit d = 4, M above the
    // small-batch range) go through the pre-pass that writes the tiled layout
    const bool skinny = !var && use_skinny(M, N);
    const bool tiled = x_dtype == UNISVQ_BF16 && !var && !skinny;
    if (x_dtype == UNISVQ_BF16) {
        _Float16* wxh = reinterpret_cast<_Float16*>(ws);
        ws += align256(static_cast<size_t>(tiled ? (M + 15) / 16 * 16 : M) * K * 2);
        float* winv = reinterpret_cast<float*>(ws);
        ws += align256(static_cast<size_t>(M) * 4);
        const hipError_t e = tiled ? launch_scale<true>(K, M, static_cast<const uint16_t*>(x), wxh, winv, s)
                                   : launch_scale<false>(K, M, static_cast<const uint16_t*>(x), wxh, winv, s);
        if (e != hipSuccess) return K > 65536 ? UNISVQ_EUNSUP : UNISVQ_EHIP;
        xh = wxh;
        inv = winv;
    }
    if (skinny)
        return launch_skinny(N, K, packed, affine, affine_one, M, xh, inv, y, y_dtype, s) == hipSuccess
                   ? UNISVQ_OK
                   : UNISVQ_EHIP;
    float* partial = reinterpret_cast<float*>(ws);
    // The activation buffer is addressed with 32-bit offsets: slice M.  The
    // workspace was sized for the whole product, which has far more than 256
    // tiles when it needs slicing; so no slice (the last one may be small)
    // splits K.
    const int64_t max_rows = kMaxBufferBytes / (2 * K) / 256 * 256;
    const bool sliced = M > max_rows;
    for (int64_t m0 = 0; m0 < M; m0 += max_rows) {
        const int64_t mc = M - m0 < max_rows ? M - m0 : max_rows;
        const _Float16* xs = xh + m0 * K;
        const float* is = inv ? inv + m0 : nullptr;
        void* ys = static_cast<uint8_t*>(y) + m0 * N * (y_dtype == UNISVQ_F32 ? 4 : 2);
        GemmPlan p = plan_gemm(N, K, mc);
        if (sliced) {
            p.splits = 1;
            p.gps = static_cast<int>(K / kGroup);
        }
        hipError_t e;
        if (var && bits == 3 && d == 4)
            e = launch_tiles_var<3, 4>(p, N, K, packed, affine, affine_one, mc, xs, is, ys, y_dtype, partial, s);
        else if (var && bits == 2 && d == 8)
            e = launch_tiles_var<2, 8>(p, N, K, packed, affine, affine_one, mc, xs, is, ys, y_dtype, partial, s);
        else if (var && bits == 3 && d == 8)
            e = launch_tiles_var<3, 8>(p, N, K, packed, affine, affine_one, mc, xs, is, ys, y_dtype, partial, s);
        else if (var)
            return UNISVQ_EUNSUP;
        else if (affine && tiled)
            e = p.mi == 2 ? launch_tiles<2, true, 2, 4, true>(p, N, K, packed, affine, affine_one, mc, xs, is, ys,
                                                              y_dtype, partial, s)
                          : launch_tiles<1, true, 2, 4, true>(p, N, K, packed, affine, affine_one, mc, xs, is, ys,
                                                              y_dtype, partial, s);
        else if (affine)
            e = p.mi == 2 ? launch_tiles<2, true>(p, N, K, packed, affine, affine_one, mc, xs, is, ys, y_dtype, partial, s)
                          : launch_tiles<1, true>(p, N, K, packed, affine, affine_one, mc, xs, is, ys, y_dtype, partial, s);
        else if (tiled)
            e = p.mi == 2 ? launch_tiles<2, false, 2, 4, true>(p, N, K, packed, nullptr, 0, mc, xs, is, ys, y_dtype,
                                                               partial, s)
                          : launch_tiles<1, false, 2, 4, true>(p, N, K, packed, nullptr, 0, mc, xs, is, ys, y_dtype,
                                                               partial, s);
        else
            e = p.mi == 2 ? launch_tiles<2, false>(p, N, K, packed, nullptr, 0, mc, xs, is, ys, y_dtype, partial, s)
                          : launch_tiles<1, false>(p, N, K, packed, nullptr, 0, mc, xs, is, ys, y_dtype, partial, s);
        if (e != hipSuccess) return UNISVQ_EHIP;
    }
    return UNISVQ_OK;
}

}  // namespace

int launch_gemm(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, void* workspace, hipStream_t s) {
    return gemm_common(N, K, packed, nullptr, 0, M, x, x_dtype, y, y_dtype, workspace, s);
}

size_t gemm_batch_workspace_bytes(const GemmBatchProblem* probs, int count, int64_t M, int x_dtype) {
    size_t b = 0;
    for (int i = 0; i < count; ++i) b += align256(gemm_workspace_bytes(probs[i].N, probs[i].K, M, x_dtype));
    return b;
}

int launch_gemm_batch(const GemmBatchProblem* probs, int count, int64_t M, int x_dtype, int y_dtype, void* workspace,
                      hipStream_t s) {
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    bool sliced = false;
    for (int i = 0; i < count; ++i) sliced = sliced || M > kMaxBufferBytes / (2 * probs[i].K) / 256 * 256;
    int64_t rows = 0;
    for (int i = 0; i < count; ++i) rows += probs[i].N;
    const bool skinny = use_skinny(M, rows);
    if (!skinny && sliced) {
        // activations above 2 GiB: one product at a time, in token slices
        for (int i = 0; i < count; ++i) {
            const GemmBatchProblem& q = probs[i];
            const int st = gemm_common(q.N, q.K, q.packed, nullptr, 0, M, q.x, x_dtype, q.y, y_dtype, ws, s);
            if (st != UNISVQ_OK) return st;
            ws += align256(gemm_workspace_bytes(q.N, q.K, M, x_dtype));
        }
        return UNISVQ_OK;
    }
    if (!skinny) {
        // one tiled launch (and one reduction) for the whole batch: the bf16
        // pre-pass of each problem into its slice, then the tiles planned
        // over the batch (a K split only as far as the batch's tiles leave
        // CUs idle; never more splits than the problem alone would take, so
        // the partials fit its slice)
        const GemmPlan p0 = plan_gemm(probs[0].N, probs[0].K, M);
        TileBatch b{};
        b.count = count;
        b.M = static_cast<int>(M);
        b.m_tiles = p0.m_tiles;
        b.y_dtype = y_dtype;
        int64_t tiles = 0;
        for (int i = 0; i < count; ++i) tiles += static_cast<int64_t>(p0.m_tiles) * ((probs[i].N + kBN - 1) / kBN);
        for (int i = 0; i < count; ++i) {
            const GemmBatchProblem& q = probs[i];
            uint8_t* slice = ws;
            ws += align256(gemm_workspace_bytes(q.N, q.K, M, x_dtype));
            const _Float16* xh = static_cast<const _Float16*>(q.x);
            const float* inv = nullptr;
            if (x_dtype == UNISVQ_BF16) {
                _Float16* wxh = reinterpret_cast<_Float16*>(slice);
                slice += align256(static_cast<size_t>((M + 15) / 16 * 16) * q.K * 2);
                float* winv = reinterpret_cast<float*>(slice);
                slice += align256(static_cast<size_t>(M) * 4);
                if (launch_scale<true>(q.K, M, static_cast<const uint16_t*>(q.x), wxh, winv, s) != hipSuccess)
                    return q.K > 65536 ? UNISVQ_EUNSUP : UNISVQ_EHIP;
                xh = wxh;
                inv = winv;
            }
            const int groups = static_cast<int>(q.K / kGroup);
            const int packets = (groups + 1) / 2;
            int splits = 1, gps = groups;
            if (tiles < 256 && groups >= 4) {
                const int fill = static_cast<int>((256 + tiles - 1) / tiles);
                const int want = fill > (packets + 3) / 4 ? fill : (packets + 3) / 4;
                const int sp = want < packets ? want : packets;
                gps = 2 * ((packets + sp - 1) / sp);
                splits = (groups + gps - 1) / gps;
            }
            b.p[i] = TileProb{q.packed, nullptr, xh, inv, nullptr, reinterpret_cast<float*>(slice), q.y, 0,
                              static_cast<int>(q.N), static_cast<int>(q.K),
                              static_cast<int>((q.N + kBN - 1) / kBN), splits, gps, 0};
        }
        const bool tx = x_dtype == UNISVQ_BF16;
        hipError_t e;
        if (p0.mi == 2)
            e = tx ? launch_tile_batch<2, false, 2, 4, true>(b, s) : launch_tile_batch<2, false>(b, s);
        else
            e = tx ? launch_tile_batch<1, false, 2, 4, true>(b, s) : launch_tile_batch<1, false>(b, s);
        return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
    }
    if (M <= kGemvMaxM) {
        GemvProblem g[kMaxBatch];
        for (int i = 0; i < count; ++i)
            g[i] = GemvProblem{probs[i].packed, probs[i].x, probs[i].y, static_cast<int>(probs[i].N),
                               static_cast<int>(probs[i].K), 0, nullptr, 0};
        const int st = launch_gemv_batch(g, count, M, x_dtype, y_dtype, s);
        if (st != UNISVQ_EUNSUP) return st;  // else K too long for its LDS: the small-batch kernel
    }
    SkinnyProblem sp[kMaxBatch];
    for (int i = 0; i < count; ++i) {
        const GemmBatchProblem& q = probs[i];
        sp[i] = SkinnyProblem{q.packed, nullptr, 0, static_cast<const _Float16*>(q.x), nullptr, q.y, q.N, q.K};
        if (x_dtype == UNISVQ_BF16) {
            // the problem's own scaled fp16 copy (row-major at this size), or
            // that of an earlier problem with the same activations (one copy
            // keeps them shared, so that workgroups may span the problems)
            int same = -1;
            for (int j = 0; j < i && same < 0; ++j)
                if (probs[j].x == q.x && probs[j].K == q.K) same = j;
            if (same >= 0) {
                sp[i].x = sp[same].x;
                sp[i].inv_scale = sp[same].inv_scale;
            } else {
                _Float16* wxh = reinterpret_cast<_Float16*>(ws);
                float* winv = reinterpret_cast<float*>(ws + align256(static_cast<size_t>(M) * q.K * 2));
                if (launch_scale<false>(q.K, M, static_cast<const uint16_t*>(q.x), wxh, winv, s) != hipSuccess)
                    return q.K > 65536 ? UNISVQ_EUNSUP : UNISVQ_EHIP;
                sp[i].x = wxh;
                sp[i].inv_scale = winv;
            }
        }
        ws += align256(gemm_workspace_bytes(q.N, q.K, M, x_dtype));
    }
    return launch_skinny_batch(sp, count, M, y_dtype, s) == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int launch_gemm_shared(int64_t N, int64_t K, const uint8_t* packed_codes, const uint8_t* affine,
                       int affine_one, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                       void* workspace, hipStream_t s) {
    return gemm_common(N, K, packed_codes, affine, affine_one, M, x, x_dtype, y, y_dtype, workspace, s);
}

// Eq. 9 fold (row-shared pairs, any M): workspace = the tiled x' copy
// (tokens padded to 16), one scale and one bias term per token, and the
// fp32 partials when the product is split along K.
size_t gemm_fold_workspace_bytes(int64_t N, int64_t K, int64_t M) {
    const GemmPlan p = plan_gemm(N, K, M);
    const size_t part = p.splits > 1 ? static_cast<size_t>(p.splits) * M * N * 4 : 0;
    return align256(static_cast<size_t>((M + 15) / 16 * 16) * K * 2) + 2 * align256(static_cast<size_t>(M) * 4) + part;
}

int launch_gemm_fold(int64_t N, int64_t K, const uint8_t* packed_codes, const uint8_t* affine, int affine_one,
                     int64_t M, const void* x, int x_dtype, void* y, int y_dtype, void* workspace, hipStream_t s) {
    const int64_t mpad = (M + 15) / 16 * 16;
    if (mpad * K * 2 > kMaxBufferBytes) return UNISVQ_EUNSUP;  // one 32-bit addressed activation buffer
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    _Float16* xh = reinterpret_cast<_Float16*>(ws);
    ws += align256(static_cast<size_t>(mpad) * K * 2);
    float* inv = reinterpret_cast<float*>(ws);
    ws += align256(static_cast<size_t>(M) * 4);
    float* bias = reinterpret_cast<float*>(ws);
    ws += align256(static_cast<size_t>(M) * 4);
    float* partial = reinterpret_cast<float*>(ws);
    const dim3 grid(static_cast<unsigned>(mpad / 16 * 2)), block(1024);
    const uint16_t* xb = static_cast<const uint16_t*>(x);
    const int k = static_cast<int>(K), m = static_cast<int>(M);
    if (x_dtype == UNISVQ_BF16)
        hipLaunchKernelGGL(fold_tiles_kernel<true>, grid, block, 0, s, xb, k, m, affine, affine_one, xh, inv, bias);
    else
        hipLaunchKernelGGL(fold_tiles_kernel<false>, grid, block, 0, s, xb, k, m, affine, affine_one, xh, inv, bias);
    if (hipGetLastError() != hipSuccess) return UNISVQ_EHIP;
    const GemmPlan p = plan_gemm(N, K, M);
    const hipError_t e =
        p.mi == 2 ? launch_tiles<2, true, 2, 4, true, true>(p, N, K, packed_codes, affine, affine_one, M, xh, inv, y,
                                                            y_dtype, partial, s, bias)
                  : launch_tiles<1, true, 2, 4, true, true>(p, N, K, packed_codes, affine, affine_one, M, xh, inv, y,
                                                            y_dtype, partial, s, bias);
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int launch_gemm_var(int64_t N, int64_t K, int bits, int d, const uint8_t* packed_codes, const uint8_t* affine,
                    int affine_one, int64_t M, const void* x, int x_dtype, void* y, int y_dtype, void* workspace,
                    hipStream_t s) {
    return gemm_common(N, K, packed_codes, affine, affine_one, M, x, x_dtype, y, y_dtype, workspace, s, bits, d);
}

}  // namespace unisvq
