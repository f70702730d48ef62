// Pack / unpack between the canonical arrays and packed format v1, and
// between codes plus row-shared pairs and the codes-only format with its
// shared affine block.
//
// All are bit-exact permutations: codes keep their two low bits, the fp16
// A and B words are moved unchanged (storage of Sec. 3.1: 2-bit codes plus
// 40 bytes of affine parameters per set).
#include "common.hpp"

namespace unisvq {
namespace {

// Byte offsets of the three parts of one packet slot for group g of a row
// block (relative to the start of the row block).
struct SlotPlace {
    int64_t code, affine, bias;
};

__device__ inline SlotPlace place(int groups, int g, int s) {
    const int p = g >> 1, j = g & 1;
    const int64_t pkt = static_cast<int64_t>(p) * kPacketBytes;
    const bool half = (groups & 1) && g == groups - 1;
    SlotPlace sp;
    if (!half) {
        sp.code = pkt + 16 * s + 8 * j;
        sp.affine = pkt + kPacketAffineOff + 16 * s + 8 * j;
        sp.bias = pkt + kPacketBiasOff + 4 * s + 2 * j;
    } else {
        sp.code = pkt + 8 * s;
        sp.affine = pkt + kHalfAffineOff + 8 * s;
        sp.bias = pkt + kHalfBiasOff + 2 * s;
    }
    return sp;
}

// One thread per (row block, group, slot): gathers component b of the 32
// vectors of row r, the A column A[r][g][0..3][b] and B[r][g][b].
__global__ void pack_kernel(int64_t N, int64_t K, const uint8_t* __restrict__ codes,
                            const uint16_t* __restrict__ A, const uint16_t* __restrict__ B,
                            uint8_t* __restrict__ packed, int32_t* __restrict__ bad) {
    const int groups = static_cast<int>(K / kGroup);
    const int64_t total = (N / kRowBlock) * groups * 64;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int s = static_cast<int>(idx & 63);
    const int64_t t = idx >> 6;
    const int g = static_cast<int>(t % groups);
    const int64_t rb = t / groups;
    const int64_t r = rb * kRowBlock + (s >> 2);
    const int b = s & 3;

    const uint8_t* q = codes + r * K + static_cast<int64_t>(g) * kGroup + b;
    uint64_t field = 0;
    int nbad = 0;
#pragma unroll
    for (int v = 0; v < 32; ++v) {
        const uint32_t c = q[4 * v];
        nbad += c > 3u;
        field |= static_cast<uint64_t>(c & 3u) << (2 * v);
    }
    const int64_t set = r * groups + g;
    uint64_t acol = 0;
#pragma unroll
    for (int a = 0; a < 4; ++a) acol |= static_cast<uint64_t>(A[(set * 4 + a) * 4 + b]) << (16 * a);
    const uint16_t bias = B[set * 4 + b];

    uint8_t* blk = packed + rb * groups * static_cast<int64_t>(kGroupBlockBytes);
    const SlotPlace sp = place(groups, g, s);
    *reinterpret_cast<uint64_t*>(blk + sp.code) = field;
    *reinterpret_cast<uint64_t*>(blk + sp.affine) = acol;
    *reinterpret_cast<uint16_t*>(blk + sp.bias) = bias;
    if (bad && nbad) atomicAdd(bad, nbad);
}

__global__ void unpack_kernel(int64_t N, int64_t K, const uint8_t* __restrict__ packed,
                              uint8_t* __restrict__ codes, uint16_t* __restrict__ A,
                              uint16_t* __restrict__ B) {
    const int groups = static_cast<int>(K / kGroup);
    const int64_t total = (N / kRowBlock) * groups * 64;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int s = static_cast<int>(idx & 63);
    const int64_t t = idx >> 6;
    const int g = static_cast<int>(t % groups);
    const int64_t rb = t / groups;
    const int64_t r = rb * kRowBlock + (s >> 2);
    const int b = s & 3;

    const uint8_t* blk = packed + rb * groups * static_cast<int64_t>(kGroupBlockBytes);
    const SlotPlace sp = place(groups, g, s);
    const uint64_t field = *reinterpret_cast<const uint64_t*>(blk + sp.code);
    const uint64_t acol = *reinterpret_cast<const uint64_t*>(blk + sp.affine);
    const uint16_t bias = *reinterpret_cast<const uint16_t*>(blk + sp.bias);

    uint8_t* q = codes + r * K + static_cast<int64_t>(g) * kGroup + b;
#pragma unroll
    for (int v = 0; v < 32; ++v) q[4 * v] = static_cast<uint8_t>((field >> (2 * v)) & 3u);
    const int64_t set = r * groups + g;
#pragma unroll
    for (int a = 0; a < 4; ++a) A[(set * 4 + a) * 4 + b] = static_cast<uint16_t>(acol >> (16 * a));
    B[set * 4 + b] = bias;
}

// ---- codes-only format and the shared affine block ----

__device__ inline int64_t code_place(int groups, int g, int s) {
    const int64_t pkt = static_cast<int64_t>(g >> 1) * kCodePacketBytes;
    const bool half = (groups & 1) && g == groups - 1;
    return half ? pkt + 8 * s : pkt + 16 * s + 8 * (g & 1);
}

// One thread per (row block, group, slot): the code field only.
__global__ void pack_codes_kernel(int64_t N, int64_t K, const uint8_t* __restrict__ codes,
                                  uint8_t* __restrict__ packed, int32_t* __restrict__ bad) {
    const int groups = static_cast<int>(K / kGroup);
    const int64_t total = (N / kRowBlock) * groups * 64;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int s = static_cast<int>(idx & 63);
    const int64_t t = idx >> 6;
    const int g = static_cast<int>(t % groups);
    const int64_t rb = t / groups;
    const int64_t r = rb * kRowBlock + (s >> 2);
    const uint8_t* q = codes + r * K + static_cast<int64_t>(g) * kGroup + (s & 3);
    uint64_t field = 0;
    int nbad = 0;
#pragma unroll
    for (int v = 0; v < 32; ++v) {
        const uint32_t c = q[4 * v];
        nbad += c > 3u;
        field |= static_cast<uint64_t>(c & 3u) << (2 * v);
    }
    uint8_t* blk = packed + rb * groups * static_cast<int64_t>(kCodeGroupBlockBytes);
    *reinterpret_cast<uint64_t*>(blk + code_place(groups, g, s)) = field;
    if (bad && nbad) atomicAdd(bad, nbad);
}

__global__ void unpack_codes_kernel(int64_t N, int64_t K, const uint8_t* __restrict__ packed,
                                    uint8_t* __restrict__ codes) {
    const int groups = static_cast<int>(K / kGroup);
    const int64_t total = (N / kRowBlock) * groups * 64;
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int s = static_cast<int>(idx & 63);
    const int64_t t = idx >> 6;
    const int g = static_cast<int>(t % groups);
    const int64_t rb = t / groups;
    const int64_t r = rb * kRowBlock + (s >> 2);
    const uint8_t* blk = packed + rb * groups * static_cast<int64_t>(kCodeGroupBlockBytes);
    const uint64_t field = *reinterpret_cast<const uint64_t*>(blk + code_place(groups, g, s));
    uint8_t* q = codes + r * K + static_cast<int64_t>(g) * kGroup + (s & 3);
#pragma unroll
    for (int v = 0; v < 32; ++v) q[4 * v] = static_cast<uint8_t>((field >> (2 * v)) & 3u);
}

// One thread per (record R, component b, group j of the record): column b of
// A and B[b] of group 2R + j (pair 0 for both groups when there is a single
// pair; zeros for a group past the last).
__global__ void pack_affine_kernel(int records, int groups, int affine_one, const uint16_t* __restrict__ A,
                                   const uint16_t* __restrict__ B, uint8_t* __restrict__ out) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= records * 8) return;
    const int R = idx >> 3, b = (idx >> 1) & 3, j = idx & 1;
    const int g = 2 * R + j;
    const int src = affine_one ? 0 : g;
    const bool valid = affine_one || g < groups;
    uint8_t* rec = out + static_cast<int64_t>(R) * kAffineRecordBytes;
    uint16_t* acol = reinterpret_cast<uint16_t*>(rec + 16 * b + 8 * j);
#pragma unroll
    for (int a = 0; a < 4; ++a) acol[a] = valid ? A[(src * 4 + a) * 4 + b] : uint16_t{0};
    *reinterpret_cast<uint16_t*>(rec + kRecordBiasOff + 4 * b + 2 * j) = valid ? B[src * 4 + b] : uint16_t{0};
}

// One thread per (pair, component b).
__global__ void unpack_affine_kernel(int pairs, int affine_one, const uint8_t* __restrict__ in,
                                     uint16_t* __restrict__ A, uint16_t* __restrict__ B) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= pairs * 4) return;
    const int g = idx >> 2, b = idx & 3;
    const int R = affine_one ? 0 : g >> 1, j = affine_one ? 0 : g & 1;
    const uint8_t* rec = in + static_cast<int64_t>(R) * kAffineRecordBytes;
    const uint16_t* acol = reinterpret_cast<const uint16_t*>(rec + 16 * b + 8 * j);
#pragma unroll
    for (int a = 0; a < 4; ++a) A[(g * 4 + a) * 4 + b] = acol[a];
    B[g * 4 + b] = *reinterpret_cast<const uint16_t*>(rec + kRecordBiasOff + 4 * b + 2 * j);
}

}  // namespace

hipError_t launch_pack_shared(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* codes,
                              const uint16_t* A, const uint16_t* B, uint8_t* packed_codes,
                              uint8_t* packed_affine, int32_t* bad, hipStream_t s) {
    const int64_t total = (N / kRowBlock) * (K / kGroup) * 64;
    const int threads = 256;
    hipLaunchKernelGGL(pack_codes_kernel, dim3(static_cast<unsigned>((total + threads - 1) / threads)),
                       dim3(threads), 0, s, N, K, codes, packed_codes, bad);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    const int groups = static_cast<int>(K / kGroup);
    const int one = affine_groups == 1;
    const int records = one ? 1 : (groups + 1) / 2;
    hipLaunchKernelGGL(pack_affine_kernel, dim3(static_cast<unsigned>((records * 8 + threads - 1) / threads)),
                       dim3(threads), 0, s, records, groups, one, A, B, packed_affine);
    return hipGetLastError();
}

hipError_t launch_unpack_shared(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* packed_codes,
                                const uint8_t* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B,
                                hipStream_t s) {
    const int64_t total = (N / kRowBlock) * (K / kGroup) * 64;
    const int threads = 256;
    hipLaunchKernelGGL(unpack_codes_kernel, dim3(static_cast<unsigned>((total + threads - 1) / threads)),
                       dim3(threads), 0, s, N, K, packed_codes, codes);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    const int pairs = static_cast<int>(affine_groups);
    hipLaunchKernelGGL(unpack_affine_kernel, dim3(static_cast<unsigned>((pairs * 4 + threads - 1) / threads)),
                       dim3(threads), 0, s, pairs, affine_groups == 1 ? 1 : 0, packed_affine, A, B);
    return hipGetLastError();
}

hipError_t launch_pack(int64_t N, int64_t K, const uint8_t* codes, const uint16_t* A,
                       const uint16_t* B, uint8_t* packed, int32_t* bad, hipStream_t s) {
    const int64_t total = (N / kRowBlock) * (K / kGroup) * 64;
    const int threads = 256;
    const int64_t blocks = (total + threads - 1) / threads;
    hipLaunchKernelGGL(pack_kernel, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0, s, N, K,
                       codes, A, B, packed, bad);
    return hipGetLastError();
}

hipError_t launch_unpack(int64_t N, int64_t K, const uint8_t* packed, uint8_t* codes,
                         uint16_t* A, uint16_t* B, hipStream_t s) {
    const int64_t total = (N / kRowBlock) * (K / kGroup) * 64;
    const int threads = 256;
    const int64_t blocks = (total + threads - 1) / threads;
    hipLaunchKernelGGL(unpack_kernel, dim3(static_cast<unsigned>(blocks)), dim3(threads), 0, s, N,
                       K, packed, codes, A, B);
    return hipGetLastError();
}

}  // namespace unisvq
