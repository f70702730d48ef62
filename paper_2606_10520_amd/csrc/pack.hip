// Pack / unpack between the canonical arrays and packed format v1.
//
// Both are bit-exact permutations: codes keep their two low bits, the fp16
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

}  // namespace

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
