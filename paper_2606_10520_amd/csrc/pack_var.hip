// Pack / unpack for the format variants (b-bit codes, b = 2, 3: Sec. 5.2.5;
// d-dimensional vectors, d = 4, 8: Sec. 5.2.3) with row-shared pairs: the
// variant codes-only layout and its shared affine block (variant format
// block in unisvq.h).  Bit-exact permutations: codes keep their b low bits,
// the fp16 words of A and B are moved unchanged.
#include "common.hpp"

namespace unisvq {
namespace {

// Offsets (within the row block) of the low and high fields of slot s, group g.
__device__ inline void var_fields(int bits, int groups, int g, int s, int64_t& lo, int64_t& hi) {
    const int64_t P = static_cast<int64_t>(g >> 1) * 2 * var_group_bytes(bits);
    const bool half = (groups & 1) && g == groups - 1;
    lo = half ? P + 8 * s : P + 16 * s + 8 * (g & 1);
    hi = half ? P + kVarHalfHiOff + 4 * s : P + kVarHiOff + 8 * s + 4 * (g & 1);
}

// Column (within the row) of code (h, u) of lane index j in group g.
template <int D>
__device__ inline int64_t var_col(int g, int h, int u, int j) {
    return static_cast<int64_t>(g) * kGroup + (D == 4 ? 4 * (16 * h + u) + j : 8 * u + 4 * h + j);
}

// Bit of code (h, u) in the high field: 8n + 4m + 2h + p for u = 4n + 2m + p.
__device__ inline int hi_bit(int h, int u) { return 8 * (u >> 2) + 4 * ((u >> 1) & 1) + 2 * h + (u & 1); }

// One thread per (row block, group, slot).
template <int BITS, int D>
__global__ void pack_var_codes_kernel(int64_t N, int64_t K, const uint8_t* __restrict__ codes,
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
    const int j = s & 3;
    const uint8_t* row = codes + r * K;
    uint32_t lo[2] = {0u, 0u}, hi = 0u;
    int nbad = 0;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            const uint32_t c = row[var_col<D>(g, h, u, j)];
            nbad += c >= (1u << BITS);
            lo[h] |= (c & 3u) << (2 * u);
            if (BITS == 3) hi |= ((c >> 2) & 1u) << hi_bit(h, u);
        }
    uint8_t* blk = packed + rb * groups * static_cast<int64_t>(var_group_bytes(BITS));
    int64_t plo, phi;
    var_fields(BITS, groups, g, s, plo, phi);
    *reinterpret_cast<uint2*>(blk + plo) = uint2{lo[0], lo[1]};
    if (BITS == 3) *reinterpret_cast<uint32_t*>(blk + phi) = hi;
    if (bad && nbad) atomicAdd(bad, nbad);
}

template <int BITS, int D>
__global__ void unpack_var_codes_kernel(int64_t N, int64_t K, const uint8_t* __restrict__ packed,
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
    const int j = s & 3;
    const uint8_t* blk = packed + rb * groups * static_cast<int64_t>(var_group_bytes(BITS));
    int64_t plo, phi;
    var_fields(BITS, groups, g, s, plo, phi);
    const uint2 lo = *reinterpret_cast<const uint2*>(blk + plo);
    const uint32_t hi = BITS == 3 ? *reinterpret_cast<const uint32_t*>(blk + phi) : 0u;
    uint8_t* row = codes + r * K;
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int u = 0; u < 16; ++u) {
            uint32_t c = ((h ? lo.y : lo.x) >> (2 * u)) & 3u;
            if (BITS == 3) c |= ((hi >> hi_bit(h, u)) & 1u) << 2;
            row[var_col<D>(g, h, u, j)] = static_cast<uint8_t>(c);
        }
}

// Record offsets of A[a][b] and B[a] of the record's group jj: lane view
// (read by the matrix-vector kernel, lane j = b % 4) and row view (read by
// the weight decode of the tiled product).
template <int D>
__device__ inline int lane_a(int jj, int a, int b) {
    return D == 4 ? 16 * b + 8 * jj + 2 * a : 64 * (b & 3) + 32 * jj + 16 * (b >> 2) + 2 * a;
}
template <int D>
__device__ inline int lane_b(int jj, int a) {
    return D == 4 ? kRecordBiasOff + 4 * a + 2 * jj : kVarBiasOff8 + 8 * (a & 3) + 4 * jj + 2 * (a >> 2);
}
template <int D>
__device__ inline int row_a(int jj, int a, int b) {
    return var_row_view_off(D) + jj * var_row_view_group_bytes(D) + 2 * (D * a + b);
}
template <int D>
__device__ inline int row_b(int jj, int a) {
    return var_row_view_off(D) + jj * var_row_view_group_bytes(D) + 2 * D * D + 2 * a;
}

// One thread per (record R, group jj of the record, component a): row a of
// A and B[a], in both views (pair 0 for both groups when there is a single
// pair; zeros for a group past the last).
template <int D>
__global__ void pack_var_affine_kernel(int records, int groups, int affine_one, const uint16_t* __restrict__ A,
                                       const uint16_t* __restrict__ B, uint8_t* __restrict__ out) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= records * 2 * D) return;
    const int a = idx % D, jj = (idx / D) & 1, R = idx / (2 * D);
    const int g = 2 * R + jj;
    const int src = affine_one ? 0 : g;
    const bool valid = affine_one || g < groups;
    uint8_t* rec = out + static_cast<int64_t>(R) * var_record_bytes(D);
#pragma unroll
    for (int b = 0; b < D; ++b) {
        const uint16_t v = valid ? A[(src * D + a) * D + b] : uint16_t{0};
        *reinterpret_cast<uint16_t*>(rec + lane_a<D>(jj, a, b)) = v;
        *reinterpret_cast<uint16_t*>(rec + row_a<D>(jj, a, b)) = v;
    }
    const uint16_t v = valid ? B[src * D + a] : uint16_t{0};
    *reinterpret_cast<uint16_t*>(rec + lane_b<D>(jj, a)) = v;
    *reinterpret_cast<uint16_t*>(rec + row_b<D>(jj, a)) = v;
}

// One thread per (pair, component a), from the lane view.
template <int D>
__global__ void unpack_var_affine_kernel(int pairs, int affine_one, const uint8_t* __restrict__ in,
                                         uint16_t* __restrict__ A, uint16_t* __restrict__ B) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= pairs * D) return;
    const int g = idx / D, a = idx % D;
    const int R = affine_one ? 0 : g >> 1, jj = affine_one ? 0 : g & 1;
    const uint8_t* rec = in + static_cast<int64_t>(R) * var_record_bytes(D);
#pragma unroll
    for (int b = 0; b < D; ++b) A[(g * D + a) * D + b] = *reinterpret_cast<const uint16_t*>(rec + lane_a<D>(jj, a, b));
    B[g * D + a] = *reinterpret_cast<const uint16_t*>(rec + lane_b<D>(jj, a));
}

template <int BITS, int D>
hipError_t pack_var(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* codes, const uint16_t* A,
                    const uint16_t* B, uint8_t* packed_codes, uint8_t* packed_affine, int32_t* bad, hipStream_t s) {
    const int64_t total = (N / kRowBlock) * (K / kGroup) * 64;
    hipLaunchKernelGGL((pack_var_codes_kernel<BITS, D>), dim3(static_cast<unsigned>((total + 255) / 256)), dim3(256),
                       0, s, N, K, codes, packed_codes, bad);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    const int groups = static_cast<int>(K / kGroup);
    const int one = affine_groups == 1;
    const int records = one ? 1 : (groups + 1) / 2;
    const int threads = records * 2 * D;
    hipLaunchKernelGGL(pack_var_affine_kernel<D>, dim3((threads + 255) / 256), dim3(256), 0, s, records, groups, one,
                       A, B, packed_affine);
    return hipGetLastError();
}

template <int BITS, int D>
hipError_t unpack_var(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* packed_codes,
                      const uint8_t* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B, hipStream_t s) {
    const int64_t total = (N / kRowBlock) * (K / kGroup) * 64;
    hipLaunchKernelGGL((unpack_var_codes_kernel<BITS, D>), dim3(static_cast<unsigned>((total + 255) / 256)),
                       dim3(256), 0, s, N, K, packed_codes, codes);
    if (hipGetLastError() != hipSuccess) return hipErrorLaunchFailure;
    const int pairs = static_cast<int>(affine_groups);
    const int threads = pairs * D;
    hipLaunchKernelGGL(unpack_var_affine_kernel<D>, dim3((threads + 255) / 256), dim3(256), 0, s, pairs,
                       affine_groups == 1 ? 1 : 0, packed_affine, A, B);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_var_pack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const uint8_t* codes,
                           const uint16_t* A, const uint16_t* B, uint8_t* packed_codes, uint8_t* packed_affine,
                           int32_t* bad, hipStream_t s) {
    if (bits == 3 && d == 4) return pack_var<3, 4>(N, K, affine_groups, codes, A, B, packed_codes, packed_affine, bad, s);
    if (bits == 2 && d == 8) return pack_var<2, 8>(N, K, affine_groups, codes, A, B, packed_codes, packed_affine, bad, s);
    if (bits == 3 && d == 8) return pack_var<3, 8>(N, K, affine_groups, codes, A, B, packed_codes, packed_affine, bad, s);
    return hipErrorInvalidValue;
}

hipError_t launch_var_unpack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups,
                             const uint8_t* packed_codes, const uint8_t* packed_affine, uint8_t* codes,
                             uint16_t* A, uint16_t* B, hipStream_t s) {
    if (bits == 3 && d == 4) return unpack_var<3, 4>(N, K, affine_groups, packed_codes, packed_affine, codes, A, B, s);
    if (bits == 2 && d == 8) return unpack_var<2, 8>(N, K, affine_groups, packed_codes, packed_affine, codes, A, B, s);
    if (bits == 3 && d == 8) return unpack_var<3, 8>(N, K, affine_groups, packed_codes, packed_affine, codes, A, B, s);
    return hipErrorInvalidValue;
}

}  // namespace unisvq
