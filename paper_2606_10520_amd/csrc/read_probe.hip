// Bandwidth reference: a plain read of given device byte ranges with the
// loads the decode kernels stream their weights with.  Not part of the
// method; the benchmark times it over the buffers of a product launch to give
// the read rate those very bytes reach in the same launch structure.
#include "common.hpp"

namespace unisvq {
namespace {

// Geometry from a sweep of plain reads over the 7B decoder launches (4 to
// 8 KB per workgroup, 64 to 1024 threads, 1 to 8 loads per thread): 128
// threads with 4 loads each was within 1% of the fastest.
constexpr int kReadThreads = 128;
constexpr int kReadLoads = 4;  // 16-byte loads per thread, all issued before any is used
constexpr uint32_t kReadChunk = kReadThreads * kReadLoads * 16;  // 8 KB per workgroup

struct ReadBatch {
    const uint8_t* p[kMaxBatch];
    uint32_t bytes[kMaxBatch];
    int wg_begin[kMaxBatch];
    int count;
};

// STORE: each wavefront stores the XOR of its words to its own sink word;
// otherwise nothing is written (an empty asm consumes the value, so the loads
// stay).
template <bool STORE>
__global__ __launch_bounds__(kReadThreads) void read_kernel(const ReadBatch b, uint32_t* __restrict__ sink) {
    const int bid = blockIdx.x;
    const uint8_t* p = b.p[0];
    uint32_t bytes = b.bytes[0];
    int wg0 = 0;
#pragma unroll
    for (int i = 1; i < kMaxBatch; ++i) {
        if (i < b.count && bid >= b.wg_begin[i]) {
            p = b.p[i];
            bytes = b.bytes[i];
            wg0 = b.wg_begin[i];
        }
    }
    const __amdgpu_buffer_rsrc_t r = make_rsrc(p, bytes);
    const uint32_t base = static_cast<uint32_t>(bid - wg0) * kReadChunk + 16u * threadIdx.x;
    uint4 v[kReadLoads];
#pragma unroll
    for (int u = 0; u < kReadLoads; ++u) v[u] = ld128_stream(r, base + static_cast<uint32_t>(u) * (kReadThreads * 16));
    uint32_t acc = 0;
#pragma unroll
    for (int u = 0; u < kReadLoads; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    if constexpr (STORE) {
#pragma unroll
        for (int d = 32; d >= 1; d >>= 1) acc ^= static_cast<uint32_t>(__shfl_xor(static_cast<int>(acc), d));
        // one word per wavefront: a store each, no contention
        if ((threadIdx.x & 63) == 0) sink[bid * (kReadThreads / 64) + (threadIdx.x >> 6)] = acc;
    } else {
        asm volatile("" ::"v"(acc));
    }
}

}  // namespace

int64_t read_sink_words(const int64_t* bytes, int count) {
    int64_t wgs = 0;
    for (int i = 0; i < count; ++i) wgs += (bytes[i] + kReadChunk - 1) / kReadChunk;
    return wgs * (kReadThreads / 64);
}

int launch_read(const uint8_t* const* ptrs, const int64_t* bytes, int count, uint32_t* sink, bool store,
                hipStream_t s) {
    ReadBatch b{};
    int wgs = 0;
    for (int i = 0; i < count; ++i) {
        b.p[i] = ptrs[i];
        b.bytes[i] = static_cast<uint32_t>(bytes[i]);
        b.wg_begin[i] = wgs;
        wgs += static_cast<int>((bytes[i] + kReadChunk - 1) / kReadChunk);
    }
    b.count = count;
    if (wgs == 0) return UNISVQ_OK;
    if (store)
        hipLaunchKernelGGL(read_kernel<true>, dim3(static_cast<unsigned>(wgs)), dim3(kReadThreads), 0, s, b, sink);
    else
        hipLaunchKernelGGL(read_kernel<false>, dim3(static_cast<unsigned>(wgs)), dim3(kReadThreads), 0, s, b, sink);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

}  // namespace unisvq
