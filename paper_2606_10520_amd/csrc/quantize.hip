// Nearest-codeword quantisation on gfx950 (the quantiser of Sec. 3.2.2
// without Hessian feedback): every vector of d = 4 consecutive weights of a
// row takes the codes q of the affine-lattice point A q + B closest to it.
//
// One thread per vector tries all 256 codewords.  The decision is an integer,
// so it is taken in fp64 with one fixed sequence of operations per candidate
// i (q_b = bits 2b, 2b+1 of i): c_a = B_a + A_a0 q_0 + A_a1 q_1 + A_a2 q_2 +
// A_a3 q_3 summed left to right (each product of an fp16 parameter and a small
// integer is exact, so contracting a product into an fma changes nothing),
// e_a = c_a - w_a, d = fma(e_a, e_a, d) over a = 0..3; candidates are visited
// in increasing index and only a strictly smaller distance replaces the best,
// so ties go to the lowest index q_0 + 4 q_1 + 16 q_2 + 64 q_3.
#include "common.hpp"

namespace unisvq {
namespace {

__device__ inline double half_bits_to_double(uint16_t h) {
    return static_cast<double>(static_cast<float>(__builtin_bit_cast(_Float16, h)));
}

// affine_groups == 0: one pair per (row, group); else row-shared pairs (1 per
// matrix, or one per group).
__global__ __launch_bounds__(256) void quantize_kernel(int64_t N, int64_t K, const float* __restrict__ W,
                                                       const uint16_t* __restrict__ A,
                                                       const uint16_t* __restrict__ B, int64_t affine_groups,
                                                       uint32_t* __restrict__ codes) {
    const int64_t vecs = N * (K / 4);
    const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= vecs) return;
    const int64_t r = idx / (K / 4);
    const int64_t v = idx - r * (K / 4);
    const int64_t groups = K / kGroup;
    const int64_t g = (4 * v) / kGroup;
    const int64_t set = affine_groups == 0 ? r * groups + g : (affine_groups == 1 ? 0 : g);

    double a[16], b[4], w[4];
#pragma unroll
    for (int i = 0; i < 16; ++i) a[i] = half_bits_to_double(A[set * 16 + i]);
#pragma unroll
    for (int i = 0; i < 4; ++i) b[i] = half_bits_to_double(B[set * 4 + i]);
    const float4 wf = *reinterpret_cast<const float4*>(W + r * K + 4 * v);
    w[0] = wf.x;
    w[1] = wf.y;
    w[2] = wf.z;
    w[3] = wf.w;

    int best = 0;
    double dbest = 0.0;
    for (int i = 0; i < 256; ++i) {
        const double q0 = static_cast<double>(i & 3), q1 = static_cast<double>((i >> 2) & 3);
        const double q2 = static_cast<double>((i >> 4) & 3), q3 = static_cast<double>((i >> 6) & 3);
        double d = 0.0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            double c = b[k];
            c = c + a[4 * k + 0] * q0;
            c = c + a[4 * k + 1] * q1;
            c = c + a[4 * k + 2] * q2;
            c = c + a[4 * k + 3] * q3;
            const double e = c - w[k];
            d = __builtin_fma(e, e, d);
        }
        if (i == 0 || d < dbest) {
            dbest = d;
            best = i;
        }
    }
    // codes of the four components, one byte each (q_b at byte b)
    codes[idx] = static_cast<uint32_t>(best & 3) | (static_cast<uint32_t>((best >> 2) & 3) << 8) |
                 (static_cast<uint32_t>((best >> 4) & 3) << 16) | (static_cast<uint32_t>((best >> 6) & 3) << 24);
}

}  // namespace

hipError_t launch_quantize(int64_t N, int64_t K, const float* W, const uint16_t* A, const uint16_t* B,
                           int64_t affine_groups, uint8_t* codes, hipStream_t s) {
    const int64_t vecs = N * (K / 4);
    const int threads = 256;
    hipLaunchKernelGGL(quantize_kernel, dim3(static_cast<unsigned>((vecs + threads - 1) / threads)), dim3(threads),
                       0, s, N, K, W, A, B, affine_groups, reinterpret_cast<uint32_t*>(codes));
    return hipGetLastError();
}

}  // namespace unisvq
