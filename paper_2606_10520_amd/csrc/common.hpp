// Internal declarations shared by the libunisvq translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "unisvq.h"

namespace unisvq {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Packed format v1 geometry (see the format block in unisvq.h).
constexpr int kGroup = 128;            // input columns per (A, B) set
constexpr int kRowBlock = 16;          // rows per row block
constexpr int kGroupBlockBytes = 1152; // one group of one row block: 16 rows * 72 B
constexpr int kPacketBytes = 2304;     // two groups
constexpr int kPacketAffineOff = 1024; // A columns inside a full packet
constexpr int kPacketBiasOff = 2048;   // B values inside a full packet
constexpr int kHalfAffineOff = 512;
constexpr int kHalfBiasOff = 1024;

// Launchers (host side).  Each returns the hipError_t of the launch.
hipError_t launch_pack(int64_t N, int64_t K, const uint8_t* codes, const uint16_t* A,
                       const uint16_t* B, uint8_t* packed, int32_t* bad, hipStream_t s);
hipError_t launch_unpack(int64_t N, int64_t K, const uint8_t* packed, uint8_t* codes,
                         uint16_t* A, uint16_t* B, hipStream_t s);

// Matrix-vector path: returns UNISVQ_EUNSUP if the shape does not fit the
// kernel (LDS budget), else maps the launch result to a status.
int launch_gemv(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x,
                int x_dtype, void* y, int y_dtype, hipStream_t s);
int launch_gemm(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x,
                int x_dtype, void* y, int y_dtype, hipStream_t s);

// Output store in the requested dtype (fp32 -> fp16 / bf16 round to nearest even).
__device__ inline void store_out(void* y, int64_t idx, float v, int y_dtype) {
    if (y_dtype == UNISVQ_F32)
        static_cast<float*>(y)[idx] = v;
    else if (y_dtype == UNISVQ_F16)
        static_cast<_Float16*>(y)[idx] = static_cast<_Float16>(v);
    else
        static_cast<__bf16*>(y)[idx] = static_cast<__bf16>(v);
}

}  // namespace unisvq
