// Internal declarations shared by the libunisvq translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "unisvq.h"

namespace unisvq {

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));

// Raw buffer access: a resource descriptor carries the buffer's size, and the
// hardware returns zeros for any read beyond it instead of faulting, so loads
// need no guarding branches (which would also serialise the wait counters).
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0),
                                             static_cast<int>(bytes), 0x00020000);
}
__device__ inline uint4 ld128(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
    return uint4{static_cast<uint32_t>(v.x), static_cast<uint32_t>(v.y), static_cast<uint32_t>(v.z),
                 static_cast<uint32_t>(v.w)};
}
__device__ inline uint2 ld64(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const i32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
    return uint2{static_cast<uint32_t>(v.x), static_cast<uint32_t>(v.y)};
}
__device__ inline uint32_t ld32(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
__device__ inline uint32_t ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

// Streaming variants for data read exactly once (the weight stream of the
// decode kernels): the non-temporal cache policy keeps it from displacing
// what is reused (activations, outputs) in L2 and the MALL.
constexpr int kNonTemporal = 2;
__device__ inline uint4 ld128_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kNonTemporal);
    return uint4{static_cast<uint32_t>(v.x), static_cast<uint32_t>(v.y), static_cast<uint32_t>(v.z),
                 static_cast<uint32_t>(v.w)};
}
__device__ inline uint2 ld64_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    const i32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kNonTemporal);
    return uint2{static_cast<uint32_t>(v.x), static_cast<uint32_t>(v.y)};
}
__device__ inline uint32_t ld32_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return static_cast<uint32_t>(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kNonTemporal));
}
__device__ inline uint32_t ld16_stream(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kNonTemporal);
}

// Largest buffer a 32-bit buffer offset addresses.
constexpr int64_t kMaxBufferBytes = (int64_t{1} << 31) - 1;
// A buffer offset past the end of every buffer the kernels address (all are
// below 2^31 bytes): such a load returns zeros.
constexpr uint32_t kOutOfRange = 0x80000000u;

// Packed format v1 geometry (see the format block in unisvq.h).
constexpr int kGroup = 128;            // input columns per (A, B) set
constexpr int kRowBlock = 16;          // rows per row block
constexpr int kGroupBlockBytes = 1152; // one group of one row block: 16 rows * 72 B
constexpr int kPacketBytes = 2304;     // two groups
constexpr int kPacketAffineOff = 1024; // A columns inside a full packet
constexpr int kPacketBiasOff = 2048;   // B values inside a full packet
constexpr int kHalfAffineOff = 512;
constexpr int kHalfBiasOff = 1024;

// Codes-only format (affine pairs shared by all rows, held in a separate
// block of 80-byte records, one per pair of groups; see unisvq.h).
constexpr int kCodeGroupBlockBytes = 512;  // one group of one row block: 16 rows * 32 B
constexpr int kCodePacketBytes = 1024;     // two groups
constexpr int kAffineRecordBytes = 80;     // A columns (64 B) and B values (16 B) of two groups
constexpr int kRecordBiasOff = 64;

// Variant codes-only format: b-bit codes (b = 2, 3) and d-dimensional vectors
// (d = 4, 8) with row-shared pairs (variant format block in unisvq.h).
constexpr int var_group_bytes(int bits) { return bits == 3 ? 768 : 512; }  // one group of a row block
constexpr int kVarHiOff = 1024;     // high fields inside a full packet
constexpr int kVarHalfHiOff = 512;  // high fields inside a half packet
constexpr int var_record_bytes(int d) { return d == 4 ? 160 : 576; }
constexpr int kVarBiasOff8 = 256;                                 // lane-view B values, d = 8
constexpr int var_row_view_off(int d) { return d == 4 ? 80 : 288; }  // row view of a record
constexpr int var_row_view_group_bytes(int d) { return 2 * (d * d + d); }

// Launchers (host side).  Each returns the hipError_t of the launch.
hipError_t launch_pack(int64_t N, int64_t K, const uint8_t* codes, const uint16_t* A,
                       const uint16_t* B, uint8_t* packed, int32_t* bad, hipStream_t s);
hipError_t launch_unpack(int64_t N, int64_t K, const uint8_t* packed, uint8_t* codes,
                         uint16_t* A, uint16_t* B, hipStream_t s);
hipError_t launch_pack_shared(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* codes,
                              const uint16_t* A, const uint16_t* B, uint8_t* packed_codes,
                              uint8_t* packed_affine, int32_t* bad, hipStream_t s);
hipError_t launch_unpack_shared(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* packed_codes,
                                const uint8_t* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B,
                                hipStream_t s);

// Variant format pack / unpack (codes uint8 [N][K]; A, B fp16 bits [Ga][d][d], [Ga][d]).
hipError_t launch_var_pack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const uint8_t* codes,
                           const uint16_t* A, const uint16_t* B, uint8_t* packed_codes, uint8_t* packed_affine,
                           int32_t* bad, hipStream_t s);
hipError_t launch_var_unpack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups,
                             const uint8_t* packed_codes, const uint8_t* packed_affine, uint8_t* codes,
                             uint16_t* A, uint16_t* B, hipStream_t s);

// Nearest-codeword quantisation (codes uint8 [N][K], 4-byte aligned).
hipError_t launch_quantize(int64_t N, int64_t K, const float* W, const uint16_t* A, const uint16_t* B,
                           int64_t affine_groups, uint8_t* codes, hipStream_t s);

// LDLQ (Eq. 7) with the caller's feedback factor U (fp64 [K][K]); workspace
// of ldlq_workspace_bytes(N, K) bytes.
size_t ldlq_workspace_bytes(int64_t N, int64_t K);
hipError_t launch_ldlq(int64_t N, int64_t K, const float* W, const double* U, const uint16_t* A, const uint16_t* B,
                       int64_t affine_groups, uint8_t* codes, void* workspace, hipStream_t s);

// Block LDL^T factorisation H = U D U^T (4 x 4 pivot blocks, fp64 [K][K]);
// workspace of ldl_workspace_bytes(K) bytes.
size_t ldl_workspace_bytes(int64_t K);
hipError_t launch_ldl(int64_t K, const double* H, double* U, double* D, int32_t* info, void* workspace,
                      hipStream_t s);

// Randomized Hadamard transform of M rows of length n (mode 0: input side,
// signs first; mode 1: output side, signs last); UNISVQ_EUNSUP when n has no
// supported Hadamard construction or exceeds the LDS row.
int launch_rht(int64_t n, int64_t M, const void* x, int x_dtype, const signed char* signs, int mode, void* y,
               int y_dtype, hipStream_t s);

// One problem of a (possibly batched) matrix-vector launch.
struct GemvProblem {
    const uint8_t* packed;   // full format, or codes only when `affine` is set
    const void* x;
    void* y;
    int N, K;
    int rb_begin;            // first workgroup index of this problem (set by the launcher)
    const uint8_t* affine;   // shared affine block (codes-only format), else null
    int affine_one;          // 1: one pair for the whole matrix
};
constexpr int kMaxBatch = 8;

// Matrix-vector path: returns UNISVQ_EUNSUP if the shape does not fit the
// kernel (LDS budget), else maps the launch result to a status.
int launch_gemv_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype,
                      hipStream_t s);
int launch_gemv(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x,
                int x_dtype, void* y, int y_dtype, hipStream_t s);
// The same for variant weights (every problem with `bits`-bit codes and
// d-dimensional vectors, codes-only with its shared affine block).
int launch_gemv_rht_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype,
                          const signed char* const* signs, hipStream_t s);
int launch_gemv_var_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype, int bits, int d,
                          hipStream_t s);
// Prefill path.  Device workspace (16-byte aligned) of
// gemm_workspace_bytes(N, K, M, x_dtype) bytes: for bf16 activations an fp16
// copy of x plus one scale per token, and for products split along K the
// fp32 partial sums.  0 means none is needed.
size_t gemm_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype);
int launch_gemm(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x,
                int x_dtype, void* y, int y_dtype, void* workspace, hipStream_t s);
// launch_gemm with the library's own fixed scratch array as the workspace
// (noalloc_scratch_bytes() per device); UNISVQ_ESCRATCH when the product
// needs more.
size_t noalloc_scratch_bytes();
int launch_gemm_noalloc(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype, void* y,
                        int y_dtype, hipStream_t s);
// The same with codes-only weights and a shared affine block.
int launch_gemm_shared(int64_t N, int64_t K, const uint8_t* packed_codes, const uint8_t* affine,
                       int affine_one, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                       void* workspace, hipStream_t s);
// Eq. 9 fold with row-shared pairs (any M): a pre-pass multiplies the
// activations by A and sums their bias terms, the tiled kernel multiplies by
// the bare codes.  Workspace of gemm_fold_workspace_bytes(N, K, M) bytes.
size_t gemm_fold_workspace_bytes(int64_t N, int64_t K, int64_t M);
int launch_gemm_fold(int64_t N, int64_t K, const uint8_t* packed_codes, const uint8_t* affine, int affine_one,
                     int64_t M, const void* x, int x_dtype, void* y, int y_dtype, void* workspace, hipStream_t s);
// Variant weights: every M > 4 goes to the tiled kernel (K split for small
// M), so the workspace differs from gemm_workspace_bytes.
size_t gemm_var_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype);
int launch_gemm_var(int64_t N, int64_t K, int bits, int d, const uint8_t* packed_codes, const uint8_t* affine,
                    int affine_one, int64_t M, const void* x, int x_dtype, void* y, int y_dtype, void* workspace,
                    hipStream_t s);
// Small-batch kernel (M <= kSkinnyMaxM) on fp16 activations; inv_scale
// (per token, may be null) multiplies the results.  Up to kGemvMaxM tokens
// unisvq_gemm runs the matrix-vector kernel instead (measured on the 7B
// decoder step: 1 token 29 us against 44, 3 tokens 40 against 46, 4 tokens
// 50 against 46), falling back to the small-batch kernel where the
// matrix-vector kernel's LDS cannot hold the activations.
constexpr int64_t kSkinnyMaxM = 32;
constexpr int64_t kGemvMaxM = 3;
hipError_t launch_skinny(int64_t N, int64_t K, const uint8_t* packed, const uint8_t* affine, int affine_one,
                         int64_t M, const _Float16* x, const float* inv_scale, void* y, int y_dtype, hipStream_t s);
// Several independent small-batch products (same M, the same weight format)
// in one launch.
struct SkinnyProblem {
    const uint8_t* packed;
    const uint8_t* affine;
    int affine_one;
    const _Float16* x;
    const float* inv_scale;
    void* y;
    int64_t N, K;
};
hipError_t launch_skinny_batch(const SkinnyProblem* probs, int count, int64_t M, int y_dtype, hipStream_t s);
// unisvq_gemm over a batch of problems (same M and dtypes): one launch of the
// small-batch kernel for M <= kSkinnyMaxM, else one tiled launch (and one
// reduction) for the batch, after the bf16 pre-passes.
// Problem i uses the workspace bytes [off_i, off_i + gemm_workspace_bytes(i)),
// off_i the 256-aligned sum of the earlier ones (gemm_batch_workspace_bytes).
struct GemmBatchProblem {
    const uint8_t* packed;
    const void* x;
    void* y;
    int64_t N, K;
};
size_t gemm_batch_workspace_bytes(const GemmBatchProblem* probs, int count, int64_t M, int x_dtype);
int launch_gemm_batch(const GemmBatchProblem* probs, int count, int64_t M, int x_dtype, int y_dtype, void* workspace,
                      hipStream_t s);

// Raise a kernel's dynamic-LDS limit on the current device, once per
// (kernel, device): `done` is the calling site's bitmask of devices already
// set up (devices past 63 are set up on every call).  Returns a status.
inline int ensure_lds_limit(const void* fn, int bytes, std::atomic<uint64_t>& done) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return UNISVQ_EHIP;
    const uint64_t bit = dev >= 0 && dev < 64 ? uint64_t{1} << dev : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return UNISVQ_OK;
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) != hipSuccess) return UNISVQ_EHIP;
    done.fetch_or(bit, std::memory_order_acq_rel);
    return UNISVQ_OK;
}

// Bandwidth reference: reads `count` byte ranges once (ptrs 16-byte aligned,
// sizes multiples of 16 below 2^31); with `store` each wavefront stores the
// XOR of the words it read to its own sink word (read_sink_words of them),
// without it nothing is written.
int64_t read_sink_words(const int64_t* bytes, int count);
int launch_read(const uint8_t* const* ptrs, const int64_t* bytes, int count, uint32_t* sink, bool store,
                hipStream_t s);

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
