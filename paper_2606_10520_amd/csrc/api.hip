// C entry points of libunisvq: argument validation (host only, before any
// HIP call) and dispatch to the kernels.
#include <cstring>

#include "common.hpp"

namespace {

bool shape_ok(int64_t N, int64_t K) {
    return N >= unisvq::kRowBlock && K >= unisvq::kGroup && N % unisvq::kRowBlock == 0 &&
           K % unisvq::kGroup == 0 && N <= (int64_t{1} << 31) - 1 && K <= (int64_t{1} << 31) - 1;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool x_dtype_ok(int t) { return t == UNISVQ_F16 || t == UNISVQ_BF16; }
bool y_dtype_ok(int t) { return t == UNISVQ_F16 || t == UNISVQ_BF16 || t == UNISVQ_F32; }

// Common checks of the two product entry points.
int check_product(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype,
                  const void* y, int y_dtype) {
    if (!packed || !x || !y) return UNISVQ_EINVAL;
    if (M < 1 || M > (int64_t{1} << 31) - 1) return UNISVQ_EINVAL;
    if (!x_dtype_ok(x_dtype) || !y_dtype_ok(y_dtype)) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!aligned(packed, 16) || !aligned(x, 16)) return UNISVQ_EALIGN;
    // the kernels address the packed matrix with 32-bit buffer offsets
    if (static_cast<int64_t>(unisvq_packed_bytes(N, K)) > unisvq::kMaxBufferBytes) return UNISVQ_EUNSUP;
    if (!aligned(y, y_dtype == UNISVQ_F32 ? 4 : 2)) return UNISVQ_EALIGN;
    return UNISVQ_OK;
}

// Row-shared affine parameters: one pair per matrix or one per group.
bool affine_groups_ok(int64_t K, int64_t ga) { return ga == 1 || ga == K / unisvq::kGroup; }

int check_shared(int64_t N, int64_t K, int64_t affine_groups, const void* codes, const void* affine, int64_t M,
                 const void* x, int x_dtype, const void* y, int y_dtype) {
    if (!codes || !affine || !x || !y) return UNISVQ_EINVAL;
    if (M < 1 || M > (int64_t{1} << 31) - 1) return UNISVQ_EINVAL;
    if (!x_dtype_ok(x_dtype) || !y_dtype_ok(y_dtype)) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(codes, 16) || !aligned(affine, 16) || !aligned(x, 16)) return UNISVQ_EALIGN;
    if (static_cast<int64_t>(unisvq_codes_bytes(N, K)) > unisvq::kMaxBufferBytes) return UNISVQ_EUNSUP;
    if (!aligned(y, y_dtype == UNISVQ_F32 ? 4 : 2)) return UNISVQ_EALIGN;
    return UNISVQ_OK;
}

// Format variants: (bits, d) = (3, 4), (2, 8), (3, 8).
bool var_ok(int bits, int d) { return (bits == 2 || bits == 3) && (d == 4 || d == 8) && !(bits == 2 && d == 4); }

int64_t var_codes_size(int64_t N, int64_t K, int bits) {
    return (N / unisvq::kRowBlock) * (K / unisvq::kGroup) * unisvq::var_group_bytes(bits);
}

int check_var(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* codes, const void* affine,
              int64_t M, const void* x, int x_dtype, const void* y, int y_dtype) {
    if (!codes || !affine || !x || !y) return UNISVQ_EINVAL;
    if (M < 1 || M > (int64_t{1} << 31) - 1) return UNISVQ_EINVAL;
    if (!x_dtype_ok(x_dtype) || !y_dtype_ok(y_dtype)) return UNISVQ_EINVAL;
    if (!var_ok(bits, d)) return UNISVQ_EUNSUP;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(codes, 16) || !aligned(affine, 16) || !aligned(x, 16)) return UNISVQ_EALIGN;
    if (var_codes_size(N, K, bits) > unisvq::kMaxBufferBytes) return UNISVQ_EUNSUP;
    if (!aligned(y, y_dtype == UNISVQ_F32 ? 4 : 2)) return UNISVQ_EALIGN;
    return UNISVQ_OK;
}

}  // namespace

extern "C" {

int unisvq_version(void) { return UNISVQ_FORMAT_VERSION; }

const char* unisvq_status_string(int status) {
    switch (status) {
        case UNISVQ_OK: return "ok";
        case UNISVQ_EINVAL: return "invalid argument";
        case UNISVQ_ESHAPE: return "invalid shape (need N % 16 == 0, K % 128 == 0)";
        case UNISVQ_EUNSUP: return "unsupported configuration";
        case UNISVQ_EALIGN: return "misaligned pointer";
        case UNISVQ_EHIP: return "HIP runtime error";
        case UNISVQ_EWORKSPACE: return "workspace too small";
        case UNISVQ_ESCRATCH: return "product needs more than the fixed scratch of unisvq_gemm_noalloc";
        default: return "unknown status";
    }
}

size_t unisvq_packed_bytes(int64_t N, int64_t K) {
    if (!shape_ok(N, K)) return 0;
    return static_cast<size_t>(N / unisvq::kRowBlock) * static_cast<size_t>(K / unisvq::kGroup) *
           unisvq::kGroupBlockBytes;
}

int unisvq_pack(int64_t N, int64_t K, const uint8_t* codes, const uint16_t* A, const uint16_t* B,
                void* packed, int32_t* bad_codes, void* stream) {
    if (!codes || !A || !B || !packed) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!aligned(packed, 16) || !aligned(A, 2) || !aligned(B, 2) || (bad_codes && !aligned(bad_codes, 4)))
        return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_pack(N, K, codes, A, B, static_cast<uint8_t*>(packed), bad_codes,
                                             static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int unisvq_unpack(int64_t N, int64_t K, const void* packed, uint8_t* codes, uint16_t* A, uint16_t* B,
                  void* stream) {
    if (!codes || !A || !B || !packed) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!aligned(packed, 16) || !aligned(A, 2) || !aligned(B, 2)) return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_unpack(N, K, static_cast<const uint8_t*>(packed), codes, A, B,
                                               static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int unisvq_gemv(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, void* stream) {
    const int st = check_product(N, K, packed, M, x, x_dtype, y, y_dtype);
    if (st != UNISVQ_OK) return st;
    if (M > 4) return UNISVQ_EUNSUP;
    return unisvq::launch_gemv(N, K, static_cast<const uint8_t*>(packed), M, x, x_dtype, y, y_dtype,
                               static_cast<hipStream_t>(stream));
}

int unisvq_gemv_batched(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype,
                        int y_dtype, void* stream) {
    if (!problems || count < 1) return UNISVQ_EINVAL;
    if (count > UNISVQ_MAX_BATCH) return UNISVQ_EUNSUP;
    unisvq::GemvProblem probs[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        const unisvq_gemv_problem& q = problems[i];
        const int st = check_product(q.N, q.K, q.packed, M, q.x, x_dtype, q.y, y_dtype);
        if (st != UNISVQ_OK) return st;
        probs[i] = unisvq::GemvProblem{static_cast<const uint8_t*>(q.packed), q.x, q.y,
                                       static_cast<int>(q.N), static_cast<int>(q.K), 0};
    }
    if (M > 4) return UNISVQ_EUNSUP;
    return unisvq::launch_gemv_batch(probs, count, M, x_dtype, y_dtype, static_cast<hipStream_t>(stream));
}

int unisvq_gemv_rht_batched(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype, int y_dtype,
                            const int8_t* const* signs, void* stream) {
    if (!problems || count < 1 || !signs) return UNISVQ_EINVAL;
    if (count > UNISVQ_MAX_BATCH) return UNISVQ_EUNSUP;
    unisvq::GemvProblem probs[UNISVQ_MAX_BATCH];
    const signed char* sg[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        const unisvq_gemv_problem& q = problems[i];
        const int st = check_product(q.N, q.K, q.packed, M, q.x, x_dtype, q.y, y_dtype);
        if (st != UNISVQ_OK) return st;
        if (!signs[i]) return UNISVQ_EINVAL;
        if (q.K != problems[0].K || (q.K != 4096 && q.K != 8192)) return UNISVQ_EUNSUP;
        probs[i] = unisvq::GemvProblem{static_cast<const uint8_t*>(q.packed), q.x, q.y,
                                       static_cast<int>(q.N), static_cast<int>(q.K), 0};
        sg[i] = reinterpret_cast<const signed char*>(signs[i]);
    }
    if (M > 4) return UNISVQ_EUNSUP;
    return unisvq::launch_gemv_rht_batch(probs, count, M, x_dtype, y_dtype, sg, static_cast<hipStream_t>(stream));
}

size_t unisvq_gemm_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype) {
    if (!shape_ok(N, K) || M < 1 || M > (int64_t{1} << 31) - 1 || !x_dtype_ok(x_dtype)) return 0;
    return unisvq::gemm_workspace_bytes(N, K, M, x_dtype);
}

int unisvq_gemm(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, void* workspace, size_t workspace_bytes, void* stream) {
    const int st = check_product(N, K, packed, M, x, x_dtype, y, y_dtype);
    if (st != UNISVQ_OK) return st;
    if (x_dtype == UNISVQ_BF16 && K > 65536) return UNISVQ_EUNSUP;  // the bf16 pre-pass holds a row in registers
    const size_t need = unisvq::gemm_workspace_bytes(N, K, M, x_dtype);
    if (need) {
        if (!workspace || workspace_bytes < need) return UNISVQ_EWORKSPACE;
        if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    }
    return unisvq::launch_gemm(N, K, static_cast<const uint8_t*>(packed), M, x, x_dtype, y, y_dtype,
                               workspace, static_cast<hipStream_t>(stream));
}

namespace {

// Validate a batch of product descriptors and convert them (count checked by the caller).
int batch_problems(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype, int y_dtype,
                   unisvq::GemmBatchProblem* out) {
    for (int i = 0; i < count; ++i) {
        const unisvq_gemv_problem& q = problems[i];
        const int st = check_product(q.N, q.K, q.packed, M, q.x, x_dtype, q.y, y_dtype);
        if (st != UNISVQ_OK) return st;
        if (x_dtype == UNISVQ_BF16 && q.K > 65536) return UNISVQ_EUNSUP;
        out[i] = unisvq::GemmBatchProblem{static_cast<const uint8_t*>(q.packed), q.x, q.y, q.N, q.K};
    }
    return UNISVQ_OK;
}

}  // namespace

size_t unisvq_gemm_batched_workspace_bytes(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype) {
    if (!problems || count < 1 || count > UNISVQ_MAX_BATCH || M < 1 || !x_dtype_ok(x_dtype)) return 0;
    unisvq::GemmBatchProblem probs[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        if (!shape_ok(problems[i].N, problems[i].K)) return 0;
        probs[i] = unisvq::GemmBatchProblem{nullptr, nullptr, nullptr, problems[i].N, problems[i].K};
    }
    return unisvq::gemm_batch_workspace_bytes(probs, count, M, x_dtype);
}

int unisvq_gemm_batched(const unisvq_gemv_problem* problems, int count, int64_t M, int x_dtype, int y_dtype,
                        void* workspace, size_t workspace_bytes, void* stream) {
    if (!problems || count < 1) return UNISVQ_EINVAL;
    if (count > UNISVQ_MAX_BATCH) return UNISVQ_EUNSUP;
    unisvq::GemmBatchProblem probs[UNISVQ_MAX_BATCH];
    const int st = batch_problems(problems, count, M, x_dtype, y_dtype, probs);
    if (st != UNISVQ_OK) return st;
    const size_t need = unisvq::gemm_batch_workspace_bytes(probs, count, M, x_dtype);
    if (need) {
        if (!workspace || workspace_bytes < need) return UNISVQ_EWORKSPACE;
        if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    }
    return unisvq::launch_gemm_batch(probs, count, M, x_dtype, y_dtype, workspace, static_cast<hipStream_t>(stream));
}

/* ---- row-shared affine parameters ---- */

size_t unisvq_codes_bytes(int64_t N, int64_t K) {
    if (!shape_ok(N, K)) return 0;
    return static_cast<size_t>(N / unisvq::kRowBlock) * static_cast<size_t>(K / unisvq::kGroup) *
           unisvq::kCodeGroupBlockBytes;
}

size_t unisvq_shared_affine_bytes(int64_t K, int64_t affine_groups) {
    if (K < unisvq::kGroup || K % unisvq::kGroup || K > (int64_t{1} << 31) - 1) return 0;
    if (!affine_groups_ok(K, affine_groups)) return 0;
    const int64_t records = affine_groups == 1 ? 1 : (K / unisvq::kGroup + 1) / 2;
    return static_cast<size_t>(records) * unisvq::kAffineRecordBytes;
}

int unisvq_pack_shared(int64_t N, int64_t K, int64_t affine_groups, const uint8_t* codes, const uint16_t* A,
                       const uint16_t* B, void* packed_codes, void* packed_affine, int32_t* bad_codes,
                       void* stream) {
    if (!codes || !A || !B || !packed_codes || !packed_affine) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(packed_codes, 16) || !aligned(packed_affine, 16) || !aligned(A, 2) || !aligned(B, 2) ||
        (bad_codes && !aligned(bad_codes, 4)))
        return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_pack_shared(N, K, affine_groups, codes, A, B,
                                                    static_cast<uint8_t*>(packed_codes),
                                                    static_cast<uint8_t*>(packed_affine), bad_codes,
                                                    static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int unisvq_unpack_shared(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                         const void* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B, void* stream) {
    if (!codes || !A || !B || !packed_codes || !packed_affine) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(packed_codes, 16) || !aligned(packed_affine, 16) || !aligned(A, 2) || !aligned(B, 2))
        return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_unpack_shared(N, K, affine_groups, static_cast<const uint8_t*>(packed_codes),
                                                      static_cast<const uint8_t*>(packed_affine), codes, A, B,
                                                      static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int unisvq_gemv_shared(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                       const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                       void* stream) {
    const unisvq_gemv_shared_problem p{N, K, affine_groups, packed_codes, packed_affine, x, y};
    return unisvq_gemv_shared_batched(&p, 1, M, x_dtype, y_dtype, stream);
}

int unisvq_gemv_shared_batched(const unisvq_gemv_shared_problem* problems, int count, int64_t M, int x_dtype,
                               int y_dtype, void* stream) {
    if (!problems || count < 1) return UNISVQ_EINVAL;
    if (count > UNISVQ_MAX_BATCH) return UNISVQ_EUNSUP;
    unisvq::GemvProblem probs[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        const unisvq_gemv_shared_problem& q = problems[i];
        const int st = check_shared(q.N, q.K, q.affine_groups, q.packed_codes, q.packed_affine, M, q.x, x_dtype,
                                    q.y, y_dtype);
        if (st != UNISVQ_OK) return st;
        probs[i] = unisvq::GemvProblem{static_cast<const uint8_t*>(q.packed_codes), q.x, q.y,
                                       static_cast<int>(q.N), static_cast<int>(q.K), 0,
                                       static_cast<const uint8_t*>(q.packed_affine), q.affine_groups == 1 ? 1 : 0};
    }
    if (M > 4) return UNISVQ_EUNSUP;
    return unisvq::launch_gemv_batch(probs, count, M, x_dtype, y_dtype, static_cast<hipStream_t>(stream));
}

int unisvq_gemm_shared(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                       const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                       void* workspace, size_t workspace_bytes, void* stream) {
    const int st = check_shared(N, K, affine_groups, packed_codes, packed_affine, M, x, x_dtype, y, y_dtype);
    if (st != UNISVQ_OK) return st;
    if (x_dtype == UNISVQ_BF16 && K > 65536) return UNISVQ_EUNSUP;  // the bf16 pre-pass holds a row in registers
    const size_t need = unisvq::gemm_workspace_bytes(N, K, M, x_dtype);
    if (need) {
        if (!workspace || workspace_bytes < need) return UNISVQ_EWORKSPACE;
        if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    }
    return unisvq::launch_gemm_shared(N, K, static_cast<const uint8_t*>(packed_codes),
                                      static_cast<const uint8_t*>(packed_affine), affine_groups == 1 ? 1 : 0, M, x,
                                      x_dtype, y, y_dtype, workspace, static_cast<hipStream_t>(stream));
}

size_t unisvq_gemm_fold_workspace_bytes(int64_t N, int64_t K, int64_t M) {
    if (!shape_ok(N, K) || M < 1) return 0;
    return unisvq::gemm_fold_workspace_bytes(N, K, M);
}

int unisvq_gemm_shared_fold(int64_t N, int64_t K, int64_t affine_groups, const void* packed_codes,
                            const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                            void* workspace, size_t workspace_bytes, void* stream) {
    const int st = check_shared(N, K, affine_groups, packed_codes, packed_affine, M, x, x_dtype, y, y_dtype);
    if (st != UNISVQ_OK) return st;
    const size_t need = unisvq::gemm_fold_workspace_bytes(N, K, M);
    if (!workspace || workspace_bytes < need) return UNISVQ_EWORKSPACE;
    if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    return unisvq::launch_gemm_fold(N, K, static_cast<const uint8_t*>(packed_codes),
                                    static_cast<const uint8_t*>(packed_affine), affine_groups == 1 ? 1 : 0, M, x,
                                    x_dtype, y, y_dtype, workspace, static_cast<hipStream_t>(stream));
}

/* ---- format variants ---- */

size_t unisvq_var_codes_bytes(int64_t N, int64_t K, int bits, int d) {
    if (!shape_ok(N, K) || !var_ok(bits, d)) return 0;
    return static_cast<size_t>(var_codes_size(N, K, bits));
}

size_t unisvq_var_affine_bytes(int64_t K, int64_t affine_groups, int bits, int d) {
    if (K < unisvq::kGroup || K % unisvq::kGroup || K > (int64_t{1} << 31) - 1) return 0;
    if (!var_ok(bits, d) || !affine_groups_ok(K, affine_groups)) return 0;
    const int64_t records = affine_groups == 1 ? 1 : (K / unisvq::kGroup + 1) / 2;
    return static_cast<size_t>(records) * unisvq::var_record_bytes(d);
}

int unisvq_var_pack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const uint8_t* codes,
                    const uint16_t* A, const uint16_t* B, void* packed_codes, void* packed_affine, int32_t* bad_codes,
                    void* stream) {
    if (!codes || !A || !B || !packed_codes || !packed_affine) return UNISVQ_EINVAL;
    if (!var_ok(bits, d)) return UNISVQ_EUNSUP;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(packed_codes, 16) || !aligned(packed_affine, 16) || !aligned(A, 2) || !aligned(B, 2) ||
        (bad_codes && !aligned(bad_codes, 4)))
        return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_var_pack(N, K, bits, d, affine_groups, codes, A, B,
                                                 static_cast<uint8_t*>(packed_codes),
                                                 static_cast<uint8_t*>(packed_affine), bad_codes,
                                                 static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int unisvq_var_unpack(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* packed_codes,
                      const void* packed_affine, uint8_t* codes, uint16_t* A, uint16_t* B, void* stream) {
    if (!codes || !A || !B || !packed_codes || !packed_affine) return UNISVQ_EINVAL;
    if (!var_ok(bits, d)) return UNISVQ_EUNSUP;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (!affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(packed_codes, 16) || !aligned(packed_affine, 16) || !aligned(A, 2) || !aligned(B, 2))
        return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_var_unpack(N, K, bits, d, affine_groups,
                                                   static_cast<const uint8_t*>(packed_codes),
                                                   static_cast<const uint8_t*>(packed_affine), codes, A, B,
                                                   static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

int unisvq_var_gemv(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* packed_codes,
                    const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                    void* stream) {
    const unisvq_gemv_shared_problem p{N, K, affine_groups, packed_codes, packed_affine, x, y};
    return unisvq_var_gemv_batched(&p, 1, bits, d, M, x_dtype, y_dtype, stream);
}

int unisvq_var_gemv_batched(const unisvq_gemv_shared_problem* problems, int count, int bits, int d, int64_t M,
                            int x_dtype, int y_dtype, void* stream) {
    if (!problems || count < 1) return UNISVQ_EINVAL;
    if (count > UNISVQ_MAX_BATCH) return UNISVQ_EUNSUP;
    unisvq::GemvProblem probs[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        const unisvq_gemv_shared_problem& q = problems[i];
        const int st = check_var(q.N, q.K, bits, d, q.affine_groups, q.packed_codes, q.packed_affine, M, q.x,
                                 x_dtype, q.y, y_dtype);
        if (st != UNISVQ_OK) return st;
        probs[i] = unisvq::GemvProblem{static_cast<const uint8_t*>(q.packed_codes), q.x, q.y,
                                       static_cast<int>(q.N), static_cast<int>(q.K), 0,
                                       static_cast<const uint8_t*>(q.packed_affine), q.affine_groups == 1 ? 1 : 0};
    }
    if (M > 4) return UNISVQ_EUNSUP;
    return unisvq::launch_gemv_var_batch(probs, count, M, x_dtype, y_dtype, bits, d,
                                         static_cast<hipStream_t>(stream));
}

size_t unisvq_var_gemm_workspace_bytes(int64_t N, int64_t K, int64_t M, int x_dtype) {
    if (!shape_ok(N, K) || M < 1 || M > (int64_t{1} << 31) - 1 || !x_dtype_ok(x_dtype)) return 0;
    return unisvq::gemm_var_workspace_bytes(N, K, M, x_dtype);
}

int unisvq_var_gemm(int64_t N, int64_t K, int bits, int d, int64_t affine_groups, const void* packed_codes,
                    const void* packed_affine, int64_t M, const void* x, int x_dtype, void* y, int y_dtype,
                    void* workspace, size_t workspace_bytes, void* stream) {
    const int st = check_var(N, K, bits, d, affine_groups, packed_codes, packed_affine, M, x, x_dtype, y, y_dtype);
    if (st != UNISVQ_OK) return st;
    if (x_dtype == UNISVQ_BF16 && K > 65536) return UNISVQ_EUNSUP;  // the bf16 pre-pass holds a row in registers
    const size_t need = unisvq::gemm_var_workspace_bytes(N, K, M, x_dtype);
    if (need) {
        if (!workspace || workspace_bytes < need) return UNISVQ_EWORKSPACE;
        if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    }
    return unisvq::launch_gemm_var(N, K, bits, d, static_cast<const uint8_t*>(packed_codes),
                                   static_cast<const uint8_t*>(packed_affine), affine_groups == 1 ? 1 : 0, M, x,
                                   x_dtype, y, y_dtype, workspace, static_cast<hipStream_t>(stream));
}

/* ---- nearest-codeword quantisation ---- */

int unisvq_quantize(int64_t N, int64_t K, const float* W, const uint16_t* A, const uint16_t* B,
                    int64_t affine_groups, uint8_t* codes, void* stream) {
    if (!W || !A || !B || !codes) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (affine_groups != 0 && !affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(W, 16) || !aligned(A, 2) || !aligned(B, 2) || !aligned(codes, 4)) return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_quantize(N, K, W, A, B, affine_groups, codes,
                                                 static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

/* ---- LDLQ ---- */

size_t unisvq_ldlq_workspace_bytes(int64_t N, int64_t K) {
    if (!shape_ok(N, K)) return 0;
    return unisvq::ldlq_workspace_bytes(N, K);
}

int unisvq_ldlq(int64_t N, int64_t K, const float* W, const double* U, const uint16_t* A, const uint16_t* B,
                int64_t affine_groups, uint8_t* codes, void* workspace, size_t workspace_bytes, void* stream) {
    if (!W || !U || !A || !B || !codes) return UNISVQ_EINVAL;
    if (!shape_ok(N, K)) return UNISVQ_ESHAPE;
    if (affine_groups != 0 && !affine_groups_ok(K, affine_groups)) return UNISVQ_EINVAL;
    if (!aligned(W, 16) || !aligned(U, 16) || !aligned(A, 2) || !aligned(B, 2) || !aligned(codes, 4))
        return UNISVQ_EALIGN;
    if (!workspace || workspace_bytes < unisvq::ldlq_workspace_bytes(N, K)) return UNISVQ_EWORKSPACE;
    if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_ldlq(N, K, W, U, A, B, affine_groups, codes, workspace,
                                             static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

/* ---- block LDL^T factorisation of the Hessian ---- */

size_t unisvq_ldl_workspace_bytes(int64_t K) {
    if (K < unisvq::kGroup || K % unisvq::kGroup || K > 32768) return 0;
    return unisvq::ldl_workspace_bytes(K);
}

int unisvq_ldl(int64_t K, const double* H, double* U, double* D, int32_t* info, void* workspace,
               size_t workspace_bytes, void* stream) {
    if (!H || !U) return UNISVQ_EINVAL;
    if (K < unisvq::kGroup || K % unisvq::kGroup || K > 32768) return UNISVQ_ESHAPE;
    if (!aligned(H, 16) || !aligned(U, 16) || (D && !aligned(D, 8)) || (info && !aligned(info, 4)))
        return UNISVQ_EALIGN;
    // U may be H itself (in place) but must not overlap it otherwise; D and
    // info must not overlap either of them
    const uintptr_t bytes = static_cast<uintptr_t>(K) * static_cast<uintptr_t>(K) * 8;
    const uintptr_t h0 = reinterpret_cast<uintptr_t>(H), u0 = reinterpret_cast<uintptr_t>(U);
    if (h0 != u0 && h0 < u0 + bytes && u0 < h0 + bytes) return UNISVQ_EINVAL;
    auto clash = [&](const void* p, uintptr_t n) {
        const uintptr_t q = reinterpret_cast<uintptr_t>(p);
        return (q < h0 + bytes && h0 < q + n) || (q < u0 + bytes && u0 < q + n);
    };
    if ((D && clash(D, static_cast<uintptr_t>(K) * 4 * 8)) || (info && clash(info, 4))) return UNISVQ_EINVAL;
    if (!workspace || workspace_bytes < unisvq::ldl_workspace_bytes(K)) return UNISVQ_EWORKSPACE;
    if (!aligned(workspace, 16)) return UNISVQ_EALIGN;
    const hipError_t e = unisvq::launch_ldl(K, H, U, D, info, workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

/* ---- randomized Hadamard transform ---- */

int unisvq_rht(int64_t n, int64_t M, const void* x, int x_dtype, const int8_t* signs, int mode, void* y, int y_dtype,
               void* stream) {
    if (!x || !signs || !y) return UNISVQ_EINVAL;
    if (n < 1 || M < 1 || M > 65535 || (mode != 0 && mode != 1)) return UNISVQ_EINVAL;
    if (!y_dtype_ok(x_dtype) || !y_dtype_ok(y_dtype)) return UNISVQ_EINVAL;  // F16, BF16 or F32 on both sides
    const size_t xb = x_dtype == UNISVQ_F32 ? 4 : 2, yb = y_dtype == UNISVQ_F32 ? 4 : 2;
    if (!aligned(x, xb) || !aligned(y, yb)) return UNISVQ_EALIGN;
    // x and y may not overlap: several workgroups read a row while others write it
    const uintptr_t x0 = reinterpret_cast<uintptr_t>(x), y0 = reinterpret_cast<uintptr_t>(y);
    const uintptr_t x1 = x0 + static_cast<uintptr_t>(n * M) * xb, y1 = y0 + static_cast<uintptr_t>(n * M) * yb;
    if (x0 < y1 && y0 < x1) return UNISVQ_EINVAL;
    return unisvq::launch_rht(n, M, x, x_dtype, reinterpret_cast<const signed char*>(signs), mode, y, y_dtype,
                              static_cast<hipStream_t>(stream));
}

/* ---- the product without a caller workspace ---- */

size_t unisvq_noalloc_scratch_bytes(void) { return unisvq::noalloc_scratch_bytes(); }

int unisvq_gemm_noalloc(int64_t N, int64_t K, const void* packed, int64_t M, const void* x, int x_dtype, void* y,
                        int y_dtype, void* stream) {
    const int st = check_product(N, K, packed, M, x, x_dtype, y, y_dtype);
    if (st != UNISVQ_OK) return st;
    if (x_dtype == UNISVQ_BF16 && K > 65536) return UNISVQ_EUNSUP;  // as unisvq_gemm
    return unisvq::launch_gemm_noalloc(N, K, static_cast<const uint8_t*>(packed), M, x, x_dtype, y, y_dtype,
                                       static_cast<hipStream_t>(stream));
}

/* ---- bandwidth reference ---- */

int64_t unisvq_read_sink_words(const unisvq_byte_range* ranges, int count) {
    if (!ranges || count < 1 || count > UNISVQ_MAX_BATCH) return 0;
    int64_t bytes[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        if (ranges[i].bytes < 0 || ranges[i].bytes > unisvq::kMaxBufferBytes) return 0;
        bytes[i] = ranges[i].bytes;
    }
    return unisvq::read_sink_words(bytes, count);
}

int unisvq_read_bytes(const unisvq_byte_range* ranges, int count, int store, uint32_t* sink, int64_t sink_words,
                      void* stream) {
    if (!ranges || count < 1 || (store && !sink)) return UNISVQ_EINVAL;
    if (count > UNISVQ_MAX_BATCH) return UNISVQ_EUNSUP;
    if (store && !aligned(sink, 4)) return UNISVQ_EALIGN;
    const uint8_t* ptrs[UNISVQ_MAX_BATCH];
    int64_t bytes[UNISVQ_MAX_BATCH];
    for (int i = 0; i < count; ++i) {
        if (ranges[i].bytes < 0 || ranges[i].bytes % 16 || ranges[i].bytes > unisvq::kMaxBufferBytes)
            return UNISVQ_EINVAL;
        if (ranges[i].bytes > 0 && !ranges[i].ptr) return UNISVQ_EINVAL;
        if (!aligned(ranges[i].ptr, 16)) return UNISVQ_EALIGN;
        ptrs[i] = static_cast<const uint8_t*>(ranges[i].ptr);
        bytes[i] = ranges[i].bytes;
    }
    if (store && sink_words < unisvq::read_sink_words(bytes, count)) return UNISVQ_EWORKSPACE;
    return unisvq::launch_read(ptrs, bytes, count, sink, store != 0, static_cast<hipStream_t>(stream));
}

}  // extern "C"
