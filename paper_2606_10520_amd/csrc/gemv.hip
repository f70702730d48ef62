// Decode-phase product for the 2-bit, d = 4 formats (per-(row, group) pairs
// in packed format v1, or codes-only with row-shared pairs): launch planning
// and entry points.  The kernel is in gemv_kernel.hpp.
#include "gemv_kernel.hpp"

namespace unisvq {
namespace {

// QX (packets per wavefront whose activations load up front): 1, 2, 4, 8
// for one token, up to 4 for two, up to 2 for three or four (plan_qx).
template <typename XT, bool SHARED, int WAVES, int MT, int PF>
int launch_qx(const GemvBatch& b, int blocks, int maxK, int qx, hipStream_t s) {
    if (qx <= 1) return launch_cfg<XT, SHARED, WAVES, MT, PF, 1>(b, blocks, maxK, s);
    if constexpr (MT >= 3) {
        return launch_cfg<XT, SHARED, WAVES, MT, PF, 2>(b, blocks, maxK, s);
    } else {
        if (qx == 2) return launch_cfg<XT, SHARED, WAVES, MT, PF, 2>(b, blocks, maxK, s);
        if constexpr (MT == 2) {
            return launch_cfg<XT, SHARED, WAVES, MT, PF, 4>(b, blocks, maxK, s);
        } else {
            if (qx == 4) return launch_cfg<XT, SHARED, WAVES, MT, PF, 4>(b, blocks, maxK, s);
            return launch_cfg<XT, SHARED, WAVES, MT, PF, 8>(b, blocks, maxK, s);
        }
    }
}

template <typename XT, bool SHARED, int WAVES, int MT>
int launch_pf(const GemvBatch& b, int blocks, int maxK, const GemvPlan& p, hipStream_t s) {
    if (p.pf == 2) return launch_qx<XT, SHARED, WAVES, MT, 2>(b, blocks, maxK, p.qx, s);
    return launch_qx<XT, SHARED, WAVES, MT, 4>(b, blocks, maxK, p.qx, s);
}

template <typename XT, bool SHARED, int MT>
int launch_waves(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    const GemvPlan p = plan_gemv(blocks, minK / kGroup, maxK / kGroup, b.M);
    if (MT == 1 && p.waves == 16) return launch_pf<XT, SHARED, 16, 1>(b, blocks, maxK, p, s);
    return launch_pf<XT, SHARED, 8, MT>(b, blocks, maxK, p, s);
}

// The token count is a template parameter (no per-token guards in the loop).
template <typename XT, bool SHARED>
int launch_tokens(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    if (b.M == 1) return launch_waves<XT, SHARED, 1>(b, blocks, minK, maxK, s);
    if (b.M == 2) return launch_waves<XT, SHARED, 2>(b, blocks, minK, maxK, s);
    if (b.M == 3) return launch_waves<XT, SHARED, 3>(b, blocks, minK, maxK, s);
    return launch_waves<XT, SHARED, 4>(b, blocks, minK, maxK, s);
}

}  // namespace

int launch_gemv_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype,
                      hipStream_t s) {
    if (M > 4 || count < 1 || count > kMaxBatch) return UNISVQ_EUNSUP;
    GemvBatch b{};
    int blocks = 0, maxK = 0, minK = 1 << 30;
    for (int i = 0; i < count; ++i) {
        b.p[i] = probs[i];
        b.p[i].rb_begin = blocks;
        blocks += probs[i].N / kRowBlock;
        maxK = probs[i].K > maxK ? probs[i].K : maxK;
        minK = probs[i].K < minK ? probs[i].K : minK;
    }
    b.count = count;
    b.M = static_cast<int>(M);
    b.y_dtype = y_dtype;
    // every problem of a batch has the same weight format (checked by the caller)
    const bool shared = probs[0].affine != nullptr;
    if (x_dtype == UNISVQ_F16)
        return shared ? launch_tokens<_Float16, true>(b, blocks, minK, maxK, s)
                      : launch_tokens<_Float16, false>(b, blocks, minK, maxK, s);
    return shared ? launch_tokens<__bf16, true>(b, blocks, minK, maxK, s)
                  : launch_tokens<__bf16, false>(b, blocks, minK, maxK, s);
}

int launch_gemv(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype,
                void* y, int y_dtype, hipStream_t s) {
    GemvProblem p{packed, x, y, static_cast<int>(N), static_cast<int>(K), 0, nullptr, 0};
    return launch_gemv_batch(&p, 1, M, x_dtype, y_dtype, s);
}

}  // namespace unisvq
