// Matrix-vector product with the input-side randomized Hadamard transform of
// Eq. 5 fused in (2-bit d = 4 weights with per-(row, group) pairs, K = 4096
// or 8192): each workgroup transforms the activation rows itself while its
// first packets are in flight, so the rotated layer needs no separate input
// launch.  The kernel is gemv_kernel with RHTK = log2(K) (gemv_kernel.hpp).
#include <cmath>

#include "gemv_kernel.hpp"

namespace unisvq {
namespace {

template <typename XT, int WAVES, int MT, int PF, int KLOG>
int launch_rht_cfg(const GemvBatch& b, int blocks, hipStream_t s) {
    const size_t lds = gemv_rht_lds_bytes(1 << KLOG, MT, WAVES);
    if (lds > kMaxLds) return UNISVQ_EUNSUP;
    static std::atomic<uint64_t> attr_done{0};
    const int st = ensure_lds_limit(reinterpret_cast<const void*>(&gemv_kernel<XT, WAVES, MT, PF, 1, 1, false, 2, 4, KLOG>),
                                    static_cast<int>(kMaxLds), attr_done);
    if (st != UNISVQ_OK) return st;
    hipLaunchKernelGGL((gemv_kernel<XT, WAVES, MT, PF, 1, 1, false, 2, 4, KLOG>), dim3(static_cast<unsigned>(blocks)),
                       dim3(WAVES * 64), lds, s, b);
    return hipGetLastError() == hipSuccess ? UNISVQ_OK : UNISVQ_EHIP;
}

// The launch geometry of the plain product (plan_gemv): the same wavefront
// split of K, hence the same summation order, so the fused product equals
// the two-launch path to the bit.
template <typename XT, int KLOG>
int launch_rht_tokens(const GemvBatch& b, int blocks, hipStream_t s) {
    const int groups = (1 << KLOG) / kGroup;
    const GemvPlan p = plan_gemv(blocks, groups, groups, b.M);
    if (b.M == 1) {
        if (p.waves == 16)
            return p.pf == 4 ? launch_rht_cfg<XT, 16, 1, 4, KLOG>(b, blocks, s) : launch_rht_cfg<XT, 16, 1, 2, KLOG>(b, blocks, s);
        return p.pf == 4 ? launch_rht_cfg<XT, 8, 1, 4, KLOG>(b, blocks, s) : launch_rht_cfg<XT, 8, 1, 2, KLOG>(b, blocks, s);
    }
    if (b.M == 2) return launch_rht_cfg<XT, 8, 2, 2, KLOG>(b, blocks, s);
    if (b.M == 3) return launch_rht_cfg<XT, 8, 3, 2, KLOG>(b, blocks, s);
    return launch_rht_cfg<XT, 8, 4, 2, KLOG>(b, blocks, s);
}

}  // namespace

int launch_gemv_rht_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype,
                          const signed char* const* signs, hipStream_t s) {
    if (M > 4 || count < 1 || count > kMaxBatch) return UNISVQ_EUNSUP;
    const int K = probs[0].K;
    if (K != 4096 && K != 8192) return UNISVQ_EUNSUP;
    GemvBatch b{};
    int blocks = 0;
    for (int i = 0; i < count; ++i) {
        if (probs[i].K != K) return UNISVQ_EUNSUP;
        b.p[i] = probs[i];
        b.p[i].rb_begin = blocks;
        blocks += probs[i].N / kRowBlock;
        b.signs[i] = signs[i];
    }
    b.count = count;
    b.M = static_cast<int>(M);
    b.y_dtype = y_dtype;
    // the same value as the standalone transform's normalisation
    b.rht_norm = static_cast<float>(1.0 / std::sqrt(static_cast<double>(K)));
    if (x_dtype == UNISVQ_F16)
        return K == 4096 ? launch_rht_tokens<_Float16, 12>(b, blocks, s) : launch_rht_tokens<_Float16, 13>(b, blocks, s);
    return K == 4096 ? launch_rht_tokens<__bf16, 12>(b, blocks, s) : launch_rht_tokens<__bf16, 13>(b, blocks, s);
}

}  // namespace unisvq
