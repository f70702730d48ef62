// Decode-phase product for the format variants: b-bit codes (b = 2, 3;
// Sec. 5.2.5) and d-dimensional vectors (d = 4, 8; Sec. 5.2.3), codes-only
// with row-shared pairs.  Same kernel as the 2-bit, d = 4 path
// (gemv_kernel.hpp), instantiated for each (b, d).
#include "gemv_kernel.hpp"

namespace unisvq {
namespace {

// (b = 2, d = 4 is the codes-only format of the main path, not a variant.)
// Geometry: 8 wavefronts per 16-row block and 2 packets in flight (a d = 8
// packet holds 64 bytes of A columns per lane); the activations of the run's
// packets load up front (plan_qx).
template <typename XT, int BITS, int D, int MT>
int launch_var_mt(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    (void)minK;
    const int per = (maxK / kGroup / 2 + 7) / 8;
    const int qx = plan_qx(per + ((maxK / kGroup) & 1), MT);
    if (qx <= 1) return launch_cfg<XT, true, 8, MT, 2, 1, BITS, D>(b, blocks, maxK, s);
    if (qx == 2) return launch_cfg<XT, true, 8, MT, 2, 2, BITS, D>(b, blocks, maxK, s);
    return launch_cfg<XT, true, 8, MT, 2, (MT > 1 ? 4 : 8), BITS, D>(b, blocks, maxK, s);
}

template <typename XT, int BITS, int D>
int launch_var_tokens(const GemvBatch& b, int blocks, int minK, int maxK, hipStream_t s) {
    if (b.M == 1) return launch_var_mt<XT, BITS, D, 1>(b, blocks, minK, maxK, s);
    if (b.M == 2) return launch_var_mt<XT, BITS, D, 2>(b, blocks, minK, maxK, s);
    if (b.M == 3) return launch_var_mt<XT, BITS, D, 3>(b, blocks, minK, maxK, s);
    return launch_var_mt<XT, BITS, D, 4>(b, blocks, minK, maxK, s);
}

template <typename XT>
int launch_var_format(const GemvBatch& b, int blocks, int minK, int maxK, int bits, int d, hipStream_t s) {
    if (bits == 3 && d == 4) return launch_var_tokens<XT, 3, 4>(b, blocks, minK, maxK, s);
    if (bits == 2 && d == 8) return launch_var_tokens<XT, 2, 8>(b, blocks, minK, maxK, s);
    if (bits == 3 && d == 8) return launch_var_tokens<XT, 3, 8>(b, blocks, minK, maxK, s);
    return UNISVQ_EUNSUP;
}

}  // namespace

int launch_gemv_var_batch(const GemvProblem* probs, int count, int64_t M, int x_dtype, int y_dtype, int bits, int d,
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
    if (x_dtype == UNISVQ_F16) return launch_var_format<_Float16>(b, blocks, minK, maxK, bits, d, s);
    return launch_var_format<__bf16>(b, blocks, minK, maxK, bits, d, s);
}

}  // namespace unisvq
