// Walsh-Hadamard butterflies in registers and across the lanes of a
// wavefront (gfx950), shared by the standalone transform and the matrix-
// vector kernel's fused input transform.  Internal header.
#pragma once

#include "common.hpp"

namespace unisvq {
namespace {

// The value of lane (lane ^ D), all on the vector ALU.  Inside a row of 16
// lanes through DPP: quad permutes for D = 1, 2; for D = 4 the lanes with
// bit 2 clear take row_shl:4 (lane + 4) and the others row_shr:4 (lane - 4);
// for D = 8 row_ror:8 (rotation by half a row is lane ^ 8).  Across rows
// through gfx950's row swaps with both operands the value itself: the
// 16-lane swap (odd rows of the first operand with even rows of the second)
// leaves rows (0, 0, 2, 2) in the first result and (1, 1, 3, 3) in the
// second; the 32-lane swap (upper half of the first with lower half of the
// second) leaves halves (0, 0) and (1, 1).
template <int D>
__device__ inline float lane_xor(float v, int lane) {
    const int b = __builtin_bit_cast(int, v);
    if constexpr (D == 1)
        return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(b, 0xB1, 0xf, 0xf, false));
    else if constexpr (D == 2)
        return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(b, 0x4E, 0xf, 0xf, false));
    else if constexpr (D == 4) {
        const int up = __builtin_amdgcn_mov_dpp(b, 0x104, 0xf, 0xf, false);    // row_shl:4
        const int down = __builtin_amdgcn_mov_dpp(b, 0x114, 0xf, 0xf, false);  // row_shr:4
        return __builtin_bit_cast(float, (lane & 4) ? down : up);
    } else if constexpr (D == 8) {
        return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(b, 0x128, 0xf, 0xf, false));  // row_ror:8
    } else if constexpr (D == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(static_cast<unsigned>(b), static_cast<unsigned>(b), false, false);
        return __builtin_bit_cast(float, (lane & 16) ? r[0] : r[1]);
    } else {
        static_assert(D == 32, "lane distances 1 .. 32");
        const auto r = __builtin_amdgcn_permlane32_swap(static_cast<unsigned>(b), static_cast<unsigned>(b), false, false);
        return __builtin_bit_cast(float, (lane & 32) ? r[0] : r[1]);
    }
}

// Butterflies over register-index bit J (registers r and r | 1 << J).
template <int R, int J>
__device__ inline void reg_stage(float (&v)[R]) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (r & (1 << J)) continue;
        const float a = v[r], b = v[r | (1 << J)];
        v[r] = a + b;
        v[r | (1 << J)] = a - b;
    }
}

template <int R, int J0, int J1>
__device__ inline void reg_stages(float (&v)[R]) {
    if constexpr (J0 < J1) {
        reg_stage<R, J0>(v);
        reg_stages<R, J0 + 1, J1>(v);
    }
}

template <int R, int D>
__device__ inline void lane_stage(float (&v)[R], int lane) {
    const bool hi = lane & D;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float p = lane_xor<D>(v[r], lane);
        v[r] = hi ? p - v[r] : v[r] + p;
    }
}

}  // namespace
}  // namespace unisvq
