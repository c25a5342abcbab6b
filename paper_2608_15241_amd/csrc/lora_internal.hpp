// Pieces of the LoRA projection shared between source files of the library.
#pragma once
#include <cstddef>
#include <cstdint>

#include "common.hpp"

namespace localk {

// The long-chunk shrink on its own, for G (1..4) projections of one x:
// P[g][z][t][j] = the sum over K slice z of x[t][k] A[g][a_t][j][k] for token
// t's own adapter a_t (tokens without one are not written), j < r_max,
// z < *slices. token_shrink_bytes is the workspace it needs (the partial
// sums first, then a bitmap area); K is a multiple of 64 and T >= 1.
size_t token_shrink_bytes(int64_t T, int64_t K, int r_max, int G, int* slices);
local_status_t token_shrink(const uint16_t* x, int64_t T, int64_t K, int G,
                            const uint16_t* const* A, int n_ad, int r_max, const int32_t* idx,
                            void* ws, hipStream_t s);

}  // namespace localk
