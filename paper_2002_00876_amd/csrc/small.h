// small.h -- limits and launchers of the fused single-launch path (small.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tsc {

constexpr int kSmallMaxLabels = 32;     // one wave computes a whole 32 x 32 product
constexpr int kSmallMaxEdges = 1024;
constexpr int kSmallMaxLevels = 12;     // ceil(log2(kSmallMaxEdges)) + 2
constexpr size_t kSmallLdsBytes = 159 * 1024;   // dynamic LDS; static holds the tree table

// exact number of tree nodes over all levels for E leaves (levels of ceil(E / 2^l))
__host__ __device__ inline int64_t small_tree_nodes(int64_t E) {
    int64_t total = E, n = E;
    while (n > 1) { n = (n + 1) / 2; total += n; }
    return total;
}

size_t small_log_lds_bytes(int64_t E, int64_t C);
size_t small_max_lds_bytes(int64_t E, int64_t C);
// true when every sequence of (N, C) fits the fused path's LDS budget
bool small_path_fits(int64_t N, int64_t C);

hipError_t launch_small_log(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                            int64_t C, float* logZ, float* marg, hipStream_t s);
hipError_t launch_small_max(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                            int64_t C, int32_t* path, float* score, hipStream_t s);
// both passes in one launch of 2B workgroups (marginals in the first B, Viterbi in the rest)
hipError_t launch_small_both(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                             int64_t C, float* logZ, float* marg, int32_t* path, float* score,
                             hipStream_t s);

}  // namespace tsc
