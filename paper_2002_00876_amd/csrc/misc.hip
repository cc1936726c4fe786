// misc.hip -- the degenerate N == 1 case: no edges, every label is free.
// log Z = log C (Sec. 5.2: the first and last label are summed over), the max score is
// the empty sum 0 and the lowest label 0 is the argmax.
#include "device.h"
#include "internal.h"
#include "ts_chain.h"

namespace tsc {
namespace {

__global__ void k_single_token(int64_t B, int64_t N, int64_t C, float* logZ, int32_t* path,
                               float* score) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= B) return;
    if (logZ) logZ[b] = logf((float)C);
    if (path) {
        path[b * N] = 0;
        for (int64_t n = 1; n < N; ++n) path[b * N + n] = -1;
    }
    if (score) score[b] = 0.f;
}

}  // namespace

hipError_t launch_single_token(int64_t B, int64_t N, int64_t C, int op, float* logZ,
                               int32_t* path, float* score, hipStream_t s) {
    (void)op;
    const int threads = 256;
    hipLaunchKernelGGL(k_single_token, dim3((unsigned)((B + threads - 1) / threads)),
                       dim3(threads), 0, s, B, N, C, logZ, path, score);
    return hipGetLastError();
}

}  // namespace tsc
