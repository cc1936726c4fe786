// semimarkov.hip -- the semi-Markov CRF (Table 1, "Semi-Markov": segment labels, parts
// N K C^2) on the same parallel scan as the linear chain (Sec. 6a notes that the scan
// carries over to semi-Markov models).
//
// Segment potentials sp[b, t, k-1, i, j] score a segment of length k that starts at step t
// with label j after a segment labelled i (steps t = 0..E-1 are the chain's edges, E = L-1;
// the first segment follows a free initial label).  The segmentation is a linear chain over
// K*C expanded states s = (c, r) = r*C + c at each boundary: c is the label of the segment
// in progress and r the steps it still has to run.  Per step t the expanded edge is
//   (i, 0) -> (j, k-1): sp[t, k-1, i, j]   (a segment of length k starts at step t)
//   (c, r) -> (c, r-1): 0                  (r >= 1: the segment runs on)
// and -inf otherwise; at step 0 only states with r = 0 may start (no segment in progress),
// and after the last step only states with r = 0 may end (no segment overruns the end).
// Every segmentation is exactly one expanded path with the same score, so the chain's log Z,
// marginals and Viterbi over the expanded edges give the semi-Markov ones:
//   mu_semi[t, k-1, i, j] = mu_chain[t, (i,0), (j,k-1)],
//   a segment starts at step t iff r_t = 0, and its length is r_{t+1} + 1.
// Ordering the states r-major makes the chain's lowest-index backtrace take, at every
// segment end, the shortest segment and then the lowest previous label among the maximisers.
// One token: log Z = log C (a free label), where the expanded chain would give log(K C).
#include "device.h"
#include "internal.h"

namespace tsc {
namespace {

constexpr int kSemiThreads = 256;

// one workgroup per valid step (b, t); waves over expanded rows, lanes over columns
__global__ __launch_bounds__(kSemiThreads) void k_semi_expand(const float* sp,
                                                              const int32_t* lengths,
                                                              int64_t N, int K, int C,
                                                              float* xp) {
    const int64_t E = N - 1;
    const int64_t b = blockIdx.x / E, t = blockIdx.x % E;
    const int64_t Eb = clamp_len(lengths, b, N) - 1;
    if (t >= Eb) return;   // padding steps are never read by the chain
    const int KC = K * C;
    const float* src = sp + (size_t)(b * E + t) * K * C * C;
    float* dst = xp + (size_t)(b * E + t) * KC * KC;
    const bool first = t == 0, last = t == Eb - 1;
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    for (int s = w; s < KC; s += kSemiThreads / kWave) {
        const int r = s / C, i = s - r * C;
        float* row = dst + (size_t)s * KC;
        for (int col = lane; col < KC; col += kWave) {
            const int rn = col / C, j = col - rn * C;
            float v = -INFINITY;
            if (!(first && r > 0) && !(last && rn > 0)) {
                if (r == 0) v = src[((size_t)rn * C + i) * C + j];
                else if (j == i && rn == r - 1) v = 0.f;
            }
            row[col] = v;
        }
    }
}

// mu_semi[b, t, k, i, j] = mu_chain[b, t, i, k*C + j] (row (i, 0) of the expanded edge);
// padding steps are 0 in the chain's marginals already
__global__ __launch_bounds__(kSemiThreads) void k_semi_gather(const float* xm, int K, int C,
                                                              float* marg) {
    const int64_t bt = blockIdx.x;
    const int KC = K * C;
    const float* src = xm + (size_t)bt * KC * KC;
    float* dst = marg + (size_t)bt * K * C * C;
    const int n = K * C * C;
    for (int e = threadIdx.x; e < n; e += kSemiThreads) {
        const int k = e / (C * C), rem = e - k * C * C, i = rem / C, j = rem - i * C;
        dst[e] = src[(size_t)i * KC + k * C + j];
    }
}

// one-token sequences: log Z = log C
__global__ void k_semi_single(const int32_t* lengths, int64_t B, int64_t N, int C, float* logZ) {
    const int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (b < B && clamp_len(lengths, b, N) == 1) logZ[b] = logf((float)C);
}

// expanded Viterbi path xs[b, n] = r_n * C + c_n  ->  labels path[b, n] = c_n and segment
// lengths seglen[b, t] = r_{t+1} + 1 where r_t = 0 (else 0); -1 past the sequence
__global__ void k_semi_decode(const int32_t* xs, const int32_t* lengths, int64_t B, int64_t N,
                              int C, int32_t* path, int32_t* seglen) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= B * N) return;
    const int64_t b = idx / N, n = idx % N;
    const int64_t L = clamp_len(lengths, b, N);
    const int32_t* x = xs + b * N;
    path[idx] = n < L ? x[n] % C : -1;
    if (n < N - 1) {
        int32_t g = -1;
        if (n < L - 1) g = (x[n] / C == 0) ? x[n + 1] / C + 1 : 0;
        seglen[b * (N - 1) + n] = g;
    }
}

}  // namespace

hipError_t launch_semi_expand(const float* sp, const int32_t* lengths, int64_t B, int64_t N,
                              int64_t K, int64_t C, float* xp, hipStream_t s) {
    hipLaunchKernelGGL(k_semi_expand, dim3((unsigned)(B * (N - 1))), dim3(kSemiThreads), 0, s,
                       sp, lengths, N, (int)K, (int)C, xp);
    return hipGetLastError();
}

hipError_t launch_semi_gather(const float* xm, int64_t B, int64_t N, int64_t K, int64_t C,
                              float* marg, hipStream_t s) {
    hipLaunchKernelGGL(k_semi_gather, dim3((unsigned)(B * (N - 1))), dim3(kSemiThreads), 0, s,
                       xm, (int)K, (int)C, marg);
    return hipGetLastError();
}

hipError_t launch_semi_single(const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                              float* logZ, hipStream_t s) {
    hipLaunchKernelGGL(k_semi_single, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s,
                       lengths, B, N, (int)C, logZ);
    return hipGetLastError();
}

hipError_t launch_semi_decode(const int32_t* xs, const int32_t* lengths, int64_t B, int64_t N,
                              int64_t C, int32_t* path, int32_t* seglen, hipStream_t s) {
    hipLaunchKernelGGL(k_semi_decode, dim3((unsigned)((B * N + 255) / 256)), dim3(256), 0, s,
                       xs, lengths, B, N, (int)C, path, seglen);
    return hipGetLastError();
}

}  // namespace tsc
