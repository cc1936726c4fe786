// sequential.hip -- the left-to-right forward algorithm (Sec. 5.2), the serial ordering the
// paper's Fig. 4a compares the parallel scan against:
//   alpha_0 = 0,  alpha_{t+1}(j) = LSE_i (alpha_t(i) + l[t][i][j]),  log Z = LSE_j alpha_{L-1}(j).
// Depth L - 1 instead of ceil(log2(L - 1)), work C^2 per step instead of C^3 per product.
// alpha is kept shifted to max 0 with the running shift in float64.
//   C <= 64: one wave per sequence; lane j owns alpha(j) and column j of each edge, whose
//            next column is loaded while the current step computes; alpha(i) reaches every
//            lane by readlane.
//   C > 64:  one workgroup of C threads per sequence, alpha in LDS, a barrier per step.
#include "device.h"
#include "internal.h"

namespace tsc {
namespace {

template <int CP>
__global__ __launch_bounds__(kWave) void k_seq_logz_wave(const float* pot, const int32_t* lengths,
                                                         int64_t N, int64_t C, float* logZ) {
    const int64_t b = blockIdx.x, E = N - 1;
    const int64_t Eb = clamp_len(lengths, b, N) - 1;
    const int c = (int)C, lane = threadIdx.x, j = min(lane, c - 1);
    const float* col = pot + (size_t)b * E * c * c + j;   // column j of edge 0
    float a = lane < c ? 0.f : -INFINITY;                  // alpha(lane), shifted
    double off = 0.0;
    float x[CP];
#pragma unroll
    for (int i = 0; i < CP; ++i) x[i] = Eb > 0 ? col[(size_t)min(i, c - 1) * c] : 0.f;
    for (int64_t t = 0; t < Eb; ++t) {
        // prefetch column j of edge t + 1
        float xn[CP];
        const float* nc = col + (size_t)min(t + 1, Eb - 1) * c * c;
#pragma unroll
        for (int i = 0; i < CP; ++i) xn[i] = nc[(size_t)min(i, c - 1) * c];
        // y(j) = LSE_i alpha(i) + l[t][i][j]
        float v[CP];
        float m = -INFINITY;
#pragma unroll
        for (int i = 0; i < CP; ++i) {
            const float ai = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(a), i));
            v[i] = i < c ? ai + x[i] : -INFINITY;
            m = fmaxf(m, v[i]);
        }
        const float sh = safe_shift(m);
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < CP; ++i) s += fexp(v[i] - sh);
        const float y = (lane < c && s > 0.f) ? sh + flog(s) : -INFINITY;
        const float ys = safe_shift(wave_max(y));
        a = y - ys;
        off += (double)ys;
#pragma unroll
        for (int i = 0; i < CP; ++i) x[i] = xn[i];
    }
    const float m = safe_shift(wave_max(a));
    const float s = wave_sum(lane < c ? fexp(a - m) : 0.f);
    if (lane == 0) logZ[b] = s > 0.f ? (float)(off + (double)m + (double)flog(s)) : -INFINITY;
}

constexpr int kSeqThreads = 256;

__global__ __launch_bounds__(kSeqThreads) void k_seq_logz_block(const float* pot,
                                                                const int32_t* lengths,
                                                                int64_t N, int64_t C,
                                                                float* logZ) {
    __shared__ float alpha[kMaxLabels];
    __shared__ float red[kSeqThreads / kWave];
    const int64_t b = blockIdx.x, E = N - 1;
    const int64_t Eb = clamp_len(lengths, b, N) - 1;
    const int c = (int)C, j = threadIdx.x, w = j / kWave, lane = j % kWave;
    if (j < c) alpha[j] = 0.f;
    double off = 0.0;
    __syncthreads();
    for (int64_t t = 0; t < Eb; ++t) {
        const float* M = pot + (size_t)(b * E + t) * c * c;
        float y = -INFINITY;
        if (j < c) {
            float m = -INFINITY, s = 0.f;
            int i = 0;
            for (; i + 8 <= c; i += 8) {
                float v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) v[u] = alpha[i + u] + M[(size_t)(i + u) * c + j];
                lse_fold<8>(m, s, v);
            }
            for (; i < c; ++i) {
                float v[1] = {alpha[i] + M[(size_t)i * c + j]};
                lse_fold<1>(m, s, v);
            }
            y = lse_val(m, s);
        }
        const float wm = wave_max(y);
        if (lane == 0) red[w] = wm;
        __syncthreads();   // also: every thread has read alpha
        float ys = red[0];
        for (int q = 1; q < kSeqThreads / kWave; ++q) ys = fmaxf(ys, red[q]);
        ys = safe_shift(ys);
        if (j < c) alpha[j] = y - ys;
        off += (double)ys;
        __syncthreads();
    }
    float a = j < c ? alpha[j] : -INFINITY;
    const float wm = wave_max(a);
    if (lane == 0) red[w] = wm;
    __syncthreads();
    float m = red[0];
    for (int q = 1; q < kSeqThreads / kWave; ++q) m = fmaxf(m, red[q]);
    m = safe_shift(m);
    __syncthreads();
    const float ws = wave_sum(j < c ? fexp(a - m) : 0.f);
    if (lane == 0) red[w] = ws;
    __syncthreads();
    if (j == 0) {
        float s = 0.f;
        for (int q = 0; q < kSeqThreads / kWave; ++q) s += red[q];
        logZ[b] = s > 0.f ? (float)(off + (double)m + (double)flog(s)) : -INFINITY;
    }
}

}  // namespace

hipError_t launch_logz_sequential(const float* pot, const int32_t* lengths, int64_t B,
                                  int64_t N, int64_t C, float* logZ, hipStream_t s) {
    const dim3 g((unsigned)B);
    if (C <= 8) hipLaunchKernelGGL(k_seq_logz_wave<8>, g, dim3(kWave), 0, s, pot, lengths, N, C, logZ);
    else if (C <= 16) hipLaunchKernelGGL(k_seq_logz_wave<16>, g, dim3(kWave), 0, s, pot, lengths, N, C, logZ);
    else if (C <= 32) hipLaunchKernelGGL(k_seq_logz_wave<32>, g, dim3(kWave), 0, s, pot, lengths, N, C, logZ);
    else if (C <= 64) hipLaunchKernelGGL(k_seq_logz_wave<64>, g, dim3(kWave), 0, s, pot, lengths, N, C, logZ);
    else hipLaunchKernelGGL(k_seq_logz_block, g, dim3(kSeqThreads), 0, s, pot, lengths, N, C, logZ);
    return hipGetLastError();
}

}  // namespace tsc
