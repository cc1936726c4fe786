// derived.hip -- quantities read off the outputs of the hot path:
//   entropy of each sequence's label distribution (the quantity of Table 2's "Entropy"
//   semiring) from the edge marginals by the chain rule of entropy of a Markov chain:
//     H = H(z_0) + sum_t H(z_{t+1} | z_t),   m_t(i) = sum_j mu[t,i,j],
//     H(z_0) = -sum_i m_0(i) log m_0(i),  H(z_{t+1} | z_t) = -sum_{i,j} mu log(mu / m_t(i));
//   log-probability of a given label sequence (Sec. 5.1): log p(z) = sum_t l[t,z_t,z_{t+1}] - A;
//   samples by forward filtering, backward sampling (the distribution of Table 2's "Sample"
//   semiring) from the edge marginals: z_{L-1} ~ sum_i mu[L-2,i,.], then
//   z_t | z_{t+1} = j ~ mu[t,.,j] (the Markov property), each draw by inverse CDF with a
//   caller-supplied uniform: the smallest k whose inclusive prefix sum exceeds u * total.
// Every term of H is >= 0, so the sum has no cancellation.  Reductions run in a fixed
// order (no atomics): per-edge partials first, then one pass per sequence.
#include "device.h"
#include "internal.h"

namespace tsc {
namespace {

constexpr int kEntThreads = 256;

// one workgroup per valid edge: part[b][t] = H(z_{t+1} | z_t) (+ H(z_0) for t = 0).  Each
// wave takes kGroup rows of mu_t at a time, lanes over j (kPer = ceil(C / 64) values of a
// row per lane): all the group's loads are issued before any reduction, so a wave keeps
// kGroup * kPer coalesced row loads in flight.  Per row:
//   m = sum_j p,   m * H(row / m) = -sum_j p (log p - log m).
// Entries (and rows) below the smallest normal float are left out: each such term is below
// 1e-36, and the hardware logarithm reads a subnormal input as zero (its log as -inf).
constexpr int kGroup = 8;
constexpr float kTiny = 1.17549435e-38f;   // the smallest normal float

template <int kPer>
__global__ __launch_bounds__(kEntThreads) void k_entropy_edges(const float* mu,
                                                               const int32_t* lengths,
                                                               int64_t N, int64_t C,
                                                               double* part) {
    __shared__ double red[kEntThreads / kWave];
    const int64_t E = N - 1;
    const int64_t b = blockIdx.x / E, t = blockIdx.x % E;
    if (t >= clamp_len(lengths, b, N) - 1) return;
    const int c = (int)C;
    const float* m = mu + (size_t)(b * E + t) * c * c;
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    double acc = 0.0;
    for (int i0 = w * kGroup; i0 < c; i0 += (kEntThreads / kWave) * kGroup) {
        float v[kGroup][kPer];
#pragma unroll
        for (int g = 0; g < kGroup; ++g)
#pragma unroll
            for (int q = 0; q < kPer; ++q) {
                const int i = i0 + g, j = q * kWave + lane;
                v[g][q] = (i < c && j < c) ? m[(size_t)i * c + j] : 0.f;
            }
        float h = 0.f;
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
            float rs = 0.f;
#pragma unroll
            for (int q = 0; q < kPer; ++q) rs += v[g][q];
            const float mi = wave_sum(rs);
            if (!(mi >= kTiny)) continue;   // wave-uniform
            const float lm = flog(mi);
            float hg = 0.f;
#pragma unroll
            for (int q = 0; q < kPer; ++q)
                if (v[g][q] >= kTiny) hg -= v[g][q] * (flog(v[g][q]) - lm);
            if (t == 0 && lane == 0) hg -= mi * lm;
            h += hg;
        }
        acc += (double)wave_sum(h);
    }
    if (lane == 0) red[w] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double s = 0.0;
        for (int i = 0; i < kEntThreads / kWave; ++i) s += red[i];
        part[b * E + t] = s;
    }
}

// one workgroup per sequence: H = the sum of its edges' partials (log C for one token), in
// a fixed order -- thread k sums edges k, k + 256, ..., then waves and lanes combine in a
// fixed tree -- so the result does not depend on scheduling
__global__ __launch_bounds__(kEntThreads) void k_entropy_sum(const double* part,
                                                             const int32_t* lengths,
                                                             int64_t N, int64_t C, float* H) {
    __shared__ double red[kEntThreads / kWave];
    const int64_t b = blockIdx.x, E = N - 1, Eb = clamp_len(lengths, b, N) - 1;
    if (Eb == 0) {
        if (threadIdx.x == 0) H[b] = logf((float)C);
        return;
    }
    double s = 0.0;
    for (int64_t t = threadIdx.x; t < Eb; t += kEntThreads) s += part[b * E + t];
    s = wave_sum_d(s);
    if (threadIdx.x % kWave == 0) red[threadIdx.x / kWave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double tot = 0.0;
        for (int i = 0; i < kEntThreads / kWave; ++i) tot += red[i];
        H[b] = (float)tot;
    }
}

// one workgroup per sequence: log p(z) = sum_{t < L-1} l[t, z_t, z_{t+1}] - log Z.  Labels
// are clamped into [0, C) so that the gather stays in bounds (the caller promises valid
// labels; TS_CHECK=1 validates them on the host).
__global__ __launch_bounds__(kEntThreads) void k_log_density(const float* pot,
                                                             const int32_t* lengths,
                                                             const int32_t* labels,
                                                             const float* logZ, int64_t N,
                                                             int64_t C, float* out) {
    __shared__ double red[kEntThreads / kWave];
    const int64_t b = blockIdx.x, E = N - 1;
    const int64_t Eb = clamp_len(lengths, b, N) - 1;
    const int32_t* z = labels + b * N;
    double s = 0.0;
    for (int64_t t = threadIdx.x; t < Eb; t += kEntThreads) {
        const int64_t i = min(max((int64_t)z[t], (int64_t)0), C - 1);
        const int64_t j = min(max((int64_t)z[t + 1], (int64_t)0), C - 1);
        s += (double)pot[((b * E + t) * C + i) * C + j];
    }
    s = wave_sum_d(s);
    const int w = threadIdx.x / kWave;
    if (threadIdx.x % kWave == 0) red[w] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double tot = 0.0;
        for (int i = 0; i < kEntThreads / kWave; ++i) tot += red[i];
        out[b] = (float)(tot - (double)logZ[b]);
    }
}

// Inverse-CDF draw over the c weights w[k * stride] by one wave: lane l holds labels l,
// l + 64, ... (kMaxLabels / 64 chunks in registers).  The total is the scan's own final
// prefix, so u < 1 always lands inside it; a label of weight 0 is never taken (the prefix
// test also asks w > 0), and if rounding leaves no positive label past u * total the last
// positive label is taken.  All weights 0: label 0.
constexpr int kChunks = kMaxLabels / kWave;

__device__ int draw_wave(const float* w, int stride, int c, float u, int lane) {
    float p[kChunks], wk[kChunks];
    float carry = 0.f;
#pragma unroll
    for (int q = 0; q < kChunks; ++q) {
        const int k = q * kWave + lane;
        if (q * kWave >= c) {   // wave-uniform: chunks past c hold nothing
            wk[q] = 0.f;
            p[q] = carry;
            continue;
        }
        wk[q] = k < c ? w[(size_t)k * stride] : 0.f;
        float x = wk[q];
#pragma unroll
        for (int d = 1; d < kWave; d <<= 1) {
            const float o = __shfl_up(x, d, kWave);
            if (lane >= d) x += o;
        }
        p[q] = x + carry;
        carry = __shfl(p[q], kWave - 1, kWave);
    }
    const float tot = carry;
    if (!(tot > 0.f)) return 0;
    const float x = u * tot;
    int last = 0;
#pragma unroll
    for (int q = 0; q < kChunks; ++q) {
        const uint64_t hit = __ballot(wk[q] > 0.f && p[q] > x);
        if (hit) return q * kWave + __builtin_ctzll(hit);
        const uint64_t pos = __ballot(wk[q] > 0.f);
        if (pos) last = q * kWave + 63 - __builtin_clzll(pos);
    }
    return last;
}

constexpr int kSampleWaves = 4;

__global__ __launch_bounds__(kSampleWaves * kWave) void k_sample(const float* mu,
                                                                 const int32_t* lengths,
                                                                 const float* uniforms,
                                                                 int64_t S, int64_t B,
                                                                 int64_t N, int64_t C,
                                                                 int32_t* paths) {
    __shared__ float colsum[kSampleWaves][kMaxLabels];
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t sb = (int64_t)blockIdx.x * kSampleWaves + w;
    if (sb >= S * B) return;
    const int64_t b = sb % B, E = N - 1;
    const int64_t L = clamp_len(lengths, b, N);
    const int c = (int)C;
    const float* u = uniforms + sb * N;
    int32_t* z = paths + sb * N;
    for (int64_t n = L + lane; n < N; n += kWave) z[n] = -1;
    // the last token: column sums of the last edge's marginal (uniform for one token)
    float* cs = colsum[w];
    for (int j = lane; j < c; j += kWave) {
        float s = 1.f;
        if (L > 1) {
            const float* last = mu + (size_t)(b * E + (L - 2)) * c * c;
            s = 0.f;
            for (int i = 0; i < c; ++i) s += last[(size_t)i * c + j];
        }
        cs[j] = s;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int zn = draw_wave(cs, 1, c, u[L - 1], lane);
    if (lane == 0) z[L - 1] = zn;
    for (int64_t t = L - 2; t >= 0; --t) {
        const float* col = mu + (size_t)(b * E + t) * c * c + zn;   // mu[t][.][z_{t+1}]
        zn = draw_wave(col, c, c, u[t], lane);
        if (lane == 0) z[t] = zn;
    }
}

}  // namespace

hipError_t launch_sample(const float* mu, const int32_t* lengths, const float* uniforms,
                         int64_t S, int64_t B, int64_t N, int64_t C, int32_t* paths,
                         hipStream_t s) {
    const int64_t waves = S * B;
    hipLaunchKernelGGL(k_sample, dim3((unsigned)((waves + kSampleWaves - 1) / kSampleWaves)),
                       dim3(kSampleWaves * kWave), 0, s, mu, lengths, uniforms, S, B, N, C, paths);
    return hipGetLastError();
}

hipError_t launch_entropy(const float* mu, const int32_t* lengths, int64_t B, int64_t N,
                          int64_t C, double* part, float* H, hipStream_t s) {
    if (N > 1) {
        const dim3 g((unsigned)(B * (N - 1))), blk(kEntThreads);
        if (C <= kWave)
            hipLaunchKernelGGL(k_entropy_edges<1>, g, blk, 0, s, mu, lengths, N, C, part);
        else if (C <= 2 * kWave)
            hipLaunchKernelGGL(k_entropy_edges<2>, g, blk, 0, s, mu, lengths, N, C, part);
        else
            hipLaunchKernelGGL(k_entropy_edges<4>, g, blk, 0, s, mu, lengths, N, C, part);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_entropy_sum, dim3((unsigned)B), dim3(kEntThreads), 0, s, part, lengths,
                       N, C, H);
    return hipGetLastError();
}

hipError_t launch_log_density(const float* pot, const int32_t* lengths, const int32_t* labels,
                              const float* logZ, int64_t B, int64_t N, int64_t C, float* out,
                              hipStream_t s) {
    hipLaunchKernelGGL(k_log_density, dim3((unsigned)B), dim3(kEntThreads), 0, s, pot, lengths,
                       labels, logZ, N, C, out);
    return hipGetLastError();
}

}  // namespace tsc
