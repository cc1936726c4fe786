// node_scan.hip -- log Z from the nodes of one tree level by the left-to-right recursion
// over them (Sec. 5.2's dynamic program, applied to the level's node products instead of
// the edges): for short sequences of many labels the upper tree levels are launches of a
// few small products, each bound by its memory round trips, while K nodes cost K dependent
// vector steps of C^2 work in one launch.  The up-sweep stops at level l (chunks of 2^l
// edges, l >= 1) and this kernel finishes the sequence:
//   v_0 = 0,  v_{q+1}[j] = LSE_i (v_q[i] + ro_q[i] + core_q[i][j]) + co_q[j],
//   log Z = LSE_j v_K[j].
// v is kept unshifted in float64 (it carries the running log Z, one entry per thread); the
// row weights v[i] + ro[i] - W (W about their maximum) are formed in float64, rounded once
// and stored to LDS by their row's thread, so the products read one float per row.  One
// workgroup per sequence, three barriers per step: node q + 2 is loaded into registers while
// node q is used from LDS (and node q + 1, loaded during the step before, is stored to the
// other LDS buffer), so a load has a whole step to arrive; the next step's W is reduced
// together with the step's result, then the next weights are formed.
#include <algorithm>

#include "device.h"
#include "internal.h"

namespace tsc {
namespace {

constexpr int kNsThreads = 512;
constexpr int kNsParts = kNsThreads / kNodeScanMaxLabels;   // threads per column, each a part of the rows
constexpr int kNsRegs = kNodeScanMaxLabels * kNodeScanMaxLabels / kNsThreads;   // node values per thread

struct NodeScanArgs {
    const float* core;     // [B * nodes][C][C] level-l nodes
    const double* ro;      // [B * nodes][C]
    const double* co;
    int64_t nodes;         // node stride per sequence
    const int32_t* lengths;
    int64_t N, C;
    int level;
    float* logZ;
};

template <bool kVec>
__global__ __launch_bounds__(kNsThreads) void k_node_scan_log(NodeScanArgs a) {
    extern __shared__ __align__(16) float nsm[];            // two node buffers [C][C]
    __shared__ double ros[2][kNodeScanMaxLabels];           // their ro vectors
    __shared__ float wsf[kNodeScanMaxLabels];               // row weights v_q[i] + ro_q[i] - W_q
    __shared__ float pm[kNsParts][kNodeScanMaxLabels], ps[kNsParts][kNodeScanMaxLabels];
    __shared__ float red[2][kNsThreads / kWave];
    __shared__ float sred[kNsThreads / kWave];
    const int64_t b = blockIdx.x;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C, CC = C * C, tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
    if (Eb <= 0) {
        if (tid == 0) a.logZ[b] = logf((float)C);
        return;
    }
    const int64_t S = (int64_t)1 << a.level, K = (Eb + S - 1) / S;
    const size_t base = (size_t)b * a.nodes;
    // block maximum of doubles, rounded to float (a shift: any value near the maximum
    // serves, as it is added back exactly): a barrier, then every thread reads the waves'
    // maxima.  The two slots alternate between steps; a slot is written again only after the
    // next step's first barrier, so one barrier per call suffices.
    auto block_max = [&](double x, int slot) {
        const float xf = wave_max_fast((float)x);
        if (lane == 0) red[slot][w] = xf;
        __syncthreads();
        float m = red[slot][0];
#pragma unroll
        for (int q = 1; q < kNsThreads / kWave; ++q) m = fmaxf(m, red[slot][q]);
        return (double)m;
    };
    // node q into registers: the thread's values idx = tid + kNsThreads * r (float4 groups
    // with kVec), and ro, co of line tid
    float xv[kNsRegs];
    double rov = 0.0, cov = 0.0;
    auto fetch = [&](int64_t q) {
        const float* src = a.core + (base + q) * (size_t)CC;
        if constexpr (kVec) {
#pragma unroll
            for (int r = 0; r < kNsRegs / 4; ++r) {
                const int i4 = tid + kNsThreads * r;
                if (4 * i4 < CC) {
                    const float4 v = reinterpret_cast<const float4*>(src)[i4];
                    xv[4 * r] = v.x;
                    xv[4 * r + 1] = v.y;
                    xv[4 * r + 2] = v.z;
                    xv[4 * r + 3] = v.w;
                }
            }
        } else {
#pragma unroll
            for (int r = 0; r < kNsRegs; ++r) {
                const int i = tid + kNsThreads * r;
                if (i < CC) xv[r] = src[i];
            }
        }
        if (tid < C) {
            rov = a.ro[(base + q) * C + tid];
            cov = a.co[(base + q) * C + tid];
        }
    };
    auto put = [&](int buf) {
        float* dst = nsm + buf * CC;
        if constexpr (kVec) {
#pragma unroll
            for (int r = 0; r < kNsRegs / 4; ++r) {
                const int i4 = tid + kNsThreads * r;
                if (4 * i4 < CC)
                    reinterpret_cast<float4*>(dst)[i4] = make_float4(xv[4 * r], xv[4 * r + 1], xv[4 * r + 2], xv[4 * r + 3]);
            }
        } else {
#pragma unroll
            for (int r = 0; r < kNsRegs; ++r) {
                const int i = tid + kNsThreads * r;
                if (i < CC) dst[i] = xv[r];
            }
        }
        if (tid < C) ros[buf][tid] = rov;
    };
    // v_0 = 0; W_0 = max_i (v_0[i] + ro_0[i])
    fetch(0);
    double co_cur = cov, co_next = 0.0;
    put(0);
    double W = safe_shift_d(block_max(tid < C ? rov : -INFINITY, 0));
    if (tid < C) wsf[tid] = (float)(rov - W);
    __syncthreads();
    if (K > 1) fetch(1);
    const int j = tid % kNodeScanMaxLabels, part = tid / kNodeScanMaxLabels;
    const int rows = (C + kNsParts - 1) / kNsParts;
    const int i0 = min(C, part * rows), i1 = min(C, i0 + rows);
    double vlast = -INFINITY;   // v_K[tid] after the last step
    for (int64_t q = 0; q < K; ++q) {
        const int cur = (int)(q & 1);
        const float* M = nsm + cur * CC;
        const double* ro = ros[cur];
        // node q + 1 (in registers since the step before) into the other buffer, which was
        // last read in step q - 1; then node q + 2's loads
        double ro_next = -INFINITY;
        if (q + 1 < K) {
            put(cur ^ 1);
            ro_next = rov;
            co_next = cov;
        }
        if (q + 2 < K) fetch(q + 2);
        // y[j] = LSE_i (v[i] + ro[i] - W + M[i][j]) over this thread's part of the rows (the
        // row weights from LDS); eight rows' reads in flight
        if (j < C) {
            float m = -INFINITY, s = 0.f;
            int i = i0;
            for (; i + 8 <= i1; i += 8) {
                float x[8];
#pragma unroll
                for (int r = 0; r < 8; ++r) x[r] = M[(i + r) * C + j];
#pragma unroll
                for (int r = 0; r < 8; ++r) x[r] += wsf[i + r];
                lse_fold<8>(m, s, x);
            }
            for (; i < i1; ++i) {
                const float x[1] = {wsf[i] + M[i * C + j]};
                lse_fold<1>(m, s, x);
            }
            pm[part][j] = m;
            ps[part][j] = s;
        }
        __syncthreads();
        // z[j] = co[j] + W + y[j] = v_{q+1}[j]; the next step's W = max_j (z[j] + ro_{q+1}[j])
        double z = -INFINITY;
        if (tid < C) {
            float m = -INFINITY, s = 0.f;
#pragma unroll
            for (int r = 0; r < kNsParts; ++r) {
                const float m2 = pm[r][tid], s2 = ps[r][tid];
                if (m2 == -INFINITY) continue;
                if (m == -INFINITY) {
                    m = m2;
                    s = s2;
                } else {
                    const float nm = fmaxf(m, m2);
                    s = s * fexp(m - nm) + s2 * fexp(m2 - nm);
                    m = nm;
                }
            }
            if (m != -INFINITY) z = co_cur + W + (double)m + (double)flog(s);
        }
        vlast = z;
        W = safe_shift_d(block_max(q + 1 < K ? z + ro_next : z, (int)((q + 1) & 1)));
        if (q + 1 < K) {
            if (tid < C) wsf[tid] = (float)(z + ro_next - W);
            __syncthreads();
        }
        co_cur = co_next;
    }
    // log Z = LSE_j v_K[j]; W is max_j v_K[j]
    const float e = tid < C && vlast != -INFINITY ? fexp((float)(vlast - W)) : 0.f;
    const float se = wave_sum(e);
    if (lane == 0) sred[w] = se;
    __syncthreads();
    if (tid == 0) {
        float t = 0.f;
        for (int q = 0; q < kNsThreads / kWave; ++q) t += sred[q];
        a.logZ[b] = t > 0.f ? (float)(W + (double)flog(t)) : -INFINITY;
    }
}

template <bool kVec>
hipError_t allow_ns_lds() {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)k_node_scan_log<kVec>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)(2 * sizeof(float) * kNodeScanMaxLabels * kNodeScanMaxLabels));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_node_scan(const Plan& p, const int32_t* lengths, float* logZ, hipStream_t s) {
    const int l = p.scan_level;
    NodeScanArgs a{p.core[l], p.ro[l], p.co[l], p.Np >> l, lengths, p.N, p.C, l, logZ};
    const size_t lds = 2 * sizeof(float) * p.C * p.C;
    hipError_t e;
    if (p.C % 4 == 0) {
        e = allow_ns_lds<true>();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_node_scan_log<true>, dim3((unsigned)p.B), dim3(kNsThreads), lds, s, a);
    } else {
        e = allow_ns_lds<false>();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_node_scan_log<false>, dim3((unsigned)p.B), dim3(kNsThreads), lds, s, a);
    }
    return hipGetLastError();
}

}  // namespace tsc
