// chunk.hip -- the lowest levels of the log-semiring tree for label sets of at most 64
// (padded to 64), one workgroup per chunk of S = 2^lc consecutive edges of a sequence
// (lc = the plan's chunk level, at most kChunkLog).
//
// Up (k_chunk_up): the workgroup folds the chunk's valid edges into their product
//   P = l_{t0} (x) l_{t0+1} (x) ... (x) l_{t1-1}
// in the log semiring (any bracketing of the associative product gives the same node,
// Sec. 6a), keeping P in LDS between products, and writes only that product: the tree
// node of level lc.  Each leaf is read from memory once and the levels below lc are never
// formed.  A product is the exp-shifted GEMM of the tree kernels (Sec. 6c's operation),
//   S[a][c] = sum_k exp(P[a][k] + coh[k] - sa[a]) exp(l[k][c] - sb[c]),
//   core = log S,  ro' = ro + max co + sa,  co' = sb,
// on the fp32 matrix cores, one 32 x 32 block per wave; S < 2^-80 is recomputed exactly.
//
// Marginals (k_chunk_form): given the outside vectors of the chunk's node (u, the forward
// message into its first edge, and v, the backward message out of its last edge), the
// workgroup recomputes the messages inside the chunk
//   alpha_{t0} = u,  alpha_{t+1} = alpha_t (x) l_t     (left to right),
//   beta_{t1} = v,   beta_t = l_t (x) beta_{t+1}        (right to left),
// and forms each edge's marginal (Sec. 5.1: p(z_p = 1) = dA/dl_p) during the right-to-left
// pass, while the edge is in registers:
//   mu_t[i][j] = exp(alpha_t[i] + l_t[i][j] + beta_{t+1}[j] - n_t),
//   n_t = LSE_j (y_t[j] + beta_{t+1}[j]),  y_t = alpha_t (x) l_t before its shift,
// a local normaliser per edge, so constant errors in alpha_t or beta_{t+1} cancel exactly.
// Vectors are kept shifted: alpha_{t+1} = y_t - h_t with h_t the largest of the columns'
// maxima, each entry formed as (m - h_t) + log s from its log-sum-exp state (m, s), so no
// message ever passes through a large unshifted value; then n_t - h_t = LSE_j (alpha_{t+1}[j]
// + beta_{t+1}[j]) and mu_t[i][j] = exp((l_t[i][j] - h_t) + alpha_t[i] + beta_{t+1}[j] -
// (n_t - h_t)), the two large terms cancelling first.  The same for beta_t.
//
// Layout of a 64 x 64 matrix in registers (loads and the leaf's uses): thread t holds rows
// (t >> 4) + 16 i, i < 4, and columns 4 (t & 15) .. + 3 as four float4; rows and columns
// past C hold -inf (the semiring zero), so padding needs no masks in the arithmetic.
#include "device.h"
#include "internal.h"

namespace tsc {

namespace {

constexpr int kCP = 64;              // labels padded to 64
constexpr int kCT = 256;             // threads: 4 waves, one 32 x 32 output block each
constexpr int kLD = kCP + 4;         // LDS row stride: 16-byte rows, conflict-free b128 reads
constexpr float kChunkUnderflow = 0x1p-80f;

typedef float f16v __attribute__((ext_vector_type(16)));

template <bool kVec>
__device__ __forceinline__ void load_mat(const float* __restrict__ M, int C, float4 (&x)[4]) {
    const int rg = threadIdx.x >> 4, c = 4 * (threadIdx.x & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = rg + 16 * i;
        const float* p = M + (size_t)r * C + c;
        if constexpr (kVec) {
            x[i] = (r < C && c < C) ? *(const float4*)p
                                    : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
        } else {
            x[i].x = (r < C && c + 0 < C) ? p[0] : -INFINITY;
            x[i].y = (r < C && c + 1 < C) ? p[1] : -INFINITY;
            x[i].z = (r < C && c + 2 < C) ? p[2] : -INFINITY;
            x[i].w = (r < C && c + 3 < C) ? p[3] : -INFINITY;
        }
    }
}

__device__ __forceinline__ float f4get(const float4& v, int q) {
    return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
}

// (m, s) += (m2, s2) for log-sum-exp states value = m + log s (m = -inf: empty)
__device__ __forceinline__ void lse_acc(float& m, float& s, float m2, float s2) {
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) { m = m2; s = s2; return; }
    const float nm = fmaxf(m, m2);
    s = s * fexp(m - nm) + s2 * fexp(m2 - nm);
    m = nm;
}

// log-sum-exp state of four values
__device__ __forceinline__ void lse4(float v0, float v1, float v2, float v3, float& m, float& s) {
    m = fmaxf(fmaxf(v0, v1), fmaxf(v2, v3));
    s = m == -INFINITY ? 0.f
                       : fexp(v0 - m) + fexp(v1 - m) + fexp(v2 - m) + fexp(v3 - m);
}

// merge of the states held by lanes lane and lane ^ o
__device__ __forceinline__ void lse_xor(float& m, float& s, int o) {
    const float m2 = __shfl_xor(m, o, kWave), s2 = __shfl_xor(s, o, kWave);
    lse_acc(m, s, m2, s2);
}

// log-sum-exp over the 64 lanes of a wave (every lane gets the result)
__device__ __forceinline__ float wave_lse64(float x) {
    const float m = wave_max(x);
    const float sh = safe_shift(m);
    const float s = wave_sum(x == -INFINITY ? 0.f : fexp(x - sh));
    return m == -INFINITY ? -INFINITY : sh + flog(s);
}

struct ChunkUpArgs {
    const float* pot;
    const int32_t* lengths;
    int64_t N, C;
    int lc;              // chunk level: a chunk is 2^lc edges
    int64_t nodes;       // nodes per sequence at level lc
    float* core;         // level-lc nodes (one output tile per line: partial maxima [nodes][C][1])
    double* ro;
    double* co;
    float* pmr;
    float* pmc;
};

// max over the four lanes of a quad (DPP quad permutations)
__device__ __forceinline__ float quad_max(float x) {
    x = fmaxf(x, dpp_f(x, 0xB1));
    return fmaxf(x, dpp_f(x, 0x4E));
}
// value of lanes l and l ^ 16 / l ^ 32 combined by max (one lane swap each)
__device__ __forceinline__ float max_x16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_x32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// per-wave partial column maxima of the matrix in registers (the wave's 16 rows) into red[w]
__device__ __forceinline__ void col_partials(const float4 (&x)[4], float (*red)[kCP]) {
    const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x >> 6;
    float m4[4];
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
        const float m = fmaxf(fmaxf(f4get(x[0], qq), f4get(x[1], qq)),
                              fmaxf(f4get(x[2], qq), f4get(x[3], qq)));
        m4[qq] = max_x32(max_x16(m));
    }
    if (lane < 16) *(float4*)&red[w][4 * lane] = make_float4(m4[0], m4[1], m4[2], m4[3]);
}

template <bool kVec>
__global__ __launch_bounds__(kCT, 4) void k_chunk_up(ChunkUpArgs a) {
    __shared__ __align__(16) float P[kCP * kLD];       // the running product's core
    __shared__ __align__(16) float Bt[kCP * kLD];      // right operand, transposed: Bt[c][k]
    __shared__ __align__(16) float red[4][kCP];         // per-wave partial column maxima
    __shared__ __align__(16) float sa[kCP], sb[kCP], cop[kCP];
    __shared__ double rop[kCP];
    __shared__ float cmaxp[1];
    const int64_t b = blockIdx.x / a.nodes, q = blockIdx.x % a.nodes;
    const int64_t E = a.N - 1, Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t S = (int64_t)1 << a.lc, t0 = q * S;
    if (t0 >= Eb) return;   // node absent: all padding
    const int64_t t1 = min(t0 + S, Eb);
    const int C = (int)a.C, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid >> 6;
    const int rg = tid >> 4, c4 = tid & 15;
    const size_t CC = (size_t)C * C;
    const float* leaves = a.pot + (size_t)(b * E) * CC;
    const size_t pn = (size_t)(b * a.nodes + q);

    // P = leaf t0 (ro = co = 0); the next leaf into registers and its column partials
    float4 x[4];
    load_mat<kVec>(leaves + (size_t)t0 * CC, C, x);
#pragma unroll
    for (int i = 0; i < 4; ++i) *(float4*)(P + (rg + 16 * i) * kLD + 4 * c4) = x[i];
    if (tid < kCP) {
        rop[tid] = 0.0;
        cop[tid] = 0.f;
    }
    if (tid == 0) cmaxp[0] = 0.f;
    if (t0 + 1 < t1) {
        load_mat<kVec>(leaves + (size_t)(t0 + 1) * CC, C, x);
        col_partials(x, red);
    }
    __syncthreads();

    const int wm = w >> 1, wn = w & 1;
    const int arow = wm * 32 + (lane & 31), kofs = 4 * (lane >> 5);
    constexpr float kL2E = 1.4426950408889634f;
    for (int64_t t = t0 + 1; t < t1; ++t) {
        const float cm = cmaxp[0];
        // -- A: column shifts from the four waves' partials and the right operand, transposed,
        // into Bt; row shifts of P (a quad of lanes per row); the next leaf's loads
        {
            float sq[4];
            const float4 r0 = *(const float4*)&red[0][4 * c4], r1 = *(const float4*)&red[1][4 * c4];
            const float4 r2 = *(const float4*)&red[2][4 * c4], r3 = *(const float4*)&red[3][4 * c4];
#pragma unroll
            for (int qq = 0; qq < 4; ++qq)
                sq[qq] = safe_shift(fmaxf(fmaxf(f4get(r0, qq), f4get(r1, qq)),
                                          fmaxf(f4get(r2, qq), f4get(r3, qq))));
            if (rg == 0) *(float4*)&sb[4 * c4] = make_float4(sq[0], sq[1], sq[2], sq[3]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int qq = 0; qq < 4; ++qq)
                    Bt[(4 * c4 + qq) * kLD + rg + 16 * i] = fexp(f4get(x[i], qq) - sq[qq]);
        }
        {
            const int ar = tid >> 2, kp = 16 * (tid & 3);
            float m = -INFINITY;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const float4 p4 = *(const float4*)(P + ar * kLD + kp + 4 * u);
                const float4 o4 = *(const float4*)(cop + kp + 4 * u);
                m = fmaxf(m, fmaxf(fmaxf(p4.x + (o4.x - cm), p4.y + (o4.y - cm)),
                                   fmaxf(p4.z + (o4.z - cm), p4.w + (o4.w - cm))));
            }
            m = quad_max(m);
            if ((tid & 3) == 0) sa[ar] = safe_shift(m);
        }
        if (t + 1 < t1) load_mat<kVec>(leaves + (size_t)(t + 1) * CC, C, x);
        __syncthreads();
        // -- B: S = A'' B'' for the wave's 32 x 32 block; the left operand is exponentiated
        // from P as it is read: A''[a][k] = exp2(fma(P + co - max co, log2 e, -sa log2 e)).
        // Lanes 0-31 contribute k..k+3 of each 8-wide k step, lanes 32-63 k+4..k+7.
        f16v acc;
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[r] = 0.f;
        {
            const float nsa = -sa[arow] * kL2E;
            const float* ap = P + arow * kLD + kofs;
            const float* op = cop + kofs;
            const float* bp = Bt + (wn * 32 + (lane & 31)) * kLD + kofs;
#pragma unroll
            for (int kk = 0; kk < kCP; kk += 8) {
                const float4 p4 = *(const float4*)(ap + kk), o4 = *(const float4*)(op + kk);
                const float4 bv = *(const float4*)(bp + kk);
                const float a0 = __builtin_amdgcn_exp2f(fmaf(p4.x + (o4.x - cm), kL2E, nsa));
                const float a1 = __builtin_amdgcn_exp2f(fmaf(p4.y + (o4.y - cm), kL2E, nsa));
                const float a2 = __builtin_amdgcn_exp2f(fmaf(p4.z + (o4.z - cm), kL2E, nsa));
                const float a3 = __builtin_amdgcn_exp2f(fmaf(p4.w + (o4.w - cm), kL2E, nsa));
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, bv.x, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, bv.y, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a2, bv.z, acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a3, bv.w, acc, 0, 0, 0);
            }
        }
        float smin = INFINITY;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            const int col = wn * 32 + (lane & 31);
            if (row < C && col < C) smin = fminf(smin, acc[r]);
        }
        // (also the barrier after every wave's reads of P and Bt)
        const bool any_under = __syncthreads_or(!(smin >= kChunkUnderflow));
        // -- C: the product's core log S into P; entries whose terms all underflowed are
        // recomputed exactly (a rare path: all reads of P before any write)
        float val[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            const int col = wn * 32 + (lane & 31);
            val[r] = (row < C && col < C) ? flog(acc[r]) : -INFINITY;
        }
        if (any_under) {
#pragma unroll 1
            for (int r = 0; r < 16; ++r) {
                const int row = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                const int col = wn * 32 + (lane & 31);
                if (row >= C || col >= C || acc[r] >= kChunkUnderflow) continue;
                const float* lcol = leaves + (size_t)t * CC + col;
                const float sr = sa[row], sc = sb[col];
                float mq = -INFINITY;
                for (int k = 0; k < C; ++k)
                    mq = fmaxf(mq, (P[row * kLD + k] + (cop[k] - cm) - sr) + (lcol[(size_t)k * C] - sc));
                float v = -INFINITY;
                if (mq != -INFINITY) {
                    float sum = 0.f;
                    for (int k = 0; k < C; ++k)
                        sum += fexp((P[row * kLD + k] + (cop[k] - cm) - sr) + (lcol[(size_t)k * C] - sc) - mq);
                    v = mq + flog(sum);
                }
                val[r] = v;
            }
            __syncthreads();
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            const int col = wn * 32 + (lane & 31);
            P[row * kLD + col] = val[r];
        }
        if (tid < kCP) {   // wave 0 only: its reads of cmaxp and cop precede its updates
            rop[tid] = tid < C ? rop[tid] + (double)cm + (double)sa[tid] : 0.0;
            const float sbt = tid < C ? sb[tid] : -INFINITY;
            const float ncm = safe_shift(wave_max_fast(sbt));
            cop[tid] = tid < C ? sbt : 0.f;
            if (tid == 0) cmaxp[0] = ncm;
        }
        if (t + 1 < t1) col_partials(x, red);
        __syncthreads();
    }

    // ---- the node: core, offsets and the partial maxima of its rows and columns
    float* Pc = a.core + pn * CC;
    for (int idx = tid; idx < kCP * kCP; idx += kCT) {
        const int r = idx >> 6, c = idx & (kCP - 1);
        if (r < C && c < C) Pc[(size_t)r * C + c] = P[r * kLD + c];
    }
    if (tid < C) {
        a.ro[pn * C + tid] = rop[tid];
        a.co[pn * C + tid] = (double)cop[tid];
    }
    {
        // rows and columns: a quad of lanes per line, sixteen entries each
        const int line = tid >> 2, part = 16 * (tid & 3);
        float mr = -INFINITY, mc = -INFINITY;
        for (int u = 0; u < 16; ++u) {
            const int k = part + u;
            if (k < C) {
                mr = fmaxf(mr, P[line * kLD + k] + cop[k]);
                mc = fmaxf(mc, P[k * kLD + line] + (float)rop[k]);
            }
        }
        mr = quad_max(mr);
        mc = quad_max(mc);
        if ((tid & 3) == 0 && line < C) {
            a.pmr[pn * C + line] = mr;
            a.pmc[pn * C + line] = mc;
        }
    }
}

struct ChunkFormArgs {
    const float* pot;
    const int32_t* lengths;
    int64_t N, C;
    int lc;
    int64_t nodes;       // nodes per sequence at level lc
    const float* u;      // outside vectors of the level-lc nodes; nullptr: zeros (lc is the root)
    const float* v;
    float* marg;
};

constexpr int kMaxChunk = 1 << kChunkLog;

// merges of log-sum-exp states across lanes: DPP within rows of 16 lanes, lane swaps across
// rows; the merge is symmetric, so both lanes of a pair hold the same state afterwards
__device__ __forceinline__ void lse_dpp(float& m, float& s, int ctrl) {
    lse_acc(m, s, dpp_f(m, ctrl), dpp_f(s, ctrl));
}
__device__ __forceinline__ void lse_x16(float& m, float& s) {
    const auto rm = __builtin_amdgcn_permlane16_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    const auto rs = __builtin_amdgcn_permlane16_swap(__float_as_uint(s), __float_as_uint(s), false, false);
    m = __uint_as_float(rm[0]);
    s = __uint_as_float(rs[0]);
    lse_acc(m, s, __uint_as_float(rm[1]), __uint_as_float(rs[1]));
}
__device__ __forceinline__ void lse_x32(float& m, float& s) {
    const auto rm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    const auto rs = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
    m = __uint_as_float(rm[0]);
    s = __uint_as_float(rs[0]);
    lse_acc(m, s, __uint_as_float(rm[1]), __uint_as_float(rs[1]));
}

// Every wave turns the four waves' partial states (m, s) of the 64 lines into the shifted
// vector (m - h) + log s, h = the largest m (lane c holds line c); returns lane c's entry.
__device__ __forceinline__ float shifted_from_partials(const float (*pm)[kCP], const float (*ps)[kCP],
                                                       int C, float* h_out) {
    const int c = threadIdx.x & (kWave - 1);
    float m = pm[0][c], s = ps[0][c];
    lse_acc(m, s, pm[1][c], ps[1][c]);
    lse_acc(m, s, pm[2][c], ps[2][c]);
    lse_acc(m, s, pm[3][c], ps[3][c]);
    if (c >= C) m = -INFINITY;
    const float h = safe_shift(wave_max_fast(m));
    *h_out = h;
    return m == -INFINITY ? -INFINITY : (m - h) + flog(s);
}

template <bool kVec>
__global__ __launch_bounds__(kCT) void k_chunk_form(ChunkFormArgs a) {
    __shared__ __align__(16) float al[kMaxChunk + 1][kCP];   // alpha_t, shifted (t - t0)
    __shared__ float hs[kMaxChunk];                          // h_t: the shift of alpha_{t+1}
    __shared__ __align__(16) float pm[2][4][kCP], ps[2][4][kCP];   // partial states, ping-pong
    const int64_t b = blockIdx.x / a.nodes, q = blockIdx.x % a.nodes;
    const int64_t E = a.N - 1, Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t S = (int64_t)1 << a.lc, t0 = q * S;
    const int64_t tall = min(t0 + S, E);
    const int C = (int)a.C, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid >> 6;
    const int rg = tid >> 4, c4 = tid & 15;
    const size_t CC = (size_t)C * C;
    // padding edges of the chunk are exactly 0
    for (int64_t t = max(t0, Eb); t < tall; ++t) {
        float* o = a.marg + (size_t)(b * E + t) * CC;
        if (kVec) {
            for (size_t idx = tid; idx < CC / 4; idx += kCT)
                *(float4*)(o + 4 * idx) = make_float4(0.f, 0.f, 0.f, 0.f);
        } else {
            for (size_t idx = tid; idx < CC; idx += kCT) o[idx] = 0.f;
        }
    }
    if (t0 >= Eb) return;
    const int64_t t1 = min(t0 + S, Eb);
    const float* leaves = a.pot + (size_t)(b * E) * CC;
    float* out = a.marg + (size_t)(b * E) * CC;
    const size_t nv = (size_t)(b * a.nodes + q) * C;
    // alpha_{t0} = u: lane c of every wave holds entry c; each thread picks its rows
    // rg + 16 i from those lanes
    float acur = lane < C ? (a.u ? a.u[nv + lane] : 0.f) : -INFINITY;
    if (tid < kCP) al[0][tid] = acur;
    float ar[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) ar[i] = __shfl(acur, rg + 16 * i, kWave);
    float4 x[4], xn[4];
    load_mat<kVec>(leaves + (size_t)t0 * CC, C, x);

    // ---- left to right: y_t[c] = LSE_r (alpha_t[r] + l_t[r][c]); alpha_{t+1} = y_t - h_t
    for (int64_t t = t0; t < t1; ++t) {
        const int k = (int)(t - t0), par = k & 1;
        if (t + 1 < t1) load_mat<kVec>(leaves + (size_t)(t + 1) * CC, C, xn);
        float mq[4], sq[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            lse4(ar[0] + f4get(x[0], qq), ar[1] + f4get(x[1], qq), ar[2] + f4get(x[2], qq),
                 ar[3] + f4get(x[3], qq), mq[qq], sq[qq]);
            lse_x16(mq[qq], sq[qq]);
            lse_x32(mq[qq], sq[qq]);
        }
        if (lane < 16) {
            *(float4*)&pm[par][w][4 * lane] = make_float4(mq[0], mq[1], mq[2], mq[3]);
            *(float4*)&ps[par][w][4 * lane] = make_float4(sq[0], sq[1], sq[2], sq[3]);
        }
        __syncthreads();
        float h;
        const float anext = shifted_from_partials(pm[par], ps[par], C, &h);
        if (w == 0) {
            al[k + 1][lane] = anext;
            if (lane == 0) hs[k] = h;
        }
        // this thread's rows of alpha_{t+1}: rows rg + 16 i live in lanes rg + 16 i of the wave
#pragma unroll
        for (int i = 0; i < 4; ++i) ar[i] = __shfl(anext, rg + 16 * i, kWave);
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = xn[i];
    }
    __syncthreads();   // al and hs complete

    // ---- right to left: the marginals of edge t from registers, then
    // beta_t[r] = (m_r - h) + log s_r, the row states of l_t[r][c] + beta_{t+1}[c]
    float bcur = lane < C ? (a.v ? a.v[nv + lane] : 0.f) : -INFINITY;   // lane c: beta_{t+1}[c]
    load_mat<kVec>(leaves + (size_t)(t1 - 1) * CC, C, x);
    for (int64_t t = t1 - 1; t >= t0; --t) {
        const int k = (int)(t - t0), par = k & 1;
        if (t > t0) load_mat<kVec>(leaves + (size_t)(t - 1) * CC, C, xn);
        // the edge's normaliser less h_t (lane c holds column c)
        const float n = wave_lse64(lane < C ? al[k + 1][lane] + bcur : -INFINITY);
        const float h = hs[k];
        float bq[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) bq[qq] = __shfl(bcur, 4 * c4 + qq, kWave);
        float* o = out + (size_t)t * CC;
        float zm[4], zs[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int r = rg + 16 * i;
            const float ai = al[k][r];
            float4 mu;
            mu.x = fexp((x[i].x - h) + ai + bq[0] - n);
            mu.y = fexp((x[i].y - h) + ai + bq[1] - n);
            mu.z = fexp((x[i].z - h) + ai + bq[2] - n);
            mu.w = fexp((x[i].w - h) + ai + bq[3] - n);
            if (n == -INFINITY) mu = make_float4(0.f, 0.f, 0.f, 0.f);
            if (r < C) {
                float* p = o + (size_t)r * C + 4 * c4;
                if constexpr (kVec) {
                    if (4 * c4 < C) *(float4*)p = mu;
                } else {
                    if (4 * c4 + 0 < C) p[0] = mu.x;
                    if (4 * c4 + 1 < C) p[1] = mu.y;
                    if (4 * c4 + 2 < C) p[2] = mu.z;
                    if (4 * c4 + 3 < C) p[3] = mu.w;
                }
            }
            // row state over this thread's four columns, merged over the row's 16 lanes
            lse4(x[i].x + bq[0], x[i].y + bq[1], x[i].z + bq[2], x[i].w + bq[3], zm[i], zs[i]);
            lse_dpp(zm[i], zs[i], 0xB1);
            lse_dpp(zm[i], zs[i], 0x4E);
            lse_dpp(zm[i], zs[i], 0x141);
            lse_dpp(zm[i], zs[i], 0x140);
        }
        // lane c4 == 0 of row group rg holds rows rg + 16 i: wave w covers rows 4w .. 4w+3
        // (+ 16 i); stored as pm[par][i][r] so that every wave reads four partials per row
        if (c4 == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                pm[par][i][rg + 16 * i] = zm[i];
                ps[par][i][rg + 16 * i] = zs[i];
            }
        }
        __syncthreads();
        // every row r has exactly one state, in slot i = r / 16; the other slots are empty
        {
            const int r = lane;
            const int i = r >> 4;
            float m = pm[par][i][r], s2 = ps[par][i][r];
            if (r >= C) m = -INFINITY;
            const float hb = safe_shift(wave_max_fast(m));
            bcur = m == -INFINITY ? -INFINITY : (m - hb) + flog(s2);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) x[i] = xn[i];
    }
}

}  // namespace

bool chunk_path(int64_t C, bool masks) { return !masks && C <= kCP; }

hipError_t launch_chunk_up(const Plan& p, const float* pot, const int32_t* lengths,
                           hipStream_t s) {
    ChunkUpArgs a{};
    a.pot = pot; a.lengths = lengths; a.N = p.N; a.C = p.C;
    a.lc = p.lc;
    a.nodes = p.Np >> p.lc;
    a.core = p.core[p.lc]; a.ro = p.ro[p.lc]; a.co = p.co[p.lc];
    a.pmr = p.pmr[p.lc]; a.pmc = p.pmc[p.lc];
    const dim3 grid((unsigned)(p.B * a.nodes));
    if (p.C % 4 == 0)
        hipLaunchKernelGGL(k_chunk_up<true>, grid, dim3(kCT), 0, s, a);
    else
        hipLaunchKernelGGL(k_chunk_up<false>, grid, dim3(kCT), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_chunk_form(const Plan& p, const float* pot, const int32_t* lengths,
                             float* marg, hipStream_t s) {
    ChunkFormArgs a{};
    a.pot = pot; a.lengths = lengths; a.N = p.N; a.C = p.C;
    a.lc = p.lc;
    a.nodes = p.Np >> p.lc;
    a.u = p.lc < p.D ? p.u[p.lc] : nullptr;
    a.v = p.lc < p.D ? p.v[p.lc] : nullptr;
    a.marg = marg;
    const dim3 grid((unsigned)(p.B * a.nodes));
    if (p.C % 4 == 0)
        hipLaunchKernelGGL(k_chunk_form<true>, grid, dim3(kCT), 0, s, a);
    else
        hipLaunchKernelGGL(k_chunk_form<false>, grid, dim3(kCT), 0, s, a);
    return hipGetLastError();
}

}  // namespace tsc
