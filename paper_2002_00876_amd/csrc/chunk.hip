// chunk.hip -- log Z and the marginals for label sets of at most 64 (padded to 64) in
// chunks of S = 2^lc consecutive edges of a sequence (lc = the plan's chunk level, at most
// kChunkLog): the chunk products (k_chunk_up, one workgroup per chunk), the forward and
// backward recursions over each sequence's chunk products (k_chunk_scan), and the
// messages and marginals inside each chunk from its boundary vectors (k_chunk_form).
//
// Up (k_chunk_up): the workgroup folds the chunk's valid edges into their product
//   P = l_{t0} (x) l_{t0+1} (x) ... (x) l_{t1-1}
// in the log semiring (any bracketing of the associative product gives the same node,
// Sec. 6a), keeping P in LDS between products, and writes only that product: the tree
// node of level lc.  Each leaf is read from memory once and the levels below lc are never
// formed.  A product is the exp-shifted GEMM of the tree kernels (Sec. 6c's operation),
//   S[a][c] = sum_k exp(P[a][k] + coh[k] - sa[a]) exp(l[k][c] - sb[c]),
//   core = log S,  ro' = ro + max co + sa,  co' = sb,
// on the fp32 matrix cores, a 16-row strip per wave; S < 2^-80 is recomputed exactly.
//
// Across chunks (k_chunk_scan): see the kernel.
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
// + beta_{t+1}[j]) and, with w_t[i][j] = (l_t[i][j] - h_t) + beta_{t+1}[j] (the two large
// terms cancelling first) and z_i = max_j w_t[i][j],
//   mu_t[i][j] = exp(w_t[i][j] - z_i) exp(z_i + alpha_t[i] - (n_t - h_t)),
// where the first factor is also the term of row i's log-sum-exp state that gives beta_t[i]:
// one exponential per entry for both.  The same shifting for beta_t.
//
// Layout of a 64 x 64 matrix in registers (loads and the leaf's uses): thread t holds rows
// (t >> 4) + 16 i, i < 4, and columns 4 (t & 15) .. + 3 as four float4; rows and columns
// past C hold -inf (the semiring zero), so padding needs no masks in the arithmetic.
#include "device.h"
#include "internal.h"

namespace tsc {

namespace {

constexpr int kCP = 64;              // labels padded to 64
constexpr int kCT = 256;             // threads: 4 waves
constexpr int kLD = kCP + 4;         // LDS row stride: 16-byte rows, conflict-free b128 reads
constexpr float kChunkUnderflow = 0x1p-80f;

typedef float f16v __attribute__((ext_vector_type(16)));

template <bool kVec, bool kFull = false>
__device__ __forceinline__ void load_mat(const float* __restrict__ M, int C, float4 (&x)[4]) {
    const int rg = threadIdx.x >> 4, c = 4 * (threadIdx.x & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = rg + 16 * i;
        const float* p = M + (size_t)r * C + c;
        if constexpr (kFull) {
            x[i] = *(const float4*)p;
        } else if constexpr (kVec) {
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
    float* core;         // level-lc nodes
    double* ro;
    double* co;
    int32_t* lin;        // per node: 1 when core holds S itself (linear path), 0 for log S
};

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

// max over the 16 lanes of a DPP row (quad swaps, then the mirrors within 8 and 16)
__device__ __forceinline__ float row16_max(float x) {
    x = fmaxf(x, dpp_f(x, 0xB1));
    x = fmaxf(x, dpp_f(x, 0x4E));
    x = fmaxf(x, dpp_f(x, 0x141));
    return fmaxf(x, dpp_f(x, 0x140));
}

// LDS of the exact path
struct ExactSmem {
    float P[kCP * kLD];       // the running product's core
    float Bt[kCP * kLD];      // right operand, transposed: Bt[c][k]
    float red[4][kCP];        // per-wave partial column maxima
    float sbuf[2][kCP];       // column shifts (= co) of the products
    float sa[kCP];            // row shifts of the next product
    double rop[kCP];
};

// ---- the exact path: every product in the log domain
// Products as 16-row strips: wave w owns rows 16 w .. 16 w + 15 of every product and all 64
// columns (four 16 x 16 blocks of v_mfma_f32_16x16x4f32), so each row of P is read,
// exponentiated and rewritten by one wave only, and the next product's row shifts come out
// of the epilogue with in-wave reductions.  Lanes 16 g .. 16 g + 15 contribute the indices
// k + 4 g .. k + 4 g + 3 of each 16-wide step (one 16-byte read of P and of each block of
// the transposed right operand).
template <bool kVec>
__device__ void chunk_up_exact(const ChunkUpArgs& a, int64_t b, int64_t t0, int64_t t1,
                               size_t pn, ExactSmem& sm) {
    float* P = sm.P;
    float* Bt = sm.Bt;
    float (*red)[kCP] = sm.red;
    float (*sbuf)[kCP] = sm.sbuf;
    float* sa = sm.sa;
    double* rop = sm.rop;
    const int64_t E = a.N - 1;
    const int C = (int)a.C, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid >> 6;
    const int rg = tid >> 4, c4 = tid & 15;
    const int lr = lane & 15, lg = lane >> 4;      // strip row / column within a block; group
    const int arow = 16 * w + lr;                  // the row this lane feeds to the products
    const size_t CC = (size_t)C * C;
    const float* leaves = a.pot + (size_t)(b * E) * CC;
    constexpr float kL2E = 1.4426950408889634f;

    // P = leaf t0 (ro = co = 0); the next leaf into registers and its column partials
    float4 x[4];
    load_mat<kVec>(leaves + (size_t)t0 * CC, C, x);
#pragma unroll
    for (int i = 0; i < 4; ++i) *(float4*)(P + (rg + 16 * i) * kLD + 4 * c4) = x[i];
    if (tid < kCP) {
        rop[tid] = 0.0;
        sbuf[1][tid] = 0.f;
    }
    if (t0 + 1 < t1) {
        load_mat<kVec>(leaves + (size_t)(t0 + 1) * CC, C, x);
        col_partials(x, red);
    }
    __syncthreads();
    {
        // row shifts of the first product: lane group lg scans columns 16 lg .. 16 lg + 15
        float m = -INFINITY;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float4 p4 = *(const float4*)(P + arow * kLD + 16 * lg + 4 * u);
            m = fmaxf(m, fmaxf(fmaxf(p4.x, p4.y), fmaxf(p4.z, p4.w)));
        }
        m = max_x32(max_x16(m));
        if (lg == 0) sa[arow] = safe_shift(m);
    }

    const int np = (int)(t1 - t0 - 1);
    for (int p = 0; p < np; ++p) {
        const int64_t t = t0 + 1 + p;
        const int cur = p & 1, prv = cur ^ 1;
        // -- A: column shifts of leaf t from the four waves' partials and the right operand,
        // transposed, into Bt; the next leaf's loads
        {
            float sq[4];
            const float4 r0 = *(const float4*)&red[0][4 * c4], r1 = *(const float4*)&red[1][4 * c4];
            const float4 r2 = *(const float4*)&red[2][4 * c4], r3 = *(const float4*)&red[3][4 * c4];
#pragma unroll
            for (int qq = 0; qq < 4; ++qq)
                sq[qq] = safe_shift(fmaxf(fmaxf(f4get(r0, qq), f4get(r1, qq)),
                                          fmaxf(f4get(r2, qq), f4get(r3, qq))));
            if (rg == 0) *(float4*)&sbuf[cur][4 * c4] = make_float4(sq[0], sq[1], sq[2], sq[3]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int qq = 0; qq < 4; ++qq)
                    Bt[(4 * c4 + qq) * kLD + rg + 16 * i] = fexp(f4get(x[i], qq) - sq[qq]);
        }
        if (t + 1 < t1) load_mat<kVec>(leaves + (size_t)(t + 1) * CC, C, x);
        __syncthreads();
        // -- B: S = A'' B'' for the wave's strip; A''[a][k] = exp2(fma(P + co - max co,
        // log2 e, -sa log2 e)) formed as P is read
        const float cm = safe_shift(wave_max_fast(lane < C ? sbuf[prv][lane] : -INFINITY));
        const float sar = sa[arow];
        typedef float f4v __attribute__((ext_vector_type(4)));
        f4v acc[4];
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[n] = (f4v){0.f, 0.f, 0.f, 0.f};
        {
            const float nsa = -sar * kL2E;
            const float* ap = P + arow * kLD + 4 * lg;
            const float* op = sbuf[prv] + 4 * lg;
            const float* bp = Bt + lr * kLD + 4 * lg;
#pragma unroll
            for (int kk = 0; kk < kCP; kk += 16) {
                const float4 p4 = *(const float4*)(ap + kk), o4 = *(const float4*)(op + kk);
                float4 bv[4];
#pragma unroll
                for (int n = 0; n < 4; ++n) bv[n] = *(const float4*)(bp + 16 * n * kLD + kk);
                const float a0 = __builtin_amdgcn_exp2f(fmaf(p4.x + (o4.x - cm), kL2E, nsa));
                const float a1 = __builtin_amdgcn_exp2f(fmaf(p4.y + (o4.y - cm), kL2E, nsa));
                const float a2 = __builtin_amdgcn_exp2f(fmaf(p4.z + (o4.z - cm), kL2E, nsa));
                const float a3 = __builtin_amdgcn_exp2f(fmaf(p4.w + (o4.w - cm), kL2E, nsa));
#pragma unroll
                for (int n = 0; n < 4; ++n) {
                    acc[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, bv[n].x, acc[n], 0, 0, 0);
                    acc[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, bv[n].y, acc[n], 0, 0, 0);
                    acc[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a2, bv[n].z, acc[n], 0, 0, 0);
                    acc[n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a3, bv[n].w, acc[n], 0, 0, 0);
                }
            }
        }
        // -- C: the product's core log S (entry (16 w + 4 lg + r, 16 n + lr) of acc[n][r]);
        // entries whose terms all underflowed are recomputed exactly from P before it is
        // overwritten (a rare path); then the wave's rows of P, ro and the next row shifts
        float val[4][4], smin = INFINITY;
#pragma unroll
        for (int n = 0; n < 4; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * w + 4 * lg + r, col = 16 * n + lr;
                const bool ok = row < C && col < C;
                val[n][r] = ok ? flog(acc[n][r]) : -INFINITY;
                if (ok) smin = fminf(smin, acc[n][r]);
            }
        if (__builtin_amdgcn_ballot_w64(!(smin >= kChunkUnderflow))) {
#pragma unroll 1
            for (int n = 0; n < 4; ++n)
#pragma unroll 1
                for (int r = 0; r < 4; ++r) {
                    const int row = 16 * w + 4 * lg + r, col = 16 * n + lr;
                    if (row >= C || col >= C || acc[n][r] >= kChunkUnderflow) continue;
                    const float* lcol = leaves + (size_t)t * CC + col;
                    const float sr = sa[row], sc = sbuf[cur][col];
                    float mq = -INFINITY;
                    for (int k = 0; k < C; ++k)
                        mq = fmaxf(mq, (P[row * kLD + k] + (sbuf[prv][k] - cm) - sr) +
                                           (lcol[(size_t)k * C] - sc));
                    float v = -INFINITY;
                    if (mq != -INFINITY) {
                        float sum = 0.f;
                        for (int k = 0; k < C; ++k)
                            sum += fexp((P[row * kLD + k] + (sbuf[prv][k] - cm) - sr) +
                                        (lcol[(size_t)k * C] - sc) - mq);
                        v = mq + flog(sum);
                    }
                    val[n][r] = v;
                }
        }
        const float cmn = safe_shift(wave_max_fast(lane < C ? sbuf[cur][lane] : -INFINITY));
        float sbc[4];
#pragma unroll
        for (int n = 0; n < 4; ++n) sbc[n] = sbuf[cur][16 * n + lr];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * w + 4 * lg + r;
            float m = -INFINITY;
#pragma unroll
            for (int n = 0; n < 4; ++n) {
                P[row * kLD + 16 * n + lr] = val[n][r];
                m = fmaxf(m, val[n][r] + sbc[n]);
            }
            m = row16_max(m);
            if (lr == 0) {
                if (row < C) rop[row] += (double)cm + (double)sa[row];
                sa[row] = safe_shift(m - cmn);
            }
        }
        if (t + 1 < t1) col_partials(x, red);
        __syncthreads();
    }

    // ---- the node: core and offsets
    const float* cop = sbuf[(np - 1) & 1];   // co of the last product (zeros for one edge)
    float* Pc = a.core + pn * CC;
    if (tid == 0) a.lin[pn] = 0;
    for (int idx = tid; idx < kCP * kCP; idx += kCT) {
        const int r = idx >> 6, c = idx & (kCP - 1);
        if (r < C && c < C) Pc[(size_t)r * C + c] = P[r * kLD + c];
    }
    if (tid < C) {
        a.ro[pn * C + tid] = rop[tid];
        a.co[pn * C + tid] = (double)cop[tid];
    }
}

// ---- the fast path: the running product in the linear domain, in the accumulators
// P_p = P_{p-1} (x) l_p is kept as P[a][c] = ro[a] + log S[a][c] + co[c] with S in fp32
// linear form, every row of S scaled to a maximum in [1/2, 1) by a power of two (exact; ro
// counts the powers), and co = CO + cb (CO a float64 scalar, cb <= 0).  Then
//   S_p = S_{p-1} B_p,   B_p[k][c] = exp(cb_{p-1}[k] + l_p[k][c] - s_p[c]),
//   s_p[c] = max_k (cb_{p-1}[k] + l_p[k][c]),   CO_p = CO_{p-1} + max s_p,  cb_p = s_p - max s_p,
// so the chain itself needs neither exp nor log: B_p depends on the leaves only and is
// prepared one product ahead, while the product runs on the matrix cores.  The product is
// formed transposed, T_p = B_p^T T_{p-1} with T = S^T: wave w owns the columns a = 16 w ..
// 16 w + 15 of T, and the accumulators of v_mfma_f32_16x16x4f32 (lane l: T[16 m + 4 (l / 16)
// + r][16 w + l % 16]) are exactly the right operand of the next product, so T never leaves
// the registers (T_0 = B_0^T is read from LDS).  The result equals the exact path's up to
// rounding as long as every entry of every S_p (rows of S_{p-1} at most 1, columns of B_p at
// most 1) is at least 2^-80: then nothing below fp32's normal range ever enters a sum that
// matters.  Otherwise the path reports failure and the chunk is redone by the exact path.
struct LinSmem {
    float bt[2][kCP * kCP];   // B of two products, transposed (bt[c][k]), 16-byte groups swizzled
    float red[2][4][kCP];     // per-wave partial column maxima of two leaves
};

// dword offset of element (c, 4 kg .. 4 kg + 3) of a transposed operand: the 16-byte groups of
// a row are permuted by c, so that both the writes (lanes: 16 consecutive 4-column groups) and
// the reads (lanes: 16 consecutive rows c) touch 16 distinct 16-byte bank groups
__device__ __forceinline__ int bt_off(int c, int kg) { return c * kCP + 4 * (kg ^ ((c ^ (c >> 2)) & 15)); }

// thread t: rows 4 (t >> 4) + i, columns 4 (t & 15) .. + 3 (past C: -inf)
template <bool kVec, bool kFull>
__device__ __forceinline__ void load_rows4(const float* __restrict__ M, int C, float4 (&x)[4]) {
    const int r0 = 4 * (threadIdx.x >> 4), c = 4 * (threadIdx.x & 15);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = r0 + i;
        const float* p = M + (size_t)r * C + c;
        if constexpr (kFull) {
            x[i] = *(const float4*)p;
        } else if constexpr (kVec) {
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

template <bool kVec, bool kFull>
__device__ bool chunk_up_linear(const ChunkUpArgs& a, int64_t b, int64_t t0, int64_t t1,
                                size_t pn, LinSmem& sm, int (&flag)[2]) {
    typedef float f4v __attribute__((ext_vector_type(4)));
    const int64_t E = a.N - 1;
    const int C = (int)a.C, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid >> 6;
    const int rg = tid >> 4, c4 = tid & 15;        // leaf layout: rows 4 rg + i, columns 4 c4 + q
    const int lr = lane & 15, g = lane >> 4;       // product layout
    const int ac = 16 * w + lr;                    // the column of T (row of S) of this lane
    const size_t CC = (size_t)C * C;
    const float* leaves = a.pot + (size_t)(b * E) * CC;
    const int np = (int)(t1 - t0);

    float4 lf[4];          // a leaf on its way from memory
    float v[4][4];         // cb[k] + l[k][c] of the next leaf to prepare
    float cbr[4];          // cb at the thread's rows 4 rg + i (of the last prepared leaf)
    float cbc[4];          // cb at the thread's columns 4 c4 + q
    double CO = 0.0;

    // (the leaf work runs in log2 units: v, cb and CO below are natural-log values times
    // log2 e, so that every entry of B is one exp2)
    constexpr float kL2E = 1.4426950408889634f;
    auto make_v = [&]() {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[i][0] = fmaf(lf[i].x, kL2E, cbr[i]);
            v[i][1] = fmaf(lf[i].y, kL2E, cbr[i]);
            v[i][2] = fmaf(lf[i].z, kL2E, cbr[i]);
            v[i][3] = fmaf(lf[i].w, kL2E, cbr[i]);
        }
    };
    // the wave's column maxima of v (its 16 rows) into red[par][w]
    auto partials = [&](int par) {
        float m4[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
            m4[q] = max_x32(max_x16(fmaxf(fmaxf(v[0][q], v[1][q]), fmaxf(v[2][q], v[3][q]))));
        if (lane < 16) *(float4*)&sm.red[par][w][4 * c4] = make_float4(m4[0], m4[1], m4[2], m4[3]);
    };
    // B of the leaf whose v is in registers (column maxima from red[par]) into bt[buf]; cb of
    // that leaf at the thread's rows and columns; CO
    auto prep = [&](int par, int buf) {
        float sc[4], sr[4];
        {
            const float4 r0 = *(const float4*)&sm.red[par][0][4 * c4], r1 = *(const float4*)&sm.red[par][1][4 * c4];
            const float4 r2 = *(const float4*)&sm.red[par][2][4 * c4], r3 = *(const float4*)&sm.red[par][3][4 * c4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                sc[q] = fmaxf(fmaxf(f4get(r0, q), f4get(r1, q)), fmaxf(f4get(r2, q), f4get(r3, q)));
        }
        {
            const float4 r0 = *(const float4*)&sm.red[par][0][4 * rg], r1 = *(const float4*)&sm.red[par][1][4 * rg];
            const float4 r2 = *(const float4*)&sm.red[par][2][4 * rg], r3 = *(const float4*)&sm.red[par][3][4 * rg];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                sr[i] = fmaxf(fmaxf(f4get(r0, i), f4get(r1, i)), fmaxf(f4get(r2, i), f4get(r3, i)));
        }
        // max over all columns: the sixteen lanes of a DPP row hold every column once
        const float M = safe_shift(row16_max(fmaxf(fmaxf(sc[0], sc[1]), fmaxf(sc[2], sc[3]))));
        float* bt = sm.bt[buf];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float sh = safe_shift(sc[q]);
            *(float4*)(bt + bt_off(4 * c4 + q, rg)) =
                make_float4(__builtin_amdgcn_exp2f(v[0][q] - sh), __builtin_amdgcn_exp2f(v[1][q] - sh),
                            __builtin_amdgcn_exp2f(v[2][q] - sh), __builtin_amdgcn_exp2f(v[3][q] - sh));
            cbc[q] = sc[q] - M;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) cbr[i] = sr[i] - M;
        CO += (double)M;
    };

    // prologue: B_0 (cb_{-1} = 0) and the column maxima of leaf 1
    load_rows4<kVec, kFull>(leaves + (size_t)t0 * CC, C, lf);
#pragma unroll
    for (int i = 0; i < 4; ++i) cbr[i] = 0.f;
    make_v();
    partials(0);
    if (np > 1) load_rows4<kVec, kFull>(leaves + (size_t)(t0 + 1) * CC, C, lf);
    __syncthreads();
    prep(0, 0);
    if (np > 1) {
        make_v();
        partials(1);
        if (np > 2) load_rows4<kVec, kFull>(leaves + (size_t)(t0 + 2) * CC, C, lf);
    }
    __syncthreads();

    f4v T[4];
    int esum = 0;
    const int xb = 64 * lr + 4 * (g ^ lr ^ (lr >> 2));
    const int cl = ac < C ? C - 4 * g : 0;   // entry (16 m + 4 g + r, ac) is real iff 16 m + r < cl

    for (int p = 0; p < np; ++p) {
        const int cur = p & 1;
        // leaf p + 1's B into the other buffer (the product below reads this one)
        if (p + 1 < np) prep((p + 1) & 1, cur ^ 1);
        // T_p = B_p^T T_{p-1}: k-step 16 mp + 4 g + j of this lane is T[mp][j] on the right and
        // bt[16 mb + lr][16 mp + 4 g + j] on the left
        // (bt_off(16 mb + lr, 4 mp + g) = 1024 mb + (xb ^ 16 (mp ^ mb)), xb = 64 lr + 4 (g ^ lr ^ lr / 4))
        const float* bt = sm.bt[cur];
        f4v U[4];
        if (p == 0) {
            // T_0 = B_0^T, read from the transposed buffer (entry (c, k = ac))
#pragma unroll
            for (int m = 0; m < 4; ++m)
#pragma unroll
                for (int r = 0; r < 4; ++r) U[m][r] = bt[bt_off(16 * m + 4 * g + r, ac >> 2) + (ac & 3)];
        } else {
#pragma unroll
            for (int m = 0; m < 4; ++m) U[m] = (f4v){0.f, 0.f, 0.f, 0.f};
            // (each left operand is read one step ahead of its four products; the products form
            // a scheduling region of their own with that order imposed)
            __builtin_amdgcn_sched_barrier(0);
            float4 av[2];
            av[0] = *(const float4*)(bt + xb);
#pragma unroll
            for (int st = 0; st < 16; ++st) {
                const int mp = st >> 2, mb = st & 3;
                if (st + 1 < 16) {
                    const int mp1 = (st + 1) >> 2, mb1 = (st + 1) & 3;
                    av[(st + 1) & 1] = *(const float4*)(bt + 1024 * mb1 + (xb ^ (16 * (mp1 ^ mb1))));
                }
                const float4 a4 = av[st & 1];
                U[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.x, T[mp][0], U[mb], 0, 0, 0);
                U[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.y, T[mp][1], U[mb], 0, 0, 0);
                U[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.z, T[mp][2], U[mb], 0, 0, 0);
                U[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.w, T[mp][3], U[mb], 0, 0, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
#pragma unroll
            for (int st = 1; st < 15; ++st) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
            }
            __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
            __builtin_amdgcn_sched_barrier(0);
        }
        // leaf p + 2's column maxima (its load was issued a product ago), leaf p + 3's load
        if (p + 2 < np) {
            make_v();
            partials(p & 1);
            if (p + 3 < np) load_rows4<kVec, kFull>(leaves + (size_t)(t0 + p + 3) * CC, C, lf);
        }
        // scale column ac of T (row ac of S) by the power of two that brings its maximum into
        // [1/2, 1); any real entry below 2^-80 sends the chunk to the exact path
        float mx = 0.f, mn = INFINITY;
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                mx = fmaxf(mx, U[m][r]);
                if (kFull || 16 * m + r < cl) mn = fminf(mn, U[m][r]);
            }
        mx = max_x32(max_x16(mx));
        if (__builtin_amdgcn_ballot_w64(!(mn >= kChunkUnderflow)) && lane == 0) flag[cur] = 1;
        const int e = mx > 0.f ? ((__float_as_int(mx) >> 23) & 0xff) - 126 : 0;
        const float sc = __int_as_float((127 - e) << 23);
#pragma unroll
        for (int m = 0; m < 4; ++m) T[m] = U[m] * sc;
        esum += e;
        __syncthreads();
        if (flag[cur]) return false;   // (a flag is written only before the barrier of its parity)
    }

    // the node in linear form: S itself (lane: row ac, columns 16 m + 4 g + r; every real
    // entry in [2^-87, 1)), ro, co
    if (tid == 0) a.lin[pn] = 1;
    if (ac < C) {
        float* row = a.core + pn * CC + (size_t)ac * C;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int c0 = 16 * m + 4 * g;
            if constexpr (kVec) {
                if (c0 < C) *(float4*)(row + c0) = make_float4(T[m][0], T[m][1], T[m][2], T[m][3]);
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (c0 + r < C) row[c0 + r] = T[m][r];
            }
        }
        if (g == 0) a.ro[pn * C + ac] = (double)esum * 0.6931471805599453;
    }
    if (rg == 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (4 * c4 + q < C) a.co[pn * C + 4 * c4 + q] = (CO + (double)cbc[q]) * 0.6931471805599453;
    }
    return true;
}

union ChunkUpSmem {
    ExactSmem exact;
    LinSmem lin;
};

template <bool kVec, bool kFull>
__global__ __launch_bounds__(kCT, 4) void k_chunk_up(ChunkUpArgs a) {
    __shared__ ChunkUpSmem sm;
    __shared__ int flag[2];
    const int64_t b = blockIdx.x / a.nodes, q = blockIdx.x % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t S = (int64_t)1 << a.lc, t0 = q * S;
    if (t0 >= Eb) return;   // node absent: all padding
    const int64_t t1 = min(t0 + S, Eb);
    const size_t pn = (size_t)(b * a.nodes + q);
    if (threadIdx.x < 2) flag[threadIdx.x] = 0;
    __syncthreads();
    if (!chunk_up_linear<kVec, kFull>(a, b, t0, t1, pn, sm.lin, flag))
        chunk_up_exact<kVec>(a, b, t0, t1, pn, sm.exact);
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

// Reductions across lanes: max first, then one exponential per value and a sum (so a
// log-sum-exp over lanes costs one exponential per value).  Sums over lanes l and l ^ 16 /
// l ^ 32 by lane swaps; over the 16 lanes of a DPP row by quad swaps and the mirrors within
// 8 and 16.
__device__ __forceinline__ float sum_x16(float x) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_x32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float row16_sum(float x) {
    x += dpp_f(x, 0xB1);
    x += dpp_f(x, 0x4E);
    x += dpp_f(x, 0x141);
    return x + dpp_f(x, 0x140);
}

// Every wave turns the four waves' partial states (m, s) of the 64 lines into the shifted
// vector (m - h) + log s, h = the largest m (lane c holds line c); returns lane c's entry.
__device__ __forceinline__ float shifted_from_partials(const float (*pm)[kCP], const float (*ps)[kCP],
                                                       int C, float* h_out) {
    const int c = threadIdx.x & (kWave - 1);
    const float m0 = pm[0][c], m1 = pm[1][c], m2 = pm[2][c], m3 = pm[3][c];
    float m = fmaxf(fmaxf(m0, m1), fmaxf(m2, m3));
    float s = 0.f;
    if (m != -INFINITY)
        s = ps[0][c] * fexp(m0 - m) + ps[1][c] * fexp(m1 - m) + ps[2][c] * fexp(m2 - m) +
            ps[3][c] * fexp(m3 - m);
    if (c >= C) m = -INFINITY;
    const float h = safe_shift(wave_max_fast(m));
    *h_out = h;
    return m == -INFINITY ? -INFINITY : (m - h) + flog(s);
}

template <bool kVec, bool kFull>
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
    float4 x[4], xn[4], xs[4], xs2[4];
    load_mat<kVec, kFull>(leaves + (size_t)t0 * CC, C, x);

    // ---- left to right: y_t[c] = LSE_r (alpha_t[r] + l_t[r][c]); alpha_{t+1} = y_t - h_t
    for (int64_t t = t0; t < t1; ++t) {
        const int k = (int)(t - t0), par = k & 1;
        if (t + 1 < t1) load_mat<kVec, kFull>(leaves + (size_t)(t + 1) * CC, C, xn);
        // the wave's state (m, s) of each of the thread's columns over the wave's 16 rows
        float mq[4], sq[4];
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const float v0 = ar[0] + f4get(x[0], qq), v1 = ar[1] + f4get(x[1], qq);
            const float v2 = ar[2] + f4get(x[2], qq), v3 = ar[3] + f4get(x[3], qq);
            const float m = max_x32(max_x16(fmaxf(fmaxf(v0, v1), fmaxf(v2, v3))));
            const float sh = safe_shift(m);
            mq[qq] = m;
            sq[qq] = sum_x32(sum_x16(fexp(v0 - sh) + fexp(v1 - sh) + fexp(v2 - sh) + fexp(v3 - sh)));
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
        // the chunk's last three edges stay in registers for the right-to-left pass
        if (t + 1 < t1) {
            if (t + 2 == t1) {
#pragma unroll
                for (int i = 0; i < 4; ++i) xs[i] = x[i];
            }
            if (t + 3 == t1) {
#pragma unroll
                for (int i = 0; i < 4; ++i) xs2[i] = x[i];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) x[i] = xn[i];
        }
    }
    __syncthreads();   // al and hs complete

    // ---- right to left: the marginals of edge t from registers, then
    // beta_t[r] = (m_r - hb) + log s_r from the row states (m_r, s_r) of w_t[r][.]
    float bcur = lane < C ? (a.v ? a.v[nv + lane] : 0.f) : -INFINITY;   // lane c: beta_{t+1}[c]
    for (int64_t t = t1 - 1; t >= t0; --t) {    // (x holds edge t1 - 1, xs t1 - 2, xs2 t1 - 3)
        const int k = (int)(t - t0), par = k & 1;
        if (t > t0) {
            if (t + 1 == t1) {
#pragma unroll
                for (int i = 0; i < 4; ++i) xn[i] = xs[i];
            } else if (t + 2 == t1) {
#pragma unroll
                for (int i = 0; i < 4; ++i) xn[i] = xs2[i];
            } else {
                load_mat<kVec, kFull>(leaves + (size_t)(t - 1) * CC, C, xn);
            }
        }
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
            // row state of (l_t[r][c] - h) + beta_{t+1}[c] over the row's 64 columns (the 16
            // lanes of the row group); its exponentials serve the marginals as well:
            // mu[r][c] = exp(v_c - sh) * exp(sh + alpha_t[r] - (n_t - h)) <= 1
            const float v0 = (x[i].x - h) + bq[0], v1 = (x[i].y - h) + bq[1],
                        v2 = (x[i].z - h) + bq[2], v3 = (x[i].w - h) + bq[3];
            zm[i] = row16_max(fmaxf(fmaxf(v0, v1), fmaxf(v2, v3)));
            const float sh = safe_shift(zm[i]);
            const float e0 = fexp(v0 - sh), e1 = fexp(v1 - sh), e2 = fexp(v2 - sh), e3 = fexp(v3 - sh);
            zs[i] = row16_sum((e0 + e1) + (e2 + e3));
            const float f = n == -INFINITY ? 0.f : fexp((sh + ai) - n);
            const float4 mu = make_float4(e0 * f, e1 * f, e2 * f, e3 * f);
            if (kFull || r < C) {
                float* p = o + (size_t)r * C + 4 * c4;
                if constexpr (kVec) {
                    if (kFull || 4 * c4 < C) *(float4*)p = mu;
                } else {
                    if (4 * c4 + 0 < C) p[0] = mu.x;
                    if (4 * c4 + 1 < C) p[1] = mu.y;
                    if (4 * c4 + 2 < C) p[2] = mu.z;
                    if (4 * c4 + 3 < C) p[3] = mu.w;
                }
            }
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


// ---------------------------------------------------------------- across the chunks
// The chunk nodes M_0, ..., M_{K-1} of a sequence (K = ceil(E_b / S), M_q = ro + core + co
// the product of the edges of chunk q) form a shorter chain with the same log partition and
// the same messages at the chunk boundaries.  One workgroup per sequence runs its forward
// recursion and another its backward recursion (Sec. 5's dynamic program, over chunks):
//   u_0 = 0,      u_{q+1}[j] = LSE_i (u_q[i] + M_q[i][j]),        log Z = LSE_j u_K[j],
//   v_{K-1} = 0,  v_{q-1}[i] = LSE_j (M_q[i][j] + v_q[j]),
// the outside vectors of the chunk nodes (u_q the forward message into chunk q's first edge,
// v_q the backward message out of its last edge), carried in float64 shifted to max 0 and
// stored as float; the shifts are summed in float64 for log Z.  The matrices are independent of the vectors, so
// they are loaded kScanAhead steps ahead of their use and each step costs one barrier.
struct ChunkScanArgs {
    const float* core;    // [B * nodes][C][C]: the chunk nodes, or the potentials when lc == 0
    const double* ro;     // [B * nodes][C] (nullptr: zeros, lc == 0)
    const double* co;
    const int32_t* lin;   // per node: core holds S (1) or log S (0); nullptr: log S
    int64_t nodes;        // node stride per sequence
    const int32_t* lengths;
    int64_t N, C;
    int lc;
    float* logZ;          // [B] or nullptr
    float* u;             // [B * nodes][C] or nullptr
    float* v;             // [B * nodes][C] or nullptr (no backward workgroups)
};

constexpr int kScanAhead = 4;

template <bool kVec>
__global__ __launch_bounds__(kCT) void k_chunk_scan(ChunkScanArgs a) {
    __shared__ __align__(16) float pm[2][4][kCP], ps[2][4][kCP];
    const bool fwd = blockIdx.x < gridDim.x / (a.v ? 2 : 1) || !a.v;
    const int64_t B = a.v ? gridDim.x / 2 : gridDim.x;
    const int64_t b = fwd ? blockIdx.x : blockIdx.x - B;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C, tid = threadIdx.x, lane = tid & (kWave - 1), w = tid >> 6;
    const int rg = tid >> 4, c4 = tid & 15;
    if (Eb <= 0) {
        if (fwd && tid == 0 && a.logZ) a.logZ[b] = logf((float)C);
        return;
    }
    const int64_t S = (int64_t)1 << a.lc, K = (Eb + S - 1) / S;
    const size_t CC = (size_t)C * C, base = (size_t)b * a.nodes;
    const bool lv = lane < C;
    // the matrices of the next kScanAhead steps in registers (step k uses slot k % kScanAhead)
    float4 x[kScanAhead][4];
    double rr[kScanAhead], cr[kScanAhead];
    int lf[kScanAhead];
    auto fetch = [&](int slot, int64_t step) {
        const int64_t q = fwd ? step : K - 1 - step;
        if (step >= (fwd ? K : K - 1)) return;
        lf[slot] = a.lin ? a.lin[base + q] : 0;
        load_mat<kVec>(a.core + (base + q) * CC, C, x[slot]);
        rr[slot] = (a.ro && lv) ? a.ro[(base + q) * C + lane] : 0.0;
        cr[slot] = (a.co && lv) ? a.co[(base + q) * C + lane] : 0.0;
    };
#pragma unroll
    for (int s = 0; s < kScanAhead; ++s) fetch(s, s);
    double cur = lv ? 0.0 : -INFINITY;  // lane c: entry c of u_q (forward) or v_q (backward),
                                        // shifted to max 0 (float64: see the log steps)
    double acc = 0.0;
    if (w == 0 && lv) {
        if (fwd && a.u) a.u[base * C + lane] = 0.f;
        if (!fwd) a.v[(base + K - 1) * C + lane] = 0.f;
    }
    const int64_t steps = fwd ? K : K - 1;
    for (int64_t k0 = 0; k0 < steps; k0 += kScanAhead) {
#pragma unroll
        for (int s = 0; s < kScanAhead; ++s) {
            const int64_t k = k0 + s;
            if (k >= steps) break;
            const int par = (int)(k & 1);
            float4 m4[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) m4[i] = x[s][i];
            const double ro = rr[s], co = cr[s];
            const bool lin = lf[s] != 0;
            fetch(s, k + kScanAhead);
            if (lin) {
                // linear node (every real entry of S in [2^-87, 1), padding read as -inf -> 0):
                // the weights exp(w - W) times S, summed; one exponential per lane
                const double wd = lv ? (fwd ? cur + ro : co + cur) : -INFINITY;
                const float W = safe_shift(wave_max_fast((float)wd));
                const float ew = lv ? fexp((float)(wd - (double)W)) : 0.f;
                float y;
                if (fwd) {
                    float er[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) er[i] = __shfl(ew, rg + 16 * i, kWave);
                    float yq[4];
#pragma unroll
                    for (int qq = 0; qq < 4; ++qq)
                        yq[qq] = sum_x32(sum_x16(er[0] * fmaxf(f4get(m4[0], qq), 0.f) + er[1] * fmaxf(f4get(m4[1], qq), 0.f) +
                                                 er[2] * fmaxf(f4get(m4[2], qq), 0.f) + er[3] * fmaxf(f4get(m4[3], qq), 0.f)));
                    if (lane < 16) *(float4*)&ps[par][w][4 * lane] = make_float4(yq[0], yq[1], yq[2], yq[3]);
                    __syncthreads();
                    y = (ps[par][0][lane] + ps[par][1][lane]) + (ps[par][2][lane] + ps[par][3][lane]);
                } else {
                    float bq[4];
#pragma unroll
                    for (int qq = 0; qq < 4; ++qq) bq[qq] = __shfl(ew, 4 * c4 + qq, kWave);
                    float zs[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        zs[i] = row16_sum(fmaxf(m4[i].x, 0.f) * bq[0] + fmaxf(m4[i].y, 0.f) * bq[1] +
                                          fmaxf(m4[i].z, 0.f) * bq[2] + fmaxf(m4[i].w, 0.f) * bq[3]);
                    if (c4 == 0) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) ps[par][i][rg + 16 * i] = zs[i];
                    }
                    __syncthreads();
                    y = ps[par][lane >> 4][lane];
                }
                const double z = (lv && y > 0.f) ? (fwd ? co : ro) + (double)flog(y) : -INFINITY;
                const float Z = safe_shift(wave_max_fast((float)z));
                cur = z - (double)Z;
                if (fwd) {
                    acc += (double)W + (double)Z;
                    if (a.u && w == 0 && lv && k + 1 < K) a.u[(base + k + 1) * C + lane] = (float)cur;
                } else {
                    const int64_t q = K - 1 - k;
                    if (w == 0 && lv) a.v[(base + q - 1) * C + lane] = (float)cur;
                }
            } else if (fwd) {
                // log node: w[i] = u[i] + ro[i], shifted; column states over the thread's four
                // rows.  A term w[i] + core[i][j] that matters can add two large values of
                // opposite sign (far-apart offsets): it is formed in float64 and rounded once.
                const double wd = lv ? cur + ro : -INFINITY;
                const float W = safe_shift(wave_max_fast((float)wd));
                const double wdel = lv ? wd - (double)W : -INFINITY;
                double ar[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) ar[i] = __shfl(wdel, rg + 16 * i, kWave);
                float mq[4], sq[4];
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    const float v0 = (float)(ar[0] + (double)f4get(m4[0], qq));
                    const float v1 = (float)(ar[1] + (double)f4get(m4[1], qq));
                    const float v2 = (float)(ar[2] + (double)f4get(m4[2], qq));
                    const float v3 = (float)(ar[3] + (double)f4get(m4[3], qq));
                    const float m = max_x32(max_x16(fmaxf(fmaxf(v0, v1), fmaxf(v2, v3))));
                    const float sh = safe_shift(m);
                    mq[qq] = m;
                    sq[qq] = sum_x32(sum_x16(fexp(v0 - sh) + fexp(v1 - sh) + fexp(v2 - sh) +
                                             fexp(v3 - sh)));
                }
                if (lane < 16) {
                    *(float4*)&pm[par][w][4 * lane] = make_float4(mq[0], mq[1], mq[2], mq[3]);
                    *(float4*)&ps[par][w][4 * lane] = make_float4(sq[0], sq[1], sq[2], sq[3]);
                }
                __syncthreads();
                // column `lane`: merge the four waves' states, add co, shift to max 0
                const float n0 = pm[par][0][lane], n1 = pm[par][1][lane];
                const float n2 = pm[par][2][lane], n3 = pm[par][3][lane];
                const float m = fmaxf(fmaxf(n0, n1), fmaxf(n2, n3));
                double z = -INFINITY;
                if (lv && m != -INFINITY) {
                    const float s = ps[par][0][lane] * fexp(n0 - m) + ps[par][1][lane] * fexp(n1 - m) +
                                    ps[par][2][lane] * fexp(n2 - m) + ps[par][3][lane] * fexp(n3 - m);
                    z = co + (double)m + (double)flog(s);
                }
                const float Z = safe_shift(wave_max_fast((float)z));
                cur = z - (double)Z;
                acc += (double)W + (double)Z;
                if (a.u && w == 0 && lv && k + 1 < K) a.u[(base + k + 1) * C + lane] = (float)cur;
            } else {
                // log node: w[j] = co[j] + v[j], shifted; row states over the 16 lanes of a
                // row group (terms formed in float64, as above)
                const double wd = lv ? co + cur : -INFINITY;
                const float W = safe_shift(wave_max_fast((float)wd));
                const double wdel = lv ? wd - (double)W : -INFINITY;
                double bq[4];
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) bq[qq] = __shfl(wdel, 4 * c4 + qq, kWave);
                float zm[4], zs[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float v0 = (float)((double)m4[i].x + bq[0]), v1 = (float)((double)m4[i].y + bq[1]);
                    const float v2 = (float)((double)m4[i].z + bq[2]), v3 = (float)((double)m4[i].w + bq[3]);
                    zm[i] = row16_max(fmaxf(fmaxf(v0, v1), fmaxf(v2, v3)));
                    const float sh = safe_shift(zm[i]);
                    zs[i] = row16_sum(fexp(v0 - sh) + fexp(v1 - sh) + fexp(v2 - sh) + fexp(v3 - sh));
                }
                if (c4 == 0) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        pm[par][i][rg + 16 * i] = zm[i];
                        ps[par][i][rg + 16 * i] = zs[i];
                    }
                }
                __syncthreads();
                // row `lane` has one state, in slot lane / 16
                const float m = pm[par][lane >> 4][lane];
                double z = -INFINITY;
                if (lv && m != -INFINITY) z = ro + (double)m + (double)flog(ps[par][lane >> 4][lane]);
                const float Z = safe_shift(wave_max_fast((float)z));
                cur = z - (double)Z;
                const int64_t q = K - 1 - k;   // node q gave v_{q-1}
                if (w == 0 && lv) a.v[(base + q - 1) * C + lane] = (float)cur;
            }
        }
    }
    if (fwd && a.logZ) {
        const float l = wave_lse64((float)cur);
        if (tid == 0) a.logZ[b] = l == -INFINITY ? -INFINITY : (float)(acc + (double)l);
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
    a.core = p.core[p.lc]; a.ro = p.ro[p.lc]; a.co = p.co[p.lc]; a.lin = p.clin;
    const dim3 grid((unsigned)(p.B * a.nodes));
    if (p.C == kCP)
        hipLaunchKernelGGL((k_chunk_up<true, true>), grid, dim3(kCT), 0, s, a);
    else if (p.C % 4 == 0)
        hipLaunchKernelGGL((k_chunk_up<true, false>), grid, dim3(kCT), 0, s, a);
    else
        hipLaunchKernelGGL((k_chunk_up<false, false>), grid, dim3(kCT), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_chunk_scan(const Plan& p, const float* pot, const int32_t* lengths,
                             float* logZ, hipStream_t s) {
    ChunkScanArgs a{};
    if (p.lc > 0) {
        a.core = p.core[p.lc]; a.ro = p.ro[p.lc]; a.co = p.co[p.lc]; a.lin = p.clin;
        a.nodes = p.Np >> p.lc;
    } else {
        a.core = pot; a.ro = nullptr; a.co = nullptr;   // one edge per chunk: the leaves
        a.nodes = p.E;
    }
    a.lengths = lengths; a.N = p.N; a.C = p.C; a.lc = p.lc;
    a.logZ = logZ; a.u = p.u[p.lc]; a.v = p.v[p.lc];
    if (!a.logZ && !a.u) return hipSuccess;
    const dim3 grid((unsigned)(a.v ? 2 * p.B : p.B));
    if (p.C % 4 == 0)
        hipLaunchKernelGGL(k_chunk_scan<true>, grid, dim3(kCT), 0, s, a);
    else
        hipLaunchKernelGGL(k_chunk_scan<false>, grid, dim3(kCT), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_chunk_form(const Plan& p, const float* pot, const int32_t* lengths,
                             float* marg, hipStream_t s) {
    ChunkFormArgs a{};
    a.pot = pot; a.lengths = lengths; a.N = p.N; a.C = p.C;
    a.lc = p.lc;
    a.nodes = p.Np >> p.lc;
    a.u = p.u[p.lc];
    a.v = p.v[p.lc];
    a.marg = marg;
    const dim3 grid((unsigned)(p.B * a.nodes));
    if (p.C == kCP)
        hipLaunchKernelGGL((k_chunk_form<true, true>), grid, dim3(kCT), 0, s, a);
    else if (p.C % 4 == 0)
        hipLaunchKernelGGL((k_chunk_form<true, false>), grid, dim3(kCT), 0, s, a);
    else
        hipLaunchKernelGGL((k_chunk_form<false, false>), grid, dim3(kCT), 0, s, a);
    return hipGetLastError();
}

}  // namespace tsc
