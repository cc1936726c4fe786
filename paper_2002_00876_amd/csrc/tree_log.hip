// tree_log.hip -- log-semiring (logsumexp, +) tree over the edges of each sequence:
// the up-sweep of C x C semiring matrix products (Torch-Struct Sec. 6a / Fig. 3; the
// product is the Sec. 6c operation V = log sum_n exp(T + U)), the root log-sum-exp
// (Sec. 5.2: A sums over the first and last label), the outside (down) sweep that
// yields every edge's forward and backward messages, and the per-edge marginals
// (Sec. 5.1: p(z_p = 1) = dA/dl_p).
//
// Node representation (levels >= 1): P[a][c] = ro[a] + co[c] + core[a][c], ro/co in
// float64, core in float32.  The product P = L (x) R is evaluated as an exp-shifted
// dense GEMM on the matrix cores (fp32 MFMA; for 128-wide full tiles, bf16 MFMA over a
// three-part bf16 split of each float32 operand, which keeps float32 precision):
//   A'[a][b] = core_L[a][b] + (co_L[b] - max co_L),   B'[b][c] = core_R[b][c] + (ro_R[b] - max ro_R)
//   rA[a] = max_b A'[a][b],  cB[c] = max_b B'[b][c]
//   S[a][c] = sum_b exp(A'[a][b] - rA[a]) * exp(B'[b][c] - cB[c])          (MFMA)
//   core_P = log S,  ro_P[a] = ro_L[a] + max co_L + rA[a],  co_P[c] = co_R[c] + max ro_R + cB[c]
// Every exponent is <= 0, so nothing overflows; S < 2^-80 (all terms underflowing) is
// recomputed exactly by a direct max-shifted log-sum-exp over b.
#include <type_traits>

#include "device.h"
#include "internal.h"

namespace tsc {

namespace {

constexpr int kUpThreads = 256;  // 4 waves; each owns a (TM/2) x (TM/2) quarter of the tile
constexpr int kSlice = 32;       // contraction indices staged per step
constexpr bool kUpBf16 = true;   // 128-wide full tiles: products from bf16 parts (see k_up_log_full)
constexpr float kUnderflow = 0x1p-80f;

typedef float f16v __attribute__((ext_vector_type(16)));


__device__ __forceinline__ size_t mat_off(int64_t b, int64_t k, int64_t nodes, int64_t C) {
    return (size_t)(b * nodes + k) * (size_t)C * (size_t)C;
}

// Row and column maxima of the valid leaves (the exp shifts of the level-1 products):
// lrmax[b][t][i] = max_j l[t][i][j] for a left operand (even t), lcmax[b][t][j] =
// max_i l[t][i][j] for a right operand (odd t), and both for an unpaired last leaf (which
// is carried up unchanged and may be consumed on either side).  Without finiteness masks
// and with C <= 128: rows (C = 64 or 128) take C / 4 lanes of 16-byte loads and a DPP
// maximum each, so a wave covers 4 or 2 rows per pass; columns take one thread per column
// and part of the rows (256 / C parts, combined through LDS).  Otherwise one wave per row
// (16-byte loads along it) and one thread per column over all rows.  Column loads are
// coalesced across threads.
struct LeafMaxArgs {
    const float* pot;
    const int32_t* lengths;
    int64_t N, C;
    float* lrmax;
    float* lcmax;
    uint64_t* rbits;   // [B, E, C, bw] finiteness of the left leaves' rows
    uint64_t* cbits;   // [B, E, C, bw] finiteness of the right leaves' columns
    int bw;
    int32_t* wide;     // [B, E] max |finite entry| > kWideMag, or nullptr
};

// Block-wide flag of the leaf's largest finite magnitude (every thread passes the maximum
// over the entries it read; waves' maxima meet in red[], one per wave)
__device__ __forceinline__ void leaf_wide_flag(const LeafMaxArgs& a, int64_t edge, float am, float* red) {
    am = wave_max(am);
    const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[w] = am;
    __syncthreads();
    if (threadIdx.x == 0) {
        float m = red[0];
        for (int q = 1; q < nw; ++q) m = fmaxf(m, red[q]);
        a.wide[edge] = m > kWideMag;
    }
}
// |x| for finite x, 0 for -inf (structural zeros carry no magnitude)
__device__ __forceinline__ float fin_abs(float x) { return x == -INFINITY ? 0.f : fabsf(x); }

template <bool kVec, bool kBits>
__global__ __launch_bounds__(256) void k_leaf_max(LeafMaxArgs a) {
    const int64_t E = a.N - 1;
    const int64_t b = blockIdx.x / E, t = blockIdx.x % E;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    if (t >= Eb) return;
    const bool left = (t & 1) == 0, right = (t & 1) == 1 || t + 1 == Eb;
    const int C = (int)a.C;
    const float* leaf = a.pot + (size_t)(b * E + t) * C * C;
    const int tid = threadIdx.x, w = tid / kWave, lane = tid % kWave;
    const bool masks = kBits && (a.cbits || a.rbits);
    const bool split = !masks && C <= 128;
    float am = 0.f;   // largest finite magnitude among the entries this thread read
    if (right && split) {
        __shared__ float part[256];
        const int P = 256 / C, p = tid / C, c = tid - p * C;   // C <= 128: P >= 2
        float cm = -INFINITY;
        if (p < P) {
#pragma unroll 8
            for (int i = p; i < C; i += P) {
                const float x = leaf[(size_t)i * C + c];
                cm = fmaxf(cm, x);
                am = fmaxf(am, fin_abs(x));
            }
        }
        part[tid] = cm;
        __syncthreads();
        if (tid < C) {
            for (int q = 1; q < P; ++q) cm = fmaxf(cm, part[q * C + tid]);
            a.lcmax[(size_t)(b * E + t) * C + tid] = cm;
        }
    } else if (right && tid < C) {
        float cm = -INFINITY;
#pragma unroll 8
        for (int i = 0; i < C; ++i) {
            const float x = leaf[(size_t)i * C + tid];
            cm = fmaxf(cm, x);
            am = fmaxf(am, fin_abs(x));
        }
        a.lcmax[(size_t)(b * E + t) * C + tid] = cm;
        if (kBits && a.cbits) {
            bool hole = false;   // a -inf entry in the column
            for (int i = 0; i < C; ++i) hole |= leaf[(size_t)i * C + tid] == -INFINITY;
            uint64_t* cb = a.cbits + ((size_t)(b * E + t) * C + tid) * a.bw;
            for (int q = 0; q < a.bw; ++q) {
                const int i1 = min(C, 64 * q + 64);
                uint64_t bits = i1 - 64 * q == 64 ? ~0ull : (1ull << (i1 - 64 * q)) - 1;
                if (hole) {
                    bits = 0;
                    for (int i = 64 * q; i < i1; ++i)
                        bits |= (uint64_t)(leaf[(size_t)i * C + tid] > -INFINITY) << (i - 64 * q);
                }
                cb[q] = bits;
            }
        }
    }
    if (left && kVec && split && (C == 64 || C == 128)) {
        float* rmax = a.lrmax + (size_t)(b * E + t) * C;
        const int lpr = C >> 2, rpw = kWave / lpr;   // lanes per row (16 or 32), rows per pass
        const int sub = lane / lpr, col = 4 * (lane - sub * lpr);
        for (int i0 = w * rpw; i0 < C; i0 += (256 / kWave) * rpw) {
            const int i = i0 + sub;
            const float4 v = *reinterpret_cast<const float4*>(leaf + (size_t)i * C + col);
            float m = fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w));
            am = fmaxf(am, fmaxf(fmaxf(fin_abs(v.x), fin_abs(v.y)), fmaxf(fin_abs(v.z), fin_abs(v.w))));
            m = fmaxf(m, dpp_f(m, 0xB1));    // within each row of 16 lanes
            m = fmaxf(m, dpp_f(m, 0x4E));
            m = fmaxf(m, dpp_f(m, 0x141));
            m = fmaxf(m, dpp_f(m, 0x140));
            if (lpr == 32) m = fmaxf(m, __shfl_xor(m, 16, kWave));
            if (lane - sub * lpr == 0) rmax[i] = m;
        }
    } else if (left) {
        float* rmax = a.lrmax + (size_t)(b * E + t) * C;
        for (int i = w; i < C; i += 256 / kWave) {
            const float* row = leaf + (size_t)i * C;
            float m = -INFINITY;
            if (kVec) {
                for (int j = 4 * lane; j < C; j += 4 * kWave) {
                    const float4 v = *reinterpret_cast<const float4*>(row + j);
                    m = fmaxf(m, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
                    am = fmaxf(am, fmaxf(fmaxf(fin_abs(v.x), fin_abs(v.y)), fmaxf(fin_abs(v.z), fin_abs(v.w))));
                }
            } else {
                for (int j = lane; j < C; j += kWave) {
                    m = fmaxf(m, row[j]);
                    am = fmaxf(am, fin_abs(row[j]));
                }
            }
            m = wave_max(m);
            if (lane == 0) rmax[i] = m;
            if (!kBits || !a.rbits) continue;   // (no products: one edge per sequence)
            bool h = false;
            for (int j = lane; j < C; j += kWave) h |= row[j] == -INFINITY;
            const bool hole = __ballot(h) != 0;   // wave-uniform
            uint64_t* rb = a.rbits + ((size_t)(b * E + t) * C + i) * a.bw;
            for (int q = 0; q < a.bw; ++q) {
                const int j = 64 * q + lane;
                const uint64_t bits = __ballot(j < C && (!hole || row[min(j, C - 1)] > -INFINITY));
                if (lane == q) rb[q] = bits;
            }
        }
    }
    if (a.wide) {
        __shared__ float wred[256 / kWave];
        leaf_wide_flag(a, b * E + t, am, wred);
    }
}

// The same maxima for C <= 128 without finiteness masks, one leaf per workgroup with every
// load in flight at once: the leaf goes to LDS (row stride C + 1, conflict-free for rows and
// columns alike), then thread t < C reduces row t and thread 128 + t column t.  (Looping
// over a leaf's rows or columns with a few loads in flight leaves a small launch -- a few
// sequences of short chains -- bound by memory latency, not bandwidth.)
constexpr int kLeafLdsMaxLabels = 128;
constexpr int kLeafLdsThreads = 256;
constexpr int64_t kLeafLdsMaxEdges = 8192;   // B * (N - 1) up to which it is used

template <bool kVec>
__global__ __launch_bounds__(kLeafLdsThreads) void k_leaf_max_lds(LeafMaxArgs a) {
    extern __shared__ float T[];   // [C][C + 1]
    const int64_t E = a.N - 1;
    const int64_t b = blockIdx.x / E, t = blockIdx.x % E;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    if (t >= Eb) return;
    const bool left = (t & 1) == 0, right = (t & 1) == 1 || t + 1 == Eb;
    const int C = (int)a.C, CC = C * C, LD = C + 1, tid = threadIdx.x;
    const float* leaf = a.pot + (size_t)(b * E + t) * CC;
    float am = 0.f;   // largest finite magnitude among the entries this thread loaded
    if constexpr (kVec) {
        // C % 4 == 0: a float4 never straddles two rows
        constexpr int kQ = kLeafLdsMaxLabels * kLeafLdsMaxLabels / 4 / kLeafLdsThreads;
        const int C4 = CC / 4;
        float4 v[kQ];
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int i4 = tid + q * kLeafLdsThreads;
            if (i4 < C4) v[q] = reinterpret_cast<const float4*>(leaf)[i4];
        }
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int i4 = tid + q * kLeafLdsThreads;
            if (i4 < C4) {
                am = fmaxf(am, fmaxf(fmaxf(fin_abs(v[q].x), fin_abs(v[q].y)),
                                     fmaxf(fin_abs(v[q].z), fin_abs(v[q].w))));
                const int r = (4 * i4) / C, c = 4 * i4 - r * C;
                float* d = T + r * LD + c;
                d[0] = v[q].x;
                d[1] = v[q].y;
                d[2] = v[q].z;
                d[3] = v[q].w;
            }
        }
    } else {
        constexpr int kQ = kLeafLdsMaxLabels * kLeafLdsMaxLabels / kLeafLdsThreads;
        float v[kQ];
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int i = tid + q * kLeafLdsThreads;
            if (i < CC) v[q] = leaf[i];
        }
#pragma unroll
        for (int q = 0; q < kQ; ++q) {
            const int i = tid + q * kLeafLdsThreads;
            if (i < CC) {
                am = fmaxf(am, fin_abs(v[q]));
                const int r = i / C;
                T[r * LD + i - r * C] = v[q];
            }
        }
    }
    __syncthreads();
    if (a.wide) {
        __shared__ float wred[kLeafLdsThreads / kWave];
        leaf_wide_flag(a, b * E + t, am, wred);
    }
    // four running maxima per line: a short dependency chain
    const bool isrow = tid < kLeafLdsMaxLabels;
    const int line = isrow ? tid : tid - kLeafLdsMaxLabels;
    if (line >= C || !(isrow ? left : right)) return;
    const int base = isrow ? line * LD : line, stride = isrow ? 1 : LD;
    float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    int e = 0;
    for (; e + 4 <= C; e += 4)
#pragma unroll
        for (int u = 0; u < 4; ++u) m[u] = fmaxf(m[u], T[base + (e + u) * stride]);
    for (; e < C; ++e) m[0] = fmaxf(m[0], T[base + e * stride]);
    (isrow ? a.lrmax : a.lcmax)[(size_t)(b * E + t) * C + line] = fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3]));
}

// One tree level of the log-semiring up-sweep, P = L (x) R for every present node.
// A workgroup computes one TM x TM output tile of one node, streaming the contraction
// index in slices of 32 through double-buffered LDS:
//   A''[a][b] = exp(core_L[a][b] + (co_L[b] - max co_L) - sa[a])
//   B''[b][c] = exp(core_R[b][c] + (ro_R[b] - max ro_R) - sb[c])
//   S = A'' B''  (fp32 MFMA 32x32x2),  core_P = log S,
//   ro_P[a] = ro_L[a] + max co_L + sa[a],  co_P[c] = co_R[c] + max ro_R + sb[c].
// The shifts sa (row maxima of core_L + co_L - max co_L) and sb (column maxima of core_R +
// ro_R - max ro_R) are known before the first slice: each producer leaves partial maxima
// of its tile's rows (pmr: max over the tile's columns of core + co) and columns (pmc: max
// over the tile's rows of core + ro), and the leaves' maxima come from k_leaf_max.  A shift
// only has to bound its line from above (nothing overflows) and be close to its maximum;
// S < 2^-80 (every term underflowed) is recomputed exactly by a direct log-sum-exp.
struct UpLogArgs {
    const float* ccore;   // children (level l-1) core, or the potentials when l == 1
    const double* cro;    // nullptr when l == 1 (leaves have ro = co = 0)
    const double* cco;
    const float* cpmr;    // children row maxima [cnodes][C][cntile] (l == 1: leaf maxima)
    const float* cpmc;    // children column maxima [cnodes][C][cntile]
    int64_t cnodes;       // child node stride per sequence
    int cntile;           // partial maxima per line of a child (1 for the leaves)
    const uint64_t* crbits;   // children's row / column finiteness bitmasks
    const uint64_t* ccbits;
    uint64_t* rbits;      // the outputs' bitmasks (nullptr at the root level)
    uint64_t* cbits;
    int bw;               // words per bitmask line
    float* core;          // outputs (level l)
    double* ro;
    double* co;
    float* pmr;           // [nodes][C][ntile]
    float* pmc;
    int64_t nodes;        // nodes per sequence at level l
    const int32_t* lengths;
    int64_t B, N, C;
    int level;
    int ntile;            // tiles per matrix dimension
    int64_t nlogical;     // B * nodes * ntile^2
    int64_t ngrid;        // node_grid(B * nodes, ntile^2)
};

// The largest partial maxima of two lines (cnt >= 1 partials each at p and at r).  The first four partials of both lines are loaded before any is used
// (indexes past cnt - 1 repeat the last partial, which leaves a maximum unchanged), so the
// usual case (at most four tiles per line in the child level) costs one memory round trip
// instead of one per partial.
constexpr int kPartialsAtOnce = 4;
__device__ __forceinline__ void partials_max2(const float* p, const float* r, int cnt, float& mp,
                                              float& mr) {
    float vp[kPartialsAtOnce], vr[kPartialsAtOnce];
#pragma unroll
    for (int q = 0; q < kPartialsAtOnce; ++q) {
        const int i = min(q, cnt - 1);
        vp[q] = p[i];
        vr[q] = r[i];
    }
    mp = fmaxf(fmaxf(vp[0], vp[1]), fmaxf(vp[2], vp[3]));
    mr = fmaxf(fmaxf(vr[0], vr[1]), fmaxf(vr[2], vr[3]));
    for (int q = kPartialsAtOnce; q < cnt; ++q) {
        mp = fmaxf(mp, p[q]);
        mr = fmaxf(mr, r[q]);
    }
}

template <int TM>
struct UpSmem {
    static constexpr int LDA = kSlice + 4, LDB = TM + 4, LDT = TM + 1;
    static constexpr int kBuf = TM * LDA + kSlice * LDB;          // one A + B slice
    static constexpr int kTileF = TM * LDT;                       // epilogue tile
    static constexpr int kMain = (2 * kBuf > kTileF ? 2 * kBuf : kTileF);
    // coh, roh [kMaxLabels]; sa, sb, cof, rof [TM]; red [2 doubles per wave]
    static constexpr int kFloats = kMain + 2 * kMaxLabels + 4 * TM + 4 * (kUpThreads / kWave);
    static constexpr size_t kBytes = sizeof(float) * kFloats;
};

template <int TM, bool VEC, bool kBits>
__global__ __launch_bounds__(kUpThreads) void k_up_log(UpLogArgs a) {
    using Sm = UpSmem<TM>;
    constexpr int LDA = Sm::LDA, LDB = Sm::LDB, LDT = Sm::LDT;
    constexpr int BR = TM / 64;                 // 32 x 32 blocks per wave per dimension
    constexpr int QW = TM / 2;                  // a wave's quarter edge
    extern __shared__ __align__(16) float smem[];
    const int ntiles = a.ntile * a.ntile;
    const int64_t lid = xcd_node_swizzle(blockIdx.x, ntiles);
    if (lid >= a.nlogical) return;
    const int tile = (int)(lid % ntiles);
    const int64_t node = lid / ntiles;
    const int64_t b = node / a.nodes, k = node % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;  // node absent: all padding
    const int C = (int)a.C;
    const int tm = tile / a.ntile, tn = tile % a.ntile;
    const int a0 = tm * TM, c0 = tn * TM;
    const int tid = threadIdx.x;
    const int nt = a.ntile, cnt = a.cntile;

    const int64_t cl = b * a.cnodes + 2 * k, cr = cl + 1, pn = b * a.nodes + k;
    const float* Lc = a.ccore + (size_t)cl * C * C;
    float* Pc = a.core + (size_t)pn * C * C;
    double* Pro = a.ro + (size_t)pn * C;
    double* Pco = a.co + (size_t)pn * C;
    float* Pmr = a.pmr + (size_t)pn * C * nt;
    float* Pmc = a.pmc + (size_t)pn * C * nt;

    const bool right = (2 * k + 1) * half < Eb;
    if (!right) {
        // the right half is padding: the node equals its left child (tile, offsets and
        // the partial maxima, re-tiled)
        for (int idx = tid; idx < TM * TM; idx += kUpThreads) {
            const int r = a0 + idx / TM, c = c0 + idx % TM;
            if (r < C && c < C) Pc[(size_t)r * C + c] = Lc[(size_t)r * C + c];
        }
        if (tn == 0)
            for (int i = tid; i < TM; i += kUpThreads)
                if (a0 + i < C) Pro[a0 + i] = a.cro ? a.cro[(size_t)cl * C + a0 + i] : 0.0;
        if (tm == 0)
            for (int i = tid; i < TM; i += kUpThreads)
                if (c0 + i < C) Pco[c0 + i] = a.cco ? a.cco[(size_t)cl * C + c0 + i] : 0.0;
        if (tm == 0 && tn == 0)
            for (int i = tid; i < C * nt; i += kUpThreads) {
                // only the maximum over a line's partials is ever read: partial 0 takes it
                const int line = i / nt, p = i % nt;
                const float* sr = a.cpmr + ((size_t)cl * C + line) * cnt;
                const float* sc = a.cpmc + ((size_t)cl * C + line) * cnt;
                float mr = -INFINITY, mc = -INFINITY;
                if (p == 0)
                    for (int q = 0; q < cnt; ++q) {
                        mr = fmaxf(mr, sr[q]);
                        mc = fmaxf(mc, sc[q]);
                    }
                Pmr[i] = mr;
                Pmc[i] = mc;
            }
        if (kBits && tm == 0 && tn == 0 && a.rbits)
            for (int i = tid; i < C * a.bw; i += kUpThreads) {
                a.rbits[(size_t)pn * C * a.bw + i] = a.crbits[(size_t)cl * C * a.bw + i];
                a.cbits[(size_t)pn * C * a.bw + i] = a.ccbits[(size_t)cl * C * a.bw + i];
            }
        return;
    }
    const float* Rc = a.ccore + (size_t)cr * C * C;
    const double* Lro = a.cro ? a.cro + (size_t)cl * C : nullptr;
    const double* Lco = a.cco ? a.cco + (size_t)cl * C : nullptr;
    const double* Rro = a.cro ? a.cro + (size_t)cr * C : nullptr;
    const double* Rco = a.cco ? a.cco + (size_t)cr * C : nullptr;

    float* coh = smem + Sm::kMain;       // [kMaxLabels] co_L - max co_L
    float* roh = coh + kMaxLabels;       // [kMaxLabels] ro_R - max ro_R
    float* sa = roh + kMaxLabels;        // [TM] row shifts of the tile
    float* sb = sa + TM;                 // [TM] column shifts
    float* cof = sb + TM;                // [TM] co_P of the tile's columns (float)
    float* rof = cof + TM;               // [TM] ro_P of the tile's rows (float)
    double* red = reinterpret_cast<double*>(rof + TM);

    // ---- staging of one slice [ks, ks + 32) of A'' (TM x 32) and B'' (32 x TM): the
    // loads of the next slice are issued before the current slice's products
    constexpr int GA = kSlice / 4, NA = TM * GA / kUpThreads;   // float4 groups per thread
    constexpr int GB = TM / 4, NB = kSlice * GB / kUpThreads;
    float4 va[NA], vb[NB];
    auto load = [&](int ks) {
#pragma unroll
        for (int it = 0; it < NA; ++it) {
            const int idx = tid + it * kUpThreads;
            const int r = a0 + idx / GA, col = ks + 4 * (idx % GA);
            const float* p = Lc + (size_t)min(r, C - 1) * C;
            if (VEC) {
                va[it] = *(const float4*)(p + min(col, C - 4));
            } else {
                va[it].x = p[min(col + 0, C - 1)];
                va[it].y = p[min(col + 1, C - 1)];
                va[it].z = p[min(col + 2, C - 1)];
                va[it].w = p[min(col + 3, C - 1)];
            }
        }
#pragma unroll
        for (int it = 0; it < NB; ++it) {
            const int idx = tid + it * kUpThreads;
            const int kk = ks + idx / GB, col = c0 + 4 * (idx % GB);
            const float* p = Rc + (size_t)min(kk, C - 1) * C;
            if (VEC) {
                vb[it] = *(const float4*)(p + min(col, C - 4));
            } else {
                vb[it].x = p[min(col + 0, C - 1)];
                vb[it].y = p[min(col + 1, C - 1)];
                vb[it].z = p[min(col + 2, C - 1)];
                vb[it].w = p[min(col + 3, C - 1)];
            }
        }
    };
    // the staged groups of one part: parts p of P take the A groups [p NA / P, (p+1) NA / P)
    // and the B groups likewise, so the exponentials of a slice can be spread over the
    // product steps of the previous one
    auto store_part = [&](int ks, int buf, int part, int nparts) {
        float* As = smem + buf * Sm::kBuf;
        float* Bs = As + TM * LDA;
#pragma unroll
        for (int it = part * NA / nparts; it < (part + 1) * NA / nparts; ++it) {
            const int idx = tid + it * kUpThreads;
            const int r = idx / GA, cl4 = 4 * (idx % GA), col = ks + cl4;
            const bool rok = a0 + r < C;
            const float s = sa[r];
            float4 x;
            x.x = (rok && col + 0 < C) ? fexp(va[it].x + coh[col + 0] - s) : 0.f;
            x.y = (rok && col + 1 < C) ? fexp(va[it].y + coh[col + 1] - s) : 0.f;
            x.z = (rok && col + 2 < C) ? fexp(va[it].z + coh[col + 2] - s) : 0.f;
            x.w = (rok && col + 3 < C) ? fexp(va[it].w + coh[col + 3] - s) : 0.f;
            *(float4*)(As + r * LDA + cl4) = x;
        }
#pragma unroll
        for (int it = part * NB / nparts; it < (part + 1) * NB / nparts; ++it) {
            const int idx = tid + it * kUpThreads;
            const int kr = idx / GB, cl4 = 4 * (idx % GB), kk = ks + kr, col = c0 + cl4;
            const bool kok = kk < C;
            const float rh = kok ? roh[kk] : 0.f;
            float4 x;
            x.x = (kok && col + 0 < C) ? fexp(vb[it].x + rh - sb[cl4 + 0]) : 0.f;
            x.y = (kok && col + 1 < C) ? fexp(vb[it].y + rh - sb[cl4 + 1]) : 0.f;
            x.z = (kok && col + 2 < C) ? fexp(vb[it].z + rh - sb[cl4 + 2]) : 0.f;
            x.w = (kok && col + 3 < C) ? fexp(vb[it].w + rh - sb[cl4 + 3]) : 0.f;
            *(float4*)(Bs + kr * LDB + cl4) = x;
        }
    };
    auto store = [&](int ks, int buf) { store_part(ks, buf, 0, 1); };

    // ---- offsets of the contracted index, shifted to max 0, and the tile's shifts.  Every
    // global read of this part goes out at once, together with the first slice (whose
    // exponentials are the first use of the shifts): one memory round trip before the loop.
    load(0);
    static_assert(kMaxLabels <= kUpThreads, "one offset of the contracted index per thread");
    const double lco = (Lco && tid < C) ? Lco[tid] : -INFINITY;
    const double rro = (Rro && tid < C) ? Rro[tid] : -INFINITY;
    float pa = -INFINITY, pb = -INFINITY;   // maxima of the partials of row a0 + tid, column c0 + tid
    if (tid < TM) {   // (lines past C read line C - 1 and are discarded)
        partials_max2(a.cpmr + ((size_t)cl * C + min(a0 + tid, C - 1)) * cnt,
                      a.cpmc + ((size_t)cr * C + min(c0 + tid, C - 1)) * cnt, cnt, pa, pb);
        if (a0 + tid >= C) pa = -INFINITY;
        if (c0 + tid >= C) pb = -INFINITY;
    }
    // both maxima in one block reduction
    {
        const double lw = wave_max_d(lco), rw = wave_max_d(rro);
        const int w = tid / kWave;
        if ((tid & (kWave - 1)) == 0) {
            red[2 * w] = lw;
            red[2 * w + 1] = rw;
        }
    }
    __syncthreads();
    double lmax = red[0], rmax = red[1];
#pragma unroll
    for (int w = 1; w < kUpThreads / kWave; ++w) {
        lmax = fmax(lmax, red[2 * w]);
        rmax = fmax(rmax, red[2 * w + 1]);
    }
    const double coLshift = Lco ? safe_shift_d(lmax) : 0.0;
    const double roRshift = Rro ? safe_shift_d(rmax) : 0.0;
    if (tid < C) {
        coh[tid] = Lco ? (float)(lco - coLshift) : 0.f;
        roh[tid] = Rro ? (float)(rro - roRshift) : 0.f;
    }
    if (tid < TM) {
        sa[tid] = safe_shift(a0 + tid < C ? pa - (float)coLshift : -INFINITY);
        sb[tid] = safe_shift(c0 + tid < C ? pb - (float)roRshift : -INFINITY);
    }
    __syncthreads();

    // ---- products: wave (wm, wn) owns rows wm*QW.., columns wn*QW.. as BR x BR blocks.
    // Within each 8-wide k step lanes 0-31 contribute k..k+3 and lanes 32-63 k+4..k+7 (one
    // 16-byte LDS read of A per block row); B uses the same k assignment.
    const int w = tid / kWave, lane = tid % kWave;
    const int wm = w >> 1, wn = w & 1;
    f16v acc[BR][BR];
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int j = 0; j < BR; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    const int nslices = (C + kSlice - 1) / kSlice;
    store(0, 0);   // (slice 0 was loaded before the shifts)
    __syncthreads();
    for (int s = 0; s < nslices; ++s) {
        const int buf = s & 1;
        if (s + 1 < nslices) load((s + 1) * kSlice);
        const float* As = smem + buf * Sm::kBuf;
        const float* Bs = As + TM * LDA;
        const float* ap = As + (wm * QW + (lane & 31)) * LDA + 4 * (lane >> 5);
        const float* bp = Bs + (4 * (lane >> 5)) * LDB + wn * QW + (lane & 31);
#pragma unroll
        for (int kk = 0; kk < kSlice; kk += 8) {
            // the second half of the slice's steps carries the next slice's exponentials
            // (its loads have had the first half to arrive); they issue while the products run
            if (kk >= kSlice / 2 && s + 1 < nslices)
                store_part((s + 1) * kSlice, buf ^ 1, (kk - kSlice / 2) / 8, kSlice / 16);
            float4 av[BR];
            float bv[BR][4];
#pragma unroll
            for (int i = 0; i < BR; ++i) av[i] = *(const float4*)(ap + i * 32 * LDA + kk);
#pragma unroll
            for (int j = 0; j < BR; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) bv[j][q] = bp[(kk + q) * LDB + j * 32];
#pragma unroll
            for (int i = 0; i < BR; ++i)
#pragma unroll
                for (int j = 0; j < BR; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i].x, bv[j][0], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i].y, bv[j][1], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i].z, bv[j][2], acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i].w, bv[j][3], acc[i][j], 0, 0, 0);
                }
        }
        __syncthreads();
    }

    // ---- epilogue: core = log S into an LDS tile; entries whose S underflowed are marked
    // and recomputed afterwards by a direct log-sum-exp (a rare, non-unrolled path)
    float* T = smem;   // [TM][LDT], over the slice buffers (all reads are done)
    uint64_t under = 0;
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int j = 0; j < BR; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = wm * QW + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                const int col = wn * QW + j * 32 + (lane & 31);
                const float S = acc[i][j][r];
                T[row * LDT + col] = flog(S);
                if (!(S >= kUnderflow) && a0 + row < C && c0 + col < C)
                    under |= 1ull << ((i * BR + j) * 16 + r);
            }
    const int under_seen = under != 0;
    while (under) {
        const int bit = __builtin_ctzll(under);
        under &= under - 1;
        const int ij = bit >> 4, r = bit & 15, i = ij / BR, j = ij % BR;
        const int row = wm * QW + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        const int col = wn * QW + j * 32 + (lane & 31);
        const int gr = a0 + row, gc = c0 + col;
        if (kBits) {
            // no finite index shared by row gr of L and column gc of R: exactly -inf
            const uint64_t* lb = a.crbits + ((size_t)cl * C + gr) * a.bw;
            const uint64_t* rb = a.ccbits + ((size_t)cr * C + gc) * a.bw;
            uint64_t shared = 0;
            for (int q = 0; q < a.bw; ++q) shared |= lb[q] & rb[q];
            if (!shared) {
                T[row * LDT + col] = -INFINITY;
                continue;
            }
        }
        const float sr = sa[row], sc = sb[col];
        const float* lrow = Lc + (size_t)gr * C;
        float q = -INFINITY;
        for (int bb = 0; bb < C; ++bb)
            q = fmaxf(q, (lrow[bb] + coh[bb] - sr) + (Rc[(size_t)bb * C + gc] + roh[bb] - sc));
        float val = -INFINITY;
        if (q != -INFINITY) {
            float sum = 0.f;
            for (int bb = 0; bb < C; ++bb)
                sum += fexp((lrow[bb] + coh[bb] - sr) + (Rc[(size_t)bb * C + gc] + roh[bb] - sc) - q);
            val = q + flog(sum);
        }
        T[row * LDT + col] = val;
    }
    const bool any_under = kBits && __syncthreads_or(under_seen);
    // the output node's offsets for the tile's rows and columns
    for (int i = tid; i < TM; i += kUpThreads) {
        const double ro = a0 + i < C ? (Lro ? Lro[a0 + i] : 0.0) + coLshift + sa[i] : 0.0;
        const double co = c0 + i < C ? (Rco ? Rco[c0 + i] : 0.0) + roRshift + sb[i] : 0.0;
        rof[i] = (float)ro;
        cof[i] = (float)co;
        if (tn == 0 && a0 + i < C) Pro[a0 + i] = ro;
        if (tm == 0 && c0 + i < C) Pco[c0 + i] = co;
    }
    __syncthreads();
    // partial maxima for the next level: thread t < TM row t, TM <= t < 2 TM column t - TM
    const int nr = min(TM, C - a0), nc = min(TM, C - c0);
    // (four running maxima per line: a short dependency chain)
    if (tid < TM) {
        if (tid < nr) {
            float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
            int c = 0;
            for (; c + 4 <= nc; c += 4)
#pragma unroll
                for (int u = 0; u < 4; ++u) m[u] = fmaxf(m[u], T[tid * LDT + c + u] + cof[c + u]);
            for (; c < nc; ++c) m[0] = fmaxf(m[0], T[tid * LDT + c] + cof[c]);
            Pmr[(size_t)(a0 + tid) * nt + tn] = fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3]));
        }
    } else if (tid < 2 * TM) {
        const int c = tid - TM;
        if (c < nc) {
            float m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
            int r = 0;
            for (; r + 4 <= nr; r += 4)
#pragma unroll
                for (int u = 0; u < 4; ++u) m[u] = fmaxf(m[u], T[(r + u) * LDT + c] + rof[r + u]);
            for (; r < nr; ++r) m[0] = fmaxf(m[0], T[r * LDT + c] + rof[r]);
            Pmc[(size_t)(c0 + c) * nt + tm] = fmaxf(fmaxf(m[0], m[1]), fmaxf(m[2], m[3]));
        }
    }
    // the finiteness bitmasks of the tile's rows (the words of its columns) and columns.
    // Only entries recomputed by the fallback can be -inf: without any, every bit is set.
    if (kBits && a.rbits) {
        constexpr int kWords = TM / 64;
        auto prefix = [](int n) { return n >= 64 ? ~0ull : n <= 0 ? 0ull : (1ull << n) - 1; };
        const bool isrow = tid < TM;
        const int line = isrow ? tid : tid - TM, nl = isrow ? nr : nc, len = isrow ? nc : nr;
        if (tid < 2 * TM && line < nl) {
            uint64_t bits[kWords];
#pragma unroll
            for (int q = 0; q < kWords; ++q) bits[q] = any_under ? 0ull : prefix(len - 64 * q);
            if (any_under)
                for (int e = 0; e < len; ++e) {
                    const float v = isrow ? T[line * LDT + e] : T[e * LDT + line];
                    bits[e >> 6] |= (uint64_t)(v > -INFINITY) << (e & 63);
                }
            uint64_t* out = isrow ? a.rbits + ((size_t)pn * C + a0 + line) * a.bw + c0 / 64
                                  : a.cbits + ((size_t)pn * C + c0 + line) * a.bw + a0 / 64;
            const int w0 = (isrow ? c0 : a0) / 64;
#pragma unroll
            for (int q = 0; q < kWords; ++q)
                if (w0 + q < a.bw) out[q] = bits[q];
        }
    }
    // the tile, row by row (16-byte stores when C is a multiple of 4: tiles then start and
    // end on multiples of 4 columns)
    if (VEC) {
        constexpr int kQ = TM / 4;
        const int nc4 = nc / 4;
        for (int idx = tid; idx < nr * kQ; idx += kUpThreads) {
            const int r = idx / kQ, c4 = idx % kQ;
            if (c4 < nc4) {
                const float* t = T + r * LDT + 4 * c4;
                *(float4*)(Pc + (size_t)(a0 + r) * C + c0 + 4 * c4) = make_float4(t[0], t[1], t[2], t[3]);
            }
        }
    } else {
        for (int idx = tid; idx < nr * TM; idx += kUpThreads) {
            const int r = idx / TM, c = idx % TM;
            if (c < nc) Pc[(size_t)(a0 + r) * C + c0 + c] = T[r * LDT + c];
        }
    }
}

// The same product for levels with few output tiles, where latency, not throughput, bounds
// the launch (the upper levels, and every level of a short batch): 32 x 32 output tiles, the
// contraction split over the four waves (wave w takes slices w, w + 4, ... of 32 indices),
// each operand exponentiated in registers straight from memory (lane l holds row / column
// l % 32 at 16 consecutive contraction indices, the same indices for A and B, so the MFMA
// sums over all of them without LDS staging), and the four partial tiles summed through
// LDS.  Every global read goes out before the sequence length is known (no address depends
// on it: an absent child is read from an in-bounds node and never used), so the workgroup
// waits for memory once before its products.  Same outputs as k_up_log (core, ro, co, the
// partial maxima per 32-wide tile); no finiteness masks.
constexpr int kSmTM = 32;
constexpr int kSmSlicesPerWave = (kMaxLabels / kSlice + 3) / 4;

template <bool VEC>
__global__ __launch_bounds__(kUpThreads) void k_up_log_small(UpLogArgs a) {
    constexpr int TM = kSmTM, LDP = TM + 1, NQ = kSmSlicesPerWave;
    static_assert(kUpThreads == 4 * kWave && TM == 32, "four waves, 32 x 32 tiles");
    __shared__ float part[4][TM * LDP];   // the waves' partial tiles; part[0] then holds log S
    __shared__ float coh[kMaxLabels], roh[kMaxLabels];
    __shared__ float sa[TM], sb[TM], rof[TM], cof[TM];
    __shared__ double red[2 * (kUpThreads / kWave)];
    const int ntiles = a.ntile * a.ntile;
    const int64_t lid = xcd_node_swizzle(blockIdx.x, ntiles);
    if (lid >= a.nlogical) return;
    const int tile = (int)(lid % ntiles);
    const int64_t node = lid / ntiles;
    const int64_t b = node / a.nodes, k = node % a.nodes;
    const int C = (int)a.C, nt = a.ntile, cnt = a.cntile;
    const int tm = tile / nt, tn = tile % nt;
    const int a0 = tm * TM, c0 = tn * TM;
    const int tid = threadIdx.x, w = tid / kWave, lane = tid % kWave;
    const int r = lane & 31, h = lane >> 5;

    // children, clamped into the sequence's node range (the node or its right child may be
    // absent; that is known only once the length has arrived)
    const int64_t cl = b * a.cnodes + min(2 * k, a.cnodes - 1);
    const int64_t cr = b * a.cnodes + min(2 * k + 1, a.cnodes - 1);
    const float* Lc = a.ccore + (size_t)cl * C * C;
    const float* Rc = a.ccore + (size_t)cr * C * C;
    const double* Lro = a.cro ? a.cro + (size_t)cl * C : nullptr;
    const double* Lco = a.cco ? a.cco + (size_t)cl * C : nullptr;
    const double* Rro = a.cro ? a.cro + (size_t)cr * C : nullptr;
    const double* Rco = a.cco ? a.cco + (size_t)cr * C : nullptr;

    // ---- every global read at once: the wave's slices of A (row a0 + r) and B (column c0 + r),
    // the contracted offsets, the output lines' offsets and the children's partial maxima
    const int nslices = (C + kSlice - 1) / kSlice;
    const int ga = min(a0 + r, C - 1), gc = min(c0 + r, C - 1);
    float xa[NQ][16], xb[NQ][16];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const int kb = (w + 4 * q) * kSlice + 16 * h;   // this lane's 16 contraction indices
        if (w + 4 * q < nslices) {
            const float* pa = Lc + (size_t)ga * C;
            if (VEC) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float4 v = *(const float4*)(pa + min(kb + 4 * u, C - 4));
                    xa[q][4 * u + 0] = v.x;
                    xa[q][4 * u + 1] = v.y;
                    xa[q][4 * u + 2] = v.z;
                    xa[q][4 * u + 3] = v.w;
                }
            } else {
#pragma unroll
                for (int u = 0; u < 16; ++u) xa[q][u] = pa[min(kb + u, C - 1)];
            }
#pragma unroll
            for (int u = 0; u < 16; ++u) xb[q][u] = Rc[(size_t)min(kb + u, C - 1) * C + gc];
        }
    }
    static_assert(kMaxLabels <= kUpThreads, "one offset of the contracted index per thread");
    const double lco = (Lco && tid < C) ? Lco[tid] : -INFINITY;
    const double rro = (Rro && tid < C) ? Rro[tid] : -INFINITY;
    // thread t < TM: row a0 + t (of L, and of the output); TM <= t < 2 TM: column c0 + t - TM
    const bool isrow = tid < TM, iscol = tid >= TM && tid < 2 * TM;
    const int li = isrow ? tid : tid - TM;
    const bool lok = (isrow && a0 + li < C) || (iscol && c0 + li < C);
    double loff = 0.0;   // ro_L of the row, co_R of the column
    float pm = -INFINITY;
    if (lok) {
        loff = isrow ? (Lro ? Lro[a0 + li] : 0.0) : (Rco ? Rco[c0 + li] : 0.0);
        const float* pp = isrow ? a.cpmr + ((size_t)cl * C + a0 + li) * cnt
                                : a.cpmc + ((size_t)cr * C + c0 + li) * cnt;
#pragma unroll
        for (int q = 0; q < kMaxLabels / kSmTM; ++q)
            if (q < cnt) pm = fmaxf(pm, pp[q]);
    }

    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;   // node absent: all padding
    const int64_t pn = b * a.nodes + k;
    float* Pc = a.core + (size_t)pn * C * C;
    double* Pro = a.ro + (size_t)pn * C;
    double* Pco = a.co + (size_t)pn * C;
    float* Pmr = a.pmr + (size_t)pn * C * nt;
    float* Pmc = a.pmc + (size_t)pn * C * nt;
    if (!((2 * k + 1) * half < Eb)) {
        // the right half is padding: the node equals its left child (tile, offsets and the
        // partial maxima, re-tiled: only the maximum over a line's partials is ever read)
        for (int idx = tid; idx < TM * TM; idx += kUpThreads) {
            const int rr = a0 + idx / TM, cc = c0 + idx % TM;
            if (rr < C && cc < C) Pc[(size_t)rr * C + cc] = Lc[(size_t)rr * C + cc];
        }
        if (tn == 0)
            for (int i = tid; i < TM; i += kUpThreads)
                if (a0 + i < C) Pro[a0 + i] = Lro ? Lro[a0 + i] : 0.0;
        if (tm == 0)
            for (int i = tid; i < TM; i += kUpThreads)
                if (c0 + i < C) Pco[c0 + i] = Lco ? Lco[c0 + i] : 0.0;
        if (tm == 0 && tn == 0)
            for (int i = tid; i < C * nt; i += kUpThreads) {
                const int line = i / nt, pq = i % nt;
                const float* sr = a.cpmr + ((size_t)cl * C + line) * cnt;
                const float* sc = a.cpmc + ((size_t)cl * C + line) * cnt;
                float mr = -INFINITY, mc = -INFINITY;
                if (pq == 0)
                    for (int q = 0; q < cnt; ++q) {
                        mr = fmaxf(mr, sr[q]);
                        mc = fmaxf(mc, sc[q]);
                    }
                Pmr[i] = mr;
                Pmc[i] = mc;
            }
        return;
    }

    // ---- shifts: max co_L and max ro_R over the contracted index (one reduction), the tile's
    // row shifts sa (row maxima of core_L + co_L - max co_L) and column shifts sb
    {
        const double lw = wave_max_d(lco), rw = wave_max_d(rro);
        if (lane == 0) {
            red[2 * w] = lw;
            red[2 * w + 1] = rw;
        }
    }
    __syncthreads();
    double lmax = red[0], rmax = red[1];
#pragma unroll
    for (int q = 1; q < kUpThreads / kWave; ++q) {
        lmax = fmax(lmax, red[2 * q]);
        rmax = fmax(rmax, red[2 * q + 1]);
    }
    const double coLshift = Lco ? safe_shift_d(lmax) : 0.0;
    const double roRshift = Rro ? safe_shift_d(rmax) : 0.0;
    if (tid < C) {
        coh[tid] = Lco ? (float)(lco - coLshift) : 0.f;
        roh[tid] = Rro ? (float)(rro - roRshift) : 0.f;
    }
    if (isrow) sa[li] = safe_shift(lok ? pm - (float)coLshift : -INFINITY);
    if (iscol) sb[li] = safe_shift(lok ? pm - (float)roRshift : -INFINITY);
    __syncthreads();

    // ---- the wave's partial product over its slices
    f16v acc;
#pragma unroll
    for (int q = 0; q < 16; ++q) acc[q] = 0.f;
    {
        const float s_a = sa[r], s_b = sb[r];
        const bool rok = a0 + r < C, cok = c0 + r < C;
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const int kb = (w + 4 * q) * kSlice + 16 * h;
            if (w + 4 * q < nslices) {
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int kk = kb + u;
                    const bool kok = kk < C;
                    const float av = (rok && kok) ? fexp(xa[q][u] + coh[kk] - s_a) : 0.f;
                    const float bv = (cok && kok) ? fexp(xb[q][u] + roh[kk] - s_b) : 0.f;
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc, 0, 0, 0);
                }
            }
        }
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
        const int row = (q >> 2) * 8 + h * 4 + (q & 3);
        part[w][row * LDP + r] = acc[q];
    }
    __syncthreads();

    // ---- S = sum of the partial tiles, core = log S (an underflowed S, every term below
    // 2^-80, is recomputed by a direct log-sum-exp: a rare, non-unrolled path)
    const int nr = min(TM, C - a0), nc = min(TM, C - c0);
#pragma unroll
    for (int q = 0; q < TM * TM / kUpThreads; ++q) {
        const int e = tid + q * kUpThreads, row = e / TM, col = e % TM, o = row * LDP + col;
        const float S = (part[0][o] + part[1][o]) + (part[2][o] + part[3][o]);
        float val = flog(S);
        if (!(S >= kUnderflow) && row < nr && col < nc) {
            const float sr = sa[row], sc = sb[col];
            const float* lrow = Lc + (size_t)(a0 + row) * C;
            const int gcol = c0 + col;
            float mx = -INFINITY;
            for (int bb = 0; bb < C; ++bb)
                mx = fmaxf(mx, (lrow[bb] + coh[bb] - sr) + (Rc[(size_t)bb * C + gcol] + roh[bb] - sc));
            val = -INFINITY;
            if (mx != -INFINITY) {
                float sum = 0.f;
                for (int bb = 0; bb < C; ++bb)
                    sum += fexp((lrow[bb] + coh[bb] - sr) + (Rc[(size_t)bb * C + gcol] + roh[bb] - sc) - mx);
                val = mx + flog(sum);
            }
        }
        part[0][o] = val;
    }
    // the output node's offsets for the tile's rows and columns
    if (lok) {
        const double off = isrow ? loff + coLshift + sa[li] : loff + roRshift + sb[li];
        (isrow ? rof : cof)[li] = (float)off;
        if (isrow && tn == 0) Pro[a0 + li] = off;
        if (iscol && tm == 0) Pco[c0 + li] = off;
    } else if (isrow || iscol) {
        (isrow ? rof : cof)[li] = 0.f;
    }
    __syncthreads();

    // ---- partial maxima for the next level: four threads per line, eight entries each
    {
        const bool rowp = tid < 4 * TM;
        const int line = (rowp ? tid : tid - 4 * TM) >> 2, seg = 8 * (tid & 3);
        const float* T = part[0];
        float m = -INFINITY;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int e = seg + u;
            if (rowp ? e < nc : e < nr)
                m = fmaxf(m, rowp ? T[line * LDP + e] + cof[e] : T[e * LDP + line] + rof[e]);
        }
        m = fmaxf(m, __shfl_xor(m, 1, kWave));
        m = fmaxf(m, __shfl_xor(m, 2, kWave));
        if ((tid & 3) == 0) {
            if (rowp && line < nr) Pmr[(size_t)(a0 + line) * nt + tn] = m;
            if (!rowp && line < nc) Pmc[(size_t)(c0 + line) * nt + tm] = m;
        }
    }
    // ---- the tile, row by row (16-byte stores when C is a multiple of 4)
    {
        const int row = tid / (TM / 4), c4 = 4 * (tid % (TM / 4));
        const float* t = part[0] + row * LDP + c4;
        if (row < nr) {
            float* dst = Pc + (size_t)(a0 + row) * C + c0 + c4;
            if (VEC) {
                if (c4 < nc) *(float4*)dst = make_float4(t[0], t[1], t[2], t[3]);
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (c4 + u < nc) dst[u] = t[u];
            }
        }
    }
}

// The same product for full tiles (C a multiple of TM, no finiteness masks), scheduled for
// the matrix cores: the raw potentials of slice s + 2 are loaded during slice s (two
// register sets, so a load has a whole slice to arrive); the exponentials of slice s + 1
// are spread over the four 8-wide k groups of slice s, between their products; and each
// group's LDS operands are read before the previous group's products are issued.  No
// per-entry masks are needed: every row, column and contracted index of a tile is valid.
// An operand is exp2(fma(x, log2 e, o log2 e) - s log2 e), the thread's shifts scaled once.
template <int TM>
struct UpFullSmem {
    static constexpr int LDA = kSlice + 4, LDB = TM + 4;
    static constexpr int kBuf = TM * LDA + kSlice * LDB;
    static constexpr int kMain = 2 * kBuf;          // (the epilogue's [2][TM] maxima fit)
    // cohs, rohs [kMaxLabels]; sa, sb, cof, rof [TM]; red [2 doubles per wave]
    static constexpr int kFloats = kMain + 2 * kMaxLabels + 4 * TM + 4 * (kUpThreads / kWave);
    static constexpr size_t kBytes = sizeof(float) * kFloats;
    static constexpr int kBlocksPerCU = 2;
};

// The bf16 variant (kBf) stages each exponentiated operand x as three bf16 parts
// x = hi + mid + lo (hi = x truncated to bf16, mid = x - hi truncated, lo = x - hi - mid, which
// bf16 holds exactly: 24 significant bits, float32's own precision, and float32's exponent
// range), in slices of 16 contracted
// indices, A as [row][k] and B transposed as [column][k], and sums the six products
//   hi.hi + hi.mid + mid.hi + hi.lo + lo.hi + mid.mid
// with the bf16 matrix instructions (32x32x16, float32 accumulation), which run 16 times the
// float32 MFMA rate.  The three dropped products are below 2^-24 of |x y|, so a sum matches
// the float32 product to float32 rounding.
// Its LDS fits three workgroups per CU (52 KB each): staged lines of 32 bytes without
// padding, the two 16-byte halves of line r swapped when bit 2 xor bit 3 of r is set (so
// that rows r .. r + 7 and r .. r + 15 of one half, aligned, land on distinct 16-byte bank
// groups, whether a 16-byte access is served 8 or 16 lanes at a time), and an epilogue that
// works from the registers.
template <int TM>
struct UpBfSmem {
    static constexpr int kK = 16;                   // contracted indices per slice
    static constexpr int LDK = kK;                  // bf16 per staged line (32 bytes)
    static constexpr int kPlane = TM * LDK;         // bf16 per part plane
    static constexpr int kBufF = 6 * kPlane / 2;    // A and B, three parts each, in floats
    static constexpr int kMain = 2 * kBufF;
    static constexpr int kFloats = kMain + 2 * kMaxLabels + 4 * TM + 4 * (kUpThreads / kWave);
    static constexpr size_t kBytes = sizeof(float) * kFloats;
    static constexpr int kBlocksPerCU = 3;
};
static_assert(3 * UpBfSmem<128>::kBytes <= 160 * 1024, "three workgroups per CU");

// element offset of the 16-byte half h of staged line r (LDK = 16 bf16 per line)
__device__ __forceinline__ int bf_line_half(int r, int h) {
    return r * 16 + 8 * (h ^ (((r >> 2) ^ (r >> 3)) & 1));
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// x = hi + mid + lo exactly: hi is x truncated to its leading 8 significant bits (the upper
// half of its float encoding), mid the same of the remainder r = x - hi (exact in float, at
// most 16 significant bits), lo = r - mid (at most 8 bits, so its upper half is exact too).
// Two elements' upper halves are packed by one byte permute.
__device__ __forceinline__ void split_bf16x3(const float (&x)[8], bf16x8& hi, bf16x8& mid, bf16x8& lo) {
    typedef unsigned u4v __attribute__((ext_vector_type(4)));
    constexpr unsigned kHi = 0xffff0000u, kSel = 0x07060302u;   // upper halves of (src1, src0)
    u4v h, m, l;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const unsigned x0 = __float_as_uint(x[2 * p]), x1 = __float_as_uint(x[2 * p + 1]);
        const float r0 = x[2 * p] - __uint_as_float(x0 & kHi);
        const float r1 = x[2 * p + 1] - __uint_as_float(x1 & kHi);
        const unsigned q0 = __float_as_uint(r0), q1 = __float_as_uint(r1);
        const float t0 = r0 - __uint_as_float(q0 & kHi), t1 = r1 - __uint_as_float(q1 & kHi);
        h[p] = __builtin_amdgcn_perm(x1, x0, kSel);
        m[p] = __builtin_amdgcn_perm(q1, q0, kSel);
        l[p] = __builtin_amdgcn_perm(__float_as_uint(t1), __float_as_uint(t0), kSel);
    }
    hi = __builtin_bit_cast(bf16x8, h);
    mid = __builtin_bit_cast(bf16x8, m);
    lo = __builtin_bit_cast(bf16x8, l);
}

template <int TM, bool kBf, int kNS = 0>
__global__ __launch_bounds__(kUpThreads,
                             (kBf ? UpBfSmem<TM>::kBlocksPerCU : UpFullSmem<TM>::kBlocksPerCU))
void k_up_log_full(UpLogArgs a) {
    using Sm = std::conditional_t<kBf, UpBfSmem<TM>, UpFullSmem<TM>>;
    constexpr int BR = TM / 64;                 // 32 x 32 blocks per wave per dimension
    constexpr int QW = TM / 2;                  // a wave's quarter edge
    constexpr float kL2E = 1.4426950408889634f;
    extern __shared__ __align__(16) float smem[];
    const int ntiles = a.ntile * a.ntile;
    const int64_t lid = xcd_node_swizzle(blockIdx.x, ntiles);
    if (lid >= a.nlogical) return;
    const int tile = (int)(lid % ntiles);
    const int64_t node = lid / ntiles;
    const int64_t b = node / a.nodes, k = node % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;  // node absent: all padding
    const int C = (int)a.C;
    const int tm = tile / a.ntile, tn = tile % a.ntile;
    const int a0 = tm * TM, c0 = tn * TM;
    const int tid = threadIdx.x;
    const int nt = a.ntile, cnt = a.cntile;

    const int64_t cl = b * a.cnodes + 2 * k, cr = cl + 1, pn = b * a.nodes + k;
    const float* Lc = a.ccore + (size_t)cl * C * C;
    float* Pc = a.core + (size_t)pn * C * C;
    double* Pro = a.ro + (size_t)pn * C;
    double* Pco = a.co + (size_t)pn * C;
    float* Pmr = a.pmr + (size_t)pn * C * nt;
    float* Pmc = a.pmc + (size_t)pn * C * nt;

    if (!((2 * k + 1) * half < Eb)) {
        // the right half is padding: the node equals its left child (tile, offsets and the
        // maximum of each line's partials, kept in partial 0)
        constexpr int kQ = TM / 4;
        for (int idx = tid; idx < TM * kQ; idx += kUpThreads) {
            const int r = a0 + idx / kQ, c = c0 + 4 * (idx % kQ);
            *(float4*)(Pc + (size_t)r * C + c) = *(const float4*)(Lc + (size_t)r * C + c);
        }
        if (tn == 0)
            for (int i = tid; i < TM; i += kUpThreads)
                Pro[a0 + i] = a.cro ? a.cro[(size_t)cl * C + a0 + i] : 0.0;
        if (tm == 0)
            for (int i = tid; i < TM; i += kUpThreads)
                Pco[c0 + i] = a.cco ? a.cco[(size_t)cl * C + c0 + i] : 0.0;
        if (tm == 0 && tn == 0)
            for (int i = tid; i < C * nt; i += kUpThreads) {
                const int line = i / nt, p = i % nt;
                const float* sr = a.cpmr + ((size_t)cl * C + line) * cnt;
                const float* sc = a.cpmc + ((size_t)cl * C + line) * cnt;
                float mr = -INFINITY, mc = -INFINITY;
                if (p == 0)
                    for (int q = 0; q < cnt; ++q) {
                        mr = fmaxf(mr, sr[q]);
                        mc = fmaxf(mc, sc[q]);
                    }
                Pmr[i] = mr;
                Pmc[i] = mc;
            }
        return;
    }
    const float* Rc = a.ccore + (size_t)cr * C * C;
    const double* Lro = a.cro ? a.cro + (size_t)cl * C : nullptr;
    const double* Lco = a.cco ? a.cco + (size_t)cl * C : nullptr;
    const double* Rro = a.cro ? a.cro + (size_t)cr * C : nullptr;
    const double* Rco = a.cco ? a.cco + (size_t)cr * C : nullptr;

    float* cohs = smem + Sm::kMain;      // [kMaxLabels] (co_L - max co_L) log2 e
    float* rohs = cohs + kMaxLabels;     // [kMaxLabels] (ro_R - max ro_R) log2 e
    float* sa = rohs + kMaxLabels;       // [TM] row shifts of the tile
    float* sb = sa + TM;                 // [TM] column shifts
    float* cof = sb + TM;                // [TM] co_P of the tile's columns (float)
    float* rof = cof + TM;               // [TM] ro_P of the tile's rows (float)
    double* red = reinterpret_cast<double*>(rof + TM);

    // the offsets of the contracted index shifted to max 0, scaled by log2 e (cohs, rohs)
    // and the tile's row and column shifts; every global read of it goes out at once, after
    // the first slices' loads
    double coLshift = 0.0, roRshift = 0.0;
    auto shifts = [&]() {
        static_assert(kMaxLabels <= kUpThreads, "one offset of the contracted index per thread");
        static_assert(TM <= kUpThreads, "one output row and column per thread");
        const double lco = (Lco && tid < C) ? Lco[tid] : -INFINITY;
        const double rro = (Rro && tid < C) ? Rro[tid] : -INFINITY;
        double lro_t = 0.0, rco_t = 0.0;   // ro_L of row a0 + tid, co_R of column c0 + tid
        if (tid < TM) {
            lro_t = Lro ? Lro[a0 + tid] : 0.0;
            rco_t = Rco ? Rco[c0 + tid] : 0.0;
        }
        float pa = -INFINITY, pb = -INFINITY;
        if (tid < TM)
            partials_max2(a.cpmr + ((size_t)cl * C + a0 + tid) * cnt,
                          a.cpmc + ((size_t)cr * C + c0 + tid) * cnt, cnt, pa, pb);
        {
            const double lw = wave_max_d(lco), rw = wave_max_d(rro);
            const int w = tid / kWave;
            if ((tid & (kWave - 1)) == 0) {
                red[2 * w] = lw;
                red[2 * w + 1] = rw;
            }
        }
        __syncthreads();
        double lmax = red[0], rmax = red[1];
#pragma unroll
        for (int w = 1; w < kUpThreads / kWave; ++w) {
            lmax = fmax(lmax, red[2 * w]);
            rmax = fmax(rmax, red[2 * w + 1]);
        }
        // (the same for every thread: kept in scalar registers through the products)
        coLshift = uniform_d(Lco ? safe_shift_d(lmax) : 0.0);
        roRshift = uniform_d(Rro ? safe_shift_d(rmax) : 0.0);
        if (tid < C) {
            const float ch = Lco ? (float)(lco - coLshift) : 0.f;
            const float rh = Rro ? (float)(rro - roRshift) : 0.f;
            cohs[tid] = ch * kL2E;
            rohs[tid] = rh * kL2E;
        }
        if (tid < TM) {
            const float sav = safe_shift(pa - (float)coLshift), sbv = safe_shift(pb - (float)roRshift);
            sa[tid] = sav;
            sb[tid] = sbv;
            // the output node's offsets for the tile's rows and columns (known now; the
            // epilogue reads them from LDS)
            const double ro = lro_t + coLshift + sav;
            const double co = rco_t + roRshift + sbv;
            rof[tid] = (float)ro;
            cof[tid] = (float)co;
            if (tn == 0) Pro[a0 + tid] = ro;
            if (tm == 0) Pco[c0 + tid] = co;
        }
        __syncthreads();
    };
    const int w = tid / kWave, lane = tid % kWave;
    const int wm = w >> 1, wn = w & 1;
    f16v acc[BR][BR];
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int j = 0; j < BR; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    if constexpr (!kBf) {
        constexpr int LDA = Sm::LDA, LDB = Sm::LDB;
        // ---- per-thread staging assignment (fixed over the slices):
        //   A'' (TM x 32): rows ar + 32 it (it < NA), contracted indices ak .. ak + 3;
        //   B'' (32 x TM): contracted rows bk .. bk + NB - 1, columns bc .. bc + 3
        constexpr int GA = kSlice / 4, NA = TM * GA / kUpThreads;
        constexpr int GB = TM / 4, NB = kSlice * GB / kUpThreads;
        static_assert(NB == 4 || NB == 2, "contracted rows of a thread: one or half a float4");
        const int ar = tid / GA, ak = 4 * (tid % GA);
        const int bk = NB * (tid / GB), bc = 4 * (tid % GB);
        // loads: raw buffer loads over each child matrix (C * C floats), a fixed 32-bit byte
        // offset per thread and register and the slice's offset in a scalar register, so that
        // no address arithmetic is repeated per slice
        const __amdgpu_buffer_rsrc_t rsL = make_rsrc(Lc, C * C);
        const __amdgpu_buffer_rsrc_t rsR = make_rsrc(Rc, C * C);
        unsigned offa[NA], offb[NB];
#pragma unroll
        for (int it = 0; it < NA; ++it) offa[it] = 4u * (unsigned)((a0 + ar + 32 * it) * C + ak);
#pragma unroll
        for (int it = 0; it < NB; ++it) offb[it] = 4u * (unsigned)((bk + it) * C + c0 + bc);
        float4 ra[2][NA], rb[2][NB];
        auto gload = [&](float4 (&xa)[NA], float4 (&xb)[NB], int ks) {
#pragma unroll
            for (int it = 0; it < NA; ++it) xa[it] = buffer_load4(rsL, offa[it], 4 * ks);
#pragma unroll
            for (int it = 0; it < NB; ++it) xb[it] = buffer_load4(rsR, offb[it], 4 * ks * C);
        };
        float sas[NA], sbs[4];
        // the offsets of the staged contracted indices (A: ak..ak+3, B: bk..bk+NB-1), scaled by
        // log2 e, read from LDS once per slice
        auto offsets = [&](float (&oa)[4], float (&ob)[4], int ks) {
            const float4 x = *(const float4*)(cohs + ks + ak);
            oa[0] = x.x; oa[1] = x.y; oa[2] = x.z; oa[3] = x.w;
            if constexpr (NB == 4) {
                const float4 y = *(const float4*)(rohs + ks + bk);
                ob[0] = y.x; ob[1] = y.y; ob[2] = y.z; ob[3] = y.w;
            } else {
                const float2 y = *(const float2*)(rohs + ks + bk);
                ob[0] = y.x; ob[1] = y.y; ob[2] = ob[3] = 0.f;
            }
        };
        // exponentials of staged part `part` of `nparts` (A groups, then B groups) into buffer buf
        auto stage = [&](const float4 (&xa)[NA], const float4 (&xb)[NB], const float (&oa)[4],
                         const float (&ob)[4], int buf, int part, int nparts) {
            float* As = smem + buf * Sm::kBuf;
            float* Bs = As + TM * LDA;
#pragma unroll
            for (int it = NA * part / nparts; it < NA * (part + 1) / nparts; ++it) {
                float4 x;
                x.x = __builtin_amdgcn_exp2f(fmaf(xa[it].x, kL2E, oa[0]) - sas[it]);
                x.y = __builtin_amdgcn_exp2f(fmaf(xa[it].y, kL2E, oa[1]) - sas[it]);
                x.z = __builtin_amdgcn_exp2f(fmaf(xa[it].z, kL2E, oa[2]) - sas[it]);
                x.w = __builtin_amdgcn_exp2f(fmaf(xa[it].w, kL2E, oa[3]) - sas[it]);
                *(float4*)(As + (ar + 32 * it) * LDA + ak) = x;
            }
#pragma unroll
            for (int it = NB * part / nparts; it < NB * (part + 1) / nparts; ++it) {
                float4 x;
                x.x = __builtin_amdgcn_exp2f(fmaf(xb[it].x, kL2E, ob[it]) - sbs[0]);
                x.y = __builtin_amdgcn_exp2f(fmaf(xb[it].y, kL2E, ob[it]) - sbs[1]);
                x.z = __builtin_amdgcn_exp2f(fmaf(xb[it].z, kL2E, ob[it]) - sbs[2]);
                x.w = __builtin_amdgcn_exp2f(fmaf(xb[it].w, kL2E, ob[it]) - sbs[3]);
                *(float4*)(Bs + (bk + it) * LDB + bc) = x;
            }
        };

        // ---- the first two slices' loads and every global read of the set-up go out at once
        const int nslices = C / kSlice;   // even: C is a multiple of 64
        gload(ra[0], rb[0], 0);
        gload(ra[1], rb[1], kSlice);
        shifts();
#pragma unroll
        for (int it = 0; it < NA; ++it) sas[it] = sa[ar + 32 * it] * kL2E;
#pragma unroll
        for (int q = 0; q < 4; ++q) sbs[q] = sb[bc + q] * kL2E;
        {
            float oa[4], ob[4];
            offsets(oa, ob, 0);
            stage(ra[0], rb[0], oa, ob, 0, 0, 1);
        }
        __syncthreads();

        // ---- products: wave (wm, wn) owns rows wm*QW.., columns wn*QW.. as BR x BR blocks.
        // Within each 8-wide k group lanes 0-31 contribute k..k+3 and lanes 32-63 k+4..k+7 (one
        // 16-byte LDS read of A per block row, four reads of B per block column).
        const int aoff = (wm * QW + (lane & 31)) * LDA + 4 * (lane >> 5);
        const int boff = TM * LDA + (4 * (lane >> 5)) * LDB + wn * QW + (lane & 31);
        float4 av[2][BR];
        float bv[2][BR][4];
        auto lds_ops = [&](float4 (&xa)[BR], float (&xb)[BR][4], int buf, int kk) {
            const float* base = smem + buf * Sm::kBuf;
#pragma unroll
            for (int i = 0; i < BR; ++i) xa[i] = *(const float4*)(base + aoff + i * 32 * LDA + kk);
#pragma unroll
            for (int j = 0; j < BR; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) xb[j][q] = base[boff + (kk + q) * LDB + j * 32];
        };
        auto mfma_group = [&](const float4 (&xa)[BR], const float (&xb)[BR][4]) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < BR; ++i)
#pragma unroll
                    for (int j = 0; j < BR; ++j) {
                        const float ax = q == 0 ? xa[i].x : q == 1 ? xa[i].y : q == 2 ? xa[i].z : xa[i].w;
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(ax, xb[j][q], acc[i][j], 0, 0, 0);
                    }
        };
        // one slice: products of buffer `cur` while slice s + 1 (raw set xa1/xb1) is staged into
        // the other buffer and slice s + 2 is loaded into the set just consumed (xa0/xb0).  After
        // the last slice the staging works on stale registers into a buffer nobody reads (no
        // branch, so the products and the staging form one block the scheduler can interleave).
        // The loads are unconditional too (the last two slices reload the last one): a load
        // behind a branch makes the compiler wait for every outstanding load where the set
        // loaded the slice before is used, i.e. for the load just issued, every second slice.
        auto slice = [&](int s, int cur, float4 (&xa0)[NA], float4 (&xb0)[NB], float4 (&xa1)[NA],
                         float4 (&xb1)[NB]) {
            gload(xa0, xb0, min(s + 2, nslices - 1) * kSlice);
            float oa[4], ob[4];
            offsets(oa, ob, min(s + 1, nslices - 1) * kSlice);
            lds_ops(av[0], bv[0], cur, 0);
#pragma unroll
            for (int g = 0; g < kSlice / 8; ++g) {
                if (g + 1 < kSlice / 8) lds_ops(av[(g + 1) & 1], bv[(g + 1) & 1], cur, 8 * (g + 1));
                stage(xa1, xb1, oa, ob, cur ^ 1, g, kSlice / 8);
                mfma_group(av[g & 1], bv[g & 1]);
                // one product, then two VALU instructions (the staging), and the operand reads
                // of the next group and the staging's stores spread over the products
#pragma unroll
                for (int i = 0; i < 4 * BR * BR; ++i) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
                    if (i % 2 == 0) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    if (i % 8 == 7) __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
                }
            }
            __syncthreads();
        };
        for (int s = 0; s < nslices; s += 2) {
            slice(s, 0, ra[0], rb[0], ra[1], rb[1]);
            slice(s + 1, 1, ra[1], rb[1], ra[0], rb[0]);
        }
    } else {
        // ---- bf16 parts.  Staging: A row ar = tid / 2, contracted indices ka .. ka + 7 (two
        // 16-byte loads); B column bcol = tid % TM, contracted indices kb .. kb + 7 (eight loads,
        // each a row segment shared by the wave: coalesced)
        static_assert(TM == 128, "one A line segment and one B column segment per thread");
        constexpr int kK = Sm::kK, LDK = Sm::LDK, PL = Sm::kPlane;
        constexpr int kBufH = 2 * Sm::kBufF;   // bf16 per slice buffer
        __bf16* hsm = reinterpret_cast<__bf16*>(smem);
        const int ar = tid >> 1, ka = 8 * (tid & 1);
        const int bcol = tid & (TM - 1);
        const int kb = __builtin_amdgcn_readfirstlane(8 * (tid / TM));   // wave-uniform
        const __amdgpu_buffer_rsrc_t rsL = make_rsrc(Lc, C * C);
        const __amdgpu_buffer_rsrc_t rsR = make_rsrc(Rc, C * C);
        const unsigned offa = 4u * (unsigned)((a0 + ar) * C + ka);
        const unsigned offb = 4u * (unsigned)(c0 + bcol);
        float4 ra[2][2];
        float rb[2][8];
        auto gload = [&](float4 (&xa)[2], float (&xb)[8], int ks) {
            xa[0] = buffer_load4(rsL, offa, 4 * ks);
            xa[1] = buffer_load4(rsL, offa + 16u, 4 * ks);
#pragma unroll
            for (int j = 0; j < 8; ++j) xb[j] = buffer_load1(rsR, offb, 4 * (ks + kb + j) * C);
        };
        float sas = 0.f, sbs = 0.f;
        // staging of one slice in phases (so that the phases can go between the products of the
        // slice before): the offset vectors of its contracted indices, the exponentials of A's
        // (or B's) eight entries, then their parts into buffer buf
        struct StageRegs {
            float4 oa0, oa1, ob0, ob1;   // offsets (log2 units) of ka.., kb..
            float x[8];                  // exponentials of the phase's side
        };
        auto stage_offsets_a = [&](StageRegs& g, int ks) {
            g.oa0 = *(const float4*)(cohs + ks + ka);
            g.oa1 = *(const float4*)(cohs + ks + ka + 4);
        };
        auto stage_offsets_b = [&](StageRegs& g, int ks) {
            g.ob0 = *(const float4*)(rohs + ks + kb);
            g.ob1 = *(const float4*)(rohs + ks + kb + 4);
        };
        auto stage_exp_a = [&](StageRegs& g, const float4 (&xa)[2]) {
            g.x[0] = __builtin_amdgcn_exp2f(fmaf(xa[0].x, kL2E, g.oa0.x) - sas);
            g.x[1] = __builtin_amdgcn_exp2f(fmaf(xa[0].y, kL2E, g.oa0.y) - sas);
            g.x[2] = __builtin_amdgcn_exp2f(fmaf(xa[0].z, kL2E, g.oa0.z) - sas);
            g.x[3] = __builtin_amdgcn_exp2f(fmaf(xa[0].w, kL2E, g.oa0.w) - sas);
            g.x[4] = __builtin_amdgcn_exp2f(fmaf(xa[1].x, kL2E, g.oa1.x) - sas);
            g.x[5] = __builtin_amdgcn_exp2f(fmaf(xa[1].y, kL2E, g.oa1.y) - sas);
            g.x[6] = __builtin_amdgcn_exp2f(fmaf(xa[1].z, kL2E, g.oa1.z) - sas);
            g.x[7] = __builtin_amdgcn_exp2f(fmaf(xa[1].w, kL2E, g.oa1.w) - sas);
        };
        auto stage_exp_b = [&](StageRegs& g, const float (&xb)[8]) {
            g.x[0] = __builtin_amdgcn_exp2f(fmaf(xb[0], kL2E, g.ob0.x) - sbs);
            g.x[1] = __builtin_amdgcn_exp2f(fmaf(xb[1], kL2E, g.ob0.y) - sbs);
            g.x[2] = __builtin_amdgcn_exp2f(fmaf(xb[2], kL2E, g.ob0.z) - sbs);
            g.x[3] = __builtin_amdgcn_exp2f(fmaf(xb[3], kL2E, g.ob0.w) - sbs);
            g.x[4] = __builtin_amdgcn_exp2f(fmaf(xb[4], kL2E, g.ob1.x) - sbs);
            g.x[5] = __builtin_amdgcn_exp2f(fmaf(xb[5], kL2E, g.ob1.y) - sbs);
            g.x[6] = __builtin_amdgcn_exp2f(fmaf(xb[6], kL2E, g.ob1.z) - sbs);
            g.x[7] = __builtin_amdgcn_exp2f(fmaf(xb[7], kL2E, g.ob1.w) - sbs);
        };
        // side 0: A row ar at ka; side 1: B column bcol at kb (planes 3..5)
        auto stage_store = [&](const StageRegs& g, int side, int buf) {
            bf16x8 h, m, l;
            split_bf16x3(g.x, h, m, l);
            __bf16* d = hsm + buf * kBufH + (side ? 3 * PL + bf_line_half(bcol, kb >> 3)
                                                  : bf_line_half(ar, ka >> 3));
            *(bf16x8*)(d) = h;
            *(bf16x8*)(d + PL) = m;
            *(bf16x8*)(d + 2 * PL) = l;
        };
        auto stage = [&](const float4 (&xa)[2], const float (&xb)[8], int ks, int buf) {
            StageRegs g;
            stage_offsets_a(g, ks);
            stage_offsets_b(g, ks);
            stage_exp_a(g, xa);
            stage_store(g, 0, buf);
            stage_exp_b(g, xb);
            stage_store(g, 1, buf);
        };
        // (C = 128 or 256: the slice count is a compile-time constant, so that the slice loop
        // below unrolls completely and each slice's offsets are immediates)
        static_assert(kNS == 8 || kNS == 16, "bf16 parts: C = 128 or 256");
        constexpr int nslices = kNS;
        gload(ra[0], rb[0], 0);
        gload(ra[1], rb[1], kK);
        shifts();
        sas = sa[ar] * kL2E;
        sbs = sb[bcol] * kL2E;
        stage(ra[0], rb[0], 0, 0);
        __syncthreads();

        // ---- products: wave (wm, wn) owns rows wm*QW.., columns wn*QW.. as BR x BR blocks;
        // lane l supplies row (column) l % 32 at contracted indices 8 (l / 32) .. + 7 (the
        // lines' bits 2 and 3 are those of l % 32, as QW and 32 are multiples of 16)
        const int li = lane & 31;
        const int aoff = bf_line_half(wm * QW + li, lane >> 5), boff = bf_line_half(wn * QW + li, lane >> 5);
        // part p of A (of B) for the wave's BR blocks
        auto read_a = [&](bf16x8 (&A)[BR], int buf, int p) {
#pragma unroll
            for (int i = 0; i < BR; ++i)
                A[i] = *(const bf16x8*)(hsm + buf * kBufH + p * PL + aoff + i * 32 * LDK);
        };
        auto read_b = [&](bf16x8 (&Bv)[BR], int buf, int p) {
#pragma unroll
            for (int j = 0; j < BR; ++j)
                Bv[j] = *(const bf16x8*)(hsm + buf * kBufH + (3 + p) * PL + boff + j * 32 * LDK);
        };
        // one slice: the products of buffer cur while slice s + 1 (raw set xa1/xb1) is staged into
        // the other buffer and slice s + 2 is loaded into the set just consumed (xa0/xb0; the
        // last two slices reload the last one, without a branch: as in the float32 variant).
        // After the last slice the staging works on stale registers into a buffer nobody reads.
        // The six products of each block pair go out in six groups of BR x BR independent products
        // (different accumulators); one staging phase follows each group, fenced so that the
        // scheduler interleaves the two within the group but keeps the groups in order.
        auto slice = [&](int s, int cur, float4 (&xa0)[2], float (&xb0)[8], float4 (&xa1)[2],
                         float (&xb1)[8]) {
            // (no instruction moves between slices: the unrolled slices would otherwise
            // interleave and hold more registers than three workgroups per CU leave)
            __builtin_amdgcn_sched_barrier(0);
            gload(xa0, xb0, min(s + 2, nslices - 1) * kK);
            // the operands of the first two groups now, those of the other four during the
            // first group (fewer registers held at once)
            bf16x8 A[3][BR], Bv[3][BR];
            read_a(A[2], cur, 2);
            read_b(Bv[0], cur, 0);
            read_a(A[0], cur, 0);
            read_b(Bv[2], cur, 2);
            StageRegs g;
            // (part of A, part of B): the smaller products first
            constexpr int kTerms[6][2] = {{2, 0}, {0, 2}, {1, 1}, {1, 0}, {0, 1}, {0, 0}};
            auto term = [&](int t) {
#pragma unroll
                for (int i = 0; i < BR; ++i)
#pragma unroll
                    for (int j = 0; j < BR; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            A[kTerms[t][0]][i], Bv[kTerms[t][1]][j], acc[i][j], 0, 0, 0);
            };
            const int ks1 = min(s + 1, nslices - 1) * kK;
            // (each side's offsets are read just before that side's exponentials need them)
            term(0);
            read_a(A[1], cur, 1);
            read_b(Bv[1], cur, 1);
            stage_offsets_a(g, ks1);
            __builtin_amdgcn_sched_barrier(0);
            term(1);
            stage_exp_a(g, xa1);
            __builtin_amdgcn_sched_barrier(0);
            term(2);
            stage_store(g, 0, cur ^ 1);
            stage_offsets_b(g, ks1);
            __builtin_amdgcn_sched_barrier(0);
            term(3);
            stage_exp_b(g, xb1);
            __builtin_amdgcn_sched_barrier(0);
            term(4);
            stage_store(g, 1, cur ^ 1);
            __builtin_amdgcn_sched_barrier(0);
            term(5);
            __syncthreads();
        };
#pragma unroll
        for (int s = 0; s < nslices; s += 2) {
            slice(s, 0, ra[0], rb[0], ra[1], rb[1]);
            slice(s + 1, 1, ra[1], rb[1], ra[0], rb[0]);
        }
    }
    // ---- epilogue, from the registers: S -> log S in place (entries whose S underflowed are
    // recomputed by a direct log-sum-exp: a rare, non-unrolled path), the partial maxima for
    // the next level by lane reductions (each merged over the two waves that share its line
    // through LDS), and the tile stored straight from the registers: one store instruction of
    // a wave writes two rows' 128-byte segments.
    float smin = INFINITY;   // the lane's smallest sum: one compare per entry on the hot path
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int j = 0; j < BR; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) smin = fminf(smin, acc[i][j][r]);
    uint64_t under = 0;
    if (!(smin >= kUnderflow)) {
        // rare: which entries underflowed
#pragma unroll
        for (int i = 0; i < BR; ++i)
#pragma unroll
            for (int j = 0; j < BR; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (!(acc[i][j][r] >= kUnderflow)) under |= 1ull << ((i * BR + j) * 16 + r);
    }
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int j = 0; j < BR; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = flog(acc[i][j][r]);
    const int lc = lane & 31, lh = lane >> 5;
    while (under) {
        const int bit = __builtin_ctzll(under);
        under &= under - 1;
        const int ij = bit >> 4, rr = bit & 15, bi = ij / BR, bj = ij % BR;
        const int row = wm * QW + bi * 32 + (rr >> 2) * 8 + lh * 4 + (rr & 3);
        const int col = wn * QW + bj * 32 + lc;
        const int gr = a0 + row, gc = c0 + col;
        const float sr = sa[row], sc = sb[col];
        const float* lrow = Lc + (size_t)gr * C;
        // one term of the sum, with the contracted index's offsets formed as the staging
        // formed them (before the log2 e scale)
        auto fb_term = [&](int bb) {
            const float ch = Lco ? (float)(Lco[bb] - coLshift) : 0.f;
            const float rh = Rro ? (float)(Rro[bb] - roRshift) : 0.f;
            return (lrow[bb] + ch - sr) + (Rc[(size_t)bb * C + gc] + rh - sc);
        };
        float q = -INFINITY;
        for (int bb = 0; bb < C; ++bb) q = fmaxf(q, fb_term(bb));
        float val = -INFINITY;
        if (q != -INFINITY) {
            float sum = 0.f;
            for (int bb = 0; bb < C; ++bb) sum += fexp(fb_term(bb) - q);
            val = q + flog(sum);
        }
#pragma unroll
        for (int i = 0; i < BR; ++i)
#pragma unroll
            for (int j = 0; j < BR; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if ((i * BR + j) * 16 + r == bit) acc[i][j][r] = val;
    }
    // partial maxima: rows of T + co over the wave's columns, columns of T + ro over its rows
    // (lane l holds rows .. + 4 (l / 32) + (r & 3) of each group of 8 and column l % 32 of each
    // 32-wide block)
    float* rowp = smem;            // [2][TM], by column half wn (the slice buffers are free)
    float* colp = smem + 2 * TM;   // [2][TM], by row half wm
    float cofv[BR], cmx[BR];
#pragma unroll
    for (int j = 0; j < BR; ++j) {
        cofv[j] = cof[wn * QW + j * 32 + lc];
        cmx[j] = -INFINITY;
    }
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int row0 = wm * QW + i * 32 + g * 8 + lh * 4;
            const float4 ro4 = *(const float4*)(rof + row0);
            const float rov[4] = {ro4.x, ro4.y, ro4.z, ro4.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int r = 4 * g + q;
                float m = acc[i][0][r] + cofv[0];
#pragma unroll
                for (int j = 1; j < BR; ++j) m = fmaxf(m, acc[i][j][r] + cofv[j]);
                m = half_max32(m);
                if (lc == 0) rowp[wn * TM + row0 + q] = m;
#pragma unroll
                for (int j = 0; j < BR; ++j) cmx[j] = fmaxf(cmx[j], acc[i][j][r] + rov[q]);
            }
        }
#pragma unroll
    for (int j = 0; j < BR; ++j) {
        const float m = fmaxf(cmx[j], __shfl_xor(cmx[j], 32, kWave));
        if (lh == 0) colp[wm * TM + wn * QW + j * 32 + lc] = m;
    }
    // the merged maxima first (a barrier waits for the stores issued before it), then the
    // tile: a lane's 32-bit offset at its first row and column, each entry's row and block in
    // the scalar offset; nothing waits for these stores
    __syncthreads();
    if (tid < TM) {
        Pmr[(size_t)(a0 + tid) * nt + tn] = fmaxf(rowp[tid], rowp[TM + tid]);
    } else if (tid < 2 * TM) {
        const int c = tid - TM;
        Pmc[(size_t)(c0 + c) * nt + tm] = fmaxf(colp[c], colp[TM + c]);
    }
    const __amdgpu_buffer_rsrc_t rsP = make_rsrc(Pc, C * C);
    const unsigned pv = 4u * (unsigned)((a0 + wm * QW + lh * 4) * C + c0 + wn * QW + lc);
#pragma unroll
    for (int i = 0; i < BR; ++i)
#pragma unroll
        for (int j = 0; j < BR; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r)
                buffer_store1(acc[i][j][r], rsP, pv, 4 * ((i * 32 + (r >> 2) * 8 + (r & 3)) * C + j * 32));
}

// ---------------------------------------------------------------- root: log Z
struct RootArgs {
    const float* core;   // level D core, or the potentials when D == 0
    const double* ro;    // nullptr when D == 0
    const double* co;
    int64_t nodes;       // node stride per sequence at that level
    const int32_t* lengths;
    int64_t N, C;
    float* logZ;
};

// One workgroup per sequence: log Z = LSE_{i,j} (core[i][j] + ro[i] + co[j]) of the root.
// Latency, not bandwidth, bounds it (B workgroups): the first kRootThreads * kRootUnroll
// entries (all of them for C <= 128) are loaded before the offsets' maxima are reduced.
constexpr int kRootThreads = 1024, kRootUnroll = 16;

__global__ __launch_bounds__(kRootThreads) void k_root_log(RootArgs a) {
    __shared__ float red[2 * kRootThreads / kWave];
    __shared__ double redd[2 * kRootThreads / kWave];
    __shared__ float rof[kMaxLabels], cof[kMaxLabels];   // offsets less their maxima
    const int64_t b = blockIdx.x;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C, CC = C * C, tid = threadIdx.x;
    if (Eb == 0) {
        if (tid == 0) a.logZ[b] = logf((float)C);
        return;
    }
    const float* P = a.core + mat_off(b, 0, a.nodes, C);
    const double* ro = a.ro ? a.ro + (size_t)b * a.nodes * C : nullptr;
    const double* co = a.co ? a.co + (size_t)b * a.nodes * C : nullptr;
    float x[kRootUnroll];
    auto load = [&](int base) {
#pragma unroll
        for (int k = 0; k < kRootUnroll; ++k) {
            const int idx = base + k * kRootThreads;
            x[k] = idx < CC ? P[idx] : -INFINITY;
        }
    };
    load(tid);
    const double rv = (ro && tid < C) ? ro[tid] : -INFINITY;
    const double cv = (co && tid < C) ? co[tid] : -INFINITY;
    // both maxima in one reduction
    {
        const double rw = wave_max_d(rv), cw = wave_max_d(cv);
        if ((tid & (kWave - 1)) == 0) {
            redd[2 * (tid / kWave)] = rw;
            redd[2 * (tid / kWave) + 1] = cw;
        }
    }
    __syncthreads();
    double rm = redd[0], cm = redd[1];
#pragma unroll
    for (int w = 1; w < kRootThreads / kWave; ++w) {
        rm = fmax(rm, redd[2 * w]);
        cm = fmax(cm, redd[2 * w + 1]);
    }
    const double rs = ro ? safe_shift_d(rm) : 0.0;
    const double cs = co ? safe_shift_d(cm) : 0.0;
    if (tid < C) {
        rof[tid] = ro ? (float)(rv - rs) : 0.f;
        cof[tid] = co ? (float)(cv - cs) : 0.f;
    }
    __syncthreads();
    Lse acc = lse_empty();
    for (int base = tid;;) {
#pragma unroll
        for (int k = 0; k < kRootUnroll; ++k) {
            const int idx = base + k * kRootThreads;
            if (idx < CC) acc = lse_push(acc, x[k] + rof[idx / C] + cof[idx % C]);
        }
        base += kRootUnroll * kRootThreads;
        if (base >= CC) break;
        load(base);
    }
    acc = block_lse(acc, red);
    if (tid == 0) {
        const float l = lse_value(acc);
        a.logZ[b] = (l == -INFINITY) ? -INFINITY : (float)(rs + cs + (double)l);
    }
}

// ---------------------------------------------------------------- outside sweep
// For a present node N = L (x) R with outside vectors (u_N, v_N) -- u the forward
// message into its first edge, v the backward message out of its last edge:
//   u_L = u_N,  v_L = R (x) v_N,  u_R = u_N (x) L,  v_R = v_N
// (an absent right child leaves v_L = v_N).  Vectors are stored shifted to max 0.
//
// The two vector products of a node read one C x C matrix each, so a level is a stream
// over its child matrices: a workgroup of 512 threads takes one node, its first 256
// threads the column pass (u_R, one thread per column j, loads coalesced across j) and the
// other 256 the row pass (v_L, one thread per row i, 16-byte loads along the row).
constexpr int kVecThreads = 512;
constexpr int kHalfThreads = kVecThreads / 2;

// LSE_i (w[i] + M[i][j]) for one column j (w in LDS, M row-major in global memory), kU
// loads in flight per step
template <int kU = 8>
__device__ __forceinline__ float col_lse(const float* __restrict__ M, int C, const float* w, int j) {
    float m = -INFINITY, s = 0.f;
    int i = 0;
    for (; i + kU <= C; i += kU) {
        float x[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) x[u] = M[(size_t)(i + u) * C + j];
#pragma unroll
        for (int u = 0; u < kU; ++u) x[u] += w[i + u];
        lse_fold<kU>(m, s, x);
    }
    for (; i < C; ++i) {
        float x[1] = {M[(size_t)i * C + j] + w[i]};
        lse_fold<1>(m, s, x);
    }
    return lse_val(m, s);
}

// LSE_j (M[i][j] + w[j]) for one row i; kVec: 16-byte loads (C % 4 == 0), kV of them in
// flight per step
template <bool kVec, int kV = 4>
__device__ __forceinline__ float row_lse(const float* __restrict__ M, int C, const float* w, int i) {
    const float* row = M + (size_t)i * C;
    float m = -INFINITY, s = 0.f;
    int j = 0;
    if constexpr (kVec) {
        const float4* r4 = reinterpret_cast<const float4*>(row);
        for (; j + 4 * kV <= C; j += 4 * kV) {
            float4 v[kV];
#pragma unroll
            for (int u = 0; u < kV; ++u) v[u] = r4[j / 4 + u];
            float x[4 * kV];
#pragma unroll
            for (int u = 0; u < kV; ++u) {
                x[4 * u + 0] = v[u].x + w[j + 4 * u + 0];
                x[4 * u + 1] = v[u].y + w[j + 4 * u + 1];
                x[4 * u + 2] = v[u].z + w[j + 4 * u + 2];
                x[4 * u + 3] = v[u].w + w[j + 4 * u + 3];
            }
            lse_fold<4 * kV>(m, s, x);
        }
    }
    for (; j + 8 <= C; j += 8) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = row[j + u] + w[j + u];
        lse_fold<8>(m, s, x);
    }
    for (; j < C; ++j) {
        float x[1] = {row[j] + w[j]};
        lse_fold<1>(m, s, x);
    }
    return lse_val(m, s);
}

// The same two passes with each term w + M formed in float64 (M raw potentials, possibly
// large): the result keeps the terms' precision (float64 maximum plus a float32 log-sum)
__device__ __forceinline__ double col_lse_d(const float* __restrict__ M, int C, const float* w, int j) {
    double m = -INFINITY;
    float s = 0.f;
    int i = 0;
    for (; i + 8 <= C; i += 8) {
        double x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = (double)M[(size_t)(i + u) * C + j];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] += (double)w[i + u];
        lse_fold_d<8>(m, s, x);
    }
    for (; i < C; ++i) {
        const double x[1] = {(double)M[(size_t)i * C + j] + (double)w[i]};
        lse_fold_d<1>(m, s, x);
    }
    return lse_val_d(m, s);
}

template <bool kVec>
__device__ __forceinline__ double row_lse_d(const float* __restrict__ M, int C, const float* w, int i) {
    const float* row = M + (size_t)i * C;
    double m = -INFINITY;
    float s = 0.f;
    int j = 0;
    if constexpr (kVec) {
        const float4* r4 = reinterpret_cast<const float4*>(row);
        for (; j + 8 <= C; j += 8) {
            const float4 v0 = r4[j / 4], v1 = r4[j / 4 + 1];
            const double x[8] = {(double)v0.x + (double)w[j], (double)v0.y + (double)w[j + 1],
                                 (double)v0.z + (double)w[j + 2], (double)v0.w + (double)w[j + 3],
                                 (double)v1.x + (double)w[j + 4], (double)v1.y + (double)w[j + 5],
                                 (double)v1.z + (double)w[j + 6], (double)v1.w + (double)w[j + 7]};
            lse_fold_d<8>(m, s, x);
        }
    }
    for (; j < C; ++j) {
        const double x[1] = {(double)row[j] + (double)w[j]};
        lse_fold_d<1>(m, s, x);
    }
    return lse_val_d(m, s);
}

// Max of a double over the calling thread's half of the workgroup (each half gets its own
// result); red holds one double per wave.  Both halves call it together (it contains
// workgroup barriers).
__device__ __forceinline__ double half_max_d(double x, double* red) {
    x = wave_max_d(x);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[w] = x;
    __syncthreads();
    const int w0 = threadIdx.x < kHalfThreads ? 0 : kHalfThreads / kWave;
    double r = red[w0];
#pragma unroll
    for (int i = 1; i < kHalfThreads / kWave; ++i) r = fmax(r, red[w0 + i]);
    __syncthreads();
    return r;
}

// One outside-vector product per half-workgroup, both halves in step:
//   half 0: y[j] = co[j] + LSE_i (x[i] + ro[i] + core[i][j])     (x (x) N, column pass)
//   half 1: y[i] = ro[i] + LSE_j (core[i][j] + co[j] + x[j])     (N (x) x, row pass)
// x, w and y are this half's LDS vectors; the result shifted to max 0 goes to y and, when
// yraw is given, unshifted (as float) to yraw.  ro/co may be null (leaves).  Either half may
// be idle (active == false) but still joins the barriers.  With C = 32 or 64 (16-byte loads)
// every thread of the half works: the C lines are cut into P = 256 / C parts (rows
// i = p, p + P, ... of a column; a contiguous chunk of a row), whose partial log-sum-exps are
// merged through LDS.  (At C = 128, two parts per line were slower than one.)
// kExact (leaves of large magnitude in the marginals pass): the terms formed in float64
// (col_lse_d / row_lse_d).  yraw, when given, receives the unshifted result in float64.
template <bool kVec, bool kExact = false>
__device__ void half_vec(bool active, const float* core, const double* ro, const double* co,
                         int C, const float* x, float* w, float* y, double* red, double* yraw) {
    __shared__ float pm[kVecThreads], ps[kVecThreads];
    const bool rowPass = threadIdx.x >= kHalfThreads;
    const int t = threadIdx.x - (rowPass ? kHalfThreads : 0);
    const double* inOff = rowPass ? co : ro;
    const double* outOff = rowPass ? ro : co;
    // w = x + inOff, shifted to max 0 (float64 for the offsets)
    double wm = -INFINITY;
    if (active)
        for (int i = t; i < C; i += kHalfThreads) wm = fmax(wm, (double)x[i] + (inOff ? inOff[i] : 0.0));
    const double ws = safe_shift_d(half_max_d(wm, red));
    if (active)
        for (int i = t; i < C; i += kHalfThreads)
            w[i] = (float)((double)x[i] + (inOff ? inOff[i] : 0.0) - ws);
    __syncthreads();
    double z = -INFINITY;
    double l = -INFINITY;
    if (!kExact && kVec && (C == 32 || C == 64)) {
        const int P = kHalfThreads / C, p = t / C, c = t - p * C, nr = C / P;   // nr % 4 == 0
        float m = -INFINITY, sum = 0.f;
        if (active) {
            if (rowPass) {   // row c, columns [p nr, p nr + nr)
                const float4* r4 = reinterpret_cast<const float4*>(core + (size_t)c * C + p * nr);
                for (int q = 0; q < nr / 4; ++q) {
                    const float4 v = r4[q];
                    const int j = p * nr + 4 * q;
                    const float xs[4] = {v.x + w[j], v.y + w[j + 1], v.z + w[j + 2], v.w + w[j + 3]};
                    lse_fold<4>(m, sum, xs);
                }
            } else {         // column c, rows p, p + P, ...
                for (int k = 0; k < nr; k += 4) {
                    float xs[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int i = p + P * (k + u);
                        xs[u] = core[(size_t)i * C + c] + w[i];
                    }
                    lse_fold<4>(m, sum, xs);
                }
            }
        }
        pm[threadIdx.x] = m;
        ps[threadIdx.x] = sum;
        __syncthreads();
        if (active && t < C) {
            const int base = rowPass ? kHalfThreads : 0;
            float mm = -INFINITY;
            for (int q = 0; q < P; ++q) mm = fmaxf(mm, pm[base + q * C + t]);
            const float sh = safe_shift(mm);
            float ss = 0.f;
            for (int q = 0; q < P; ++q) ss += ps[base + q * C + t] * fexp(pm[base + q * C + t] - sh);
            l = lse_val(mm, ss);
        }
    } else if (active && t < C) {
        if constexpr (kExact)
            l = rowPass ? row_lse_d<kVec>(core, C, w, t) : col_lse_d(core, C, w, t);
        else
            // (C >= 128: 128 bytes in flight per thread, 32 loads down a column or eight
            // 16-byte loads along a row; still two workgroups per CU)
            l = rowPass ? (C >= 128 ? row_lse<kVec, 8>(core, C, w, t) : row_lse<kVec>(core, C, w, t))
                        : (C >= 128 ? col_lse<32>(core, C, w, t) : col_lse(core, C, w, t));
    }
    if (active && t < C) {
        z = (l == -INFINITY) ? -INFINITY : (outOff ? outOff[t] : 0.0) + ws + l;
        if (yraw) yraw[t] = z;
    }
    const double zs = safe_shift_d(half_max_d(z, red));
    if (active && t < C) y[t] = (z == -INFINITY) ? -INFINITY : (float)(z - zs);
    __syncthreads();
}

struct DownArgs {
    const float* uN;       // level l vectors (nullptr at the root: zeros)
    const float* vN;
    int64_t nodes;         // nodes per sequence at level l
    const float* ccore;    // children (level l-1 >= 1)
    const double* cro;
    const double* cco;
    int64_t cnodes;
    float* uC;             // child vectors (level l-1)
    float* vC;
    const int32_t* lengths;
    int64_t N, C;
    int level;
};

template <bool kVec>
__global__ __launch_bounds__(kVecThreads) void k_down_log(DownArgs a) {
    __shared__ float sx[2][kMaxLabels], sw[2][kMaxLabels], sy[2][kMaxLabels];
    __shared__ double red[kVecThreads / kWave];
    const int64_t b = blockIdx.x / a.nodes, k = blockIdx.x % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;
    const int64_t kl = 2 * k, kr = 2 * k + 1;
    const bool right = kr * half < Eb;
    const size_t nvec = (size_t)(b * a.nodes + k) * C;
    float* uL = a.uC + (size_t)(b * a.cnodes + kl) * C;
    float* vL = a.vC + (size_t)(b * a.cnodes + kl) * C;
    float* uR = a.uC + (size_t)(b * a.cnodes + kr) * C;
    float* vR = a.vC + (size_t)(b * a.cnodes + kr) * C;
    // u_L = u_N; v_R = v_N (or v_L = v_N without a right child)
    for (int i = threadIdx.x; i < C; i += kVecThreads) {
        const float u = a.uN ? a.uN[nvec + i] : 0.f, v = a.vN ? a.vN[nvec + i] : 0.f;
        uL[i] = u;
        (right ? vR : vL)[i] = v;
        sx[0][i] = u;
        sx[1][i] = v;
    }
    if (!right) return;
    __syncthreads();
    const bool rowPass = threadIdx.x >= kHalfThreads;
    const int64_t child = b * a.cnodes + (rowPass ? kr : kl);
    const float* core = a.ccore + (size_t)child * C * C;
    half_vec<kVec>(true, core, a.cro + (size_t)child * C, a.cco + (size_t)child * C, C,
                   sx[rowPass], sw[rowPass], sy[rowPass], red, nullptr);
    float* dst = rowPass ? vL : uR;
    const int t = threadIdx.x - (rowPass ? kHalfThreads : 0);
    for (int i = t; i < C; i += kHalfThreads) dst[i] = sy[rowPass][i];
}

// ---------------------------------------------------------------- marginals
// One workgroup per level-1 node (edges 2k and 2k+1), with the node's outside vectors
// (u, v): alpha_{2k} = u, beta_{2k+2} = v, and the two messages inside the pair come from
// one column pass and one row pass over the two leaves, run side by side:
//   y = u (x) leaf_{2k}   (alpha_{2k+1} = y shifted),   z = leaf_{2k+1} (x) v   (beta_{2k+1}).
// Each edge's marginal uses its own normaliser n_t = LSE_{i,j} (alpha_t[i] + l_t[i][j] +
// beta_{t+1}[j]), which is a vector log-sum-exp of the same products:
//   n_{2k} = LSE_j (y[j] + beta_{2k+1}[j]),   n_{2k+1} = LSE_i (alpha_{2k+1}[i] + z[i]),
//   mu_t[i][j] = exp(alpha_t[i] + l_t[i][j] + beta_{t+1}[j] - n_t)
// (exact: alpha_t, beta_{t+1} are the true messages up to constants, and log Z = const +
// n_t for every edge t).  The leaves are then streamed once more, 16 bytes per access.
struct FormArgs {
    const float* pot;
    const float* u1;   // level-1 vectors, nullptr when level 1 is the root (D <= 1)
    const float* v1;
    int64_t nodes1;    // nodes per sequence at level 1 (Np / 2, or 1 when D == 0)
    const int32_t* lengths;
    int64_t N, C;
    float* marg;
    const int32_t* wide;   // per edge: potentials reach kWideMag (nullptr: every edge)
};

// Whether the pair (tL, tR) of sequence b takes the float64 formation: kernels are launched
// once per formation, and a workgroup returns at once when its pair belongs to the other.
__device__ __forceinline__ bool pair_wide(const FormArgs& a, int64_t b, int64_t E, int64_t tL,
                                          bool right) {
    if (!a.wide) return true;
    return a.wide[b * E + tL] != 0 || (right && a.wide[b * E + tL + 1] != 0);
}

// The same per-pair computation with each leaf read from memory once (C <= 128, C % 4 == 0):
// the workgroup keeps both leaves in registers, in the layout write_marginal uses (thread t
// holds columns 4 (t % G) .. +3 of rows t / G + q * step, q < kR), and forms
//   y = u (x) leaf_{2k}: partial column log-sum-exps over the thread's rows, merged in LDS
//   over the `step` threads of a column group;
//   z = leaf_{2k+1} (x) v: partial row log-sum-exps over the thread's 4 columns, merged in
//   LDS over the G threads of a row;
// then the normalisers and the marginals from the registers (the second read of each leaf
// in k_form_log is gone: one read and one write per edge, the algorithmic traffic).
constexpr int kRegMaxLabels = 128;

// (m, s) += (m2, s2) for log-sum-exp states value = m + log s (m = -inf: empty)
__device__ __forceinline__ void lse_merge_into(float& m, float& s, float m2, float s2) {
    if (m2 == -INFINITY) return;
    if (m == -INFINITY) { m = m2; s = s2; return; }
    const float nm = fmaxf(m, m2);
    s = s * fexp(m - nm) + s2 * fexp(m2 - nm);
    m = nm;
}

// A state with a float64 maximum as a float32 state of the same value: m rounded to float,
// the rounding folded into s (a relative change below 2^-24).  Merging such states in float
// stays exact where it matters: maxima within a factor 2 subtract exactly, and farther ones
// weigh in by a negligible exponential.
__device__ __forceinline__ void lse_to_float(double m, float s, float& mf, float& sf) {
    if (m == -INFINITY) {
        mf = -INFINITY;
        sf = 0.f;
        return;
    }
    mf = (float)m;
    sf = s * fexp((float)(m - (double)mf));
}
__device__ __forceinline__ void lse_to_float(float m, float s, float& mf, float& sf) {
    mf = m;
    sf = s;
}

template <int kR, bool kExact>
__global__ __launch_bounds__(kVecThreads) void k_form_reg(FormArgs a) {
    using Tm = std::conditional_t<kExact, double, float>;   // type of the formed terms
    // column partials [step][C] (step * C <= 4 kVecThreads) and row partials [C][G]
    constexpr int kMaxC = kR == 2 ? 64 : kRegMaxLabels;   // kR = 2 serves C <= 64
    constexpr int kColParts = 4 * kVecThreads, kRowParts = kMaxC * kMaxC / 4;
    __shared__ float su[kRegMaxLabels], sv[kRegMaxLabels], ya[kRegMaxLabels], zb[kRegMaxLabels];
    __shared__ double yraw[kRegMaxLabels], zraw[kRegMaxLabels];
    __shared__ float pm[kColParts], ps[kColParts], qm[kRowParts], qs[kRowParts];
    __shared__ double nrm[2];
    const int64_t npairs = (a.N - 1 + 1) / 2;
    const int64_t b = blockIdx.x / npairs, k = blockIdx.x % npairs;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C;
    const int64_t E = a.N - 1;
    const int64_t tL = 2 * k, tR = 2 * k + 1;
    const size_t CC = (size_t)C * C;
    const int tid = threadIdx.x;
    if (!kExact)   // (padding edges once, by the float32 formation's launch)
        for (int64_t t = tL; t <= tR; ++t)
            if (t < E && t >= Eb) {
                float* o = a.marg + (size_t)(b * E + t) * CC;
                for (size_t idx = tid; idx < CC; idx += kVecThreads) o[idx] = 0.f;
            }
    if (tL >= Eb) return;
    const bool right = tR < Eb;
    if (pair_wide(a, b, E, tL, right) != kExact) return;
    const int G = C / 4, step = kVecThreads / G;
    const int g = tid % G, i0 = tid / G, j = 4 * g;
    const bool act = i0 < step;
    // both leaves into registers first (every load in flight together)
    const float* leafL = a.pot + (size_t)(b * E + tL) * CC;
    const float* leafR = a.pot + (size_t)(b * E + tR) * CC;
    float4 lv[kR], rv[kR];
#pragma unroll
    for (int q = 0; q < kR; ++q) {
        const int i = i0 + q * step;
        const bool ok = act && i < C;
        lv[q] = ok ? *reinterpret_cast<const float4*>(leafL + (size_t)i * C + j) : make_float4(0.f, 0.f, 0.f, 0.f);
        rv[q] = ok && right ? *reinterpret_cast<const float4*>(leafR + (size_t)i * C + j)
                            : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    for (int i = tid; i < C; i += kVecThreads) {
        su[i] = a.u1 ? a.u1[(size_t)(b * a.nodes1 + k) * C + i] : 0.f;
        sv[i] = a.v1 ? a.v1[(size_t)(b * a.nodes1 + k) * C + i] : 0.f;
    }
    __syncthreads();
    // partial log-sum-exps: columns j..j+3 of leaf_{2k} over the thread's rows (with u), and
    // each of the thread's rows of leaf_{2k+1} over its 4 columns (with v).  A term adds a raw
    // potential to a message entry; with kExact (potentials of large magnitude) it is formed
    // in float64 and rounded only after the maximum is taken off (here, in the normalisers
    // and in the marginals' exponents alike), so that float32 rounding at the potentials'
    // magnitude never enters.  (The normalisers are formed in float64 either way.)
    if (act) {
        const Tm v0 = sv[j], v1 = sv[j + 1], v2 = sv[j + 2], v3 = sv[j + 3];
        Tm xc[4][kR];   // u[i] + l_{2k}[i][j + c] of the thread's rows (-inf past C)
#pragma unroll
        for (int q = 0; q < kR; ++q) {
            const int i = i0 + q * step;
            const bool ok = i < C;
            const Tm ui = ok ? (Tm)su[i] : (Tm)-INFINITY;
            xc[0][q] = ui + (Tm)lv[q].x;
            xc[1][q] = ui + (Tm)lv[q].y;
            xc[2][q] = ui + (Tm)lv[q].z;
            xc[3][q] = ui + (Tm)lv[q].w;
            if (right && ok) {
                const Tm r[4] = {(Tm)rv[q].x + v0, (Tm)rv[q].y + v1, (Tm)rv[q].z + v2, (Tm)rv[q].w + v3};
                Tm m = -INFINITY;
                float sr = 0.f;
                lse_fold_t<4>(m, sr, r);
                lse_to_float(m, sr, qm[i * G + g], qs[i * G + g]);
            }
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            Tm m = -INFINITY;
            float sm = 0.f;
            lse_fold_t<kR>(m, sm, xc[c]);
            lse_to_float(m, sm, pm[i0 * C + j + c], ps[i0 * C + j + c]);
        }
    }
    __syncthreads();
    // merged: yraw[j] = LSE_i u[i] + l_{2k}[i][j],  zraw[i] = LSE_j l_{2k+1}[i][j] + v[j]
    if (tid < C) {
        float m = -INFINITY, sm = 0.f;
        for (int r = 0; r < step; ++r) lse_merge_into(m, sm, pm[r * C + tid], ps[r * C + tid]);
        yraw[tid] = lse_val_d(m, sm);
    } else if (right && tid >= kVecThreads / 2 && tid - kVecThreads / 2 < C) {
        const int i = tid - kVecThreads / 2;
        float m = -INFINITY, sm = 0.f;
        for (int r = 0; r < G; ++r) lse_merge_into(m, sm, qm[i * G + r], qs[i * G + r]);
        zraw[i] = lse_val_d(m, sm);
    }
    __syncthreads();
    // the messages shifted to max 0 (wave 0: alpha_{2k+1} from y, wave 1: beta_{2k+1} from z)
    const int w = tid / kWave, lane = tid % kWave;
    if (w < 2 && (w == 0 || right)) {
        const double* src = w == 0 ? yraw : zraw;
        double m = -INFINITY;
        for (int i = lane; i < C; i += kWave) m = fmax(m, src[i]);
        m = safe_shift_d(wave_max_d(m));
        float* dst = w == 0 ? ya : zb;
        for (int i = lane; i < C; i += kWave) dst[i] = (float)(src[i] - m);
    }
    __syncthreads();
    // normalisers: n_{2k} = LSE_j yraw[j] + beta_{2k+1}[j] (or + v[j] without a right edge),
    // n_{2k+1} = LSE_i alpha_{2k+1}[i] + zraw[i]
    if (w < 2 && (w == 0 || right)) {
        double m = -INFINITY;
        float sm = 0.f;
        for (int i = lane; i < C; i += kWave) {
            const double x[1] = {w == 0 ? yraw[i] + (double)(right ? zb[i] : sv[i]) : (double)ya[i] + zraw[i]};
            lse_fold_d<1>(m, sm, x);
        }
        const double mm = wave_max_d(m);
        sm = wave_sum(m == -INFINITY ? 0.f : sm * fexp((float)(m - safe_shift_d(mm))));
        if (lane == 0) nrm[w] = lse_val_d(mm, sm);
    }
    __syncthreads();
    if (!act) return;
    // the marginals from the registers (exponents formed in Tm)
    auto write = [&](const float4* lvq, const float* al, const float* be, double n, float* out) {
        const bool zero = n == -INFINITY;
        const Tm b0 = be[j], b1 = be[j + 1], b2 = be[j + 2], b3 = be[j + 3];
#pragma unroll
        for (int q = 0; q < kR; ++q) {
            const int i = i0 + q * step;
            if (i < C) {
                const Tm an = (Tm)((double)al[i] - n);
                float4 r;
                r.x = zero ? 0.f : fexp((float)(((Tm)lvq[q].x + b0) + an));
                r.y = zero ? 0.f : fexp((float)(((Tm)lvq[q].y + b1) + an));
                r.z = zero ? 0.f : fexp((float)(((Tm)lvq[q].z + b2) + an));
                r.w = zero ? 0.f : fexp((float)(((Tm)lvq[q].w + b3) + an));
                *reinterpret_cast<float4*>(out + (size_t)i * C + j) = r;
            }
        }
    };
    write(lv, su, right ? zb : sv, nrm[0], a.marg + (size_t)(b * E + tL) * CC);
    if (right) write(rv, ya, sv, nrm[1], a.marg + (size_t)(b * E + tR) * CC);
}

// The per-pair computation for C = 256, where two leaves do not fit a workgroup's registers:
// the left leaf is held in registers (1024 threads, 64 values each) and read once, the right
// one is streamed for its row pass and again for its marginals, except the rows kept in LDS
// from the first read: 1.28 reads per edge instead of 2.  Thread t = 64 w + g holds columns
// 4g .. 4g+3 of rows w + 16 q (q < 16), so
// each row of a leaf is one wave's contiguous 1 KiB: the row pass of the right leaf reduces
// within a wave, the column pass of the left leaf merges the 16 waves' states through LDS.
constexpr int kBigLabels = 256;
constexpr int kBigThreads = 1024;
// rows of the right leaf each wave keeps in LDS from its first read (of the 16 it handles):
// the second read takes them from there (7 of 16 rows: 112 KB beside the kernel's 40 KB of
// static LDS, one workgroup per CU as its registers already allow)
constexpr int kBigKeep = 7;
constexpr size_t kBigKeepBytes = sizeof(float4) * kBigKeep * (kBigThreads / kWave) * kWave;

// (m, s) += (m2, s2) for log-sum-exp states; value = m + log s, m = -inf: empty
template <typename Tm>
__device__ __forceinline__ void lse_merge_state(Tm& m, float& s, Tm m2, float s2) {
    const Tm nm = m > m2 ? m : m2;
    if (nm != (Tm)-INFINITY) {
        s = (m == (Tm)-INFINITY ? 0.f : s * fexp((float)(m - nm))) +
            (m2 == (Tm)-INFINITY ? 0.f : s2 * fexp((float)(m2 - nm)));
        m = nm;
    }
}

// (m, s) merged over the 64 lanes of a wave
template <typename Tm>
__device__ __forceinline__ void wave_lse_state(Tm& m, float& s) {
#pragma unroll
    for (int off = kWave / 2; off >= 1; off >>= 1)
        lse_merge_state(m, s, __shfl_xor(m, off, kWave), __shfl_xor(s, off, kWave));
}

// Four rows' states, each spread over the 64 lanes of a wave ((m[q], s[q]) for row q in every
// lane), merged over the wave: lane l ends with row 2 b5 + b4 (b5, b4: bits 5 and 4 of l).  A
// reduce-scatter over lane bits 5 and 4 (each lane sends the rows it gives up and keeps the
// others), then a full reduction over bits 3 .. 0: seven exchanges instead of the 24 of four
// separate wave reductions.
template <typename Tm>
__device__ __forceinline__ int wave_lse_rows4(const Tm (&m)[4], const float (&s)[4], Tm& mo, float& so) {
    const int lane = threadIdx.x & (kWave - 1);
    const bool b5 = (lane & 32) != 0, b4 = (lane & 16) != 0;
    Tm km[2];
    float ks[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {   // bit 5: keep rows {0, 1} (b5 = 0) or {2, 3}
        km[u] = b5 ? m[u + 2] : m[u];
        ks[u] = b5 ? s[u + 2] : s[u];
        const Tm sm = b5 ? m[u] : m[u + 2];
        const float ss = b5 ? s[u] : s[u + 2];
        lse_merge_state(km[u], ks[u], __shfl_xor(sm, 32, kWave), __shfl_xor(ss, 32, kWave));
    }
    mo = b4 ? km[1] : km[0];   // bit 4: keep the first (b4 = 0) or the second
    so = b4 ? ks[1] : ks[0];
    lse_merge_state(mo, so, __shfl_xor(b4 ? km[0] : km[1], 16, kWave),
                    __shfl_xor(b4 ? ks[0] : ks[1], 16, kWave));
#pragma unroll
    for (int off = 8; off >= 1; off >>= 1)
        lse_merge_state(mo, so, __shfl_xor(mo, off, kWave), __shfl_xor(so, off, kWave));
    return 2 * (int)b5 + (int)b4;
}

template <bool kExact>
__global__ __launch_bounds__(kBigThreads) void k_form_big(FormArgs a) {
    using Tm = std::conditional_t<kExact, double, float>;   // type of the formed terms
    constexpr int C = kBigLabels, G = C / 4, kW = kBigThreads / kWave, kR = C / kW;
    static_assert(G == kWave && kR * kW == C, "a row is one wave's 64 float4");
    __shared__ float su[C], sv[C], ya[C], zb[C];
    __shared__ double yraw[C], zraw[C];
    __shared__ float pm[kW][C], ps[kW][C];
    __shared__ double nrm[2];
    extern __shared__ __align__(16) float4 rkeep[];   // [kBigKeep][kW][64]: right-leaf rows
    const int64_t npairs = (a.N - 1 + 1) / 2;
    const int64_t b = blockIdx.x / npairs, k = blockIdx.x % npairs;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t E = a.N - 1;
    const int64_t tL = 2 * k, tR = 2 * k + 1;
    const size_t CC = (size_t)C * C;
    const int tid = threadIdx.x, w = tid / kWave, g = tid % kWave, j = 4 * g;
    if (!kExact)   // (padding edges once, by the float32 formation's launch)
        for (int64_t t = tL; t <= tR; ++t)
            if (t < E && t >= Eb) {
                float4* o = reinterpret_cast<float4*>(a.marg + (size_t)(b * E + t) * CC);
                for (int idx = tid; idx < C * G; idx += kBigThreads) o[idx] = make_float4(0.f, 0.f, 0.f, 0.f);
            }
    if (tL >= Eb) return;
    const bool right = tR < Eb;
    if (pair_wide(a, b, E, tL, right) != kExact) return;
    // raw buffer accesses: one 32-bit offset per thread (row w, column j), the row step
    // 16 q in a scalar offset, so that no per-row address is kept in registers
    const __amdgpu_buffer_rsrc_t rsL = make_rsrc(a.pot + (size_t)(b * E + tL) * CC, C * C);
    const __amdgpu_buffer_rsrc_t rsR = make_rsrc(a.pot + (size_t)(b * E + (right ? tR : tL)) * CC, C * C);
    const unsigned voff = 4u * (unsigned)(w * C + j);
    constexpr int kRowStep = 4 * kW * C;   // bytes between a thread's rows
    float4 lv[kR];
#pragma unroll
    for (int q = 0; q < kR; ++q) lv[q] = buffer_load4(rsL, voff, kRowStep * q);
    if (tid < C) {
        su[tid] = a.u1 ? a.u1[(size_t)(b * a.nodes1 + k) * C + tid] : 0.f;
        sv[tid] = a.v1 ? a.v1[(size_t)(b * a.nodes1 + k) * C + tid] : 0.f;
    }
    __syncthreads();
    // column pass of the left leaf: the thread's partial log-sum-exps of u[i] + l[i][j + c]
    // over its 16 rows, four rows at a time straight from the registers, merged below over
    // the 16 waves
    {
        Tm m[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        float sc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int q0 = 0; q0 < kR; q0 += 4) {
            Tm ui[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) ui[u] = su[w + kW * (q0 + u)];
            const Tm x0[4] = {ui[0] + (Tm)lv[q0].x, ui[1] + (Tm)lv[q0 + 1].x, ui[2] + (Tm)lv[q0 + 2].x, ui[3] + (Tm)lv[q0 + 3].x};
            const Tm x1[4] = {ui[0] + (Tm)lv[q0].y, ui[1] + (Tm)lv[q0 + 1].y, ui[2] + (Tm)lv[q0 + 2].y, ui[3] + (Tm)lv[q0 + 3].y};
            const Tm x2[4] = {ui[0] + (Tm)lv[q0].z, ui[1] + (Tm)lv[q0 + 1].z, ui[2] + (Tm)lv[q0 + 2].z, ui[3] + (Tm)lv[q0 + 3].z};
            const Tm x3[4] = {ui[0] + (Tm)lv[q0].w, ui[1] + (Tm)lv[q0 + 1].w, ui[2] + (Tm)lv[q0 + 2].w, ui[3] + (Tm)lv[q0 + 3].w};
            lse_fold_t<4>(m[0], sc[0], x0);
            lse_fold_t<4>(m[1], sc[1], x1);
            lse_fold_t<4>(m[2], sc[2], x2);
            lse_fold_t<4>(m[3], sc[3], x3);
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) lse_to_float(m[c], sc[c], pm[w][j + c], ps[w][j + c]);
    }
    // row pass of the right leaf (first read): z[i] = LSE_j r[i][j] + v[j], one wave per row,
    // four rows at a time merged over the wave together
    if (right) {
        const Tm v0 = sv[j], v1 = sv[j + 1], v2 = sv[j + 2], v3 = sv[j + 3];
        constexpr int kChunk = 4;   // rows of a wave in flight together
#pragma unroll
        for (int q0 = 0; q0 < kR; q0 += kChunk) {
            float4 rv[kChunk];
#pragma unroll
            for (int q = 0; q < kChunk; ++q) rv[q] = buffer_load4(rsR, voff, kRowStep * (q0 + q));
#pragma unroll
            for (int q = 0; q < kChunk; ++q)
                if (q0 + q < kBigKeep) rkeep[((q0 + q) * kW + w) * kWave + g] = rv[q];
            Tm m[kChunk];
            float sm[kChunk];
#pragma unroll
            for (int q = 0; q < kChunk; ++q) {
                const Tm r[4] = {(Tm)rv[q].x + v0, (Tm)rv[q].y + v1, (Tm)rv[q].z + v2, (Tm)rv[q].w + v3};
                m[q] = -INFINITY;
                sm[q] = 0.f;
                lse_fold_t<4>(m[q], sm[q], r);
            }
            Tm mo;
            float so;
            const int q = wave_lse_rows4(m, sm, mo, so);
            if ((g & 15) == 0)
                zraw[w + kW * (q0 + q)] = mo == (Tm)-INFINITY ? -INFINITY : (double)mo + (double)flog(so);
        }
    }
    __syncthreads();
    // merged: yraw[j] = LSE_i u[i] + l_{2k}[i][j]
    if (tid < C) {
        float m = -INFINITY, sm = 0.f;
#pragma unroll
        for (int r = 0; r < kW; ++r) lse_merge_into(m, sm, pm[r][tid], ps[r][tid]);
        yraw[tid] = lse_val_d(m, sm);
    }
    __syncthreads();
    // the messages shifted to max 0 (wave 0: alpha_{2k+1} from y, wave 1: beta_{2k+1} from z)
    if (w < 2 && (w == 0 || right)) {
        const double* src = w == 0 ? yraw : zraw;
        double m = -INFINITY;
        for (int i = g; i < C; i += kWave) m = fmax(m, src[i]);
        m = safe_shift_d(wave_max_d(m));
        float* dst = w == 0 ? ya : zb;
        for (int i = g; i < C; i += kWave) dst[i] = (float)(src[i] - m);
    }
    __syncthreads();
    // normalisers: n_{2k} = LSE_j yraw[j] + beta_{2k+1}[j] (or + v[j] without a right edge),
    // n_{2k+1} = LSE_i alpha_{2k+1}[i] + zraw[i]
    if (w < 2 && (w == 0 || right)) {
        double m = -INFINITY;
        float sm = 0.f;
        for (int i = g; i < C; i += kWave) {
            const double x[1] = {w == 0 ? yraw[i] + (double)(right ? zb[i] : sv[i]) : (double)ya[i] + zraw[i]};
            lse_fold_d<1>(m, sm, x);
        }
        const double mm = wave_max_d(m);
        sm = wave_sum(m == -INFINITY ? 0.f : sm * fexp((float)(m - safe_shift_d(mm))));
        if (g == 0) nrm[w] = lse_val_d(mm, sm);
    }
    __syncthreads();
    // the marginals: the left leaf from the registers, the right one streamed again
    auto emit = [&](const float4& x, const float* be, double n, double al) {
        if (n == -INFINITY) return make_float4(0.f, 0.f, 0.f, 0.f);
        const Tm an = (Tm)(al - n);
        float4 r;
        r.x = fexp((float)(((Tm)x.x + (Tm)be[j]) + an));
        r.y = fexp((float)(((Tm)x.y + (Tm)be[j + 1]) + an));
        r.z = fexp((float)(((Tm)x.z + (Tm)be[j + 2]) + an));
        r.w = fexp((float)(((Tm)x.w + (Tm)be[j + 3]) + an));
        return r;
    };
    {
        const __amdgpu_buffer_rsrc_t rsO = make_rsrc(a.marg + (size_t)(b * E + tL) * CC, C * C);
        const double n = nrm[0];
        const float* be = right ? zb : sv;
#pragma unroll
        for (int q = 0; q < kR; ++q)
            buffer_store4(emit(lv[q], be, n, (double)su[w + kW * q]), rsO, voff, kRowStep * q);
    }
    if (right) {
        const __amdgpu_buffer_rsrc_t rsO = make_rsrc(a.marg + (size_t)(b * E + tR) * CC, C * C);
        const double n = nrm[1];
        constexpr int kChunk = 4;
#pragma unroll
        for (int q0 = 0; q0 < kR; q0 += kChunk) {
            float4 rv[kChunk];
#pragma unroll
            for (int q = 0; q < kChunk; ++q)   // (the kept rows from LDS; each thread reads its own)
                rv[q] = q0 + q < kBigKeep ? rkeep[((q0 + q) * kW + w) * kWave + g]
                                          : buffer_load4(rsR, voff, kRowStep * (q0 + q));
#pragma unroll
            for (int q = 0; q < kChunk; ++q)
                buffer_store4(emit(rv[q], sv, n, (double)ya[w + kW * (q0 + q)]), rsO, voff,
                              kRowStep * (q0 + q));
        }
    }
}

// mu = exp(al[i] + leaf[i][j] + be[j] - n) over one C x C edge, the whole workgroup:
// thread t takes column group t % G (16 bytes when kVec, else one float) of rows t / G,
// t / G + T / G, ... so that each row is read and written contiguously
// (kExact: the exponent al[i] + leaf[i][j] + be[j] - n formed in float64, rounded once)
template <bool kVec, bool kExact>
__device__ void write_marginal(const float* __restrict__ leaf, const float* al, const float* be,
                               double n, int C, float* __restrict__ out) {
    using Tm = std::conditional_t<kExact, double, float>;
    constexpr int kW = kVec ? 4 : 1;
    const int G = C / kW, step = kVecThreads / G;
    const int g = threadIdx.x % G, i0 = threadIdx.x / G;
    if (i0 >= step) return;
    const int j = g * kW;
    Tm bj[kW];
#pragma unroll
    for (int q = 0; q < kW; ++q) bj[q] = be[j + q];
    const bool zero = n == -INFINITY;
#pragma unroll 4
    for (int i = i0; i < C; i += step) {
        const Tm an = (Tm)((double)al[i] - n);
        if constexpr (kVec) {
            const float4 v = *reinterpret_cast<const float4*>(leaf + (size_t)i * C + j);
            float4 r;
            r.x = zero ? 0.f : fexp((float)(((Tm)v.x + bj[0]) + an));
            r.y = zero ? 0.f : fexp((float)(((Tm)v.y + bj[1]) + an));
            r.z = zero ? 0.f : fexp((float)(((Tm)v.z + bj[2]) + an));
            r.w = zero ? 0.f : fexp((float)(((Tm)v.w + bj[3]) + an));
            *reinterpret_cast<float4*>(out + (size_t)i * C + j) = r;
        } else {
            const float v = leaf[(size_t)i * C + j];
            out[(size_t)i * C + j] = zero ? 0.f : fexp((float)(((Tm)v + bj[0]) + an));
        }
    }
}

template <bool kVec, bool kExact>
__global__ __launch_bounds__(kVecThreads) void k_form_log(FormArgs a) {
    __shared__ float su[kMaxLabels], sv[kMaxLabels], sy[2][kMaxLabels], sw[2][kMaxLabels];
    __shared__ double raw[2][kMaxLabels];
    __shared__ double red[kVecThreads / kWave];
    __shared__ double nrm[2];
    const int64_t npairs = (a.N - 1 + 1) / 2;
    const int64_t b = blockIdx.x / npairs, k = blockIdx.x % npairs;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C;
    const int64_t E = a.N - 1;
    const int64_t tL = 2 * k, tR = 2 * k + 1;
    const size_t CC = (size_t)C * C;
    // padding edges are exactly zero (written by the float32 formation's launch)
    if (!kExact)
        for (int64_t t = tL; t <= tR; ++t)
            if (t < E && t >= Eb) {
                float* o = a.marg + (size_t)(b * E + t) * CC;
                for (size_t idx = threadIdx.x; idx < CC; idx += kVecThreads) o[idx] = 0.f;
            }
    if (tL >= Eb) return;
    if (pair_wide(a, b, E, tL, tR < Eb) != kExact) return;
    for (int i = threadIdx.x; i < C; i += kVecThreads) {
        su[i] = a.u1 ? a.u1[(size_t)(b * a.nodes1 + k) * C + i] : 0.f;
        sv[i] = a.v1 ? a.v1[(size_t)(b * a.nodes1 + k) * C + i] : 0.f;
    }
    __syncthreads();
    const float* leafL = a.pot + (size_t)(b * E + tL) * CC;
    float* outL = a.marg + (size_t)(b * E + tL) * CC;
    const bool right = tR < Eb;
    if (!right) {
        // a lone edge: n = LSE_{i,j} (u[i] + l[i][j] + v[j]) = LSE_j (y[j] + v[j]), y = u (x) leaf
        // (column pass only; the row half idles through the barriers)
        half_vec<kVec, kExact>(threadIdx.x < kHalfThreads, leafL, nullptr, nullptr, C, su, sw[0],
                               sy[0], red, raw[0]);
        if (threadIdx.x < kWave) {
            double m = -INFINITY;
            float s = 0.f;
            for (int j = threadIdx.x; j < C; j += kWave) {
                const double x[1] = {raw[0][j] + (double)sv[j]};
                lse_fold_d<1>(m, s, x);
            }
            const double mm = wave_max_d(m);
            s = wave_sum(m == -INFINITY ? 0.f : s * fexp((float)(m - safe_shift_d(mm))));
            if (threadIdx.x == 0) nrm[0] = lse_val_d(mm, s);
        }
        __syncthreads();
        write_marginal<kVec, kExact>(leafL, su, sv, nrm[0], C, outL);
        return;
    }
    const float* leafR = a.pot + (size_t)(b * E + tR) * CC;
    float* outR = a.marg + (size_t)(b * E + tR) * CC;
    // half 0: y = u (x) leaf_{2k} -> alpha_{2k+1} (sy[0]);  half 1: z = leaf_{2k+1} (x) v ->
    // beta_{2k+1} (sy[1]); raw[] keep the unshifted log-sum-exps
    const bool rowPass = threadIdx.x >= kHalfThreads;
    half_vec<kVec, kExact>(true, rowPass ? leafR : leafL, nullptr, nullptr, C, rowPass ? sv : su,
                           sw[rowPass], sy[rowPass], red, raw[rowPass]);
    // n_{2k} = LSE_j (y[j] + beta_{2k+1}[j]) (wave 0);  n_{2k+1} = LSE_i (alpha_{2k+1}[i] + z[i]) (wave 1)
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    if (w < 2) {
        double m = -INFINITY;
        float s = 0.f;
        for (int j = lane; j < C; j += kWave) {
            const double x[1] = {w == 0 ? raw[0][j] + (double)sy[1][j] : (double)sy[0][j] + raw[1][j]};
            lse_fold_d<1>(m, s, x);
        }
        const double mm = wave_max_d(m);
        s = wave_sum(m == -INFINITY ? 0.f : s * fexp((float)(m - safe_shift_d(mm))));
        if (lane == 0) nrm[w] = lse_val_d(mm, s);
    }
    __syncthreads();
    write_marginal<kVec, kExact>(leafL, su, sy[1], nrm[0], C, outL);
    write_marginal<kVec, kExact>(leafR, sy[0], sv, nrm[1], C, outR);
}

template <int TM, bool VEC, bool kBits>
hipError_t allow_up_lds() {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)k_up_log<TM, VEC, kBits>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)UpSmem<TM>::kBytes);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    return hipSuccess;
}

template <bool kExact>
hipError_t allow_form_big_lds() {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)k_form_big<kExact>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)kBigKeepBytes);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    return hipSuccess;
}

template <bool VEC>
hipError_t allow_leaf_lds() {
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute(
            (const void*)k_leaf_max_lds<VEC>, hipFuncAttributeMaxDynamicSharedMemorySize,
            (int)(sizeof(float) * kLeafLdsMaxLabels * (kLeafLdsMaxLabels + 1)));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    return hipSuccess;
}

template <int TM, bool kBf, int kNS = 0>
hipError_t allow_up_full_lds() {
    static bool attr_set = false;
    if (!attr_set) {
        using Sm = std::conditional_t<kBf, UpBfSmem<TM>, UpFullSmem<TM>>;
        hipError_t e = hipFuncSetAttribute((const void*)k_up_log_full<TM, kBf, kNS>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)Sm::kBytes);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    return hipSuccess;
}

template <bool VEC, bool kBits>
hipError_t up_sweep_vec(const Plan& p, const float* pot, const int32_t* lengths, hipStream_t s) {
    hipError_t e = allow_up_lds<64, VEC, kBits>();
    if (e == hipSuccess && p.C > 64) e = allow_up_lds<128, VEC, kBits>();
    // full tiles (every tile edge divides C; dense chains): the scheduled kernel
    const bool full64 = !kBits && p.C % 64 == 0, full128 = !kBits && p.C % 128 == 0;
    if (e == hipSuccess && full64) e = allow_up_full_lds<64, false>();
    // (C <= kMaxLabels = 256, so full 128-wide tiles mean C = 128 or 256: 8 or 16 slices)
    static_assert(kMaxLabels <= 256, "the bf16 product is instantiated for C = 128 and 256");
    if (e == hipSuccess && full128) {
        if constexpr (kUpBf16)
            e = p.C == 128 ? allow_up_full_lds<128, true, 8>() : allow_up_full_lds<128, true, 16>();
        else
            e = allow_up_full_lds<128, false>();
    }
    if (e != hipSuccess) return e;
    // the leaves' row and column maxima (shifts of the level-1 products)
    LeafMaxArgs m{pot, lengths, p.N, p.C, p.lrmax, p.lcmax, p.rbits[0], p.cbits[0], p.bw, p.wide};
    // (the LDS-staged kernel for short batches, whose few workgroups are bound by memory
    // latency; with many edges the streaming kernel keeps more bytes in flight per CU)
    if (!kBits && p.C <= kLeafLdsMaxLabels && p.B * p.E <= kLeafLdsMaxEdges) {
        const size_t lds = sizeof(float) * p.C * (p.C + 1);
        e = allow_leaf_lds<VEC>();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((k_leaf_max_lds<VEC>), dim3((unsigned)(p.B * p.E)),
                           dim3(kLeafLdsThreads), lds, s, m);
    } else {
        hipLaunchKernelGGL((k_leaf_max<VEC, kBits>), dim3((unsigned)(p.B * p.E)), dim3(256), 0, s, m);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int top = p.scan_level > 0 ? p.scan_level : p.D;   // the levels formed
    for (int l = 1; l <= top; ++l) {
        UpLogArgs a{};
        if (l == 1) {
            a.ccore = pot; a.cro = nullptr; a.cco = nullptr; a.cnodes = p.E;
            a.cpmr = p.lrmax; a.cpmc = p.lcmax; a.cntile = 1;
        } else {
            a.ccore = p.core[l - 1]; a.cro = p.ro[l - 1]; a.cco = p.co[l - 1];
            a.cnodes = p.Np >> (l - 1);
            a.cpmr = p.pmr[l - 1]; a.cpmc = p.pmc[l - 1]; a.cntile = p.ntile[l - 1];
        }
        a.core = p.core[l]; a.ro = p.ro[l]; a.co = p.co[l];
        a.pmr = p.pmr[l]; a.pmc = p.pmc[l];
        a.crbits = p.rbits[l - 1]; a.ccbits = p.cbits[l - 1];
        a.rbits = l < p.D ? p.rbits[l] : nullptr;
        a.cbits = l < p.D ? p.cbits[l] : nullptr;
        a.bw = p.bw;
        a.nodes = p.Np >> l;
        a.lengths = lengths; a.B = p.B; a.N = p.N; a.C = p.C; a.level = l;
        const int nt = p.ntile[l];
        a.ntile = nt;
        a.nlogical = p.B * a.nodes * nt * nt;
        a.ngrid = node_grid(p.B * a.nodes, nt * nt);
        const int tm = up_tile(p.C, p.B * a.nodes, kBits);
        if (tm == kSmTM)
            hipLaunchKernelGGL((k_up_log_small<VEC>), dim3((unsigned)a.ngrid), dim3(kUpThreads), 0, s, a);
        else if (tm == 64 && full64)
            hipLaunchKernelGGL((k_up_log_full<64, false>), dim3((unsigned)a.ngrid), dim3(kUpThreads),
                               UpFullSmem<64>::kBytes, s, a);
        else if (tm == 128 && full128) {
            if constexpr (kUpBf16) {
                if (p.C == 128)
                    hipLaunchKernelGGL((k_up_log_full<128, true, 8>), dim3((unsigned)a.ngrid),
                                       dim3(kUpThreads), UpBfSmem<128>::kBytes, s, a);
                else
                    hipLaunchKernelGGL((k_up_log_full<128, true, 16>), dim3((unsigned)a.ngrid),
                                       dim3(kUpThreads), UpBfSmem<128>::kBytes, s, a);
            } else {
                hipLaunchKernelGGL((k_up_log_full<128, false>), dim3((unsigned)a.ngrid), dim3(kUpThreads),
                                   UpFullSmem<128>::kBytes, s, a);
            }
        }
        else if (tm == 64)
            hipLaunchKernelGGL((k_up_log<64, VEC, kBits>), dim3((unsigned)a.ngrid), dim3(kUpThreads),
                               UpSmem<64>::kBytes, s, a);
        else
            hipLaunchKernelGGL((k_up_log<128, VEC, kBits>), dim3((unsigned)a.ngrid), dim3(kUpThreads),
                               UpSmem<128>::kBytes, s, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

template <bool kBits>
hipError_t up_sweep_bits(const Plan& p, const float* pot, const int32_t* lengths, hipStream_t s) {
    return (p.C % 4) == 0 ? up_sweep_vec<true, kBits>(p, pot, lengths, s)
                          : up_sweep_vec<false, kBits>(p, pot, lengths, s);
}

hipError_t up_sweep(const Plan& p, const float* pot, const int32_t* lengths, hipStream_t s) {
    return p.rbits[0] ? up_sweep_bits<true>(p, pot, lengths, s)
                      : up_sweep_bits<false>(p, pot, lengths, s);
}

hipError_t root(const Plan& p, const float* pot, const int32_t* lengths, float* logZ,
                hipStream_t s) {
    RootArgs r{};
    if (p.D == 0) {
        r.core = pot; r.ro = nullptr; r.co = nullptr; r.nodes = p.E;
    } else {
        r.core = p.core[p.D]; r.ro = p.ro[p.D]; r.co = p.co[p.D]; r.nodes = p.Np >> p.D;
    }
    r.lengths = lengths; r.N = p.N; r.C = p.C; r.logZ = logZ;
    hipLaunchKernelGGL(k_root_log, dim3((unsigned)p.B), dim3(kRootThreads), 0, s, r);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_logz_tree(const Plan& p, const float* pot, const int32_t* lengths,
                            float* logZ, hipStream_t s) {
    if (p.chunk) {
        // chunk nodes from the leaves, then the recursions over the chunks (log Z and, for
        // the marginals, the chunks' outside vectors)
        hipError_t e = p.lc > 0 ? launch_chunk_up(p, pot, lengths, s) : hipSuccess;
        return e == hipSuccess ? launch_chunk_scan(p, pot, lengths, logZ, s) : e;
    }
    hipError_t e = up_sweep(p, pot, lengths, s);
    if (e != hipSuccess || !logZ) return e;
    if (p.scan_level > 0) return launch_node_scan(p, lengths, logZ, s);
    return root(p, pot, lengths, logZ, s);
}

hipError_t launch_marginals_tree(const Plan& p, const float* pot, const int32_t* lengths,
                                 float* marg, hipStream_t s) {
    // (the up-sweep has been enqueued by the caller)
    if (p.chunk) return launch_chunk_form(p, pot, lengths, marg, s);
    for (int l = p.D; l >= 2; --l) {
        DownArgs d{};
        d.uN = (l == p.D) ? nullptr : p.u[l];
        d.vN = (l == p.D) ? nullptr : p.v[l];
        d.nodes = p.Np >> l;
        d.ccore = p.core[l - 1]; d.cro = p.ro[l - 1]; d.cco = p.co[l - 1];
        d.cnodes = p.Np >> (l - 1);
        d.uC = p.u[l - 1]; d.vC = p.v[l - 1];
        d.lengths = lengths; d.N = p.N; d.C = p.C; d.level = l;
        if (p.C % 4 == 0)
            hipLaunchKernelGGL(k_down_log<true>, dim3((unsigned)(p.B * d.nodes)), dim3(kVecThreads), 0, s, d);
        else
            hipLaunchKernelGGL(k_down_log<false>, dim3((unsigned)(p.B * d.nodes)), dim3(kVecThreads), 0, s, d);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    FormArgs f{};
    f.pot = pot;
    f.u1 = (p.D >= 2) ? p.u[1] : nullptr;
    f.v1 = (p.D >= 2) ? p.v[1] : nullptr;
    f.nodes1 = (p.D >= 1) ? (p.Np >> 1) : 1;
    f.lengths = lengths; f.N = p.N; f.C = p.C; f.marg = marg; f.wide = p.wide;
    const int64_t npairs = (p.N - 1 + 1) / 2;
    const dim3 grid((unsigned)(p.B * npairs));
    // both leaves of a pair held in registers when they fit: one read of each edge.  One
    // launch per formation (float32 terms, float64 terms for pairs of large magnitude).
    if (p.C % 4 == 0 && p.C <= 64) {
        hipLaunchKernelGGL((k_form_reg<2, false>), grid, dim3(kVecThreads), 0, s, f);
        hipLaunchKernelGGL((k_form_reg<2, true>), grid, dim3(kVecThreads), 0, s, f);
    } else if (p.C % 4 == 0 && p.C <= kRegMaxLabels) {
        hipLaunchKernelGGL((k_form_reg<8, false>), grid, dim3(kVecThreads), 0, s, f);
        hipLaunchKernelGGL((k_form_reg<8, true>), grid, dim3(kVecThreads), 0, s, f);
    } else if (p.C == kBigLabels) {
        // (pairs of large magnitude: the two-read kernel, whose float64 terms fit its registers)
        hipError_t e = allow_form_big_lds<false>();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL((k_form_big<false>), grid, dim3(kBigThreads), kBigKeepBytes, s, f);
        hipLaunchKernelGGL((k_form_log<true, true>), grid, dim3(kVecThreads), 0, s, f);
    } else if (p.C % 4 == 0) {
        hipLaunchKernelGGL((k_form_log<true, false>), grid, dim3(kVecThreads), 0, s, f);
        hipLaunchKernelGGL((k_form_log<true, true>), grid, dim3(kVecThreads), 0, s, f);
    } else {
        hipLaunchKernelGGL((k_form_log<false, false>), grid, dim3(kVecThreads), 0, s, f);
        hipLaunchKernelGGL((k_form_log<false, true>), grid, dim3(kVecThreads), 0, s, f);
    }
    return hipGetLastError();
}

}  // namespace tsc
