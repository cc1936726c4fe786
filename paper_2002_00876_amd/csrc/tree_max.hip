// tree_max.hip -- the (max, +) instance of the edge tree (Torch-Struct Sec. 5.2: the
// max semiring turns the forward algorithm into the max score; Table 2 "Max"; Sec. 6a
// tree order), followed by backpointers and a lowest-index backtrace.
//
// All sums are float64.  A float64 sum of float32 potentials is exact while the partial
// sums stay within 53 significant bits (e.g. every |l| >= 2^-14 and |sum| < 2^15), so
// the tree's forward scores delta_t equal the sequential recursion's bit for bit and
// every argmax decision (and tie) is the same whatever the association order.
//
//   up-sweep:   P[a][c] = max_b L[a][b] + R[b][c]              (nodes of levels 1..D-1)
//   down-sweep: u_L = u_N, u_R = u_N (x) L                     (forward scores only)
//   leaves:     delta_t = u at edge t; bp_t[j] = lowest argmax_i delta_t[i] + l[t][i][j];
//               the last edge also gives z_{L-1} = lowest argmax_j delta_{L-1}[j] and the score
//   decode:     z_t = bp_t[z_{t+1}] by chunks: each chunk maps its end label to its start
//               label for every possible end label; one short serial walk over chunks;
//               each chunk then emits its labels.
#include <type_traits>

#include "device.h"
#include "internal.h"

namespace tsc {

namespace {

constexpr int kMT = 64;    // output tile edge
constexpr int kMK = 16;    // k slice of the narrow kernel (16: fewer staging registers, more waves)
constexpr int kMThreads = 256;
constexpr int64_t kFewTiles = 512;   // two 128-wide tiles per compute unit

struct UpMaxArgs {
    const float* leaves;    // level 1 reads the potentials
    const double* cnode;    // level >= 2 reads float64 nodes
    int64_t cnodes;
    double* node;
    int64_t nodes;
    const int32_t* lengths;
    int64_t B, N, C;
    int level, ntm;
    int64_t nlogical, ngrid;
};

// child entry (r, c) of child k of sequence b: a potential (kLeaf, level 1) or a float64 node
template <bool kLeaf>
__device__ __forceinline__ double child_at(const UpMaxArgs& a, int64_t b, int64_t k, int64_t r,
                                           int64_t c) {
    const size_t off = (size_t)(b * a.cnodes + k) * a.C * a.C + (size_t)(r * a.C + c);
    if constexpr (kLeaf) return (double)a.leaves[off];
    else return a.cnode[off];
}

// One tree level of the max-plus up-sweep in 64 x 64 output tiles (C <= 64, and the levels
// of larger C with few products): one tile per workgroup of 256 threads with 4 x 4 float64
// outputs each (small register footprint, many waves).  kLeaf: level 1 (fp32 potentials).
template <bool kLeaf>
__global__ __launch_bounds__(kMThreads) void k_up_max_narrow(UpMaxArgs a) {
    __shared__ __align__(16) double As[kMK][kMT + 2];   // As[k][row]; the padding spreads
                                                        // the transposing stores over banks
    __shared__ __align__(16) double Bs[kMK][kMT];       // Bs[k][col]
    const int ntiles = a.ntm * a.ntm;
    const int64_t lid = xcd_node_swizzle(blockIdx.x, ntiles);
    if (lid >= a.nlogical) return;
    const int tile = (int)(lid % ntiles);
    const int64_t node = lid / ntiles;
    const int64_t b = node / a.nodes, k = node % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;
    const int64_t C = a.C;
    const int tm = tile / a.ntm, tn = tile % a.ntm;
    const int64_t a0 = (int64_t)tm * kMT, c0 = (int64_t)tn * kMT;
    const int tid = threadIdx.x;
    double* P = a.node + (size_t)(b * a.nodes + k) * C * C;
    const bool right = (2 * k + 1) * half < Eb;
    if (!right) {
        for (int idx = tid; idx < kMT * kMT; idx += kMThreads) {
            const int64_t r = a0 + idx / kMT, c = c0 + idx % kMT;
            if (r < C && c < C) P[r * C + c] = child_at<kLeaf>(a, b, 2 * k, r, c);
        }
        return;
    }
    // 4 x 4 outputs per thread: rows ty * 4 .. + 3; columns in pairs, 2 tx + 32 m + {0, 1}
    // (m = 0, 1), so that the 16 lanes of a 16-byte operand read cover 256 contiguous bytes
    // (no bank conflicts) and a store of a pair by 16 lanes covers 256 contiguous bytes
    const int ty = tid / 16, tx = tid % 16;
    double acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = -INFINITY;
    constexpr int kPer = kMT * kMK / kMThreads;   // staged values per thread and operand
    using T = typename std::conditional<kLeaf, float, double>::type;
    const T* src = kLeaf ? (const T*)a.leaves : (const T*)a.cnode;
    const size_t lbase = (size_t)(b * a.cnodes + 2 * k) * C * C, rbase = lbase + (size_t)C * C;
    // the next slice's loads are in flight while the current slice is used (raw values:
    // the widening of fp32 leaves waits until they are stored)
    T va[kPer], vb[kPer];
    auto load = [&](int64_t k0) {
#pragma unroll
        for (int v = 0; v < kPer; ++v) {
            const int idx = tid + v * kMThreads;
            const int r = idx / kMK, kk = idx % kMK;
            const int64_t row = a0 + r, kg = k0 + kk;
            va[v] = (row < C && kg < C) ? src[lbase + (size_t)row * C + kg] : (T)-INFINITY;
            const int kb = idx / kMT, cc = idx % kMT;
            const int64_t col = c0 + cc, kgb = k0 + kb;
            vb[v] = (col < C && kgb < C) ? src[rbase + (size_t)kgb * C + col] : (T)-INFINITY;
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int v = 0; v < kPer; ++v) {
            const int idx = tid + v * kMThreads;
            As[idx % kMK][idx / kMK] = (double)va[v];
            Bs[idx / kMT][idx % kMT] = (double)vb[v];
        }
    };
    load(0);
    store();
    __syncthreads();
    for (int64_t k0 = 0; k0 < C; k0 += kMK) {
        const bool more = k0 + kMK < C;
        if (more) load(k0 + kMK);
#pragma unroll 2
        for (int kk = 0; kk < kMK; ++kk) {
            double av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const double2 b2 = *(const double2*)&Bs[kk][32 * m + 2 * tx];
                bv[2 * m] = b2.x;
                bv[2 * m + 1] = b2.y;
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmax(acc[i][j], av[i] + bv[j]);
        }
        if (more) {
            __syncthreads();
            store();
            __syncthreads();
        }
    }
    // 16-byte stores of a lane's column pairs when they lie inside the matrix (even C)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t r = a0 + ty * 4 + i;
        if (r >= C) continue;
        double* row = P + r * C;
#pragma unroll
        for (int m = 0; m < 2; ++m) {
            const int64_t cb = c0 + 32 * m + 2 * tx;
            if (cb + 2 <= C && (C % 2) == 0) {
                double2 v;
                v.x = acc[i][2 * m];
                v.y = acc[i][2 * m + 1];
                *(double2*)(row + cb) = v;
            } else {
                if (cb < C) row[cb] = acc[i][2 * m];
                if (cb + 1 < C) row[cb + 1] = acc[i][2 * m + 1];
            }
        }
    }
}

// One tree level of the max-plus up-sweep, P[a][c] = max_b L[a][b] + R[b][c], for one TM x TM
// output tile per workgroup of (TM/8)^2 threads, each holding 8 x 8 float64 accumulators
// (8 rows; 8 columns as 4 interleaved pairs; 64 add + 64 max per 16 operands read from LDS).
// The contraction index runs in slices of KS: A is staged transposed, As[k][row] (rows padded
// to TM + 2 doubles, which keeps the 16-byte operand reads aligned and spreads the
// transposing stores over the banks), B as is, Bs[k][col]; the next slice's global loads are
// in flight while the current one is used (kLeaf: level 1, whose fp32 potentials are widened
// when they are staged).
template <int TM, int KS, bool kLeaf>
__global__ __launch_bounds__((TM / 8) * (TM / 8)) void k_up_max(UpMaxArgs a) {
    constexpr int TPD = TM / 8, NT = TPD * TPD, LDA = TM + 2;
    constexpr int NA = TM * KS / NT;   // staged values per thread and operand
    __shared__ __align__(16) double As[KS * LDA];
    __shared__ __align__(16) double Bs[KS * TM];
    const int ntiles = a.ntm * a.ntm;
    const int64_t lid = xcd_node_swizzle(blockIdx.x, ntiles);
    if (lid >= a.nlogical) return;
    const int tile = (int)(lid % ntiles);
    const int64_t node = lid / ntiles;
    const int64_t b = node / a.nodes, k = node % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;
    const int C = (int)a.C;
    const int tm = tile / a.ntm, tn = tile % a.ntm;
    const int a0 = tm * TM, c0 = tn * TM;
    const int tid = threadIdx.x;
    double* P = a.node + (size_t)(b * a.nodes + k) * C * C;
    const bool right = (2 * k + 1) * half < Eb;
    if (!right) {
        for (int idx = tid; idx < TM * TM; idx += NT) {
            const int r = a0 + idx / TM, c = c0 + idx % TM;
            if (r < C && c < C) P[(size_t)r * C + c] = child_at<kLeaf>(a, b, 2 * k, r, c);
        }
        return;
    }
    const size_t lbase = (size_t)(b * a.cnodes + 2 * k) * C * C;
    const size_t rbase = lbase + (size_t)C * C;
    using T = typename std::conditional<kLeaf, float, double>::type;
    const T* src = kLeaf ? (const T*)a.leaves : (const T*)a.cnode;
    T ra[NA], rb[NA];   // raw values: the widening waits until they are stored
    // staging of slice [k0, k0 + KS): thread value v of A is (row idx / KS, k idx % KS) with
    // idx = tid + v * NT (consecutive threads read consecutive k), of B (k idx / TM, col idx % TM)
    auto load = [&](int k0) {
#pragma unroll
        for (int v = 0; v < NA; ++v) {
            const int idx = tid + v * NT;
            const int r = a0 + idx / KS, kk = k0 + idx % KS;
            ra[v] = (r < C && kk < C) ? src[lbase + (size_t)r * C + kk] : (T)-INFINITY;
            const int kr = k0 + idx / TM, c = c0 + idx % TM;
            rb[v] = (kr < C && c < C) ? src[rbase + (size_t)kr * C + c] : (T)-INFINITY;
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int v = 0; v < NA; ++v) {
            const int idx = tid + v * NT;
            As[(idx % KS) * LDA + idx / KS] = (double)ra[v];
            Bs[idx] = (double)rb[v];
        }
    };
    // 8 x 8 outputs per thread: rows ty * 8 .. + 7; columns in pairs, 2 tx + GW m + {0, 1}
    // (m = 0 .. 3, GW = 2 TPD), so that the TPD lanes of a 16-byte operand read cover
    // contiguous bytes (no bank conflicts) and so do the TPD lanes of a pair's store
    constexpr int GW = 2 * TPD;
    static_assert(4 * GW == TM, "four column groups of 2 TPD");
    const int ty = tid / TPD, tx = tid % TPD;
    double acc[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = -INFINITY;
    const int nslices = (C + KS - 1) / KS;
    load(0);
    store();
    __syncthreads();
    for (int s = 0; s < nslices; ++s) {
        if (s + 1 < nslices) load((s + 1) * KS);
#pragma unroll 2
        for (int kk = 0; kk < KS; ++kk) {
            double av[8], bv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) av[i] = As[kk * LDA + ty * 8 + i];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const double2 b2 = *(const double2*)(Bs + kk * TM + GW * m + 2 * tx);
                bv[2 * m] = b2.x;
                bv[2 * m + 1] = b2.y;
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                double t[8];   // eight independent sums, then eight independent maxima
#pragma unroll
                for (int j = 0; j < 8; ++j) t[j] = av[i] + bv[j];
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[i][j] = fmax(acc[i][j], t[j]);
            }
        }
        if (s + 1 < nslices) {
            __syncthreads();
            store();
            __syncthreads();
        }
    }
    // a lane's column pairs: 16-byte stores when a pair lies inside the matrix and starts on
    // a 16-byte boundary (even C), single stores at the edges
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = a0 + ty * 8 + i;
        if (r >= C) continue;
        double* row = P + (size_t)r * C;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int cb = c0 + GW * m + 2 * tx;
            if (cb + 2 <= C && (C % 2) == 0) {
                double2 v;
                v.x = acc[i][2 * m];
                v.y = acc[i][2 * m + 1];
                *(double2*)(row + cb) = v;
            } else {
                if (cb < C) row[cb] = acc[i][2 * m];
                if (cb + 1 < C) row[cb + 1] = acc[i][2 * m + 1];
            }
        }
    }
}

// ---- forward scores down the tree: u_L = u_N, u_R = u_N (x) L
struct DownMaxArgs {
    const double* uN;    // nullptr at the root (zeros)
    int64_t nodes;
    const double* cnode; // children (level l-1 >= 1)
    int64_t cnodes;
    double* uC;
    const int32_t* lengths;
    int64_t N, C;
    int level;
};

template <int kS>
__global__ __launch_bounds__(256) void k_down_max(DownMaxArgs a) {
    __shared__ double su[kMaxLabels];
    const int64_t b = blockIdx.x / a.nodes, k = blockIdx.x % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t C = a.C;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;
    for (int64_t i = threadIdx.x; i < C; i += blockDim.x)
        su[i] = a.uN ? a.uN[(size_t)(b * a.nodes + k) * C + i] : 0.0;
    __syncthreads();
    double* uL = a.uC + (size_t)(b * a.cnodes + 2 * k) * C;
    for (int64_t i = threadIdx.x; i < C; i += blockDim.x) uL[i] = su[i];
    if ((2 * k + 1) * half >= Eb) return;
    const double* L = a.cnode + (size_t)(b * a.cnodes + 2 * k) * C * C;
    double* uR = a.uC + (size_t)(b * a.cnodes + 2 * k + 1) * C;
    // kS consecutive threads per column, each over every kS-th row (four loads in flight),
    // then a max across them (exact in any order)
    const int t = (int)threadIdx.x, j = t / kS, s = t % kS;
    double m = -INFINITY;
    if (j < C) {
        int i = s;
        for (; i + 3 * kS < C; i += 4 * kS) {
            double l[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) l[u] = L[(size_t)(i + u * kS) * C + j];
#pragma unroll
            for (int u = 0; u < 4; ++u) m = fmax(m, su[i + u * kS] + l[u]);
        }
        for (; i < C; i += kS) m = fmax(m, su[i] + L[(size_t)i * C + j]);
    }
#pragma unroll
    for (int o = 1; o < kS; o <<= 1) m = fmax(m, __shfl_xor(m, o, kWave));
    if (j < C && s == 0) uR[j] = m;
}

// ---- leaves: backpointers, last label and score
struct BpArgs {
    const float* pot;
    const double* u1;   // level-1 forward vectors (nullptr when level 1 is the root)
    int64_t nodes1;
    const int32_t* lengths;
    int64_t N, C;
    uint8_t* bp;        // [B, E, C]
    int32_t* zlast;     // [B]
    float* score;       // [B]
};

// For edge t with forward scores d (shared, [C]): bp[t][j] = lowest argmax_i d[i] + l[t][i][j]
// and, into dn[j] (shared, may be nullptr), the max itself.  kS consecutive threads share a
// column (kS * C <= 256 threads): part s scans rows s, s + kS, ... in ascending order, four
// rows' loads issued together, keeping the first maximum; the parts then meet through lane
// exchanges, the lower index winning ties (all -inf gives row 0, as a serial scan would).
template <int kS>
__device__ void backpointers(const float* leaf, const double* d, int C, uint8_t* bp, double* dn) {
    const int t = (int)threadIdx.x, j = t / kS, s = t % kS;
    double best = -INFINITY;
    int arg = s;
    if (j < C) {
        int i = s;
        for (; i + 3 * kS < C; i += 4 * kS) {
            float l[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) l[u] = leaf[(size_t)(i + u * kS) * C + j];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const double v = d[i + u * kS] + (double)l[u];
                if (v > best) { best = v; arg = i + u * kS; }
            }
        }
        for (; i < C; i += kS) {
            const double v = d[i] + (double)leaf[(size_t)i * C + j];
            if (v > best) { best = v; arg = i; }
        }
    }
#pragma unroll
    for (int o = 1; o < kS; o <<= 1) {
        const double ov = __shfl_xor(best, o, kWave);
        const int oi = __shfl_xor(arg, o, kWave);
        if (ov > best || (ov == best && oi < arg)) { best = ov; arg = oi; }
    }
    if (j < C && s == 0) {
        bp[j] = (uint8_t)arg;
        if (dn) dn[j] = best;
    }
}

template <int kS>
__global__ __launch_bounds__(256) void k_bp_max(BpArgs a) {
    __shared__ double su[kMaxLabels], sr[kMaxLabels], sl[kMaxLabels];
    __shared__ double rv[4];
    __shared__ int ri[4];
    const int64_t npairs = (a.N - 1 + 1) / 2;
    const int64_t b = blockIdx.x / npairs, k = blockIdx.x % npairs;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t C = a.C, E = a.N - 1;
    if (Eb == 0) {
        if (k == 0 && threadIdx.x == 0) { a.zlast[b] = 0; a.score[b] = 0.f; }
        return;
    }
    const int64_t tL = 2 * k, tR = 2 * k + 1;
    if (tL >= Eb) return;
    for (int64_t i = threadIdx.x; i < C; i += blockDim.x)
        su[i] = a.u1 ? a.u1[(size_t)(b * a.nodes1 + k) * C + i] : 0.0;
    __syncthreads();
    const float* leafL = a.pot + (size_t)(b * E + tL) * C * C;
    const bool right = tR < Eb;
    // edge tL: delta_{tL} = u; its max gives delta_{tL+1} = delta_{tR}
    backpointers<kS>(leafL, su, (int)C, a.bp + (size_t)(b * E + tL) * C, sr);
    __syncthreads();
    const double* dlast = sr;
    if (right) {
        const float* leafR = a.pot + (size_t)(b * E + tR) * C * C;
        backpointers<kS>(leafR, sr, (int)C, a.bp + (size_t)(b * E + tR) * C, sl);
        __syncthreads();
        dlast = sl;
    }
    const int64_t tlast = right ? tR : tL;
    if (tlast != Eb - 1) return;
    // z_{L-1} = lowest argmax_j delta_{L-1}[j]
    double best = -INFINITY;
    int arg = 0x7fffffff;
    for (int64_t j = threadIdx.x; j < C; j += blockDim.x) {
        const double v = dlast[j];
        if (v > best || (v == best && j < arg)) { best = v; arg = (int)j; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        const double ov = __shfl_xor(best, o, kWave);
        const int oi = __shfl_xor(arg, o, kWave);
        if (ov > best || (ov == best && oi < arg)) { best = ov; arg = oi; }
    }
    const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) { rv[w] = best; ri[w] = arg; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int i = 1; i < nw; ++i)
            if (rv[i] > best || (rv[i] == best && ri[i] < arg)) { best = rv[i]; arg = ri[i]; }
        // every label ties at -inf when no sequence is finite: the lowest label, 0
        if (arg >= C) arg = 0;
        a.zlast[b] = arg;
        a.score[b] = (float)best;
    }
}

// ---- decode
struct DecArgs {
    const uint8_t* bp;
    const int32_t* lengths;
    int64_t N, C, chunk, nchunks;
    uint8_t* map;       // [B, nchunks, C]
    int32_t* zend;      // [B, nchunks]
    const int32_t* zlast;
    int32_t* path;      // [B, N]
};

// chunk c covers edges [c*K, min((c+1)*K, E_b)); it maps the label at position
// e_c = min((c+1)*K, E_b) to the label at position s_c = c*K, for every label at e_c.
__global__ __launch_bounds__(256) void k_dec_map(DecArgs a) {
    extern __shared__ uint8_t sbp[];
    const int64_t b = blockIdx.x / a.nchunks, c = blockIdx.x % a.nchunks;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1, E = a.N - 1;
    const int64_t s = c * a.chunk;
    if (s >= Eb) return;
    const int64_t e = min((c + 1) * a.chunk, Eb);
    const int64_t n = (e - s) * a.C;
    const uint8_t* src = a.bp + (size_t)(b * E + s) * a.C;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) sbp[i] = src[i];
    __syncthreads();
    const int64_t j = threadIdx.x;
    if (j < a.C) {
        int z = (int)j;
        for (int64_t t = e - 1; t >= s; --t) z = sbp[(t - s) * a.C + z];
        a.map[(size_t)(b * a.nchunks + c) * a.C + j] = (uint8_t)z;
    }
}

// one wave per sequence: z at every chunk end, walking the chunk maps backwards
__global__ __launch_bounds__(64) void k_dec_walk(DecArgs a) {
    extern __shared__ uint8_t smap[];
    const int64_t b = blockIdx.x;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    if (Eb == 0) {
        if (threadIdx.x == 0) a.zend[b * a.nchunks] = 0;
        return;
    }
    const int64_t last = (Eb - 1) / a.chunk;
    const int64_t n = (last + 1) * a.C;
    const uint8_t* src = a.map + (size_t)b * a.nchunks * a.C;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) smap[i] = src[i];
    __syncthreads();
    if (threadIdx.x == 0) {
        int z = a.zlast[b];
        for (int64_t c = last; c >= 0; --c) {
            a.zend[b * a.nchunks + c] = z;
            z = smap[c * a.C + z];
        }
    }
}

// each chunk writes the labels of positions (s_c, e_c] (chunk 0 also position 0) and -1
// for its positions at or past the length
__global__ __launch_bounds__(64) void k_dec_emit(DecArgs a) {
    extern __shared__ uint8_t sbp[];
    const int64_t b = blockIdx.x / a.nchunks, c = blockIdx.x % a.nchunks;
    const int64_t L = clamp_len(a.lengths, b, a.N), Eb = L - 1, E = a.N - 1;
    const int64_t s = c * a.chunk;
    int32_t* path = a.path + (size_t)b * a.N;
    // positions s+1 .. min(s+K, N-1) that lie past the last token
    for (int64_t n = s + 1 + threadIdx.x; n <= min(s + a.chunk, E); n += blockDim.x)
        if (n >= L) path[n] = -1;
    if (Eb == 0) {
        if (c == 0 && threadIdx.x == 0) path[0] = a.zend[b * a.nchunks];
        return;
    }
    if (s >= Eb) return;
    const int64_t e = min((c + 1) * a.chunk, Eb);
    const int64_t n = (e - s) * a.C;
    const uint8_t* src = a.bp + (size_t)(b * E + s) * a.C;
    for (int64_t i = threadIdx.x; i < n; i += blockDim.x) sbp[i] = src[i];
    __syncthreads();
    if (threadIdx.x == 0) {
        int z = a.zend[b * a.nchunks + c];
        path[e] = z;
        for (int64_t t = e - 1; t >= s; --t) {
            z = sbp[(t - s) * a.C + z];
            if (t > s || c == 0) path[t] = z;
        }
    }
}


}  // namespace

hipError_t launch_viterbi_tree(const Plan& p, const float* pot, const int32_t* lengths,
                               int32_t* path, float* score, hipStream_t s) {
    const int64_t C = p.C;
    // levels below the root: the forward scores start from the root with zeros and only
    // read its children's matrices
    for (int l = 1; l < p.D; ++l) {
        // 128-wide tiles above C = 64, unless a level has too few of them to give every
        // compute unit a workgroup: then the narrow kernel's 64-wide tiles (a quarter of the
        // work each, so four times the workgroups and a quarter of the latency)
        const int64_t wide = (C + 2 * kMT - 1) / (2 * kMT);
        const bool narrow = C <= kMT || p.B * (p.Np >> l) * wide * wide < kFewTiles;
        const int tmax = narrow ? kMT : 2 * kMT;
        const int ntm = (int)((C + tmax - 1) / tmax);
        UpMaxArgs a{};
        a.leaves = (l == 1) ? pot : nullptr;
        a.cnode = (l == 1) ? nullptr : p.mnode[l - 1];
        a.cnodes = (l == 1) ? p.E : (p.Np >> (l - 1));
        a.node = p.mnode[l];
        a.nodes = p.Np >> l;
        a.lengths = lengths; a.B = p.B; a.N = p.N; a.C = C; a.level = l; a.ntm = ntm;
        a.nlogical = p.B * a.nodes * ntm * ntm;
        a.ngrid = node_grid(p.B * a.nodes, ntm * ntm);
        if (narrow && l == 1)
            hipLaunchKernelGGL(k_up_max_narrow<true>, dim3((unsigned)a.ngrid), dim3(kMThreads), 0, s, a);
        else if (narrow)
            hipLaunchKernelGGL(k_up_max_narrow<false>, dim3((unsigned)a.ngrid), dim3(kMThreads), 0, s, a);
        else if (l == 1)
            hipLaunchKernelGGL((k_up_max<2 * kMT, 16, true>), dim3((unsigned)a.ngrid), dim3(256), 0, s, a);
        else
            hipLaunchKernelGGL((k_up_max<2 * kMT, 16, false>), dim3((unsigned)a.ngrid), dim3(256), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    for (int l = p.D; l >= 2; --l) {
        DownMaxArgs d{};
        d.uN = (l == p.D) ? nullptr : p.mu[l];
        d.nodes = p.Np >> l;
        d.cnode = p.mnode[l - 1];
        d.cnodes = p.Np >> (l - 1);
        d.uC = p.mu[l - 1];
        d.lengths = lengths; d.N = p.N; d.C = C; d.level = l;
        const dim3 dgrid((unsigned)(p.B * d.nodes));
        if (C <= 64) hipLaunchKernelGGL(k_down_max<4>, dgrid, dim3(256), 0, s, d);
        else if (C <= 128) hipLaunchKernelGGL(k_down_max<2>, dgrid, dim3(256), 0, s, d);
        else hipLaunchKernelGGL(k_down_max<1>, dgrid, dim3(256), 0, s, d);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    BpArgs bpa{};
    bpa.pot = pot;
    bpa.u1 = (p.D >= 2) ? p.mu[1] : nullptr;
    bpa.nodes1 = (p.D >= 1) ? (p.Np >> 1) : 1;
    bpa.lengths = lengths; bpa.N = p.N; bpa.C = C; bpa.bp = p.bp; bpa.zlast = p.zlast;
    bpa.score = score;
    const int64_t npairs = (p.N - 1 + 1) / 2;
    // as many threads per column as 256 threads allow, up to four
    const dim3 bgrid((unsigned)(p.B * npairs));
    if (C <= 64) hipLaunchKernelGGL(k_bp_max<4>, bgrid, dim3(256), 0, s, bpa);
    else if (C <= 128) hipLaunchKernelGGL(k_bp_max<2>, bgrid, dim3(256), 0, s, bpa);
    else hipLaunchKernelGGL(k_bp_max<1>, bgrid, dim3(256), 0, s, bpa);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    DecArgs d{};
    d.bp = p.bp; d.lengths = lengths; d.N = p.N; d.C = C; d.chunk = p.dec_chunk;
    d.nchunks = p.dec_nchunks; d.map = p.dec_map; d.zend = p.dec_zend; d.zlast = p.zlast;
    d.path = path;
    const size_t chunk_bytes = (size_t)p.dec_chunk * C;
    hipLaunchKernelGGL(k_dec_map, dim3((unsigned)(p.B * p.dec_nchunks)), dim3(256), chunk_bytes,
                       s, d);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dec_walk, dim3((unsigned)p.B), dim3(64), (size_t)p.dec_nchunks * C, s, d);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(k_dec_emit, dim3((unsigned)(p.B * p.dec_nchunks)), dim3(64), chunk_bytes,
                       s, d);
    return hipGetLastError();
}

}  // namespace tsc
