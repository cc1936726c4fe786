// tree_log.hip -- log-semiring (logsumexp, +) tree over the edges of each sequence:
// the up-sweep of C x C semiring matrix products (Torch-Struct Sec. 6a / Fig. 3; the
// product is the Sec. 6c operation V = log sum_n exp(T + U)), the root log-sum-exp
// (Sec. 5.2: A sums over the first and last label), the outside (down) sweep that
// yields every edge's forward and backward messages, and the per-edge marginals
// (Sec. 5.1: p(z_p = 1) = dA/dl_p).
//
// Node representation (levels >= 1): P[a][c] = ro[a] + co[c] + core[a][c], ro/co in
// float64, core in float32.  The product P = L (x) R is evaluated as an exp-shifted
// dense GEMM on the fp32 matrix cores:
//   A'[a][b] = core_L[a][b] + (co_L[b] - max co_L),   B'[b][c] = core_R[b][c] + (ro_R[b] - max ro_R)
//   rA[a] = max_b A'[a][b],  cB[c] = max_b B'[b][c]
//   S[a][c] = sum_b exp(A'[a][b] - rA[a]) * exp(B'[b][c] - cB[c])          (MFMA, fp32)
//   core_P = log S,  ro_P[a] = ro_L[a] + max co_L + rA[a],  co_P[c] = co_R[c] + max ro_R + cB[c]
// Every exponent is <= 0, so nothing overflows; S < 2^-80 (all terms underflowing) is
// recomputed exactly by a direct max-shifted log-sum-exp over b.
#include "device.h"
#include "internal.h"

namespace tsc {

namespace {

constexpr int kTile = 64;        // output tile rows = cols per workgroup
constexpr int kUpThreads = 256;  // 4 waves, each owns a 32 x 32 quadrant of the tile
constexpr float kUnderflow = 0x1p-80f;

typedef float f16v __attribute__((ext_vector_type(16)));

struct UpLogArgs {
    const float* ccore;   // children (level l-1): core, or the potentials when l == 1
    const double* cro;    // nullptr for leaves (ro = co = 0)
    const double* cco;
    int64_t cnodes;       // child node stride per sequence
    float* core;          // outputs (level l)
    double* ro;
    double* co;
    int64_t nodes;        // nodes per sequence at level l
    const int32_t* lengths;
    int64_t B, N, C;
    int level;
    int ntm;              // tiles per matrix dimension
    int kp;               // C rounded up to a multiple of 8
    int64_t nlogical;     // B * nodes * ntm * ntm
    int64_t ngrid;        // nlogical rounded up to a multiple of 8
};

inline int64_t round8(int64_t x) { return (x + 7) / 8 * 8; }

__device__ __forceinline__ size_t mat_off(int64_t b, int64_t k, int64_t nodes, int64_t C) {
    return (size_t)(b * nodes + k) * (size_t)C * (size_t)C;
}

// One tree level: workgroup = one 64 x 64 output tile of one node.  KP is C rounded up
// to 64, 128 or 256 (compile-time, so every staging loop unrolls into batched loads);
// VEC selects 16-byte global loads (C % 4 == 0).
//   LDS: As[64][KP+4]  rows a0.. of A' (k contiguous), then exp(A' - rowmax)
//        Bs[KP][64+4]  columns c0.. of B' (k-major, as stored in HBM), then exp(B' - colmax)
template <int KP, bool VEC>
__global__ __launch_bounds__(kUpThreads) void k_up_log(UpLogArgs a) {
    extern __shared__ __align__(16) float smem[];
    constexpr int LDA = KP + 4, LDB = kTile + 4;
    const int64_t lid = xcd_swizzle(blockIdx.x, a.ngrid);
    if (lid >= a.nlogical) return;
    const int ntiles = a.ntm * a.ntm;
    const int tile = (int)(lid % ntiles);
    const int64_t node = lid / ntiles;
    const int64_t b = node / a.nodes, k = node % a.nodes;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t span = (int64_t)1 << a.level, half = span >> 1;
    if (k * span >= Eb) return;  // node absent: all padding
    const int C = (int)a.C;
    const int tm = tile / a.ntm, tn = tile % a.ntm;
    const int a0 = tm * kTile, c0 = tn * kTile;
    const int tid = threadIdx.x;

    const float* Lc = a.ccore + mat_off(b, 2 * k, a.cnodes, C);
    const double* Lro = a.cro ? a.cro + (size_t)(b * a.cnodes + 2 * k) * C : nullptr;
    const double* Lco = a.cco ? a.cco + (size_t)(b * a.cnodes + 2 * k) * C : nullptr;
    float* Pc = a.core + mat_off(b, k, a.nodes, C);
    double* Pro = a.ro + (size_t)(b * a.nodes + k) * C;
    double* Pco = a.co + (size_t)(b * a.nodes + k) * C;

    const bool right = (2 * k + 1) * half < Eb;
    if (!right) {
        // the right half is padding: the node equals its left child
#pragma unroll
        for (int it = 0; it < kTile * kTile / kUpThreads; ++it) {
            const int idx = tid + it * kUpThreads;
            const int r = a0 + idx / kTile, c = c0 + idx % kTile;
            if (r < C && c < C) Pc[r * C + c] = Lc[r * C + c];
        }
        if (tn == 0)
            for (int i = tid; i < kTile; i += kUpThreads)
                if (a0 + i < C) Pro[a0 + i] = Lro ? Lro[a0 + i] : 0.0;
        if (tm == 0)
            for (int i = tid; i < kTile; i += kUpThreads)
                if (c0 + i < C) Pco[c0 + i] = Lco ? Lco[c0 + i] : 0.0;
        return;
    }
    const float* Rc = a.ccore + mat_off(b, 2 * k + 1, a.cnodes, C);
    const double* Rro = a.cro ? a.cro + (size_t)(b * a.cnodes + 2 * k + 1) * C : nullptr;
    const double* Rco = a.cco ? a.cco + (size_t)(b * a.cnodes + 2 * k + 1) * C : nullptr;

    float* As = smem;                  // [kTile][LDA]
    float* Bs = As + kTile * LDA;      // [KP][LDB]
    float* coh = Bs + KP * LDB;        // [KP] co_L - max co_L
    float* roh = coh + KP;             // [KP] ro_R - max ro_R
    float* rowm = roh + KP;            // [kTile]
    float* colm = rowm + kTile;        // [kTile]
    double* red = (double*)(colm + kTile);  // [4]

    // ---- column offsets of L and row offsets of R, shifted to max 0
    double lmax = -INFINITY, rmax = -INFINITY;
    for (int i = tid; i < C; i += kUpThreads) {
        if (Lco) lmax = fmax(lmax, Lco[i]);
        if (Rro) rmax = fmax(rmax, Rro[i]);
    }
    const double coLshift = Lco ? safe_shift_d(block_max_d(lmax, red)) : 0.0;
    const double roRshift = Rro ? safe_shift_d(block_max_d(rmax, red)) : 0.0;
    for (int i = tid; i < KP; i += kUpThreads) {
        coh[i] = (i < C && Lco) ? (float)(Lco[i] - coLshift) : 0.f;
        roh[i] = (i < C && Rro) ? (float)(Rro[i] - roRshift) : 0.f;
    }
    __syncthreads();

    // ---- stage A' = rows a0.. of L (+coh) and B' = columns c0.. of R (+roh); all loads of
    // a panel are issued before any store
    constexpr float NI = -INFINITY;
    {
        constexpr int GA = KP / 4, NA = kTile * GA / kUpThreads;
        float4 v[NA];
#pragma unroll
        for (int it = 0; it < NA; ++it) {
            const int idx = tid + it * kUpThreads;
            const int r = idx / GA, col = 4 * (idx % GA), row = a0 + r;
            if (VEC) {
                v[it] = (row < C && col < C) ? *(const float4*)(Lc + (size_t)row * C + col)
                                             : make_float4(NI, NI, NI, NI);
            } else {
                const float* p = Lc + (size_t)row * C + col;
                v[it].x = (row < C && col + 0 < C) ? p[0] : NI;
                v[it].y = (row < C && col + 1 < C) ? p[1] : NI;
                v[it].z = (row < C && col + 2 < C) ? p[2] : NI;
                v[it].w = (row < C && col + 3 < C) ? p[3] : NI;
            }
        }
#pragma unroll
        for (int it = 0; it < NA; ++it) {
            const int idx = tid + it * kUpThreads;
            const int r = idx / GA, col = 4 * (idx % GA);
            float4 x = v[it];
            x.x += coh[col]; x.y += coh[col + 1]; x.z += coh[col + 2]; x.w += coh[col + 3];
            *(float4*)(As + r * LDA + col) = x;
        }
    }
    {
        constexpr int GB = kTile / 4, NB = KP * GB / kUpThreads;
        float4 v[NB];
#pragma unroll
        for (int it = 0; it < NB; ++it) {
            const int idx = tid + it * kUpThreads;
            const int kk = idx / GB, cl = 4 * (idx % GB), col = c0 + cl;
            if (VEC) {
                v[it] = (kk < C && col < C) ? *(const float4*)(Rc + (size_t)kk * C + col)
                                            : make_float4(NI, NI, NI, NI);
            } else {
                const float* p = Rc + (size_t)kk * C + col;
                v[it].x = (kk < C && col + 0 < C) ? p[0] : NI;
                v[it].y = (kk < C && col + 1 < C) ? p[1] : NI;
                v[it].z = (kk < C && col + 2 < C) ? p[2] : NI;
                v[it].w = (kk < C && col + 3 < C) ? p[3] : NI;
            }
        }
#pragma unroll
        for (int it = 0; it < NB; ++it) {
            const int idx = tid + it * kUpThreads;
            const int kk = idx / GB, cl = 4 * (idx % GB);
            float4 x = v[it];
            const float rh = roh[kk];
            x.x += rh; x.y += rh; x.z += rh; x.w += rh;
            *(float4*)(Bs + kk * LDB + cl) = x;
        }
    }
    __syncthreads();

    // ---- row maxima of A' and column maxima of B' (4 neighbouring lanes per row/column)
    {
        const int r = tid >> 2, part = tid & 3;
        float m1 = -INFINITY, m2 = -INFINITY;
#pragma unroll
        for (int g = part; g < KP / 4; g += 4) {
            const float4 x = *(const float4*)(As + r * LDA + 4 * g);
            m1 = fmaxf(m1, fmaxf(fmaxf(x.x, x.y), fmaxf(x.z, x.w)));
        }
#pragma unroll
        for (int kk = part; kk < KP; kk += 4) m2 = fmaxf(m2, Bs[kk * LDB + r]);
        m1 = fmaxf(m1, dpp_f(m1, 0xB1));
        m1 = fmaxf(m1, dpp_f(m1, 0x4E));
        m2 = fmaxf(m2, dpp_f(m2, 0xB1));
        m2 = fmaxf(m2, dpp_f(m2, 0x4E));
        if (part == 0) {
            rowm[r] = m1;
            colm[r] = m2;
        }
    }
    __syncthreads();
    {
        constexpr int GA = KP / 4, NA = kTile * GA / kUpThreads;
#pragma unroll
        for (int it = 0; it < NA; ++it) {
            const int idx = tid + it * kUpThreads;
            const int r = idx / GA, col = 4 * (idx % GA);
            float4* p = (float4*)(As + r * LDA + col);
            float4 x = *p;
            const float s = safe_shift(rowm[r]);
            x.x = __expf(x.x - s); x.y = __expf(x.y - s); x.z = __expf(x.z - s); x.w = __expf(x.w - s);
            *p = x;
        }
        constexpr int GB = kTile / 4, NB = KP * GB / kUpThreads;
#pragma unroll
        for (int it = 0; it < NB; ++it) {
            const int idx = tid + it * kUpThreads;
            const int kk = idx / GB, cl = 4 * (idx % GB);
            float4* p = (float4*)(Bs + kk * LDB + cl);
            float4 x = *p;
            x.x = __expf(x.x - safe_shift(colm[cl]));
            x.y = __expf(x.y - safe_shift(colm[cl + 1]));
            x.z = __expf(x.z - safe_shift(colm[cl + 2]));
            x.w = __expf(x.w - safe_shift(colm[cl + 3]));
            *p = x;
        }
    }
    __syncthreads();

    // ---- S = expA * expB on the matrix cores.  Within each 8-wide k step, lanes 0-31
    // contribute k..k+3 and lanes 32-63 k+4..k+7 (one 16-byte LDS read of A per lane);
    // A and B use the same k assignment, so the sum over k is unchanged.
    const int w = tid / kWave, lane = tid % kWave;
    const int wm = w >> 1, wn = w & 1;
    f16v acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const float* ap = As + (wm * 32 + (lane & 31)) * LDA + 4 * (lane >> 5);
    const float* bp = Bs + (4 * (lane >> 5)) * LDB + wn * 32 + (lane & 31);
    const int kend = (C + 7) & ~7;
#pragma unroll 2
    for (int kk = 0; kk < kend; kk += 8) {
        const float4 av = *(const float4*)(ap + kk);
        const float b0 = bp[(kk + 0) * LDB], b1 = bp[(kk + 1) * LDB];
        const float b2 = bp[(kk + 2) * LDB], b3 = bp[(kk + 3) * LDB];
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.x, b0, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.y, b1, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.z, b2, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av.w, b3, acc, 0, 0, 0);
    }

    // ---- epilogue: core = log S (exact fallback when S underflows)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int row = wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        const int col = wn * 32 + (lane & 31);
        const int gr = a0 + row, gc = c0 + col;
        if (gr < C && gc < C) {
            const float S = acc[r];
            float val;
            if (S >= kUnderflow) {
                val = __logf(S);
            } else {
                const float sa = safe_shift(rowm[row]), sb = safe_shift(colm[col]);
                float q = -INFINITY;
                for (int bb = 0; bb < C; ++bb) {
                    const float x = (Lc[(size_t)gr * C + bb] + coh[bb] - sa) +
                                    (Rc[(size_t)bb * C + gc] + roh[bb] - sb);
                    q = fmaxf(q, x);
                }
                if (q == -INFINITY) {
                    val = -INFINITY;
                } else {
                    float s = 0.f;
                    for (int bb = 0; bb < C; ++bb) {
                        const float x = (Lc[(size_t)gr * C + bb] + coh[bb] - sa) +
                                        (Rc[(size_t)bb * C + gc] + roh[bb] - sb);
                        s += __expf(x - q);
                    }
                    val = q + __logf(s);
                }
            }
            Pc[(size_t)gr * C + gc] = val;
        }
    }
    if (tn == 0)
        for (int i = tid; i < kTile; i += kUpThreads)
            if (a0 + i < C) Pro[a0 + i] = (Lro ? Lro[a0 + i] : 0.0) + coLshift + safe_shift(rowm[i]);
    if (tm == 0)
        for (int i = tid; i < kTile; i += kUpThreads)
            if (c0 + i < C) Pco[c0 + i] = (Rco ? Rco[c0 + i] : 0.0) + roRshift + safe_shift(colm[i]);
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

__global__ __launch_bounds__(256) void k_root_log(RootArgs a) {
    __shared__ float red[16];
    __shared__ double redd[4];
    const int64_t b = blockIdx.x;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int64_t C = a.C;
    if (Eb == 0) {
        if (threadIdx.x == 0) a.logZ[b] = logf((float)C);
        return;
    }
    const float* P = a.core + mat_off(b, 0, a.nodes, C);
    const double* ro = a.ro ? a.ro + (size_t)b * a.nodes * C : nullptr;
    const double* co = a.co ? a.co + (size_t)b * a.nodes * C : nullptr;
    double rm = -INFINITY, cm = -INFINITY;
    for (int64_t i = threadIdx.x; i < C; i += blockDim.x) {
        if (ro) rm = fmax(rm, ro[i]);
        if (co) cm = fmax(cm, co[i]);
    }
    const double rs = ro ? safe_shift_d(block_max_d(rm, redd)) : 0.0;
    const double cs = co ? safe_shift_d(block_max_d(cm, redd)) : 0.0;
    Lse acc = lse_empty();
    for (int64_t idx = threadIdx.x; idx < C * C; idx += blockDim.x) {
        const int64_t i = idx / C, j = idx % C;
        float x = P[idx];
        if (ro) x += (float)(ro[i] - rs) + (float)(co[j] - cs);
        acc = lse_push(acc, x);
    }
    acc = block_lse(acc, red);
    if (threadIdx.x == 0) {
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

// LSE_i (w[i] + M[i][j]) for one column j (w in LDS, M row-major in global memory), eight
// loads in flight per step
__device__ __forceinline__ float col_lse(const float* __restrict__ M, int C, const float* w, int j) {
    float m = -INFINITY, s = 0.f;
    int i = 0;
    for (; i + 8 <= C; i += 8) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = M[(size_t)(i + u) * C + j];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] += w[i + u];
        lse_fold<8>(m, s, x);
    }
    for (; i < C; ++i) {
        float x[1] = {M[(size_t)i * C + j] + w[i]};
        lse_fold<1>(m, s, x);
    }
    return lse_val(m, s);
}

// LSE_j (M[i][j] + w[j]) for one row i; kVec: 16-byte loads (C % 4 == 0)
template <bool kVec>
__device__ __forceinline__ float row_lse(const float* __restrict__ M, int C, const float* w, int i) {
    const float* row = M + (size_t)i * C;
    float m = -INFINITY, s = 0.f;
    int j = 0;
    if constexpr (kVec) {
        const float4* r4 = reinterpret_cast<const float4*>(row);
        for (; j + 16 <= C; j += 16) {
            float4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = r4[j / 4 + u];
            float x[16];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                x[4 * u + 0] = v[u].x + w[j + 4 * u + 0];
                x[4 * u + 1] = v[u].y + w[j + 4 * u + 1];
                x[4 * u + 2] = v[u].z + w[j + 4 * u + 2];
                x[4 * u + 3] = v[u].w + w[j + 4 * u + 3];
            }
            lse_fold<16>(m, s, x);
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
// be idle (active == false) but still joins the barriers.
template <bool kVec>
__device__ void half_vec(bool active, const float* core, const double* ro, const double* co,
                         int C, const float* x, float* w, float* y, double* red, float* yraw) {
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
    if (active && t < C) {
        const float l = rowPass ? row_lse<kVec>(core, C, w, t) : col_lse(core, C, w, t);
        z = (l == -INFINITY) ? -INFINITY : (outOff ? outOff[t] : 0.0) + ws + (double)l;
        if (yraw) yraw[t] = (float)z;
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
};

// mu = exp(al[i] + leaf[i][j] + be[j] - n) over one C x C edge, the whole workgroup:
// thread t takes column group t % G (16 bytes when kVec, else one float) of rows t / G,
// t / G + T / G, ... so that each row is read and written contiguously
template <bool kVec>
__device__ void write_marginal(const float* __restrict__ leaf, const float* al, const float* be,
                               float n, int C, float* __restrict__ out) {
    constexpr int kW = kVec ? 4 : 1;
    const int G = C / kW, step = kVecThreads / G;
    const int g = threadIdx.x % G, i0 = threadIdx.x / G;
    if (i0 >= step) return;
    const int j = g * kW;
    float bj[kW];
#pragma unroll
    for (int q = 0; q < kW; ++q) bj[q] = be[j + q] - n;
    const bool zero = n == -INFINITY;
#pragma unroll 4
    for (int i = i0; i < C; i += step) {
        const float ai = al[i];
        if constexpr (kVec) {
            const float4 v = *reinterpret_cast<const float4*>(leaf + (size_t)i * C + j);
            float4 r;
            r.x = zero ? 0.f : fexp(ai + v.x + bj[0]);
            r.y = zero ? 0.f : fexp(ai + v.y + bj[1]);
            r.z = zero ? 0.f : fexp(ai + v.z + bj[2]);
            r.w = zero ? 0.f : fexp(ai + v.w + bj[3]);
            *reinterpret_cast<float4*>(out + (size_t)i * C + j) = r;
        } else {
            const float v = leaf[(size_t)i * C + j];
            out[(size_t)i * C + j] = zero ? 0.f : fexp(ai + v + bj[0]);
        }
    }
}

template <bool kVec>
__global__ __launch_bounds__(kVecThreads) void k_form_log(FormArgs a) {
    __shared__ float su[kMaxLabels], sv[kMaxLabels], sy[2][kMaxLabels], sw[2][kMaxLabels],
        raw[2][kMaxLabels];
    __shared__ double red[kVecThreads / kWave];
    __shared__ float nrm[2];
    const int64_t npairs = (a.N - 1 + 1) / 2;
    const int64_t b = blockIdx.x / npairs, k = blockIdx.x % npairs;
    const int64_t Eb = clamp_len(a.lengths, b, a.N) - 1;
    const int C = (int)a.C;
    const int64_t E = a.N - 1;
    const int64_t tL = 2 * k, tR = 2 * k + 1;
    const size_t CC = (size_t)C * C;
    // padding edges are exactly zero
    for (int64_t t = tL; t <= tR; ++t)
        if (t < E && t >= Eb) {
            float* o = a.marg + (size_t)(b * E + t) * CC;
            for (size_t idx = threadIdx.x; idx < CC; idx += kVecThreads) o[idx] = 0.f;
        }
    if (tL >= Eb) return;
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
        half_vec<kVec>(threadIdx.x < kHalfThreads, leafL, nullptr, nullptr, C, su, sw[0], sy[0],
                       red, raw[0]);
        if (threadIdx.x < kWave) {
            float m = -INFINITY, s = 0.f;
            for (int j = threadIdx.x; j < C; j += kWave) {
                float x[1] = {raw[0][j] + sv[j]};
                lse_fold<1>(m, s, x);
            }
            const float mm = wave_max(m);
            s = wave_sum(m == -INFINITY ? 0.f : s * fexp(m - safe_shift(mm)));
            if (threadIdx.x == 0) nrm[0] = lse_val(mm, s);
        }
        __syncthreads();
        write_marginal<kVec>(leafL, su, sv, nrm[0], C, outL);
        return;
    }
    const float* leafR = a.pot + (size_t)(b * E + tR) * CC;
    float* outR = a.marg + (size_t)(b * E + tR) * CC;
    // half 0: y = u (x) leaf_{2k} -> alpha_{2k+1} (sy[0]);  half 1: z = leaf_{2k+1} (x) v ->
    // beta_{2k+1} (sy[1]); raw[] keep the unshifted log-sum-exps
    const bool rowPass = threadIdx.x >= kHalfThreads;
    half_vec<kVec>(true, rowPass ? leafR : leafL, nullptr, nullptr, C, rowPass ? sv : su,
                   sw[rowPass], sy[rowPass], red, raw[rowPass]);
    // n_{2k} = LSE_j (y[j] + beta_{2k+1}[j]) (wave 0);  n_{2k+1} = LSE_i (alpha_{2k+1}[i] + z[i]) (wave 1)
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    if (w < 2) {
        float m = -INFINITY, s = 0.f;
        for (int j = lane; j < C; j += kWave) {
            float x[1] = {w == 0 ? raw[0][j] + sy[1][j] : sy[0][j] + raw[1][j]};
            lse_fold<1>(m, s, x);
        }
        const float mm = wave_max(m);
        s = wave_sum(m == -INFINITY ? 0.f : s * fexp(m - safe_shift(mm)));
        if (lane == 0) nrm[w] = lse_val(mm, s);
    }
    __syncthreads();
    write_marginal<kVec>(leafL, su, sy[1], nrm[0], C, outL);
    write_marginal<kVec>(leafR, sy[0], sv, nrm[1], C, outR);
}

template <int KP, bool VEC>
hipError_t up_sweep_kp(const Plan& p, const float* pot, const int32_t* lengths, hipStream_t s) {
    constexpr int LDA = KP + 4, LDB = kTile + 4;
    const size_t lds = sizeof(float) * (kTile * LDA + KP * LDB + 2 * KP + 2 * kTile) +
                       sizeof(double) * 4;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void*)k_up_log<KP, VEC>,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           160 * 1024);
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int64_t C = p.C;
    const int ntm = (int)((C + kTile - 1) / kTile);
    for (int l = 1; l <= p.D; ++l) {
        UpLogArgs a{};
        if (l == 1) {
            a.ccore = pot; a.cro = nullptr; a.cco = nullptr; a.cnodes = p.E;
        } else {
            a.ccore = p.core[l - 1]; a.cro = p.ro[l - 1]; a.cco = p.co[l - 1];
            a.cnodes = p.Np >> (l - 1);
        }
        a.core = p.core[l]; a.ro = p.ro[l]; a.co = p.co[l];
        a.nodes = p.Np >> l;
        a.lengths = lengths; a.B = p.B; a.N = p.N; a.C = C; a.level = l;
        a.ntm = ntm; a.kp = KP;
        a.nlogical = p.B * a.nodes * ntm * ntm;
        a.ngrid = round8(a.nlogical);
        hipLaunchKernelGGL((k_up_log<KP, VEC>), dim3((unsigned)a.ngrid), dim3(kUpThreads), lds, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t up_sweep(const Plan& p, const float* pot, const int32_t* lengths, hipStream_t s) {
    const bool vec = (p.C % 4) == 0;
    if (p.C <= 64) return vec ? up_sweep_kp<64, true>(p, pot, lengths, s) : up_sweep_kp<64, false>(p, pot, lengths, s);
    if (p.C <= 128) return vec ? up_sweep_kp<128, true>(p, pot, lengths, s) : up_sweep_kp<128, false>(p, pot, lengths, s);
    return vec ? up_sweep_kp<256, true>(p, pot, lengths, s) : up_sweep_kp<256, false>(p, pot, lengths, s);
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
    hipLaunchKernelGGL(k_root_log, dim3((unsigned)p.B), dim3(256), 0, s, r);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_logz_tree(const Plan& p, const float* pot, const int32_t* lengths,
                            float* logZ, hipStream_t s) {
    hipError_t e = up_sweep(p, pot, lengths, s);
    if (e != hipSuccess || !logZ) return e;
    return root(p, pot, lengths, logZ, s);
}

hipError_t launch_marginals_tree(const Plan& p, const float* pot, const int32_t* lengths,
                                 float* marg, hipStream_t s) {
    // (the up-sweep has been enqueued by the caller)
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
    f.lengths = lengths; f.N = p.N; f.C = p.C; f.marg = marg;
    const int64_t npairs = (p.N - 1 + 1) / 2;
    if (p.C % 4 == 0)
        hipLaunchKernelGGL(k_form_log<true>, dim3((unsigned)(p.B * npairs)), dim3(kVecThreads), 0, s, f);
    else
        hipLaunchKernelGGL(k_form_log<false>, dim3((unsigned)(p.B * npairs)), dim3(kVecThreads), 0, s, f);
    return hipGetLastError();
}

}  // namespace tsc
