// small.hip -- fused single-launch path for small label sets (C <= 32): one workgroup per
// sequence keeps that sequence's whole edge tree in LDS and runs, in one kernel,
//   log semiring: up-sweep of semiring matrix products (Sec. 6a / Fig. 3), root
//   log-sum-exp (log Z), outside sweep and per-edge marginals (Sec. 5.1 gradient identity);
//   max semiring: float64 up-sweep, forward scores, backpointers and the backtrace.
// The arithmetic is that of the multi-launch tree (tree_log.hip / tree_max.hip): node
// matrices P[a][c] = ro[a] + co[c] + core[a][c] with an exp-shifted fp32 MFMA product,
// and exact float64 max-plus for Viterbi.  Each product is computed by one wave.
//
// Tree bookkeeping for a sequence with E edges: level 0 holds the E leaves (staged from
// global memory into LDS); level l holds n_l = ceil(E / 2^l) nodes.  Node k of level l
// is a product of its two children when 2k+1 < n_{l-1} and otherwise equals its left
// child.  Products are stored in LDS slots numbered level by level.
//
// All LDS data is addressed as integer offsets into the one dynamic LDS array, so every
// access compiles to a ds_read/ds_write.
#include "device.h"
#include "internal.h"
#include "small.h"

namespace tsc {

extern __shared__ __align__(16) float ts_small_lds[];

namespace {

constexpr int kSmallThreads = 1024;  // 16 waves
constexpr int kSmallWaves = kSmallThreads / kWave;
constexpr float kUnderflow = 0x1p-80f;

typedef float f16v __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float& F(int off) { return ts_small_lds[off]; }
__device__ __forceinline__ double& Dd(int off_floats) {
    return reinterpret_cast<double*>(ts_small_lds)[off_floats >> 1];
}
__device__ __forceinline__ int align4(int off) { return (off + 3) & ~3; }
// values that are the same in every lane, moved to scalar registers
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ------------------------------------------------------------------ tree bookkeeping
struct Tree {
    int E, D;
    int n[kSmallMaxLevels + 1];      // nodes per level
    int pbase[kSmallMaxLevels + 1];  // first product slot of each level
    int vbase[kSmallMaxLevels + 1];  // first vector index of each level
    int nodes;                       // sum of n over all levels
    __device__ void init(int e) {
        E = e;
        D = 0;
        n[0] = e;
        pbase[0] = 0;
        vbase[0] = 0;
        int slots = 0, vec = e;
        while (n[D] > 1) {
            ++D;
            n[D] = (n[D - 1] + 1) / 2;
            pbase[D] = slots;
            vbase[D] = vec;
            slots += n[D - 1] / 2;
            vec += n[D];
        }
        nodes = vec;
    }
    __device__ int products(int l) const { return n[l - 1] / 2; }
    // >= 0: product slot; < 0: leaf -(h+1)
    __device__ int handle(int l, int k) const {
        while (l > 0) {
            if (k < products(l)) return pbase[l] + k;
            --l;
            k *= 2;
        }
        return -(k + 1);
    }
};

__device__ __forceinline__ void stage_leaves(const float* src, int dst, int n) {
    if ((((uintptr_t)src) & 15) == 0 && (n & 3) == 0) {
        const float4* s4 = (const float4*)src;
        float4* d4 = reinterpret_cast<float4*>(ts_small_lds + dst);
        for (int i = threadIdx.x; i < n / 4; i += blockDim.x) d4[i] = s4[i];
    } else {
        for (int i = threadIdx.x; i < n; i += blockDim.x) F(dst + i) = src[i];
    }
}

// ================================================================== log semiring
// LDS layout (float offsets): leaves [E][C][C] | slots [E-1][slotF] | vectors
// [nodes][2][C] (u then v) | per-wave scratch [16][128].  A slot holds core [C*C] (padded
// to a multiple of 2), then ro [C] and co [C] as doubles.
struct LogLayout {
    int C, CC, slotF, leaves, slots, vecs, scr;
    __device__ void init(int c, int E, int nodes) {
        C = c;
        CC = c * c;
        slotF = ((CC + 1) & ~1) + 4 * c;
        leaves = 0;
        slots = align4(E * CC);
        vecs = align4(slots + (E - 1) * slotF);
        scr = align4(vecs + nodes * 2 * c);
    }
    // a node: core offset and ro offset (-1 for a leaf: ro = co = 0)
    __device__ int core(int h) const { return h < 0 ? leaves + (-h - 1) * CC : slots + h * slotF; }
    __device__ int ro(int h) const { return h < 0 ? -1 : slots + h * slotF + ((CC + 1) & ~1); }
};

typedef float f4v __attribute__((ext_vector_type(4)));

// A team of TS waves computes P = L (x) R, the exp-shifted fp32 MFMA product, for
// C <= CP <= 32:
//   A'[a][b] = L[a][b] + (co_L[b] - max co_L), B'[b][c] = R[b][c] + (ro_R[b] - max ro_R)
//   S = sum_b exp(A' - rowmax) exp(B' - colmax); core_P = log S (exact fallback when S
//   underflows), ro_P = ro_L + max co_L + rowmax, co_P = co_R + max ro_R + colmax.
// The output is cut into 16 x 16 blocks (one for CP <= 16, four for CP = 32); team member
// `mem` computes blocks mem, mem + TS, ... with v_mfma_f32_16x16x4f32.  Every member
// derives the shifts and row/column maxima itself (same inputs, same results), so the team
// needs no synchronisation.  The offset shifts only need to be near the maximum, so they
// are reduced in fp32.
template <int CP, int TS>
__device__ __attribute__((noinline)) void team_product_log(const LogLayout& ly, int Lc, int Lro, int Rc, int Rro, int Pc,
                                 int Pro, int mem, int scr) {
    constexpr int kNB = CP <= 16 ? 1 : 4;      // 16 x 16 output blocks
    const int C = uni(ly.C);
    Lc = uni(Lc); Lro = uni(Lro); Rc = uni(Rc); Rro = uni(Rro); Pc = uni(Pc); Pro = uni(Pro);
    mem = uni(mem); scr = uni(scr);
    const int lane = threadIdx.x % kWave;
    const int coh = scr, roh = scr + 32, rA = scr + 64, cB = scr + 96;
    double lm = -INFINITY, rm = -INFINITY;
    if (lane < C) {
        if (Lro >= 0) lm = Dd(Lro + 2 * C + 2 * lane);   // co_L[lane]
        if (Rro >= 0) rm = Dd(Rro + 2 * lane);           // ro_R[lane]
    }
    const double coLs = Lro >= 0 ? (double)safe_shift(wave_max_fast((float)lm)) : 0.0;
    const double roRs = Rro >= 0 ? (double)safe_shift(wave_max_fast((float)rm)) : 0.0;
    if (lane < 32) {
        F(coh + lane) = (lane < C && Lro >= 0) ? (float)(lm - coLs) : 0.f;
        F(roh + lane) = (lane < C && Rro >= 0) ? (float)(rm - roRs) : 0.f;
    }
    wave_sync();
    // lanes 0-31: maxima of the rows of A'; lanes 32-63: maxima of the columns of B'
    {
        const int i = lane & 31, h = lane >> 5;
        const int ic = min(i, C - 1);
        const int base = h == 0 ? Lc + ic * C : Rc + ic;
        const int stride = h == 0 ? 1 : C;
        const int add = h == 0 ? coh : roh;
        float m = -INFINITY;
#pragma unroll
        for (int k = 0; k < CP; ++k)
            if (k < C) m = fmaxf(m, F(base + k * stride) + F(add + k));
        F((h == 0 ? rA : cB) + i) = (i < C) ? m : -INFINITY;
    }
    wave_sync();
    const int l16 = lane & 15, kq = lane >> 4;
#pragma unroll
    for (int blk = mem; blk < kNB; blk += TS) {
        const int r0 = (blk >> 1) * 16, c0 = (blk & 1) * 16;
        const int ia = r0 + l16, jb = c0 + l16;
        const int iac = min(ia, C - 1), jbc = min(jb, C - 1);
        const float sa = safe_shift(F(rA + iac)), sb = safe_shift(F(cB + jbc));
        f4v acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < CP; kk += 4) {
            if (kk < C) {
                const int k = kk + kq;
                const int kc = min(k, C - 1);
                const float ea = __expf(F(Lc + iac * C + kc) + F(coh + kc) - sa);
                const float eb = __expf(F(Rc + kc * C + jbc) + F(roh + kc) - sb);
                const bool ka = k < C;
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32((ka && ia < C) ? ea : 0.f,
                                                           (ka && jb < C) ? eb : 0.f, acc, 0, 0, 0);
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = r0 + 4 * kq + r, col = jb;
            if (row < C && col < C) {
                const float S = acc[r];
                float val;
                if (S >= kUnderflow) {
                    val = __logf(S);
                } else {
                    const float ra = safe_shift(F(rA + row)), cb = safe_shift(F(cB + col));
                    float q = -INFINITY;
                    for (int k = 0; k < C; ++k)
                        q = fmaxf(q, (F(Lc + row * C + k) + F(coh + k) - ra) +
                                         (F(Rc + k * C + col) + F(roh + k) - cb));
                    if (q == -INFINITY) {
                        val = -INFINITY;
                    } else {
                        float s = 0.f;
                        for (int k = 0; k < C; ++k)
                            s += __expf((F(Lc + row * C + k) + F(coh + k) - ra) +
                                        (F(Rc + k * C + col) + F(roh + k) - cb) - q);
                        val = q + __logf(s);
                    }
                }
                F(Pc + row * C + col) = val;
            }
        }
    }
    if (mem == 0 && lane < C) {
        Dd(Pro + 2 * lane) =
            (Lro >= 0 ? Dd(Lro + 2 * lane) : 0.0) + coLs + (double)safe_shift(F(rA + lane));
        Dd(Pro + 2 * C + 2 * lane) =
            (Rro >= 0 ? Dd(Rro + 2 * C + 2 * lane) : 0.0) + roRs + (double)safe_shift(F(cB + lane));
    }
    wave_sync();
}

// team size for a level with np products on kSmallWaves waves: the largest power of two
// <= waves / np, at most 4
__device__ __forceinline__ int team_size(int np) {
    const int per = kSmallWaves / max(np, 1);
    return per >= 4 ? 4 : (per >= 2 ? 2 : 1);
}

// One wave, C <= CP <= 32.  kRowSide == false: y[j] = LSE_i x[i] + N[i][j]  (y = x (x) N);
// kRowSide == true: y[i] = LSE_j N[i][j] + x[j]  (y = N (x) x).  y is shifted to max 0.
template <int CP, bool kRowSide>
__device__ void wave_vec_log(const LogLayout& ly, int x, int Nc, int Nro, int y, int scr) {
    const int C = ly.C;
    const int lane = threadIdx.x % kWave;
    // x on the left pairs with ro and the result picks up co; on the right the reverse
    const int inOff = kRowSide ? 2 * C : 0, outOff = kRowSide ? 0 : 2 * C;
    double w = -INFINITY;
    if (lane < C) w = (double)F(x + lane) + (Nro >= 0 ? Dd(Nro + inOff + 2 * lane) : 0.0);
    const double ws = (double)safe_shift(wave_max_fast((float)w));
    if (lane < C) F(scr + lane) = (w == -INFINITY) ? -INFINITY : (float)(w - ws);
    wave_sync();
    double z = -INFINITY;
    {
        const int lc = min(lane, C - 1);
        float e[CP];
        float m = -INFINITY;
#pragma unroll
        for (int t = 0; t < CP; ++t) {
            e[t] = -INFINITY;
            if (t < C) {
                e[t] = F(scr + t) + (kRowSide ? F(Nc + lc * C + t) : F(Nc + t * C + lc));
                m = fmaxf(m, e[t]);
            }
        }
        if (m != -INFINITY && lane < C) {
            float s = 0.f;
#pragma unroll
            for (int t = 0; t < CP; ++t) s += __expf(e[t] - m);
            z = (Nro >= 0 ? Dd(Nro + outOff + 2 * lane) : 0.0) + (double)(m + __logf(s));
        }
    }
    const double zs = (double)safe_shift(wave_max_fast((float)z));
    if (lane < C) F(y + lane) = (z == -INFINITY) ? -INFINITY : (float)(z - zs);
    wave_sync();
}

struct SmallLogArgs {
    const float* pot;
    const int32_t* lengths;
    int64_t N;
    int C;
    float* logZ;      // nullable
    float* marg;      // nullable: log Z only
};

template <int CP>
__global__ __launch_bounds__(kSmallThreads) void k_small_log(SmallLogArgs a) {
    const int64_t b = blockIdx.x;
    const int C = a.C;
    const int64_t E = a.N - 1;
    const int Eb = (int)(clamp_len(a.lengths, b, a.N) - 1);
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int CC = C * C;
    if (a.marg) {  // padding edges are exactly zero
        float* mz = a.marg + ((size_t)b * E + Eb) * CC;
        const size_t nz = (size_t)(E - Eb) * CC;
        for (size_t idx = threadIdx.x; idx < nz; idx += kSmallThreads) mz[idx] = 0.f;
    }
    if (Eb == 0) {
        if (a.logZ && threadIdx.x == 0) a.logZ[b] = logf((float)C);
        return;
    }
    __shared__ Tree T;
    if (threadIdx.x == 0) T.init(Eb);
    stage_leaves(a.pot + (size_t)b * E * CC, 0, Eb * CC);
    __syncthreads();
    LogLayout ly;
    ly.init(C, Eb, T.nodes);
    const int scr = ly.scr + w * 128;

    // ---- up-sweep
    for (int l = 1; l <= T.D; ++l) {
        const int np = T.products(l);
        const int ts = team_size(np), nteams = kSmallWaves / ts;
        const int team = w / ts, mem = w % ts;
        for (int k = team; k < np; k += nteams) {
            const int hl = T.handle(l - 1, 2 * k), hr = T.handle(l - 1, 2 * k + 1);
            const int s = T.pbase[l] + k;
            const int Lc = ly.core(hl), Lro = ly.ro(hl), Rc = ly.core(hr), Rro = ly.ro(hr);
            if (ts == 4) team_product_log<CP, 4>(ly, Lc, Lro, Rc, Rro, ly.core(s), ly.ro(s), mem, scr);
            else if (ts == 2) team_product_log<CP, 2>(ly, Lc, Lro, Rc, Rro, ly.core(s), ly.ro(s), mem, scr);
            else team_product_log<CP, 1>(ly, Lc, Lro, Rc, Rro, ly.core(s), ly.ro(s), mem, scr);
        }
        __syncthreads();
    }
    // ---- root: log Z = LSE_{a,c} ro[a] + co[c] + core[a][c]
    const int hroot = T.handle(T.D, 0);
    if (a.logZ && w == 0) {
        const int rc = ly.core(hroot), rr = ly.ro(hroot);
        double rm = -INFINITY, cm = -INFINITY;
        if (lane < C) {
            rm = rr >= 0 ? Dd(rr + 2 * lane) : 0.0;
            cm = rr >= 0 ? Dd(rr + 2 * C + 2 * lane) : 0.0;
        }
        const double rs = (double)safe_shift(wave_max_fast((float)rm));
        const double cs = (double)safe_shift(wave_max_fast((float)cm));
        float m = -INFINITY;
        for (int idx = lane; idx < CC; idx += kWave) {
            const int i = idx / C, j = idx % C;
            float x = F(rc + idx);
            if (rr >= 0) x += (float)(Dd(rr + 2 * i) - rs) + (float)(Dd(rr + 2 * C + 2 * j) - cs);
            m = fmaxf(m, x);
        }
        m = wave_max_fast(m);
        float s = 0.f;
        if (m != -INFINITY)
            for (int idx = lane; idx < CC; idx += kWave) {
                const int i = idx / C, j = idx % C;
                float x = F(rc + idx);
                if (rr >= 0) x += (float)(Dd(rr + 2 * i) - rs) + (float)(Dd(rr + 2 * C + 2 * j) - cs);
                s += __expf(x - m);
            }
        s = wave_sum_fast(s);
        if (lane == 0)
            a.logZ[b] = (m == -INFINITY) ? -INFINITY : (float)(rs + cs + (double)(m + __logf(s)));
    }
    if (!a.marg) return;
    // ---- outside sweep: u, v of every node (root: zeros)
    auto U = [&](int l, int k) { return ly.vecs + (T.vbase[l] + k) * 2 * C; };
    for (int idx = threadIdx.x; idx < 2 * C; idx += kSmallThreads) F(U(T.D, 0) + idx) = 0.f;
    __syncthreads();
    for (int l = T.D; l >= 1; --l) {
        const int nn = T.n[l];
        for (int task = w; task < 3 * nn; task += kSmallWaves) {
            const int k = task / 3, which = task % 3;
            const bool right = 2 * k + 1 < T.n[l - 1];
            const int uN = U(l, k), vN = uN + C;
            if (which == 0) {
                if (lane < C) {
                    F(U(l - 1, 2 * k) + lane) = F(uN + lane);
                    if (right) F(U(l - 1, 2 * k + 1) + C + lane) = F(vN + lane);
                    else F(U(l - 1, 2 * k) + C + lane) = F(vN + lane);
                }
            } else if (which == 1 && right) {   // u_R = u_N (x) L
                const int hl = T.handle(l - 1, 2 * k);
                wave_vec_log<CP, false>(ly, uN, ly.core(hl), ly.ro(hl), U(l - 1, 2 * k + 1), scr);
            } else if (which == 2 && right) {   // v_L = R (x) v_N
                const int hr = T.handle(l - 1, 2 * k + 1);
                wave_vec_log<CP, true>(ly, vN, ly.core(hr), ly.ro(hr), U(l - 1, 2 * k) + C, scr);
            }
        }
        __syncthreads();
    }
    // ---- marginals with a per-edge normaliser n_t
    // lane -> column j = lane & 31 and rows (lane >> 5) + 2q: no integer division, every
    // lane runs the same (clamped, in-bounds) loads; entries past C are masked
    constexpr int kPer = CP / 2;
    const int j = lane & 31, i0 = lane >> 5, jc = min(j, C - 1);
    for (int t = w; t < Eb; t += kSmallWaves) {
        const int al = U(0, t), be = al + C, leaf = ly.leaves + t * CC;
        const float bj = F(be + jc);
        float x[kPer];
        float m = -INFINITY;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int i = i0 + 2 * q, ic = min(i, C - 1);
            const float v = F(al + ic) + F(leaf + ic * C + jc) + bj;
            x[q] = (i < C && j < C) ? v : -INFINITY;
            m = fmaxf(m, x[q]);
        }
        m = wave_max_fast(m);
        float s = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int q = 0; q < kPer; ++q) s += __expf(x[q] - m);
        }
        s = wave_sum_fast(s);
        const float n = (m == -INFINITY) ? -INFINITY : m + __logf(s);
        float* out = a.marg + ((size_t)b * E + t) * CC;
#pragma unroll
        for (int q = 0; q < kPer; ++q) {
            const int i = i0 + 2 * q;
            if (i < C && j < C) out[i * C + j] = (n == -INFINITY) ? 0.f : __expf(x[q] - n);
        }
    }
}

// ================================================================== max semiring
// LDS layout (float offsets): leaves fp32 [E][C][C] | slots fp64 [E-1][C][C] | forward
// scores fp64 [nodes][C] | last scores fp64 [C] | backpointers u8 [E][C].
struct MaxLayout {
    int C, CC, leaves, slots, vecs, dlast, bp;
    __device__ void init(int c, int E, int nodes) {
        C = c;
        CC = c * c;
        leaves = 0;
        slots = align4(E * CC);
        vecs = slots + (E - 1) * CC * 2;
        dlast = vecs + nodes * c * 2;
        bp = dlast + 2 * c;
    }
};

// element idx of a node: a leaf in fp32 or a product slot in fp64
template <bool kLeaf>
__device__ __forceinline__ double mx(int base, int idx) {
    if constexpr (kLeaf) return (double)F(base + idx);
    else return Dd(base + 2 * idx);
}

// A team of TS waves computes P = L (x) R in (max, +), float64.  Member `mem` owns
// columns [mem*CP/TS, (mem+1)*CP/TS); within it lane (r = lane & 31, g = lane >> 5)
// computes row r on one half of that window.  Indices are clamped into the matrix so that
// every lane runs the same loads; rows and columns past C are never stored.
template <int CP, int TS, bool kLL, bool kRL>
__device__ __attribute__((noinline)) void team_product_max(int C, int Lb, int Rb, int Pb, int mem) {
    constexpr int kW = CP / TS, kH = kW > 1 ? kW / 2 : 1;   // columns per member / per lane
    constexpr int kT = kH < 4 ? kH : 4;                     // columns per lane per pass
    C = uni(C); Lb = uni(Lb); Rb = uni(Rb); Pb = uni(Pb); mem = uni(mem);
    const int lane = threadIdx.x % kWave;
    const int r = lane & 31, g = lane >> 5;
    const int c0 = mem * kW + (kW > 1 ? g * kH : 0);
    const bool active = (kW > 1 || g == 0) && r < C;
    const int rr = min(r, C - 1);
#pragma unroll
    for (int p0 = 0; p0 < kH; p0 += kT) {
        int cc[kT];
        double acc[kT];
#pragma unroll
        for (int m = 0; m < kT; ++m) {
            cc[m] = min(c0 + p0 + m, C - 1);
            acc[m] = -INFINITY;
        }
        // the loop runs over the padded size with no branch; terms past C are -inf
#pragma unroll 4
        for (int q = 0; q < CP; ++q) {
            const int qc = min(q, C - 1);
            const double x = q < C ? mx<kLL>(Lb, rr * C + qc) : -INFINITY;
#pragma unroll
            for (int m = 0; m < kT; ++m) acc[m] = fmax(acc[m], x + mx<kRL>(Rb, qc * C + cc[m]));
        }
        if (active) {
#pragma unroll
            for (int m = 0; m < kT; ++m)
                if (p0 + m < kH && c0 + p0 + m < C) Dd(Pb + 2 * (r * C + c0 + p0 + m)) = acc[m];
        }
    }
    wave_sync();
}

template <int CP, int TS>
__device__ __forceinline__ void team_product_max_any(int C, int hl, int hr, int Lb, int Rb, int Pb,
                                                     int mem) {
    if (hl < 0 && hr < 0) team_product_max<CP, TS, true, true>(C, Lb, Rb, Pb, mem);
    else if (hl < 0) team_product_max<CP, TS, true, false>(C, Lb, Rb, Pb, mem);
    else if (hr < 0) team_product_max<CP, TS, false, true>(C, Lb, Rb, Pb, mem);
    else team_product_max<CP, TS, false, false>(C, Lb, Rb, Pb, mem);
}

// One wave: y[j] = max_i x[i] + N[i][j]  (float64)
template <int CP, bool kLeaf>
__device__ void wave_vec_max(int C, int x, int Nb, int y) {
    const int lane = threadIdx.x % kWave;
    const int j = min(lane, C - 1);
    double m = -INFINITY;
#pragma unroll
    for (int i = 0; i < CP; ++i)
        if (i < C) m = fmax(m, Dd(x + 2 * i) + mx<kLeaf>(Nb, i * C + j));
    if (lane < C) Dd(y + 2 * lane) = m;
    wave_sync();
}

struct SmallMaxArgs {
    const float* pot;
    const int32_t* lengths;
    int64_t N;
    int C;
    int32_t* path;
    float* score;
};

template <int CP>
__global__ __launch_bounds__(kSmallThreads) void k_small_max(SmallMaxArgs a) {
    const int64_t b = blockIdx.x;
    const int C = a.C;
    const int64_t E = a.N - 1;
    const int L = (int)clamp_len(a.lengths, b, a.N), Eb = L - 1;
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int CC = C * C;
    int32_t* path = a.path + (size_t)b * a.N;
    for (int64_t n = L + threadIdx.x; n < a.N; n += kSmallThreads) path[n] = -1;
    if (Eb == 0) {
        if (threadIdx.x == 0) { path[0] = 0; a.score[b] = 0.f; }
        return;
    }
    __shared__ Tree T;
    if (threadIdx.x == 0) T.init(Eb);
    stage_leaves(a.pot + (size_t)b * E * CC, 0, Eb * CC);
    __syncthreads();
    MaxLayout ly;
    ly.init(C, Eb, T.nodes);
    auto base = [&](int h) { return h < 0 ? ly.leaves + (-h - 1) * CC : ly.slots + h * CC * 2; };
    // ---- up-sweep
    for (int l = 1; l <= T.D; ++l) {
        const int np = T.products(l);
        const int ts = team_size(np), nteams = kSmallWaves / ts;
        const int team = w / ts, mem = w % ts;
        for (int k = team; k < np; k += nteams) {
            const int hl = T.handle(l - 1, 2 * k), hr = T.handle(l - 1, 2 * k + 1);
            const int Pb = ly.slots + (T.pbase[l] + k) * CC * 2;
            if (ts == 4) team_product_max_any<CP, 4>(C, hl, hr, base(hl), base(hr), Pb, mem);
            else if (ts == 2) team_product_max_any<CP, 2>(C, hl, hr, base(hl), base(hr), Pb, mem);
            else team_product_max_any<CP, 1>(C, hl, hr, base(hl), base(hr), Pb, mem);
        }
        __syncthreads();
    }
    // ---- forward scores: u_L = u_N, u_R = u_N (x) L
    auto U = [&](int l, int k) { return ly.vecs + (T.vbase[l] + k) * 2 * C; };
    for (int i = threadIdx.x; i < C; i += kSmallThreads) Dd(U(T.D, 0) + 2 * i) = 0.0;
    __syncthreads();
    for (int l = T.D; l >= 1; --l) {
        const int nn = T.n[l];
        for (int task = w; task < 2 * nn; task += kSmallWaves) {
            const int k = task / 2, which = task % 2;
            const int uN = U(l, k);
            if (which == 0) {
                if (lane < C) Dd(U(l - 1, 2 * k) + 2 * lane) = Dd(uN + 2 * lane);
            } else if (2 * k + 1 < T.n[l - 1]) {
                const int hl = T.handle(l - 1, 2 * k);
                if (hl < 0) wave_vec_max<CP, true>(C, uN, base(hl), U(l - 1, 2 * k + 1));
                else wave_vec_max<CP, false>(C, uN, base(hl), U(l - 1, 2 * k + 1));
            }
        }
        __syncthreads();
    }
    // ---- backpointers: bp[t][j] = lowest argmax_i delta_t[i] + l[t][i][j]
    uint8_t* bp = reinterpret_cast<uint8_t*>(ts_small_lds + ly.bp);
    for (int t = w; t < Eb; t += kSmallWaves) {
        const int d = U(0, t), leaf = ly.leaves + t * CC;
        const int j = min(lane, C - 1);
        double best = Dd(d) + (double)F(leaf + j);
        int arg = 0;
#pragma unroll
        for (int i = 1; i < CP; ++i) {
            if (i < C) {
                const double v = Dd(d + 2 * i) + (double)F(leaf + i * C + j);
                const bool better = v > best;
                best = better ? v : best;
                arg = better ? i : arg;
            }
        }
        if (lane < C) {
            bp[t * C + lane] = (uint8_t)arg;
            if (t == Eb - 1) Dd(ly.dlast + 2 * lane) = best;
        }
    }
    __syncthreads();
    // ---- last label (lowest argmax), score, backtrace
    if (w == 0) {
        double best = lane < C ? Dd(ly.dlast + 2 * lane) : -INFINITY;
        int arg = lane < C ? lane : 0x7fffffff;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const double ov = __shfl_xor(best, o, kWave);
            const int oi = __shfl_xor(arg, o, kWave);
            if (ov > best || (ov == best && oi < arg)) { best = ov; arg = oi; }
        }
        if (lane == 0) {
            int z = arg < C ? arg : 0;
            a.score[b] = (float)best;
            path[Eb] = z;
            for (int t = Eb - 1; t >= 0; --t) {
                z = bp[t * C + z];
                path[t] = z;
            }
        }
    }
}

}  // namespace

// Both layouts are sized for the longest sequence (E = N-1 edges); a shorter sequence
// uses a prefix of each region, so the offsets computed in the kernels stay inside.
size_t small_log_lds_bytes(int64_t E, int64_t C) {
    if (E < 1) return 0;
    const int64_t CC = C * C, slotF = ((CC + 1) & ~1) + 4 * C;
    const int64_t floats = (E * CC + 3) + ((E - 1) * slotF + 3) +
                           (small_tree_nodes(E) * 2 * C + 3) + kSmallWaves * 128;
    return sizeof(float) * (size_t)floats;
}

size_t small_max_lds_bytes(int64_t E, int64_t C) {
    if (E < 1) return 0;
    const int64_t CC = C * C;
    const int64_t floats = (E * CC + 3) + (E - 1) * CC * 2 + small_tree_nodes(E) * C * 2 + 2 * C;
    return sizeof(float) * (size_t)floats + (size_t)(E * C);
}

bool small_path_fits(int64_t N, int64_t C) {
    const int64_t E = N - 1;
    if (C > kSmallMaxLabels || E < 1 || E > kSmallMaxEdges) return false;
    return small_log_lds_bytes(E, C) <= kSmallLdsBytes &&
           small_max_lds_bytes(E, C) <= kSmallLdsBytes;
}

namespace {

template <class K>
hipError_t allow_lds(K kernel) {
    return hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                               kSmallLdsBytes);
}

template <int CP>
hipError_t small_log_cp(const SmallLogArgs& a, int64_t B, size_t lds, hipStream_t s) {
    static bool attr = false;
    if (!attr) {
        hipError_t e = allow_lds(k_small_log<CP>);
        if (e != hipSuccess) return e;
        attr = true;
    }
    hipLaunchKernelGGL(k_small_log<CP>, dim3((unsigned)B), dim3(kSmallThreads), lds, s, a);
    return hipGetLastError();
}

template <int CP>
hipError_t small_max_cp(const SmallMaxArgs& a, int64_t B, size_t lds, hipStream_t s) {
    static bool attr = false;
    if (!attr) {
        hipError_t e = allow_lds(k_small_max<CP>);
        if (e != hipSuccess) return e;
        attr = true;
    }
    hipLaunchKernelGGL(k_small_max<CP>, dim3((unsigned)B), dim3(kSmallThreads), lds, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_small_log(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                            int64_t C, float* logZ, float* marg, hipStream_t s) {
    SmallLogArgs a{pot, lengths, N, (int)C, logZ, marg};
    const size_t lds = small_log_lds_bytes(N - 1, C);
    if (C <= 8) return small_log_cp<8>(a, B, lds, s);
    if (C <= 16) return small_log_cp<16>(a, B, lds, s);
    if (C <= 24) return small_log_cp<24>(a, B, lds, s);
    return small_log_cp<32>(a, B, lds, s);
}

hipError_t launch_small_max(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                            int64_t C, int32_t* path, float* score, hipStream_t s) {
    SmallMaxArgs a{pot, lengths, N, (int)C, path, score};
    const size_t lds = small_max_lds_bytes(N - 1, C);
    if (C <= 8) return small_max_cp<8>(a, B, lds, s);
    if (C <= 16) return small_max_cp<16>(a, B, lds, s);
    if (C <= 24) return small_max_cp<24>(a, B, lds, s);
    return small_max_cp<32>(a, B, lds, s);
}

}  // namespace tsc
