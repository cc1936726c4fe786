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

// coalesced copy of a sequence's valid edges into LDS, several loads in flight per thread
__device__ __forceinline__ void stage_leaves(const float* src, int dst, int n) {
    const int tid = threadIdx.x, nt = blockDim.x;
    if ((((uintptr_t)src) & 15) == 0 && (n & 3) == 0 && (dst & 3) == 0) {
        const float4* s4 = (const float4*)src;
        float4* d4 = reinterpret_cast<float4*>(ts_small_lds + dst);
        const int n4 = n / 4;
        for (int base = 0; base < n4; base += 4 * nt) {
            float4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = s4[min(base + u * nt + tid, n4 - 1)];
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (base + u * nt + tid < n4) d4[base + u * nt + tid] = v[u];
        }
    } else {
        for (int base = 0; base < n; base += 8 * nt) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = src[min(base + u * nt + tid, n - 1)];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (base + u * nt + tid < n) F(dst + base + u * nt + tid) = v[u];
        }
    }
}

typedef float f4v __attribute__((ext_vector_type(4)));

// team size for a level with np products on kSmallWaves waves: the largest power of two
// <= waves / np, at most 4
__device__ __forceinline__ int team_size(int np) {
    const int per = kSmallWaves / max(np, 1);
    return per >= 4 ? 4 : (per >= 2 ? 2 : 1);
}

// ================================================================== log semiring
// Every node is kept in the form its consumer needs, so a product needs only exp + MFMA:
//   LEFT operand  (left child of a product):  P[a][b] = ro[a] + core[a][b], max_b core[a][b] = 0
//   RIGHT operand (right child of a product): P[b][c] = co[c] + core[b][c], max_b core[b][c] = 0
//   NONE (the root): P[a][c] = ro[a] + co[c] + core[a][c]
// (an absent right child makes a node equal to its left child, so a node takes the role
// of its first ancestor that is consumed; the root is consumed by the log-sum-exp).
// For P = L (x) R with L in LEFT and R in RIGHT form:
//   S[a][c] = sum_b exp(core_L[a][b]) exp(core_R[b][c])     (fp32 MFMA, every factor <= 1)
//   P[a][c] = ro_L[a] + co_R[c] + log S[a][c]
// and the producer then normalises P into the form of its own role.  S < 2^-80 (all
// terms underflowed) is recomputed exactly by a direct max-shifted log-sum-exp over b.
//
// LDS layout (float offsets): slots [2E-1][slotF] (leaves are slots 0..E-1, products
// follow level by level) | vectors [nodes][2][C] (u then v).  A slot holds core [C*C]
// (padded to a multiple of 4), then ro [C] and co [C] as doubles.
constexpr int kLeft = 0, kRight = 1, kNone = 2;

__device__ __forceinline__ int node_role(const Tree& T, int l, int k) {
    while (l < T.D) {
        if (k & 1) return kRight;
        if (k + 1 < T.n[l]) return kLeft;
        ++l;
        k >>= 1;
    }
    return kNone;
}

struct LogLayout {
    int C, CC, slotF, coreF, vecs;
    __device__ void init(int c, int E) {
        C = c;
        CC = c * c;
        coreF = align4(CC);
        slotF = coreF + 4 * c;
        vecs = (2 * E - 1) * slotF;
    }
    __device__ int core(int slot) const { return slot * slotF; }
    __device__ int ro(int slot) const { return slot * slotF + coreF; }   // doubles: ro, then co
    __device__ int co(int slot) const { return slot * slotF + coreF + 2 * C; }
};

// slot of node (l, k): leaves are slots 0..E-1, products E + pbase[l] + k
__device__ __forceinline__ int log_slot(const Tree& T, int l, int k) {
    const int h = T.handle(l, k);
    return h < 0 ? (-h - 1) : T.E + h;
}

// Product of the LEFT node at slot sl and the RIGHT node at slot sr into slot sp, in the
// form kRole.  Output blocks are 16 x 16 (v_mfma_f32_16x16x4f32): one block for CP <= 16
// (member 0 only), four for CP > 16 shared by two waves -- by block rows when the result is
// normalised per row (LEFT, NONE) and by block columns when per column (RIGHT), so each
// wave holds whole rows (or columns) of what it normalises.
template <int CP, int kRole>
__device__ __forceinline__ void prod_log(const LogLayout& ly, int sl, int sr, int sp, int m) {
    constexpr bool kTwo = CP > 16;
    constexpr bool kColSplit = kTwo && kRole == kRight;
    constexpr int kSteps = CP / 4;
    const int C = ly.C;
    const int Lc = ly.core(sl), Lro = ly.ro(sl);
    const int Rc = ly.core(sr), Rco = ly.co(sr);
    const int Pc = ly.core(sp), Pro = ly.ro(sp), Pco = ly.co(sp);
    const int lane = threadIdx.x % kWave, l16 = lane & 15, kq = lane >> 4;
    const int rb0 = kTwo ? (kColSplit ? 0 : 16 * m) : 0, cb0 = kColSplit ? 16 * m : 0;
    const int rb1 = kColSplit ? 16 : rb0, cb1 = kColSplit ? cb0 : 16;
    const int ia0 = rb0 + l16, ia1 = rb1 + l16, jb0 = cb0 + l16, jb1 = cb1 + l16;
    // row / column base offsets (clamped into the matrix; masked below)
    const int arow0 = Lc + min(ia0, C - 1) * C, arow1 = Lc + min(ia1, C - 1) * C;
    const int bcol0 = Rc + min(jb0, C - 1), bcol1 = Rc + min(jb1, C - 1);
    float av[kSteps], bv[kSteps], cv[kSteps];
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
        const int kc = min(4 * st + kq, C - 1);
        av[st] = F(arow0 + kc);
        bv[st] = F(bcol0 + kc * C);
        if (kTwo) cv[st] = kColSplit ? F(arow1 + kc) : F(bcol1 + kc * C);
    }
    f4v acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    const bool a0ok = ia0 < C, b0ok = jb0 < C, c1ok = kColSplit ? ia1 < C : jb1 < C;
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
        const bool kv = 4 * st + kq < C;
        const float a0 = (kv && a0ok) ? fexp(av[st]) : 0.f;
        const float b0 = (kv && b0ok) ? fexp(bv[st]) : 0.f;
        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0, acc0, 0, 0, 0);
        if (kTwo) {
            const float c = (kv && c1ok) ? fexp(cv[st]) : 0.f;
            if (kColSplit) acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(c, b0, acc1, 0, 0, 0);
            else acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, c, acc1, 0, 0, 0);
        }
    }
    // log S; lane-held entries: block X rows rbX + 4 kq + r, column cbX + l16
    constexpr int kB = kTwo ? 2 : 1;
    float ls[kB][4];
    bool need = false;
#pragma unroll
    for (int x = 0; x < kB; ++x)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float S = x ? acc1[r] : acc0[r];
            const int row = (x ? rb1 : rb0) + 4 * kq + r, col = x ? jb1 : jb0;
            ls[x][r] = flog(S);
            need |= row < C && col < C && !(S >= kUnderflow);
        }
    if (need) {   // some entry underflowed (or is padding): exact recomputation
#pragma unroll
        for (int x = 0; x < kB; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = (x ? rb1 : rb0) + 4 * kq + r, col = x ? jb1 : jb0;
                const float S = x ? acc1[r] : acc0[r];
                if (!(S >= kUnderflow) && row < C && col < C) {
                    float q = -INFINITY;
                    for (int k = 0; k < C; ++k) q = fmaxf(q, F(Lc + row * C + k) + F(Rc + k * C + col));
                    float v = -INFINITY;
                    if (q != -INFINITY) {
                        float s = 0.f;
                        for (int k = 0; k < C; ++k) s += fexp(F(Lc + row * C + k) + F(Rc + k * C + col) - q);
                        v = q + flog(s);
                    }
                    ls[x][r] = v;
                }
            }
    }
    const int lc = min(lane, C - 1);
    if constexpr (kRole == kLeft) {
        // P[a][c] = ro_L[a] + co_R[c] + log S: fold co_R (shifted) in, then shift each row to max 0
        const float mco = safe_shift(wave_max_fast(lane < C ? (float)Dd(Rco + 2 * lc) : -INFINITY));
        float coh[kB];
        coh[0] = (float)(Dd(Rco + 2 * min(jb0, C - 1)) - (double)mco);
        if (kTwo) coh[kB - 1] = (float)(Dd(Rco + 2 * min(jb1, C - 1)) - (double)mco);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = rb0 + 4 * kq + r;
            float x0 = b0ok ? ls[0][r] + coh[0] : -INFINITY;
            float x1 = (kTwo && jb1 < C) ? ls[kB - 1][r] + coh[kB - 1] : -INFINITY;
            float mx = fmaxf(x0, x1);
            mx = fmaxf(mx, dpp_f(mx, 0xB1));
            mx = fmaxf(mx, dpp_f(mx, 0x4E));
            mx = fmaxf(mx, dpp_f(mx, 0x141));
            mx = fmaxf(mx, dpp_f(mx, 0x140));
            const float sh = safe_shift(mx);
            if (row < C) {
                if (b0ok) F(Pc + row * C + jb0) = x0 - sh;
                if (kTwo && jb1 < C) F(Pc + row * C + jb1) = x1 - sh;
                if (l16 == 0) Dd(Pro + 2 * row) = Dd(Lro + 2 * row) + (double)mco + (double)sh;
            }
        }
        if (m == 0 && lane < C) Dd(Pco + 2 * lane) = 0.0;
    } else if constexpr (kRole == kRight) {
        // fold ro_L (shifted) in, then shift each column to max 0
        const float mro = safe_shift(wave_max_fast(lane < C ? (float)Dd(Lro + 2 * lc) : -INFINITY));
        float xs[kB][4];
        float mx = -INFINITY;
#pragma unroll
        for (int x = 0; x < kB; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = (x ? rb1 : rb0) + 4 * kq + r;
                const float roh = (float)(Dd(Lro + 2 * min(row, C - 1)) - (double)mro);
                xs[x][r] = row < C ? ls[x][r] + roh : -INFINITY;
                mx = fmaxf(mx, xs[x][r]);
            }
        mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
        mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
        const float sh = safe_shift(mx);
        if (b0ok) {
#pragma unroll
            for (int x = 0; x < kB; ++x)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int row = (x ? rb1 : rb0) + 4 * kq + r;
                    if (row < C) F(Pc + row * C + jb0) = xs[x][r] - sh;
                }
            if (kq == 0) Dd(Pco + 2 * jb0) = Dd(Rco + 2 * jb0) + (double)mro + (double)sh;
        }
        if (m == 0 && lane < C) Dd(Pro + 2 * lane) = 0.0;
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = rb0 + 4 * kq + r;
            if (row < C) {
                if (b0ok) F(Pc + row * C + jb0) = ls[0][r];
                if (kTwo && jb1 < C) F(Pc + row * C + jb1) = ls[kB - 1][r];
            }
        }
        if (m == 0 && lane < C) {
            Dd(Pro + 2 * lane) = Dd(Lro + 2 * lane);
            Dd(Pco + 2 * lane) = Dd(Rco + 2 * lane);
        }
    }
}

// Put a staged leaf (raw potentials in slot t, ro = co = 0) into the form of its role.
template <int CP>
__device__ void normalise_leaf(int C, int slot, int role, int slotF, int coreF) {
    const int lane = threadIdx.x % kWave;
    const int c0 = slot * slotF, ro = c0 + coreF, co = ro + 2 * C;
    const int x = min(lane, C - 1);
    if (role == kNone) {
        if (lane < C) {
            Dd(ro + 2 * lane) = 0.0;
            Dd(co + 2 * lane) = 0.0;
        }
        wave_sync();
        return;
    }
    // LEFT: lane x owns row x; RIGHT: lane x owns column x.  Loads are unconditional
    // (indices clamped into the matrix) so they issue back to back.
    const int base = role == kLeft ? c0 + x * C : c0 + x;
    const int stride = role == kLeft ? 1 : C;
    float v[CP];
#pragma unroll
    for (int j = 0; j < CP; ++j) v[j] = F(base + min(j, C - 1) * stride);
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < CP; ++j) m = fmaxf(m, v[j]);   // entries past C repeat entry C-1
    const float sh = safe_shift(m);
    if (lane < C) {
#pragma unroll
        for (int j = 0; j < CP; ++j)
            if (j < C) F(base + j * stride) = v[j] - sh;
        Dd((role == kLeft ? ro : co) + 2 * lane) = (double)sh;
        Dd((role == kLeft ? co : ro) + 2 * lane) = 0.0;
    }
    wave_sync();
}

// One wave, C <= CP <= 32, node N[a][b] = ro[a] + co[b] + core[a][b] at LDS offsets
// (Nc, Nro; co follows ro).  kRowSide == false: y[j] = LSE_i x[i] + N[i][j] (y = x (x) N);
// kRowSide == true: y[i] = LSE_j N[i][j] + x[j] (y = N (x) x).  y is shifted to max 0.
template <int CP, bool kRowSide>
__device__ void wave_vec_log(int C, int x, int Nc, int Nro, int y, int scr) {
    const int lane = threadIdx.x % kWave;
    // x on the left pairs with ro and the result picks up co; on the right the reverse
    const int inOff = kRowSide ? 2 * C : 0, outOff = kRowSide ? 0 : 2 * C;
    double w = -INFINITY;
    if (lane < C) w = (double)F(x + lane) + Dd(Nro + inOff + 2 * lane);
    const double ws = (double)safe_shift(wave_max_fast((float)w));
    if (lane < C) F(scr + lane) = (w == -INFINITY) ? -INFINITY : (float)(w - ws);
    wave_sync();
    double z = -INFINITY;
    {
        const int lc = min(lane, C - 1);
        float e[CP];
#pragma unroll
        for (int t = 0; t < CP; ++t) {
            const int tc = min(t, C - 1);
            e[t] = F(scr + tc) + (kRowSide ? F(Nc + lc * C + tc) : F(Nc + tc * C + lc));
        }
        float m = -INFINITY;
#pragma unroll
        for (int t = 0; t < CP; ++t) {
            e[t] = t < C ? e[t] : -INFINITY;
            m = fmaxf(m, e[t]);
        }
        if (m != -INFINITY && lane < C) {
            float s = 0.f;
#pragma unroll
            for (int t = 0; t < CP; ++t) s += fexp(e[t] - m);
            z = Dd(Nro + outOff + 2 * lane) + (double)(m + flog(s));
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
__device__ __forceinline__ void small_log_body(const SmallLogArgs& a, const int64_t b) {
    const int C = a.C;
    const int64_t E = a.N - 1;
    const int Eb = (int)(clamp_len(a.lengths, b, a.N) - 1);
    const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int CC = C * C;
    const float* gleaf = a.pot + (size_t)b * E * CC;
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
    LogLayout ly;
    ly.init(C, Eb);
    // ---- stage the valid edges into slots 0..Eb-1 (8 loads in flight per thread)
    {
        const int n = Eb * CC;
        for (int base = 0; base < n; base += 8 * kSmallThreads) {
            float v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = gleaf[min(base + u * kSmallThreads + (int)threadIdx.x, n - 1)];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int idx = base + u * kSmallThreads + threadIdx.x;
                if (idx < n) {
                    const int t = idx / CC;
                    F(t * ly.slotF + idx - t * CC) = v[u];
                }
            }
        }
    }
    __syncthreads();
    for (int t = w; t < Eb; t += kSmallWaves)
        normalise_leaf<CP>(C, t, node_role(T, 0, t), ly.slotF, ly.coreF);
    __syncthreads();
    // ---- up-sweep: one wave per product (two for CP > 16)
    constexpr int kPer = CP > 16 ? 2 : 1;
    for (int l = 1; l <= T.D; ++l) {
        const int np = T.products(l);
        for (int task = w; task < np * kPer; task += kSmallWaves) {
            const int k = task / kPer, m = task % kPer;
            const int sl = log_slot(T, l - 1, 2 * k), sr = log_slot(T, l - 1, 2 * k + 1);
            const int sp = T.E + T.pbase[l] + k, role = node_role(T, l, k);
            if (role == kLeft) prod_log<CP, kLeft>(ly, sl, sr, sp, m);
            else if (role == kRight) prod_log<CP, kRight>(ly, sl, sr, sp, m);
            else prod_log<CP, kNone>(ly, sl, sr, sp, m);
            wave_sync();
        }
        __syncthreads();
    }
    const int rslot = log_slot(T, T.D, 0);
    auto U = [&](int l, int k) { return ly.vecs + (T.vbase[l] + k) * 2 * C; };
    // ---- root: log Z = LSE_{a,c} ro[a] + co[c] + core[a][c]   (last wave, overlapping
    // the first outside level, which does not need it)
    if (a.logZ && w == kSmallWaves - 1) {
        const int rc = ly.core(rslot), rr = ly.ro(rslot), rcc = ly.co(rslot);
        const int lc = min(lane, C - 1);
        const double rs = (double)safe_shift(wave_max_fast(lane < C ? (float)Dd(rr + 2 * lc) : -INFINITY));
        const double cs = (double)safe_shift(wave_max_fast(lane < C ? (float)Dd(rcc + 2 * lc) : -INFINITY));
        constexpr int kRows = CP / 2;
        const int j = lane & 31, i0 = lane >> 5, jc = min(j, C - 1);
        const float cj = (float)(Dd(rcc + 2 * jc) - cs);
        float x[kRows];
#pragma unroll
        for (int q = 0; q < kRows; ++q) {
            const int ic = min(i0 + 2 * q, C - 1);
            x[q] = F(rc + ic * C + jc) + (float)(Dd(rr + 2 * ic) - rs) + cj;
        }
        float m = -INFINITY;
#pragma unroll
        for (int q = 0; q < kRows; ++q) {
            x[q] = (i0 + 2 * q < C && j < C) ? x[q] : -INFINITY;
            m = fmaxf(m, x[q]);
        }
        m = wave_max_fast(m);
        float s = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int q = 0; q < kRows; ++q) s += fexp(x[q] - m);
        }
        s = wave_sum_fast(s);
        if (lane == 0)
            a.logZ[b] = (m == -INFINITY) ? -INFINITY : (float)(rs + cs + (double)(m + flog(s)));
    }
    if (!a.marg) return;
    // ---- outside sweep: u, v of every node (root: zeros)
    if (w < kSmallWaves - 1 || !a.logZ)
        for (int idx = lane; idx < 2 * C; idx += kWave)
            if (w == 0) F(U(T.D, 0) + idx) = 0.f;
    __syncthreads();
    const int scr = ly.vecs + T.nodes * 2 * C + w * 64;
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
                const int sl = log_slot(T, l - 1, 2 * k);
                wave_vec_log<CP, false>(C, uN, ly.core(sl), ly.ro(sl), U(l - 1, 2 * k + 1), scr);
            } else if (which == 2 && right) {   // v_L = R (x) v_N
                const int sr = log_slot(T, l - 1, 2 * k + 1);
                wave_vec_log<CP, true>(C, vN, ly.core(sr), ly.ro(sr), U(l - 1, 2 * k) + C, scr);
            }
        }
        __syncthreads();
    }
    // ---- marginals with a per-edge normaliser n_t; the raw edge is re-read from global
    // memory (L2).  Lane -> column j = lane & 31 and rows (lane >> 5) + 2q.
    constexpr int kRows = CP / 2;
    const int j = lane & 31, i0 = lane >> 5, jc = min(j, C - 1);
    for (int t = w; t < Eb; t += kSmallWaves) {
        const int al = U(0, t), be = al + C;
        const float* leaf = gleaf + (size_t)t * CC;
        const float bj = F(be + jc);
        float x[kRows];
#pragma unroll
        for (int q = 0; q < kRows; ++q) {
            const int i = i0 + 2 * q, ic = min(i, C - 1);
            x[q] = leaf[ic * C + jc];
        }
        float m = -INFINITY;
#pragma unroll
        for (int q = 0; q < kRows; ++q) {
            const int i = i0 + 2 * q, ic = min(i, C - 1);
            x[q] = (i < C && j < C) ? F(al + ic) + x[q] + bj : -INFINITY;
            m = fmaxf(m, x[q]);
        }
        m = wave_max_fast(m);
        float s = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int q = 0; q < kRows; ++q) s += fexp(x[q] - m);
        }
        s = wave_sum_fast(s);
        const float n = (m == -INFINITY) ? -INFINITY : m + flog(s);
        float* out = a.marg + ((size_t)b * E + t) * CC;
#pragma unroll
        for (int q = 0; q < kRows; ++q) {
            const int i = i0 + 2 * q;
            if (i < C && j < C) out[i * C + j] = (n == -INFINITY) ? 0.f : fexp(x[q] - n);
        }
    }
}

// ================================================================== max semiring
// LDS layout (float offsets): leaves fp32 [E][C][C] | product slots fp64 [E-1][C][C] |
// last leaf again in fp64 [C][C] | forward scores fp64 [nodes][C] | last scores fp64 [C] |
// backpointers u8 [E][C].  Above level 1 the only leaf that can still be an operand is the
// last one (through nodes whose right half is padding), so levels >= 2 read fp64 only.
struct MaxLayout {
    int C, CC, leaves, slots, lastc, vecs, dlast, bp;
    __device__ void init(int c, int E, int nodes) {
        C = c;
        CC = c * c;
        leaves = 0;
        slots = align4(E * CC);
        lastc = slots + (E - 1) * CC * 2;
        vecs = lastc + CC * 2;
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

// All products of level l, P = L (x) R in (max, +), float64, by the whole workgroup: every
// thread owns MR x MC output entries of one product (register-tiled loop over the inner
// index).  kLeaves: the operands are leaves (level 1, fp32); otherwise fp64 slots.
template <int MR, int MC, bool kLeaves>
__device__ void block_prod_max(const MaxLayout& ly, const Tree& T, int l) {
    const int C = ly.C, CC = ly.CC;
    const int TR = (C + MR - 1) / MR, TC = (C + MC - 1) / MC, tpp = TR * TC;
    const int total = T.products(l) * tpp;
    for (int tile = threadIdx.x; tile < total; tile += kSmallThreads) {
        const int k = tile / tpp, rem = tile - k * tpp, tr = rem / TC, tc = rem - tr * TC;
        const int hl = T.handle(l - 1, 2 * k), hr = T.handle(l - 1, 2 * k + 1);
        int lb, rb;
        if constexpr (kLeaves) {
            lb = ly.leaves + (-hl - 1) * CC;
            rb = ly.leaves + (-hr - 1) * CC;
        } else {
            lb = hl < 0 ? ly.lastc : ly.slots + hl * CC * 2;
            rb = hr < 0 ? ly.lastc : ly.slots + hr * CC * 2;
        }
        const int r0 = tr * MR, c0 = tc * MC;
        int ra[MR], cb[MC];
#pragma unroll
        for (int i = 0; i < MR; ++i) ra[i] = min(r0 + i, C - 1) * C;
#pragma unroll
        for (int j = 0; j < MC; ++j) cb[j] = min(c0 + j, C - 1);
        double acc[MR][MC];
#pragma unroll
        for (int i = 0; i < MR; ++i)
#pragma unroll
            for (int j = 0; j < MC; ++j) acc[i][j] = -INFINITY;
#pragma unroll 2
        for (int q = 0; q < C; ++q) {
            double av[MR], bv[MC];
#pragma unroll
            for (int i = 0; i < MR; ++i) av[i] = mx<kLeaves>(lb, ra[i] + q);
#pragma unroll
            for (int j = 0; j < MC; ++j) bv[j] = mx<kLeaves>(rb, q * C + cb[j]);
#pragma unroll
            for (int i = 0; i < MR; ++i)
#pragma unroll
                for (int j = 0; j < MC; ++j) acc[i][j] = fmax(acc[i][j], av[i] + bv[j]);
        }
        const int Pb = ly.slots + (T.pbase[l] + k) * CC * 2;
#pragma unroll
        for (int i = 0; i < MR; ++i)
#pragma unroll
            for (int j = 0; j < MC; ++j)
                if (r0 + i < C && c0 + j < C) Dd(Pb + 2 * ((r0 + i) * C + c0 + j)) = acc[i][j];
    }
}

// the smallest register tile that still gives every thread at most one tile
template <bool kLeaves>
__device__ void level_prod_max(const MaxLayout& ly, const Tree& T, int l) {
    const int np = T.products(l), C = ly.C;
    auto tiles = [&](int mr, int mc) { return np * ((C + mr - 1) / mr) * ((C + mc - 1) / mc); };
    if (tiles(1, 1) <= kSmallThreads) block_prod_max<1, 1, kLeaves>(ly, T, l);
    else if (tiles(1, 2) <= kSmallThreads) block_prod_max<1, 2, kLeaves>(ly, T, l);
    else if (tiles(2, 2) <= kSmallThreads) block_prod_max<2, 2, kLeaves>(ly, T, l);
    else if (tiles(2, 4) <= kSmallThreads) block_prod_max<2, 4, kLeaves>(ly, T, l);
    else block_prod_max<4, 4, kLeaves>(ly, T, l);
}

template <int CP, bool kLeaf>
__device__ void wave_vec_max(int C, int x, int Nb, int y) {
    const int lane = threadIdx.x % kWave;
    const int j = min(lane, C - 1);
    double v[CP];
#pragma unroll
    for (int i = 0; i < CP; ++i) {
        const int ic = min(i, C - 1);
        v[i] = Dd(x + 2 * ic) + mx<kLeaf>(Nb, ic * C + j);   // past C: repeats entry C-1
    }
    double m = -INFINITY;
#pragma unroll
    for (int i = 0; i < CP; ++i) m = fmax(m, v[i]);
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
__device__ __forceinline__ void small_max_body(const SmallMaxArgs& a, const int64_t b) {
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
    // the last leaf in fp64 for levels >= 2 (read only after the level-1 barrier)
    for (int i = threadIdx.x; i < CC; i += kSmallThreads)
        Dd(ly.lastc + 2 * i) = (double)F(ly.leaves + (Eb - 1) * CC + i);
    // ---- up-sweep: all threads share each level's products
    for (int l = 1; l <= T.D; ++l) {
        if (l == 1) level_prod_max<true>(ly, T, l);
        else level_prod_max<false>(ly, T, l);
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
        double v[CP];
#pragma unroll
        for (int i = 0; i < CP; ++i) {
            const int ic = min(i, C - 1);
            v[i] = Dd(d + 2 * ic) + (double)F(leaf + ic * C + j);
        }
        double best = v[0];
        int arg = 0;
#pragma unroll
        for (int i = 1; i < CP; ++i) {
            const bool better = i < C && v[i] > best;   // strict: the lowest index wins ties
            best = better ? v[i] : best;
            arg = better ? i : arg;
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

template <int CP>
__global__ __launch_bounds__(kSmallThreads) void k_small_log(SmallLogArgs a) {
    small_log_body<CP>(a, blockIdx.x);
}

template <int CP>
__global__ __launch_bounds__(kSmallThreads) void k_small_max(SmallMaxArgs a) {
    small_max_body<CP>(a, blockIdx.x);
}

// Both computations in one launch: workgroups [0, B) run the log-semiring pass of sequence
// b, workgroups [B, 2B) the max-plus pass of sequence b - B.  The two halves share nothing
// but the read-only potentials, so they run side by side on different compute units.
template <int CP>
__global__ __launch_bounds__(kSmallThreads) void k_small_both(SmallLogArgs la, SmallMaxArgs ma,
                                                             int64_t B) {
    const int64_t g = blockIdx.x;
    if (g < B) small_log_body<CP>(la, g);
    else small_max_body<CP>(ma, g - B);
}

}  // namespace

// Both layouts are sized for the longest sequence (E = N-1 edges); a shorter sequence
// uses a prefix of each region, so the offsets computed in the kernels stay inside.
size_t small_log_lds_bytes(int64_t E, int64_t C) {
    if (E < 1) return 0;
    const int64_t slotF = ((C * C + 3) & ~3) + 4 * C;
    const int64_t floats = (2 * E - 1) * slotF + small_tree_nodes(E) * 2 * C + kSmallWaves * 64;
    return sizeof(float) * (size_t)floats;
}

size_t small_max_lds_bytes(int64_t E, int64_t C) {
    if (E < 1) return 0;
    const int64_t CC = C * C;
    const int64_t floats = (E * CC + 3) + (E - 1) * CC * 2 + CC * 2 + small_tree_nodes(E) * C * 2 + 2 * C;
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

template <int CP>
hipError_t small_both_cp(const SmallLogArgs& la, const SmallMaxArgs& ma, int64_t B, size_t lds,
                         hipStream_t s) {
    static bool attr = false;
    if (!attr) {
        hipError_t e = allow_lds(k_small_both<CP>);
        if (e != hipSuccess) return e;
        attr = true;
    }
    hipLaunchKernelGGL(k_small_both<CP>, dim3((unsigned)(2 * B)), dim3(kSmallThreads), lds, s, la,
                       ma, B);
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

hipError_t launch_small_both(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                             int64_t C, float* logZ, float* marg, int32_t* path, float* score,
                             hipStream_t s) {
    SmallLogArgs la{pot, lengths, N, (int)C, logZ, marg};
    SmallMaxArgs ma{pot, lengths, N, (int)C, path, score};
    const size_t lds = std::max(small_log_lds_bytes(N - 1, C), small_max_lds_bytes(N - 1, C));
    if (C <= 8) return small_both_cp<8>(la, ma, B, lds, s);
    if (C <= 16) return small_both_cp<16>(la, ma, B, lds, s);
    if (C <= 24) return small_both_cp<24>(la, ma, B, lds, s);
    return small_both_cp<32>(la, ma, B, lds, s);
}

}  // namespace tsc
