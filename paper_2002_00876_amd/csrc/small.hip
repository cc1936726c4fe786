// small.hip -- fused single-launch path for small label sets (C <= 32): one workgroup per
// sequence keeps that sequence's whole edge tree in LDS and runs, in one kernel,
//   log semiring: up-sweep of semiring matrix products (Sec. 6a / Fig. 3), root
//   log-sum-exp (log Z), outside sweep and per-edge marginals (Sec. 5.1 gradient identity);
//   max semiring: float64 up-sweep, forward scores, backpointers and the backtrace.
// The arithmetic is that of the multi-launch tree (tree_log.hip / tree_max.hip): node
// matrices P[a][c] = ro[a] + co[c] + core[a][c] with an exp-shifted fp32 MFMA product
// (one wave per product), and exact float64 max-plus for Viterbi (the whole workgroup
// shares each level's products).  k_small_both runs both passes of a batch in one launch,
// one workgroup per sequence and pass.
//
// Tree bookkeeping for a sequence with E edges: level 0 holds the E leaves (staged from
// global memory into LDS); level l holds n_l = ceil(E / 2^l) nodes.  Node k of level l
// is a product of its two children when 2k+1 < n_{l-1} and otherwise equals its left
// child.  Products are stored in LDS slots numbered level by level.
//
// All LDS data is addressed as integer offsets into the one dynamic LDS array, so every
// access compiles to a ds_read/ds_write.
#include <type_traits>

#include "device.h"
#include "internal.h"
#include "small.h"

namespace tsc {

extern __shared__ __align__(16) float ts_small_lds[];

namespace {

constexpr int kSmallThreads = 1024;  // 16 waves
constexpr int kSmallWaves = kSmallThreads / kWave;
constexpr float kUnderflow = 0x1p-80f;

__device__ __forceinline__ float& F(int off) { return ts_small_lds[off]; }
// doubles sit at even float offsets
__device__ __forceinline__ double& Dd(int off_floats) {
    __builtin_assume((off_floats & 1) == 0);
    return reinterpret_cast<double*>(ts_small_lds)[off_floats >> 1];
}
__device__ __forceinline__ unsigned short& H(int off_halves) {
    return reinterpret_cast<unsigned short*>(ts_small_lds)[off_halves];
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
    __device__ int products(int l) const { return n[l - 1] / 2; }
};

// ================================================================== log semiring
// Every node is kept in the form its consumer needs, so a product needs only exp + MFMA:
//   LEFT operand  (left child of a product):  P[a][b] = ro[a] + core[a][b], max_b core[a][b] = 0
//   RIGHT operand (right child of a product): P[b][c] = co[c] + core[b][c], max_b core[b][c] = 0
//   NONE (the root): P[a][c] = ro[a] + co[c] + core[a][c]
// (an absent right child makes a node equal to its left child, so a node takes the role
// of its first ancestor that is consumed).  The root's matrix is never formed: log Z comes
// from its children's outside vectors, so every product is a LEFT or a RIGHT node; only
// the single leaf of a one-edge sequence is a NONE node.
// For P = L (x) R with L in LEFT and R in RIGHT form:
//   S[a][c] = sum_b exp(core_L[a][b]) exp(core_R[b][c])     (fp32 MFMA, every factor <= 1)
//   P[a][c] = ro_L[a] + co_R[c] + log S[a][c]
// and the producer then normalises P into the form of its own role.  S < 2^-80 (all
// terms underflowed) is recomputed exactly by a direct max-shifted log-sum-exp over b.
//
// One wave computes a whole product as one MFMA tile (32 x 32 for CP > 16, 16 x 16
// otherwise).  The tile's output layout gives each lane one column and a set of rows, so
// a product that is normalised per column (RIGHT) is computed as P and one
// normalised per row (LEFT) as its transpose P^T = R^T L^T: either way the lane owns the
// line it normalises, and the reduction is over its own values plus the lanes holding the
// same column.
//
// Labels are padded to CP.  A slot holds core [CP][CP + 1] (the odd row stride keeps the
// strided operand reads free of bank conflicts), then ro [CP] and co [CP] as doubles.
// Invariants, kept by every producer:
//   * ro[i] = co[i] = -inf for C <= i < CP;
//   * LEFT node: core[a][b] = -inf for a < C <= b;  RIGHT node: core[b][c] = -inf for
//     c < C <= b, so the padded part of the contracted index contributes exp(-inf) = 0;
//   * the other padding entries are never read: operand rows and columns are read through
//     indices clamped to C - 1, which makes the padded part of a product a copy of valid
//     entries (so the underflow test needs no mask).
// Outside vectors (u, v) have CP entries with -inf padding.
//
// LDS layout (float offsets): slots [2E-1][slotF] (leaves are slots 0..E-1, products
// follow level by level) | vectors [nodes][2][CP] (u then v) | per-wave scratch [16][64] |
// node table (16-bit entries).
constexpr int kLeft = 0, kRight = 1, kNone = 2;

// nodes at level l of the tree over E >= 1 leaves: ceil(E / 2^l)
__device__ __forceinline__ int lvl_n(int E, int l) { return ((E - 1) >> l) + 1; }

// role of node (l, k), from E alone (register arithmetic, no table)
__device__ __forceinline__ int role_of(int E, int l, int k) {
    while ((E - 1) >> l) {   // level l has more than one node
        if (k & 1) return kRight;
        if (k + 1 < lvl_n(E, l)) return kLeft;
        ++l;
        k >>= 1;
    }
    return kNone;
}

// The node tables of every tree of up to kTableEdges leaves, computed at compile time (the
// same walk as build_node_table below): a short sequence copies its row instead of
// computing it.
constexpr int kTableEdges = 64;

constexpr int ce_lvl_n(int E, int l) { return ((E - 1) >> l) + 1; }

constexpr int ce_nodes(int E) {
    int total = E, n = E;
    while (n > 1) { n = (n + 1) / 2; total += n; }
    return total;
}

constexpr int ce_role(int E, int l, int k) {
    while ((E - 1) >> l) {
        if (k & 1) return kRight;
        if (k + 1 < ce_lvl_n(E, l)) return kLeft;
        ++l;
        k >>= 1;
    }
    return kNone;
}

constexpr unsigned short ce_entry(int E, int i) {
    int l = 0, vb = 0, n = E, nprev = 0, pb = E;
    while (i >= vb + n) {
        if (l >= 1) pb += nprev / 2;
        vb += n;
        nprev = n;
        n = (n + 1) / 2;
        ++l;
    }
    const int k = i - vb;
    int ll = l, kk = k;
    while (ll > 0 && kk >= ce_lvl_n(E, ll - 1) / 2) {
        --ll;
        kk *= 2;
        if (ll > 0) pb -= ce_lvl_n(E, ll - 1) / 2;
    }
    const int slot = ll == 0 ? kk : pb + kk;
    return (unsigned short)(slot | (ce_role(E, l, k) << 14));
}

constexpr int ce_total() {
    int t = 0;
    for (int E = 1; E <= kTableEdges; ++E) t += ce_nodes(E);
    return t;
}

struct NodeTables {
    int off[kTableEdges + 1];
    unsigned short entry[ce_total()];
};

constexpr NodeTables ce_tables() {
    NodeTables t{};
    int o = 0;
    for (int E = 1; E <= kTableEdges; ++E) {
        t.off[E] = o;
        for (int i = 0; i < ce_nodes(E); ++i) t.entry[o + i] = ce_entry(E, i);
        o += ce_nodes(E);
    }
    return t;
}

__constant__ NodeTables kNodeTables = ce_tables();

// The node table: one 16-bit entry per node in level-major order (node (l, k) at
// vbase[l] + k) holding its slot (bits 0..13) and role (bits 14..15).  Leaves are slots
// 0..E-1; the products of level l follow those of the levels below (slots from
// pbase[l] = E + sum_{q<l} n[q-1] / 2); a node without a right child is its left child.
// One pass per node with running sums, register arithmetic only.
constexpr int kSlotMask = 0x3fff;

__device__ void build_node_table(int E, int nodes, int info) {
    // A table of at most 64 nodes is built in one pass by one wave (the one before the wave
    // that sets up the tree): every wave that runs this code issues all of its instructions,
    // whatever few lanes are active.  Larger tables: node i goes to lane i / 16 of wave i % 16.
    const int wave = (int)(threadIdx.x / kWave), lane = (int)(threadIdx.x % kWave);
    if (E <= kTableEdges) {   // precomputed: one wave copies the row
        if (wave != kSmallWaves - 2) return;
        for (int i = lane; i < nodes; i += kWave) H(info + i) = kNodeTables.entry[kNodeTables.off[E] + i];
        return;
    }
    const bool one = nodes <= kWave;
    if (one && wave != kSmallWaves - 2) return;
    for (int base = 0; base < nodes; base += one ? kWave : kSmallThreads) {
        const int i = one ? base + lane : base + lane * kSmallWaves + wave;
        if (i >= nodes) continue;
        int l = 0, vb = 0, n = E, nprev = 0, pb = E;   // pb = pbase[l] once l >= 1
        while (i >= vb + n) {
            if (l >= 1) pb += nprev / 2;
            vb += n;
            nprev = n;
            n = (n + 1) / 2;
            ++l;
        }
        const int k = i - vb;
        // follow the left-child chain down to a product or a leaf
        int ll = l, kk = k;
        while (ll > 0 && kk >= lvl_n(E, ll - 1) / 2) {
            --ll;
            kk *= 2;
            if (ll > 0) pb -= lvl_n(E, ll - 1) / 2;
        }
        const int slot = ll == 0 ? kk : pb + kk;
        H(info + i) = (unsigned short)(slot | (role_of(E, l, k) << 14));
    }
}

// Tree of E >= 1 leaves set up by one wave (lane l fills level l), instead of one thread
// walking the levels
__device__ void tree_init_wave(Tree& T, int E) {
    // lane l <= kSmallMaxLevels holds level l; vbase and pbase are prefix sums over the lanes
    const int l = threadIdx.x % kWave;
    const int n = l <= kSmallMaxLevels ? lvl_n(E, l) : 0;
    int sn = n, sp = n / 2;   // n[l] / 2 = products of level l + 1
#pragma unroll
    for (int d = 1; d <= kSmallMaxLevels; d <<= 1) {
        const int on = __shfl_up(sn, d, kWave), op = __shfl_up(sp, d, kWave);
        sn += l >= d ? on : 0;
        sp += l >= d ? op : 0;
    }
    const int sp2 = __shfl_up(sp, 2, kWave);   // products of levels 1..l-1
    if (l <= kSmallMaxLevels) {
        T.n[l] = n;
        T.vbase[l] = sn - n;
        T.pbase[l] = l >= 2 ? sp2 : 0;
    }
    if (l == 0) {
        T.E = E;
        T.D = E <= 1 ? 0 : 32 - __clz(E - 1);
        T.nodes = (int)small_tree_nodes(E);
    }
}

// Flat, coalesced copy of a sequence's first `n` potentials (all N-1 edges: the loads go
// out before the length is known) into registers; kPer loads per thread.
template <int kPer>
struct LeafBatch {
    float v[kPer];
    __device__ void load(const float* src, int base, int n) {
#pragma unroll
        for (int u = 0; u < kPer; ++u) v[u] = src[min(base + u * kSmallThreads + (int)threadIdx.x, n - 1)];
    }
    // store elements [base, min(n, base + kPer * threads)) to LDS at dst
    __device__ void store(int dst, int base, int n) const {
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int idx = base + u * kSmallThreads + threadIdx.x;
            if (idx < n) F(dst + idx) = v[u];
        }
    }
};
constexpr int kLeafBatch = 16;

template <int CP>
struct LogLayout {
    static constexpr int kLd = CP + 1;                          // core row stride
    static constexpr int kCoreF = (CP * kLd + 1) & ~1;          // doubles stay 8-byte aligned
    static constexpr int kSlotF = kCoreF + 4 * CP;
    int C, vecs, scr, info;
    __device__ void init(int c, int E) {
        C = c;
        vecs = (2 * E - 1) * kSlotF;
        scr = vecs + (int)small_tree_nodes(E) * 2 * CP;
        info = 2 * (scr + kSmallWaves * 64);   // in halves
    }
    __device__ static int core(int slot) { return slot * kSlotF; }
    __device__ static int ro(int slot) { return slot * kSlotF + kCoreF; }    // doubles
    __device__ static int co(int slot) { return slot * kSlotF + kCoreF + 2 * CP; }
};

// max / sum of x over lanes l and l ^ 32 (the same value in both lanes)
__device__ __forceinline__ float xor32_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xor32_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// MFMA tile of a CP-padded product: 32 x 32 x 2 (16 values per lane) or 16 x 16 x 4
// (4 values per lane).  Value r of lane l sits at tile row row(r), column l % kT.
template <int CP>
struct Tile {
    static constexpr int kT = CP > 16 ? 32 : 16;
    static constexpr int kK = kT == 32 ? 2 : 4;      // contraction indices per step
    static constexpr int kSteps = CP / kK;
    static constexpr int kV = kT == 32 ? 16 : 4;     // values per lane
    // values that hold a row below CP in at least one half of the wave (rows grow with r
    // for the 32-wide tile; rows at or past CP are computed from clamped operands and not
    // stored)
    static constexpr int kVr = kT == 32 ? ((CP + 7) / 8) * 4 : 4;
    __device__ static int row(int r, int lane) {
        return kT == 32 ? (r >> 2) * 8 + ((lane >> 5) << 2) + (r & 3) : ((lane >> 4) << 2) + r;
    }
};

// LSE_k row[k] + col[k * stride] over k < C, by a direct max-shifted sum: the exact value of
// a product entry whose exp-shifted terms all underflowed.  A rare path, kept out of line so
// that the products' code stays small.
__device__ __noinline__ float exact_entry(int row, int col, int stride, int C) {
    float q = -INFINITY;
    for (int k = 0; k < C; ++k) q = fmaxf(q, F(row + k) + F(col + k * stride));
    if (q == -INFINITY) return -INFINITY;
    float s = 0.f;
    for (int k = 0; k < C; ++k) s += fexp(F(row + k) + F(col + k * stride) - q);
    return q + flog(s);
}

// Product of the LEFT node at slot sl and the RIGHT node at slot sr into slot sp, in the
// form kRole (one wave).
template <int CP, int kRole>
__device__ __forceinline__ void prod_log(const LogLayout<CP>& ly, int sl, int sr, int sp) {
    static_assert(kRole == kLeft || kRole == kRight, "products below the root only");
    using Ly = LogLayout<CP>;
    using Tl = Tile<CP>;
    constexpr int kT = Tl::kT, kLd = Ly::kLd;
    constexpr bool kTrans = kRole == kLeft;   // compute P^T: lanes own rows of P
    const int C = ly.C;
    const int lane = threadIdx.x % kWave, own = lane % kT, grp = lane / kT;
    const int oc = min(own, C - 1);
    const int Lc = Ly::core(sl), Rc = Ly::core(sr), Pc = Ly::core(sp);
    // offsets of the values' own lines, read before the products so they overlap them:
    // LEFT: co_R of each value's column, RIGHT: ro_L of each value's row
    const int offBase = kRole == kLeft ? Ly::co(sr) : Ly::ro(sl);
    const float mOff =
        safe_shift(wave_max_fast(lane < C ? (float)Dd(offBase + 2 * min(lane, C - 1)) : -INFINITY));
    float oh[Tl::kVr];
#pragma unroll
    for (int r = 0; r < Tl::kVr; ++r)
        oh[r] = (float)(Dd(offBase + 2 * min(Tl::row(r, lane), CP - 1)) - (double)mOff);
    // operand values: L[own][k] and R[k][own], k = kK * st + grp
    float lv[Tl::kSteps], rv[Tl::kSteps];
#pragma unroll
    for (int st = 0; st < Tl::kSteps; ++st) {
        const int k = Tl::kK * st + grp;
        lv[st] = F(Lc + oc * kLd + k);
        rv[st] = F(Rc + k * kLd + oc);
    }
    typedef float accv __attribute__((ext_vector_type(Tl::kV)));
    accv acc = {};
#pragma unroll
    for (int st = 0; st < Tl::kSteps; ++st) {
        const float el = fexp(lv[st]), er = fexp(rv[st]);
        if constexpr (kT == 32)
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(kTrans ? er : el, kTrans ? el : er, acc, 0, 0, 0);
        else
            acc = __builtin_amdgcn_mfma_f32_16x16x4f32(kTrans ? er : el, kTrans ? el : er, acc, 0, 0, 0);
    }
    // log S; the padded part of the tile copies valid entries, so every value is tested
    float x[Tl::kVr];
    float smin = INFINITY;
#pragma unroll
    for (int r = 0; r < Tl::kVr; ++r) {
        x[r] = flog(acc[r]);
        smin = fminf(smin, acc[r]);
    }
    if (__builtin_amdgcn_ballot_w64(!(smin >= kUnderflow))) {
        // exact recomputation of underflowed entries: LSE_b core_L[a][b] + core_R[b][c]
#pragma unroll
        for (int r = 0; r < Tl::kVr; ++r) {
            if (!(acc[r] >= kUnderflow)) {
                const int other = min(Tl::row(r, lane), C - 1);
                const int a = kTrans ? oc : other, c = kTrans ? other : oc;
                x[r] = exact_entry(Lc + a * kLd, Rc + c, kLd, C);
            }
        }
    }
    const bool rowsOk = kT == 32 || Tl::row(0, lane) < CP;   // 16-wide tile, CP = 8
    {
        // fold the shifted offsets of the other index in, then shift the lane's line to max 0
        float m = -INFINITY;
#pragma unroll
        for (int r = 0; r < Tl::kVr; ++r) {
            x[r] += oh[r];
            m = fmaxf(m, x[r]);
        }
        if constexpr (kT == 32) {
            m = xor32_max(m);
        } else {
            m = fmaxf(m, __shfl_xor(m, 16, kWave));
            m = fmaxf(m, __shfl_xor(m, 32, kWave));
        }
        // lines past C become -inf (shift by +inf): the padding invariant
        const float sh = own < C ? safe_shift(m) : INFINITY;
        if (own < CP && rowsOk) {
#pragma unroll
            for (int r = 0; r < Tl::kVr; ++r) {
                const int o = Tl::row(r, lane);
                if (o < CP) F(Pc + (kTrans ? own * kLd + o : o * kLd + own)) = x[r] - sh;
            }
        }
        if (lane < CP) {
            // the lane's line offset picks up the other side's max and the shift; the other
            // offset is 0 (padding -inf)
            const int keep = kTrans ? Ly::ro(sl) : Ly::co(sr);
            const int mine = kTrans ? Ly::ro(sp) : Ly::co(sp);
            const int zero = kTrans ? Ly::co(sp) : Ly::ro(sp);
            Dd(mine + 2 * lane) = lane < C ? Dd(keep + 2 * lane) + (double)mOff + (double)sh : -INFINITY;
            Dd(zero + 2 * lane) = lane < C ? 0.0 : -INFINITY;
        }
    }
}

// Staged leaves (raw, flat at LDS offset raw) into the form of their roles: one thread per
// line (row of a LEFT or NONE leaf, column of a RIGHT leaf), which it shifts to max 0 (not
// the NONE leaf of a one-edge sequence) and whose shift it records as ro (LEFT) or co
// (RIGHT); the other offset is 0.  Lines C..CP-1 and entries C..CP-1 of a line are -inf,
// so a leaf's whole padding is -inf.
//
// Leaves normalised by rows (the even ones but a last leaf without a sibling) take the
// first half of the workgroup, leaves normalised by columns (the odd ones and that last
// leaf) the second half, so every wave runs one of the two forms with its strides known at
// compile time.
template <int CP, bool kCols>
__device__ __forceinline__ void normalise_line(const LogLayout<CP>& ly, int raw, int E, int t,
                                               int r) {
    using Ly = LogLayout<CP>;
    constexpr int kLd = Ly::kLd;
    const int C = ly.C, CC = C * C;
    const bool pad = r >= C;
    const int rc = min(r, C - 1);
    // entries past C repeat entry C - 1: the maximum is unchanged, and their stores are
    // overwritten with -inf below (no per-entry masks)
    float v[CP];
    const int line = raw + t * CC + (kCols ? rc : rc * C);
#pragma unroll
    for (int q = 0; q < CP; ++q) v[q] = F(line + min(q, C - 1) * (kCols ? C : 1));
    float m = v[0];
#pragma unroll
    for (int q = 1; q < CP; ++q) m = fmaxf(m, v[q]);
    const bool none = !kCols && E == 1;   // the root of a one-edge tree keeps its values
    const float sh = none ? 0.f : safe_shift(m);
    constexpr int kStep = kCols ? kLd : 1;
    const int base = Ly::core(t) + (kCols ? r : r * kLd);
#pragma unroll
    for (int q = 0; q < CP; ++q) F(base + q * kStep) = pad ? -INFINITY : v[q] - sh;
    for (int q = C; q < CP; ++q) F(base + q * kStep) = -INFINITY;
    const int ro = Ly::ro(t), co = Ly::co(t);
    Dd((kCols ? co : ro) + 2 * r) = pad ? -INFINITY : (double)sh;
    Dd((kCols ? ro : co) + 2 * r) = pad ? -INFINITY : 0.0;
}

template <int CP>
__device__ void normalise_leaves(const LogLayout<CP>& ly, int raw, int E) {
    constexpr int kHalf = kSmallThreads / 2;
    const int nCols = E / 2 + ((E & 1) && E > 1 ? 1 : 0);   // odd leaves + a lone last leaf
    const int nRows = E - nCols;
    const int tid = (int)threadIdx.x;
    if (tid < kHalf) {
        for (int i = tid; i < nRows * CP; i += kHalf) {
            const int q = i / CP;
            normalise_line<CP, false>(ly, raw, E, 2 * q, i - q * CP);
        }
    } else {
        for (int i = tid - kHalf; i < nCols * CP; i += kHalf) {
            const int q = i / CP;
            normalise_line<CP, true>(ly, raw, E, min(2 * q + 1, E - 1), i - q * CP);
        }
    }
}

// One wave: outside-vector product with the node at `slot` (N[i][j] = ro[i] + co[j] +
// core[i][j]).  kRowSide == false: y[j] = LSE_i x[i] + N[i][j] (y = x (x) N);
// kRowSide == true: y[i] = LSE_j N[i][j] + x[j] (y = N (x) x).  y is shifted to max 0 and
// its padding is -inf; the total shift (of the input and of the output) is returned.  Lane l
// computes output l % 32 over half l / 32 of the index.
template <int CP, bool kRowSide>
__device__ double vec_log(const LogLayout<CP>& ly, int x, int slot, int y, int scr) {
    using Ly = LogLayout<CP>;
    constexpr int kLd = Ly::kLd, kHalf = CP / 2;
    const int C = ly.C;
    const int lane = threadIdx.x % kWave, o = lane & 31, h = lane >> 5;
    const int Nc = Ly::core(slot);
    // x on the left pairs with ro and the result picks up co; on the right the reverse
    const int inOff = kRowSide ? Ly::co(slot) : Ly::ro(slot);
    const int outOff = kRowSide ? Ly::ro(slot) : Ly::co(slot);
    const int li = min(lane, CP - 1);
    const double w = lane < CP ? (double)F(x + li) + Dd(inOff + 2 * li) : -INFINITY;
    const double ws = (double)safe_shift(wave_max_fast((float)w));
    if (lane < CP) F(scr + lane) = (float)(w - ws);
    wave_sync();
    const int oc = min(o, C - 1);
    float e[kHalf];
#pragma unroll
    for (int q = 0; q < kHalf; ++q) {
        const int t = h * kHalf + q;
        e[q] = F(scr + t) + (kRowSide ? F(Nc + oc * kLd + t) : F(Nc + t * kLd + oc));
    }
    float m = -INFINITY;
#pragma unroll
    for (int q = 0; q < kHalf; ++q) m = fmaxf(m, e[q]);
    m = safe_shift(xor32_max(m));
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < kHalf; ++q) s += fexp(e[q] - m);
    s = xor32_sum(s);
    const double z = (o < C && s > 0.f) ? Dd(outOff + 2 * oc) + (double)(m + flog(s)) : -INFINITY;
    const double zs = (double)safe_shift(wave_max_fast((float)z));
    if (h == 0 && o < CP) F(y + o) = (float)(z - zs);
    wave_sync();
    return ws + zs;   // y as stored plus this is the exact x (x) N
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
    using Ly = LogLayout<CP>;
    constexpr int kLd = Ly::kLd;
    const int C = a.C;
    const int64_t E = a.N - 1;
    const int CC = C * C;
    const float* gleaf = a.pot + (size_t)b * E * CC;
    // the first loads of the potentials go out before the length is known
    LeafBatch<kLeafBatch> lb;
    lb.load(gleaf, 0, (int)E * CC);
    const int Eb = (int)(clamp_len(a.lengths, b, a.N) - 1);
    const int w = uni(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    // padding edges are exactly zero (written last: these stores would otherwise hold up
    // the first loads, which wait for all earlier memory operations)
    auto zero_padding = [&]() {
        if (!a.marg) return;
        float* mz = a.marg + ((size_t)b * E + Eb) * CC;
        const size_t nz = (size_t)(E - Eb) * CC;
        for (size_t idx = threadIdx.x; idx < nz; idx += kSmallThreads) mz[idx] = 0.f;
    };
    if (Eb == 0) {
        if (a.logZ && threadIdx.x == 0) a.logZ[b] = logf((float)C);
        zero_padding();
        return;
    }
    __shared__ Tree T;
    Ly ly;
    ly.init(C, Eb);
    const int nodes = (int)small_tree_nodes(Eb);
    // ---- tree, node table and raw leaves (staged in the product-slot region, which the
    // normalised leaves do not touch), then the leaves in the forms of their roles
    if (w == kSmallWaves - 1) tree_init_wave(T, Eb);
    build_node_table(Eb, nodes, ly.info);
    const int raw = Ly::core(Eb), n = Eb * CC;
    lb.store(raw, 0, n);
    for (int base = kLeafBatch * kSmallThreads; base < n; base += kLeafBatch * kSmallThreads) {
        lb.load(gleaf, base, n);
        lb.store(raw, base, n);
    }
    __syncthreads();
    normalise_leaves<CP>(ly, raw, Eb);
    __syncthreads();
    // the root's outside vectors (zeros, padding -inf; the root is the last node), written
    // once the raw leaves (which can reach into the vectors' region) are consumed and read
    // after the next barrier
    if (w == kSmallWaves - 1)
        for (int idx = lane; idx < 2 * CP; idx += kWave)
            F(ly.vecs + (nodes - 1) * 2 * CP + idx) = (idx % CP) < C ? 0.f : -INFINITY;
    if (T.D < 2) __syncthreads();   // no level of the up-sweep (and no barrier) follows
    // ---- up-sweep: one wave per product, below the root: the root's matrix is never needed
    // (log Z comes from its children's outside vectors)
    for (int l = 1; l < T.D; ++l) {
        const int np = uni(T.products(l));
        const int vb0 = uni(T.vbase[l - 1]), vb1 = uni(T.vbase[l]);
        for (int k = w; k < np; k += kSmallWaves) {
            const int sl = uni(H(ly.info + vb0 + 2 * k)) & kSlotMask;
            const int sr = uni(H(ly.info + vb0 + 2 * k + 1)) & kSlotMask;
            const int ip = uni(H(ly.info + vb1 + k));
            const int sp = ip & kSlotMask, role = ip >> 14;
            // below the root every node is consumed as a left or a right operand
            if (role == kLeft) prod_log<CP, kLeft>(ly, sl, sr, sp);
            else prod_log<CP, kRight>(ly, sl, sr, sp);
            wave_sync();
        }
        __syncthreads();
    }
    auto U = [&](int l, int k) { return ly.vecs + (T.vbase[l] + k) * 2 * CP; };
    // log Z stays in a register of the last wave until the end: a global store before a
    // barrier would hold the barrier up until it completes
    float lz = 0.f;
    auto store_logz = [&]() {
        if (a.logZ && w == kSmallWaves - 1 && lane == 0) a.logZ[b] = lz;
    };
    if (T.D == 0) {
        // one edge: log Z = LSE_{a,c} of the leaf itself
        if (a.logZ && w == kSmallWaves - 1) {
            const int rslot = uni(H(ly.info + T.vbase[0])) & kSlotMask;
            const int rc = Ly::core(rslot), rr = Ly::ro(rslot), rcc = Ly::co(rslot);
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
                x[q] = F(rc + ic * kLd + jc) + (float)(Dd(rr + 2 * ic) - rs) + cj;
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
            lz = (m == -INFINITY) ? -INFINITY : (float)(rs + cs + (double)(m + flog(s)));
        }
        if (!a.marg) {
            store_logz();
            return;
        }
    }
    // ---- outside sweep: u, v of every node (root: zeros, padding -inf).  With the root's
    // children L and R, log Z = LSE_{a,c} (L (x) R)[a][c] = LSE_b u_R[b] + v_L[b], where
    // u_R = 0 (x) L and v_L = R (x) 0 are the first level's outside vectors; their shifts
    // are kept in rootShift.
    // ---- marginals of edge t with a per-edge normaliser n_t, from the leaves kept in LDS:
    // l[i][j] = ro[i] + co[j] + core[i][j].  One wave per edge; lane l holds the entries
    // v = l + 64 q of the row-major C x C edge (every lane busy, contiguous stores).  The
    // edge's row terms alpha(i) + ro(i) and column terms beta(j) + co(j) go to the wave's
    // scratch first; mu = exp(x - m) / s with m the maximum and s the sum.
    constexpr int kF = (CP * CP + kWave - 1) / kWave;
    const int di = kWave / C, dj = kWave - di * C;          // the step of 64 entries
    const int i0 = lane / C, j0 = lane - i0 * C;
    const int scr = ly.scr + w * 64;
    // alpha_t at LDS offset al, beta_{t+1} at be
    auto form_edge = [&](int t, int al, int be) {
        const int lc = Ly::core(t), lro = Ly::ro(t), lco = Ly::co(t);
        if (lane < C) {
            F(scr + lane) = F(al + lane) + (float)Dd(lro + 2 * lane);
            F(scr + 32 + lane) = F(be + lane) + (float)Dd(lco + 2 * lane);
        }
        wave_sync();
        float x[kF];
        float m = -INFINITY;
        int i = i0, jj = j0;
#pragma unroll
        for (int q = 0; q < kF; ++q) {
            const int ic = min(i, C - 1);
            const float v = F(scr + ic) + F(scr + 32 + jj) + F(lc + ic * kLd + jj);
            x[q] = lane + kWave * q < CC ? v : -INFINITY;
            m = fmaxf(m, x[q]);
            jj += dj;
            i += di;
            const bool wrap = jj >= C;
            jj -= wrap ? C : 0;
            i += wrap ? 1 : 0;
        }
        m = wave_max_fast(m);
        float s = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int q = 0; q < kF; ++q) {
                x[q] = fexp(x[q] - m);
                s += x[q];
            }
        }
        s = wave_sum_fast(s);
        const float inv = m == -INFINITY ? 0.f : 1.f / s;
        float* out = a.marg + ((size_t)b * E + t) * CC;
#pragma unroll
        for (int q = 0; q < kF; ++q) {
            const int v = lane + kWave * q;
            if (v < CC) out[v] = m == -INFINITY ? 0.f : x[q] * inv;
        }
        wave_sync();   // the scratch is rewritten for the wave's next edge
    };

    __shared__ double rootShift[2];
    for (int l = T.D; l >= 1; --l) {
        const int nn = uni(T.n[l]), nprev = uni(T.n[l - 1]), vb0 = uni(T.vbase[l - 1]);
        const int ub = uni(U(l, 0)), ub0 = uni(U(l - 1, 0));
        // two tasks per node, the copies folded into them: u_L = u_N with u_R = u_N (x) L
        // (or v_L = v_N without a right child), and v_R = v_N with v_L = R (x) v_N.  On the
        // leaf level (a leaf t holds alpha_t and beta_{t+1}) each task goes on to the
        // marginals of the edge whose vectors it has just completed, reading the copied one
        // from the parent, so the copies are not needed there.
        const bool leaves = l == 1, form = leaves && a.marg;
        for (int task = w; task < 2 * nn; task += kSmallWaves) {
            const int k = task >> 1, which = task & 1;
            const bool right = 2 * k + 1 < nprev;
            const int uN = ub + k * 2 * CP, vN = uN + CP;
            const int uL = ub0 + 2 * k * 2 * CP, uR = uL + 2 * CP;
            if (which == 0) {
                if (!leaves && lane < CP) {
                    F(uL + lane) = F(uN + lane);
                    if (!right) F(uL + CP + lane) = F(vN + lane);
                }
                if (right) {   // u_R = u_N (x) L
                    const int sl = uni(H(ly.info + vb0 + 2 * k)) & kSlotMask;
                    const double zs = vec_log<CP, false>(ly, uN, sl, uR, scr);
                    if (l == T.D && lane == 0) rootShift[0] = zs;
                    if (form) form_edge(2 * k + 1, uR, vN);
                } else if (form) {
                    form_edge(2 * k, uN, vN);
                }
            } else if (right) {
                if (!leaves && lane < CP) F(uR + CP + lane) = F(vN + lane);
                // v_L = R (x) v_N
                const int sr = uni(H(ly.info + vb0 + 2 * k + 1)) & kSlotMask;
                const double zs = vec_log<CP, true>(ly, vN, sr, uL + CP, scr);
                if (l == T.D && lane == 0) rootShift[1] = zs;
                if (form) form_edge(2 * k, uN, uL + CP);
            }
        }
        __syncthreads();
        if (l == T.D) {
            if (a.logZ && w == kSmallWaves - 1) {
                const int uR = U(T.D - 1, 1), vL = U(T.D - 1, 0) + CP;
                const float xb = lane < C ? F(uR + lane) + F(vL + lane) : -INFINITY;
                const float m = wave_max_fast(xb);
                const float s = wave_sum_fast(m == -INFINITY ? 0.f : fexp(xb - m));
                lz = (m == -INFINITY) ? -INFINITY
                                      : (float)(rootShift[0] + rootShift[1] + (double)(m + flog(s)));
            }
            if (!a.marg) {   // log Z only
                store_logz();
                return;
            }
        }
    }
    // a single edge (no tree levels): its vectors are the root's zeros
    if (T.D == 0 && w == 0) form_edge(0, U(0, 0), U(0, 0) + CP);
    store_logz();
    zero_padding();
}

// ================================================================== max semiring
// LDS layout (float offsets): leaves fp32 [E][C][C] | product slots fp64 [E-1][C][C] |
// last leaf again in fp64 [C][C] | forward scores fp64 [nodes][C] | last scores fp64 [C] |
// node table (16-bit slots, as for the log semiring) | backpointers u8 [C][E rounded up to
// 32] (column-major: the backtrace reads 32 edges of a column at once; the padding edges
// map every label to itself, so the backtrace runs through whole chunks of 32).  Above
// level 1 the only leaf that can still be an operand is the last one (through nodes whose
// right half is padding), so levels >= 2 read fp64 only.
struct MaxLayout {
    int C, CC, leaves, slots, lastc, vecs, dlast, info, bp;
    __device__ void init(int c, int E, int nodes) {
        C = c;
        CC = c * c;
        leaves = 0;
        slots = align4(E * CC);
        lastc = slots + (E - 1) * CC * 2;
        vecs = lastc + CC * 2;
        dlast = vecs + nodes * c * 2;
        info = 2 * (dlast + 2 * c);             // in halves
        bp = align4(dlast + 2 * c + (nodes + 1) / 2);
    }
    // fp64 node of a level >= 1 node-table slot: a product slot or the last leaf
    __device__ int node64(int slot, int E) const {
        return slot < E ? lastc : slots + (slot - E) * CC * 2;
    }
};

// quotient x / d for 0 <= x < 2^22 and 1 <= d, with inv = 1.0f / d (float estimate, then
// corrected, so it is exact)
__device__ __forceinline__ int fdiv(int x, int d, float inv) {
    int q = (int)((float)x * inv);
    q -= q * d > x;
    q += (q + 1) * d <= x;
    return q;
}

// DPP permutation kCtrl of a float64 (both halves moved alike)
template <int kCtrl>
__device__ __forceinline__ double dpp_d(double x) {
    const uint64_t u = __double_as_longlong(x);
    const int lo = (int)(unsigned)u, hi = (int)(unsigned)(u >> 32);
    const unsigned rlo = (unsigned)__builtin_amdgcn_update_dpp(lo, lo, kCtrl, 0xF, 0xF, false);
    const unsigned rhi = (unsigned)__builtin_amdgcn_update_dpp(hi, hi, kCtrl, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)rhi << 32) | rlo));
}

// x of lane l ^ kXor within its quad of lanes (DPP quad_perm [1,0,3,2] / [2,3,0,1]), float64
template <int kXor>
__device__ __forceinline__ double quad_xor_d(double x) {
    return dpp_d<kXor == 1 ? 0xB1 : 0x4E>(x);
}

__device__ __forceinline__ double readlane_d(double x, int lane) {
    const uint64_t u = __double_as_longlong(x);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, lane);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), lane);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Maximum of a float64 over the wave (uniform result): DPP inside each row of 16 lanes
// (quad swaps, then the mirrors within 8 and within 16), readlane across the rows.  A max is
// exact, so the order of the steps does not matter.
__device__ __forceinline__ double wave_max_dpp_d(double x) {
    x = fmax(x, dpp_d<0xB1>(x));
    x = fmax(x, dpp_d<0x4E>(x));
    x = fmax(x, dpp_d<0x141>(x));
    x = fmax(x, dpp_d<0x140>(x));
    return fmax(fmax(readlane_d(x, 0), readlane_d(x, 16)), fmax(readlane_d(x, 32), readlane_d(x, 48)));
}

// All products of level l, P = L (x) R in (max, +), float64, by the whole workgroup.  The
// outputs of a product are cut into MR x MC tiles and each tile goes to a group of kS
// consecutive lanes (kS = 2 or 4, inside one DPP quad): lane s of the group takes the
// contraction indices q = s, s + kS, ... (clamped to C - 1: a repeated index leaves a max
// unchanged), and the group's partial maxima are then combined by DPP.  A max is exact in
// any order, so splitting q changes no bit of the result; it cuts the chain of dependent
// maxima and lets larger register tiles (fewer LDS reads per pair) keep enough lanes busy.
// Entries past C are computed from neighbouring data and not stored.  kLeaves: level 1
// (fp32 leaves).  kC > 0: C == kC known at compile time (strides fold into the LDS offsets
// and the index loop unrolls); 0: C at run time.
template <int MR, int MC, int kS, bool kLeaves, int kC>
__device__ void block_prod_max(const MaxLayout& ly, int E, int np, int vb0, int pbase) {
    using T = typename std::conditional<kLeaves, float, double>::type;
    static_assert(kS == 2 || kS == 4, "the q split runs inside a DPP quad");
    static_assert((MR * MC) % kS == 0, "every lane of a group stores the same count");
    constexpr int kPer = MR * MC / kS;   // entries stored per lane
    const int C = kC > 0 ? kC : ly.C, CC = C * C;
    const int TR = (C + MR - 1) / MR, TC = (C + MC - 1) / MC, tpp = TR * TC;
    const float invTpp = 1.f / (float)tpp, invTc = 1.f / (float)TC;
    const int nq = (C + kS - 1) / kS;
    const int total = np * tpp * kS;   // lanes; a multiple of kS, and so is every stride
    const int s = (int)(threadIdx.x % kS);
    const T* const nodes = reinterpret_cast<const T*>(ts_small_lds);   // element index
    double* const prod = reinterpret_cast<double*>(ts_small_lds) + ly.slots / 2;
    for (int g = threadIdx.x; g < total; g += kSmallThreads) {
        const int tile = g / kS;
        const int k = fdiv(tile, tpp, invTpp), rem = tile - k * tpp;
        const int tr = fdiv(rem, TC, invTc), tc = rem - tr * TC;
        const int sl = H(ly.info + vb0 + 2 * k) & kSlotMask, sr = H(ly.info + vb0 + 2 * k + 1) & kSlotMask;
        // element offsets of the operands (leaves: floats; fp64 nodes: doubles)
        const int lb = kLeaves ? ly.leaves + sl * CC : ly.node64(sl, E) / 2;
        const int rb = kLeaves ? ly.leaves + sr * CC : ly.node64(sr, E) / 2;
        const int r0 = tr * MR, c0 = tc * MC;
        // rows past C repeat row C - 1 (MR - 1 rows could otherwise run past the operand);
        // columns past C read at most MC - 1 entries beyond it, which stay inside the layout
        int lrow[MR];
#pragma unroll
        for (int i = 0; i < MR; ++i) lrow[i] = lb + min(r0 + i, C - 1) * C;
        const T* rp = nodes + rb + c0;       // R[q][c0 + j] = rp[q * C + j]
        double acc[MR * MC];
#pragma unroll
        for (int e = 0; e < MR * MC; ++e) acc[e] = -INFINITY;
        auto step = [&](int q) {
            double av[MR], bv[MC];
#pragma unroll
            for (int i = 0; i < MR; ++i) av[i] = (double)nodes[lrow[i] + q];
#pragma unroll
            for (int j = 0; j < MC; ++j) bv[j] = (double)rp[q * C + j];
#pragma unroll
            for (int i = 0; i < MR; ++i)
#pragma unroll
                for (int j = 0; j < MC; ++j) acc[i * MC + j] = fmax(acc[i * MC + j], av[i] + bv[j]);
        };
        if constexpr (kC > 0) {
#pragma unroll 2
            for (int i = 0; i < nq; ++i) step(min(s + kS * i, C - 1));
        } else {
            int i = 0;
            for (; i + 2 <= nq; i += 2) {   // two indices per trip: their reads go out together
                step(min(s + kS * i, C - 1));
                step(min(s + kS * (i + 1), C - 1));
            }
            if (i < nq) step(min(s + kS * i, C - 1));
        }
#pragma unroll
        for (int e = 0; e < MR * MC; ++e) acc[e] = fmax(acc[e], quad_xor_d<1>(acc[e]));
        if constexpr (kS == 4) {
#pragma unroll
            for (int e = 0; e < MR * MC; ++e) acc[e] = fmax(acc[e], quad_xor_d<2>(acc[e]));
        }
        // lane s stores the entries e = m * kS + s of the tile
        double* out = prod + (pbase + k) * CC;
#pragma unroll
        for (int m = 0; m < kPer; ++m) {
            double v = acc[m * kS];
#pragma unroll
            for (int u = 1; u < kS; ++u) v = s == u ? acc[m * kS + u] : v;
            const int e = m * kS + s, r = r0 + e / MC, c = c0 + e % MC;
            if (r < C && c < C) out[r * C + c] = v;
        }
    }
}

// Tile shape and q split of a level: the largest tiles (fewest LDS reads per pair) that still
// give at least six waves of lanes, at most one tile per lane; the widest level splits q in
// two only.
template <bool kLeaves, int kC>
__device__ void level_prod_max_c(const MaxLayout& ly, int E, int np, int vb0, int pbase) {
    const int C = ly.C;
    auto lanes = [&](int mr, int mc, int ks) {
        return np * ((C + mr - 1) / mr) * ((C + mc - 1) / mc) * ks;
    };
    constexpr int kEnough = 6 * kWave;
    if (lanes(4, 4, 4) > kSmallThreads) block_prod_max<4, 4, 2, kLeaves, kC>(ly, E, np, vb0, pbase);
    else if (lanes(4, 4, 4) >= kEnough) block_prod_max<4, 4, 4, kLeaves, kC>(ly, E, np, vb0, pbase);
    else if (lanes(2, 4, 4) >= kEnough) block_prod_max<2, 4, 4, kLeaves, kC>(ly, E, np, vb0, pbase);
    else block_prod_max<2, 2, 4, kLeaves, kC>(ly, E, np, vb0, pbase);
}

// C equal to the padded size CP takes the compile-time variant
template <bool kLeaves, int CP>
__device__ void level_prod_max(const MaxLayout& ly, int E, int np, int vb0, int pbase) {
    if (ly.C == CP) level_prod_max_c<kLeaves, CP>(ly, E, np, vb0, pbase);
    else level_prod_max_c<kLeaves, 0>(ly, E, np, vb0, pbase);
}

__device__ __forceinline__ double xor32_max_d(double x) {
    const uint64_t u = __double_as_longlong(x);
    const auto lo = __builtin_amdgcn_permlane32_swap((unsigned)u, (unsigned)u, false, false);
    const auto hi = __builtin_amdgcn_permlane32_swap((unsigned)(u >> 32), (unsigned)(u >> 32), false, false);
    const double a = __longlong_as_double((long long)(((uint64_t)hi[0] << 32) | lo[0]));
    const double b = __longlong_as_double((long long)(((uint64_t)hi[1] << 32) | lo[1]));
    return fmax(a, b);
}

// One wave: y[j] = max_i x[i] + N[i][j] with N a float64 node at Nb.  Lane l computes
// column l % 32 over half l / 32 of i; the halves meet through a cross-half max.  Past C the
// index repeats C - 1, which leaves a max unchanged.
template <int CP>
__device__ void wave_vec_max(int C, int x, int Nb, int y) {
    constexpr int kHalf = CP / 2;
    const int lane = threadIdx.x % kWave, o = lane & 31, h = lane >> 5;
    const int j = min(o, C - 1);
    double m = -INFINITY;
#pragma unroll
    for (int q = 0; q < kHalf; ++q) {
        const int ic = min(h * kHalf + q, C - 1);
        m = fmax(m, Dd(x + 2 * ic) + Dd(Nb + 2 * (ic * C + j)));
    }
    m = xor32_max_d(m);
    if (h == 0 && o < C) Dd(y + 2 * o) = m;
    wave_sync();
}

// One wave, one edge (fp32 leaf at Nb) after forward scores x (fp64): bp[j * ep] = the lowest
// i maximising x[i] + l[i][j] (the backpointer of column j; the column-major layout puts
// a column's edges next to each other), and the maximum itself into y when y >= 0 (the next
// edge's forward scores) and into dl when dl >= 0 (the last edge's scores).  Lane l takes
// column l % 32 over half l / 32 of i; the upper half wins only when strictly better.
template <int CP>
__device__ void wave_edge_argmax(int C, int x, int Nb, uint8_t* bp, int ep, int y, int dl) {
    constexpr int kHalf = CP / 2;
    const int lane = threadIdx.x % kWave, o = lane & 31, h = lane >> 5;
    const int j = min(o, C - 1);
    double best = -INFINITY;
    int arg = h * kHalf;
#pragma unroll
    for (int q = 0; q < kHalf; ++q) {
        const int i = h * kHalf + q, ic = min(i, C - 1);
        const double v = Dd(x + 2 * ic) + (double)F(Nb + ic * C + j);
        const bool better = i < C && v > best;   // strict: the lowest index wins ties
        best = better ? v : best;
        arg = better ? i : arg;
    }
    const double ob = xor32_max_d(best);   // max of both halves
    const bool upperWins = h == 0 && ob > best;
    const int oarg = __shfl_xor(arg, 32, kWave);
    if (h == 0 && o < C) {
        bp[o * ep] = (uint8_t)(upperWins ? oarg : arg);
        if (y >= 0) Dd(y + 2 * o) = ob;
        if (dl >= 0) Dd(dl + 2 * o) = ob;
    }
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
    const int CC = C * C;
    const float* gleaf = a.pot + (size_t)b * E * CC;
    // the first loads of the potentials go out before the length is known
    LeafBatch<kLeafBatch> lb;
    lb.load(gleaf, 0, (int)E * CC);
    const int L = (int)clamp_len(a.lengths, b, a.N), Eb = L - 1;
    const int w = uni(threadIdx.x / kWave), lane = threadIdx.x % kWave;
    int32_t* path = a.path + (size_t)b * a.N;
    // past the length the path is -1 (written last, as the marginals' padding)
    auto pad_path = [&]() {
        for (int64_t n = L + threadIdx.x; n < a.N; n += kSmallThreads) path[n] = -1;
    };
    if (Eb == 0) {
        if (threadIdx.x == 0) { path[0] = 0; a.score[b] = 0.f; }
        pad_path();
        return;
    }
    __shared__ Tree T;
    const int nodes = (int)small_tree_nodes(Eb);
    MaxLayout ly;
    ly.init(C, Eb, nodes);
    // ---- tree, node table and leaves (fp32, flat)
    if (w == kSmallWaves - 1) tree_init_wave(T, Eb);
    build_node_table(Eb, nodes, ly.info);
    {
        const int n = Eb * CC;
        lb.store(ly.leaves, 0, n);
        for (int base = kLeafBatch * kSmallThreads; base < n; base += kLeafBatch * kSmallThreads) {
            lb.load(gleaf, base, n);
            lb.store(ly.leaves, base, n);
        }
    }
    // the root's forward scores (zeros; the root is the last node): nothing else writes the
    // score vectors before the forward sweep
    if (w == 0 && lane < C) Dd(ly.vecs + (nodes - 1) * 2 * C + 2 * lane) = 0.0;
    // padding edges [Eb, ep) of the backpointers: z_t = z_{t+1}
    if ((int)threadIdx.x < C) {
        uint8_t* col = reinterpret_cast<uint8_t*>(ts_small_lds + ly.bp) + threadIdx.x * ((Eb + 31) & ~31);
        for (int t = Eb; t < ((Eb + 31) & ~31); ++t) col[t] = (uint8_t)threadIdx.x;
    }
    __syncthreads();
    // the last leaf in fp64 for levels >= 2 (read only after the level-1 barrier)
    for (int i = threadIdx.x; i < CC; i += kSmallThreads)
        Dd(ly.lastc + 2 * i) = (double)F(ly.leaves + (Eb - 1) * CC + i);
    // ---- up-sweep: all threads share each level's products, below the root (the forward
    // scores start from the root with zeros and only use its children's matrices)
    for (int l = 1; l < T.D; ++l) {
        const int np = uni(T.products(l)), vb0 = uni(T.vbase[l - 1]), pb = uni(T.pbase[l]);
        if (l == 1) level_prod_max<true, CP>(ly, Eb, np, vb0, pb);
        else level_prod_max<false, CP>(ly, Eb, np, vb0, pb);
        __syncthreads();
    }
    // ---- forward scores: u_L = u_N, u_R = u_N (x) L   (root: zeros, set with the leaves)
    auto U = [&](int l, int k) { return ly.vecs + (T.vbase[l] + k) * 2 * C; };
    // backpointers, column-major with ep (edges rounded up to 32) bytes per column; the
    // padding edges were set to the identity with the leaves
    uint8_t* bp = reinterpret_cast<uint8_t*>(ts_small_lds + ly.bp);
    const int ep = (Eb + 31) & ~31;
    for (int l = T.D; l >= 1; --l) {
        const int nn = uni(T.n[l]), nprev = uni(T.n[l - 1]), vb0 = uni(T.vbase[l - 1]);
        const int ub = uni(U(l, 0)), ub0 = uni(U(l - 1, 0));
        // one task per node: u_L = u_N, and u_R = u_N (x) L when there is a right child.  On
        // the leaf level the same maximisation gives the left edge's backpointers, and the
        // right edge's follow from u_R; u_L is read from the parent there (no copy).
        for (int k = w; k < nn; k += kSmallWaves) {
            const int uN = ub + k * 2 * C, uL = ub0 + 2 * k * 2 * C;
            const bool right = 2 * k + 1 < nprev;
            if (l == 1) {
                const int t = 2 * k;
                wave_edge_argmax<CP>(C, uN, ly.leaves + t * CC, bp + t, ep, right ? uL + 2 * C : -1,
                                     t == Eb - 1 ? ly.dlast : -1);
                if (right)
                    wave_edge_argmax<CP>(C, uL + 2 * C, ly.leaves + (t + 1) * CC, bp + t + 1, ep, -1,
                                         t + 1 == Eb - 1 ? ly.dlast : -1);
                continue;
            }
            if (lane < C) Dd(uL + 2 * lane) = Dd(uN + 2 * lane);
            if (right) {
                const int sl = uni(H(ly.info + vb0 + 2 * k)) & kSlotMask;
                wave_vec_max<CP>(C, uN, ly.node64(sl, Eb), uL + 2 * C);
            }
        }
        __syncthreads();
    }
    if (T.D == 0) {   // one edge: its forward scores are the root's zeros
        if (w == 0) wave_edge_argmax<CP>(C, U(0, 0), ly.leaves, bp, ep, -1, ly.dlast);
        __syncthreads();
    }
    // ---- last label (lowest argmax: the first lane holding the maximum), score, backtrace.
    // Wave 0 keeps 32 edges of backpointers at a time in registers (lane j holds column j,
    // four edges per register) and follows the path with readlane; the padding edges past
    // Eb leave the label unchanged.
    if (w == 0) {
        const double v = lane < C ? Dd(ly.dlast + 2 * lane) : -INFINITY;
        const double best = wave_max_dpp_d(v);
        const uint64_t hit = __builtin_amdgcn_ballot_w64(lane < C && v == best);
        int z = hit ? uni((int)__builtin_ctzll(hit)) : 0;
        if (lane == 0) {
            a.score[b] = (float)best;
            path[Eb] = z;
        }
        const int jc = min(lane, C - 1);
        for (int c = (Eb - 1) >> 5; c >= 0; --c) {       // edges [32 c, 32 c + 32)
            const int t0 = 32 * c;
            unsigned pk[8];
#pragma unroll
            for (int g = 0; g < 8; ++g) pk[g] = *reinterpret_cast<const unsigned*>(bp + jc * ep + t0 + 4 * g);
            int zs = 0;   // lane t - t0 records z_t
#pragma unroll
            for (int g = 7; g >= 0; --g) {
#pragma unroll
                for (int e = 3; e >= 0; --e) {
                    z = (__builtin_amdgcn_readlane(pk[g], z) >> (8 * e)) & 0xff;
                    zs = lane == 4 * g + e ? z : zs;
                }
            }
            if (lane < min(32, Eb - t0)) path[t0 + lane] = zs;
        }
    }
    pad_path();
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
    const int64_t CP = C <= 8 ? 8 : C <= 16 ? 16 : C <= 20 ? 20 : C <= 24 ? 24 : 32;   // as the launcher
    const int64_t coreF = (CP * (CP + 1) + 1) & ~1, slotF = coreF + 4 * CP;
    const int64_t floats = (2 * E - 1) * slotF + small_tree_nodes(E) * 2 * CP + kSmallWaves * 64;
    return sizeof(float) * (size_t)floats + 2 * (size_t)small_tree_nodes(E);   // + node table
}

size_t small_max_lds_bytes(int64_t E, int64_t C) {
    if (E < 1) return 0;
    const int64_t CC = C * C, nodes = small_tree_nodes(E);
    const int64_t floats = (E * CC + 3) + (E - 1) * CC * 2 + CC * 2 + nodes * C * 2 + 2 * C +
                           (nodes + 1) / 2 + 3;   // + node table, alignment of bp
    return sizeof(float) * (size_t)floats + (size_t)(((E + 31) & ~31) * C);
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
    if (C <= 20) return small_log_cp<20>(a, B, lds, s);
    if (C <= 24) return small_log_cp<24>(a, B, lds, s);
    return small_log_cp<32>(a, B, lds, s);
}

hipError_t launch_small_max(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                            int64_t C, int32_t* path, float* score, hipStream_t s) {
    SmallMaxArgs a{pot, lengths, N, (int)C, path, score};
    const size_t lds = small_max_lds_bytes(N - 1, C);
    if (C <= 8) return small_max_cp<8>(a, B, lds, s);
    if (C <= 16) return small_max_cp<16>(a, B, lds, s);
    if (C <= 20) return small_max_cp<20>(a, B, lds, s);
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
    if (C <= 20) return small_both_cp<20>(la, ma, B, lds, s);
    if (C <= 24) return small_both_cp<24>(la, ma, B, lds, s);
    return small_both_cp<32>(la, ma, B, lds, s);
}

}  // namespace tsc
