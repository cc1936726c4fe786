// internal.h -- workspace plan and kernel launchers shared by the C-ABI layer (api.cpp)
// and the HIP kernels.  Not part of the public interface.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tsc {

constexpr int kMaxLabels = 256;   // largest C (backpointers are one byte; panels fit LDS)
constexpr int kMaxLevels = 40;

// Tree over the edges of every sequence: Np = smallest power of two >= N-1 leaves,
// D = log2(Np) levels above the leaves.  Node k of level l covers edges
// [k*2^l, (k+1)*2^l); it is present for sequence b iff k*2^l < E_b = len_b - 1.
// A present node whose right child is absent equals its left child (the right
// half is all padding, i.e. the semiring identity).
//
// Log-semiring node storage (levels 1..D): the node matrix is
//   P[a][c] = ro[a] + co[c] + core[a][c]
// with ro, co in float64 and core in float32 (core = log of an exp-shifted product, so
// it stays small however long the span is).  Leaves (level 0) are the raw potentials
// with ro = co = 0.
struct Plan {
    int64_t B = 0, N = 0, C = 0, E = 0, Np = 1;
    int D = 0;
    int op = 0;
    bool fused = false;   // single-launch path of small.hip (no workspace)
    // log semiring for C <= 64 without masks (chunk.hip): k_chunk_up folds every chunk of
    // 2^lc edges into its level-lc node, k_chunk_scan runs the forward and backward
    // recursions over a sequence's chunk nodes (log Z and the chunks' outside vectors
    // u[lc], v[lc]) and k_chunk_form the marginals inside each chunk; no other level is formed
    bool chunk = false;
    int lc = 0;
    // log Z on the tree (C <= kNodeScanMaxLabels, no masks): the up-sweep stops at this level
    // and k_node_scan runs the recursion over its nodes (0: the tree up to the root)
    int scan_level = 0;
    int32_t* clin = nullptr;   // per chunk node: its core holds S (1) or log S (0)
    // log semiring, levels 1..D (index by level)
    float* core[kMaxLevels] = {};
    double* ro[kMaxLevels] = {};
    double* co[kMaxLevels] = {};
    // per-tile partial maxima of the rows (core + co) and columns (core + ro) of every node
    // of levels 1..D, [nodes][C][ntile[l]]: the exp shifts of the next level's products; and
    // the leaves' row and column maxima [B, E, C]
    float* pmr[kMaxLevels] = {};
    float* pmc[kMaxLevels] = {};
    float* lrmax = nullptr;
    float* lcmax = nullptr;
    // marginals: per edge, whether its potentials reach magnitude kWideMag (the edge's
    // messages and marginal exponents are then formed in float64), [B][E]
    int32_t* wide = nullptr;
    // finiteness bitmasks (only with masks; nullptr otherwise) of every node consumed by a
    // product (levels 0..D-1; level 0 is the leaves [B, E]): rbits [nodes][C][bw] has bit c of row a set iff entry (a, c) is
    // finite, cbits [nodes][C][bw] bit a of column c.  An entry of L (x) R is -inf exactly
    // when row a of L and column c of R share no finite index, which spares the exact
    // fallback of the exp-shifted product for structural zeros.
    uint64_t* rbits[kMaxLevels] = {};
    uint64_t* cbits[kMaxLevels] = {};
    int bw = 1;                 // 64-bit words per line: ceil(C / 64)
    int ntile[kMaxLevels] = {}; // output tiles per matrix dimension of each level (up_tile)
    // outside vectors of the nodes of levels 1..D-1 (normalised to max 0)
    float* u[kMaxLevels] = {};
    float* v[kMaxLevels] = {};
    // max semiring (float64 nodes, levels 1..D-1: the root matrix is never needed) and forward
    // vectors (levels 1..D-1)
    double* mnode[kMaxLevels] = {};
    double* mu[kMaxLevels] = {};
    uint8_t* bp = nullptr;      // [B, E, C] backpointers
    int32_t* zlast = nullptr;   // [B] label of the last token
    int64_t dec_chunk = 1;      // edges per decode chunk
    int64_t dec_nchunks = 0;    // chunks per sequence
    uint8_t* dec_map = nullptr; // [B, nchunks, C] label at chunk start given label at its end
    int32_t* dec_zend = nullptr;// [B, nchunks] label at each chunk's end position
    size_t bytes = 0;
};

constexpr int kChunkLog = 4;   // chunks of at most 16 edges
constexpr int kNodeScanMaxLabels = 128;   // the recursion over nodes keeps two nodes in LDS

// Potentials of magnitude above this make float32 rounding of a sum such as message +
// potential (about 2^-24 of the magnitude per operation) approach the marginals' absolute
// tolerance; edges that reach it take the float64 formation of those sums.
constexpr float kWideMag = 16.f;

// Whether the log-semiring tree of C labels takes the chunk kernels (C <= 64, no masks).
bool chunk_path(int64_t C, bool masks);

// Output tile edge of a level of the log-semiring up-sweep with `nodes` nodes (all
// sequences) of C labels.  32 (the latency-bound kernel, no finiteness masks) while the
// level has at most kSmallTiles such tiles -- about 4 per compute unit: there each
// workgroup's chain of memory round trips and barriers, not the chip's throughput, sets
// the time; otherwise 64 for C <= 64, and 128 above unless the level has too few 128-wide
// tiles to give every compute unit two of them: then 64 (four times the workgroups, each
// with a quarter of the work and of the latency).
constexpr int64_t kSmallTiles = 1024;
inline int up_tile(int64_t C, int64_t nodes, bool masks) {
    if (!masks) {
        const int64_t t = (C + 31) / 32;
        if (nodes * t * t <= kSmallTiles) return 32;
    }
    if (C <= 64) return 64;
    const int64_t t = (C + 127) / 128;
    return nodes * t * t < 512 ? 64 : 128;
}

// Records `msg` as the calling thread's last error (ts_last_error) and returns `code`.
int report_error(int code, const char* msg);

// Fills the plan; with base == nullptr only sizes are computed.  Returns false on overflow.
// masks: keep finiteness bitmasks of the log-semiring nodes (inputs with many structural
// -inf entries, such as the semi-Markov expansion).
bool make_plan(int op, int64_t B, int64_t N, int64_t C, void* base, Plan* p,
               bool masks = false);

// ---- launchers (return the first HIP error, hipSuccess otherwise) ----
hipError_t launch_logz_tree(const Plan& p, const float* pot, const int32_t* lengths,
                            float* logZ, hipStream_t s);
hipError_t launch_node_scan(const Plan& p, const int32_t* lengths, float* logZ, hipStream_t s);
hipError_t launch_marginals_tree(const Plan& p, const float* pot, const int32_t* lengths,
                                 float* marg, hipStream_t s);
hipError_t launch_viterbi_tree(const Plan& p, const float* pot, const int32_t* lengths,
                               int32_t* path, float* score, hipStream_t s);
hipError_t launch_chunk_up(const Plan& p, const float* pot, const int32_t* lengths,
                           hipStream_t s);
hipError_t launch_chunk_scan(const Plan&, const float*, const int32_t*, float*, hipStream_t);
hipError_t launch_chunk_form(const Plan& p, const float* pot, const int32_t* lengths,
                             float* marg, hipStream_t s);
hipError_t launch_single_token(int64_t B, int64_t N, int64_t C, int op, float* logZ,
                               int32_t* path, float* score, hipStream_t s);
// entropy from marginals mu [B, N-1, C, C]; part is [B, N-1] doubles (unused when N == 1)
hipError_t launch_entropy(const float* mu, const int32_t* lengths, int64_t B, int64_t N,
                          int64_t C, double* part, float* H, hipStream_t s);
// FFBS draws from marginals mu [B, N-1, C, C] with uniforms [S, B, N] into paths [S, B, N]
hipError_t launch_sample(const float* mu, const int32_t* lengths, const float* uniforms,
                         int64_t S, int64_t B, int64_t N, int64_t C, int32_t* paths,
                         hipStream_t s);
// semi-Markov CRF: expand segment potentials [B, N-1, K, C, C] into chain edges over K*C
// states [B, N-1, KC, KC]; gather the segment marginals back; fix one-token log Z; decode
// the expanded Viterbi path into labels [B, N] and segment lengths [B, N-1]
hipError_t launch_semi_expand(const float* sp, const int32_t* lengths, int64_t B, int64_t N,
                              int64_t K, int64_t C, float* xp, hipStream_t s);
hipError_t launch_semi_gather(const float* xm, int64_t B, int64_t N, int64_t K, int64_t C,
                              float* marg, hipStream_t s);
hipError_t launch_semi_single(const int32_t* lengths, int64_t B, int64_t N, int64_t C,
                              float* logZ, hipStream_t s);
hipError_t launch_semi_decode(const int32_t* xs, const int32_t* lengths, int64_t B, int64_t N,
                              int64_t C, int32_t* path, int32_t* seglen, hipStream_t s);
hipError_t launch_logz_sequential(const float* pot, const int32_t* lengths, int64_t B,
                                  int64_t N, int64_t C, float* logZ, hipStream_t s);
hipError_t launch_log_density(const float* pot, const int32_t* lengths, const int32_t* labels,
                              const float* logZ, int64_t B, int64_t N, int64_t C, float* out,
                              hipStream_t s);

}  // namespace tsc
