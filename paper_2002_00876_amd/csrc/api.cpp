// api.cpp -- the C ABI declared in include/ts_chain.h: argument validation, workspace
// planning and the kernel sequence of each call.  All arithmetic happens in the HIP
// kernels (tree_log.hip, tree_max.hip, small.hip); this file only checks and enqueues.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"
#include "small.h"
#include "ts_chain.h"

namespace tsc {
namespace {

thread_local std::string g_err;

ts_status fail(ts_status code, const std::string& msg) {
    g_err = msg;
    return code;
}

// Side stream of the combined marginals + Viterbi call on the multi-launch tree: one per
// device (default priority, created on first use and kept until the process ends), with an
// event for the fork from the caller's stream and one for the join back into it.  A record
// and the wait on it are made under one lock, so concurrent callers cannot interleave them
// (a wait takes the event's latest record).
constexpr int kMaxDevices = 64;
struct Side {
    hipStream_t stream = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;
Side g_side[kMaxDevices];

hipError_t side_of_current_device(Side** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_side_mu);
    Side& sd = g_side[dev];
    if (!sd.stream) {
        // all three or none: a failed creation releases what was made and is retried later
        Side made;
        e = hipEventCreateWithFlags(&made.fork, hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&made.join, hipEventDisableTiming);
        if (e == hipSuccess) e = hipStreamCreateWithFlags(&made.stream, hipStreamNonBlocking);
        if (e != hipSuccess) {
            if (made.fork) (void)hipEventDestroy(made.fork);
            if (made.join) (void)hipEventDestroy(made.join);
            return e;
        }
        sd = made;
    }
    *out = &sd;
    return hipSuccess;
}

// `to` waits for everything enqueued on `from` so far
hipError_t link(hipEvent_t ev, hipStream_t from, hipStream_t to) {
    std::lock_guard<std::mutex> lock(g_side_mu);
    hipError_t e = hipEventRecord(ev, from);
    return e == hipSuccess ? hipStreamWaitEvent(to, ev, 0) : e;
}

constexpr size_t kAlign = 256;
constexpr int64_t kMaxGridItems = (int64_t)1 << 29;   // B * N bound: grids stay below 2^31

struct Bump {
    char* base;
    size_t off = 0;
    template <class T>
    T* take(size_t count) {
        off = (off + kAlign - 1) / kAlign * kAlign;
        T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
        off += count * sizeof(T);
        return p;
    }
};

bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > INT64_MAX / a) return false;
    *out = a * b;
    return true;
}

}  // namespace

int report_error(int code, const char* msg) { return fail(code, msg); }

// The level at which log Z's up-sweep stops for the recursion over its nodes, 0 for the tree
// to the root.  A level of few small products costs about kLevelUs (its launch and memory
// round trips), a step of the recursion about kStepUs: with S = 2^l edges per node, levels
// 1..l and ceil(E / S) steps against D levels and the root's log-sum-exp.
int node_scan_level(int64_t E, int D) {
    constexpr double kLevelUs = 12.0, kStepUs = 1.0, kScanUs = 5.0, kRootUs = 10.0;
    double best = D * kLevelUs + kRootUs;
    int level = 0;
    for (int l = 1; l < D; ++l) {
        const double t = l * kLevelUs + (double)((E + (int64_t(1) << l) - 1) >> l) * kStepUs + kScanUs;
        if (t < best) {
            best = t;
            level = l;
        }
    }
    return level;
}

bool make_plan(int op, int64_t B, int64_t N, int64_t C, void* base, Plan* p, bool masks) {
    *p = Plan{};
    p->B = B; p->N = N; p->C = C; p->E = N - 1; p->op = op;
    int64_t cc, bcc;
    // every buffer below is at most B * Np * C * C * 8 bytes; bound that product
    if (!mul_ok(C, C, &cc) || !mul_ok(B, cc, &bcc) || !mul_ok(bcc, 2 * (N + 1), &cc) ||
        !mul_ok(cc, 8, &cc) || cc > ((int64_t)1 << 60))
        return false;
    // launch grids reach B * (N-1) * 4 workgroups (one per edge, or per tile of a tree
    // node); keep that within one launch's grid
    if (!mul_ok(B, N, &cc) || cc > kMaxGridItems) return false;
    if (N == 1) return true;  // no edges: no workspace
    // small label sets: one fused launch per call, tree kept in LDS, no workspace.
    // TS_PATH=tree forces the multi-launch tree (used by the tests to cover both paths).
    const char* path = std::getenv("TS_PATH");
    const bool force_tree = path && std::strcmp(path, "tree") == 0;
    if (!force_tree && small_path_fits(N, C)) {
        p->fused = true;
        return true;
    }
    int64_t Np = 1;
    int D = 0;
    while (Np < p->E) { Np <<= 1; ++D; }
    p->Np = Np; p->D = D;
    Bump bump{static_cast<char*>(base)};
    if (op == TS_OP_LOGPARTITION || op == TS_OP_MARGINALS) {
        p->chunk = chunk_path(C, masks);
        if (p->chunk) {
            // the chunk nodes (level lc; the leaves themselves when lc == 0) and, for the
            // marginals, their outside vectors
            // chunks of S = 2^lc edges.  For log Z alone the critical path is about S - 1
            // chunk products and E / S steps of the recursion over chunks; with their
            // measured costs (about 2 : 1.1) its minimum lies near S = sqrt(0.55 E).  The
            // marginals keep the longest chunks: every chunk boundary passes the messages
            // through float storage, and fewer boundaries keep wide-range inputs within
            // the marginals' absolute tolerance.
            int lc = D < kChunkLog ? D : kChunkLog;
            if (op == TS_OP_LOGPARTITION && D > 0) {
                const double sopt = std::sqrt(0.55 * (double)p->E);
                const int l2 = (int)std::lround(std::log2(sopt > 2.0 ? sopt : 2.0));
                lc = l2 < lc ? l2 : lc;
            }
            const size_t n = (size_t)B * (size_t)(Np >> lc);
            p->lc = lc;
            if (lc > 0) {
                p->core[lc] = bump.take<float>(n * C * C);
                p->ro[lc] = bump.take<double>(n * C);
                p->co[lc] = bump.take<double>(n * C);
                p->clin = bump.take<int32_t>(n);
            }
            if (op == TS_OP_MARGINALS) {
                const size_t nv = lc > 0 ? n : (size_t)B * p->E;
                p->u[lc] = bump.take<float>(nv * C);
                p->v[lc] = bump.take<float>(nv * C);
            }
            p->bytes = (bump.off + kAlign - 1) / kAlign * kAlign;
            return true;
        }
        if (op == TS_OP_LOGPARTITION && !masks && C <= kNodeScanMaxLabels && D >= 2)
            p->scan_level = node_scan_level(p->E, D);
        const int top = p->scan_level > 0 ? p->scan_level : D;   // the levels formed
        for (int l = 1; l <= top; ++l) {
            const size_t n = (size_t)B * (size_t)(Np >> l);
            const int tm = up_tile(C, (int64_t)n, masks);
            p->ntile[l] = (int)((C + tm - 1) / tm);
            p->core[l] = bump.take<float>(n * C * C);
            p->ro[l] = bump.take<double>(n * C);
            p->co[l] = bump.take<double>(n * C);
            p->pmr[l] = bump.take<float>(n * C * p->ntile[l]);
            p->pmc[l] = bump.take<float>(n * C * p->ntile[l]);
        }
        p->lrmax = bump.take<float>((size_t)B * p->E * C);
        p->lcmax = bump.take<float>((size_t)B * p->E * C);
        if (op == TS_OP_MARGINALS) p->wide = bump.take<int32_t>((size_t)B * p->E);
        p->bw = (int)((C + 63) / 64);
        for (int l = 0; masks && l < D; ++l) {
            const size_t n = l == 0 ? (size_t)B * p->E : (size_t)B * (size_t)(Np >> l);
            p->rbits[l] = bump.take<uint64_t>(n * C * p->bw);
            p->cbits[l] = bump.take<uint64_t>(n * C * p->bw);
        }
        if (op == TS_OP_MARGINALS)
            for (int l = 1; l < D; ++l) {
                const size_t n = (size_t)B * (size_t)(Np >> l);
                p->u[l] = bump.take<float>(n * C);
                p->v[l] = bump.take<float>(n * C);
            }
    } else {
        for (int l = 1; l < D; ++l) {   // the root's matrix is never formed
            const size_t n = (size_t)B * (size_t)(Np >> l);
            p->mnode[l] = bump.take<double>(n * C * C);
        }
        for (int l = 1; l < D; ++l) {
            const size_t n = (size_t)B * (size_t)(Np >> l);
            p->mu[l] = bump.take<double>(n * C);
        }
        p->bp = bump.take<uint8_t>((size_t)B * p->E * C);
        p->zlast = bump.take<int32_t>((size_t)B);
        // decode chunks: the per-sequence map table (nchunks * C bytes) and one chunk of
        // backpointers (chunk * C bytes) must each fit in 64 KiB of LDS
        int64_t K = 64;
        while (((p->E + K - 1) / K) * C > 65536) K <<= 1;
        if (K * C > 65536) return false;
        p->dec_chunk = K;
        p->dec_nchunks = (p->E + K - 1) / K;
        p->dec_map = bump.take<uint8_t>((size_t)B * p->dec_nchunks * C);
        p->dec_zend = bump.take<int32_t>((size_t)B * p->dec_nchunks);
    }
    p->bytes = (bump.off + kAlign - 1) / kAlign * kAlign;
    return true;
}

namespace {

ts_status check_dims(const float* pot, int64_t B, int64_t N, int64_t C, int op, Plan* plan) {
    if (B < 1 || N < 1 || C < 1)
        return fail(TS_ERR_BAD_DIM, "B, N and C must all be >= 1");
    if (C > kMaxLabels)
        return fail(TS_ERR_BAD_DIM, "C exceeds ts_chain_max_labels() = " +
                                        std::to_string(kMaxLabels));
    if (N > 1 && !pot) return fail(TS_ERR_NULL_ARG, "pot is NULL");
    if (!make_plan(op, B, N, C, nullptr, plan))
        return fail(TS_ERR_BAD_DIM, "problem size overflows the supported range");
    return TS_OK;
}

ts_status check_ws(size_t need, void* ws, size_t ws_bytes) {
    if (need == 0) return TS_OK;
    if (!ws) return fail(TS_ERR_NULL_ARG, "ws is NULL but the call needs a workspace");
    if (ws_bytes < need)
        return fail(TS_ERR_WORKSPACE, "workspace too small: need " + std::to_string(need) +
                                          " bytes, got " + std::to_string(ws_bytes));
    if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
        return fail(TS_ERR_WORKSPACE, "workspace must be 256-byte aligned");
    return TS_OK;
}

ts_status check_common(const float* pot, int64_t B, int64_t N, int64_t C, int op, void* ws,
                       size_t ws_bytes, Plan* plan) {
    ts_status st = check_dims(pot, B, N, C, op, plan);
    if (st == TS_OK) st = check_ws(plan->bytes, ws, ws_bytes);
    if (st == TS_OK && plan->bytes > 0) make_plan(op, B, N, C, ws, plan);
    return st;
}

ts_status check_lengths(const int32_t* lengths, int64_t B, int64_t N, hipStream_t s) {
    const char* env = std::getenv("TS_CHECK");
    if (!lengths || !env || std::strcmp(env, "1") != 0) return TS_OK;
    std::vector<int32_t> h((size_t)B);
    if (hipMemcpyAsync(h.data(), lengths, sizeof(int32_t) * B, hipMemcpyDeviceToHost, s) !=
            hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return fail(TS_ERR_HIP, "could not read lengths for TS_CHECK");
    for (int64_t b = 0; b < B; ++b)
        if (h[b] < 1 || h[b] > N)
            return fail(TS_ERR_LENGTHS, "lengths[" + std::to_string(b) + "] = " +
                                            std::to_string(h[b]) + " is outside [1, N]");
    return TS_OK;
}

ts_status check_labels(const int32_t* labels, const int32_t* lengths, int64_t B, int64_t N,
                       int64_t C, hipStream_t s) {
    const char* env = std::getenv("TS_CHECK");
    if (!env || std::strcmp(env, "1") != 0) return TS_OK;
    std::vector<int32_t> z((size_t)(B * N)), len((size_t)B, (int32_t)N);
    if (hipMemcpyAsync(z.data(), labels, sizeof(int32_t) * B * N, hipMemcpyDeviceToHost, s) !=
            hipSuccess ||
        (lengths && hipMemcpyAsync(len.data(), lengths, sizeof(int32_t) * B,
                                   hipMemcpyDeviceToHost, s) != hipSuccess) ||
        hipStreamSynchronize(s) != hipSuccess)
        return fail(TS_ERR_HIP, "could not read labels for TS_CHECK");
    for (int64_t b = 0; b < B; ++b)
        for (int64_t n = 0; n < len[b] && n < N; ++n)
            if (z[b * N + n] < 0 || z[b * N + n] >= C)
                return fail(TS_ERR_LABELS, "labels[" + std::to_string(b) + ", " +
                                               std::to_string(n) + "] = " +
                                               std::to_string(z[b * N + n]) +
                                               " is outside [0, C)");
    return TS_OK;
}

// Workspace of the derived quantities: the plan of the call they build on, then their own
// buffers (entropy: the marginals and per-edge partials; log density: log Z).
struct Derived {
    Plan base;
    size_t extra = 0, mu = 0, part = 0, logz = 0;   // byte offsets after base.bytes
};

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool plan_derived(int op, int64_t B, int64_t N, int64_t C, Derived* d) {
    const int baseOp = op == TS_OP_LOG_DENSITY ? TS_OP_LOGPARTITION : TS_OP_MARGINALS;
    if (!make_plan(baseOp, B, N, C, nullptr, &d->base)) return false;
    const size_t E = (size_t)(N - 1);
    if (op == TS_OP_ENTROPY || op == TS_OP_SAMPLE) {
        d->mu = 0;
        d->part = align_up(sizeof(float) * B * E * C * C);
        d->extra = d->part + (op == TS_OP_ENTROPY ? align_up(sizeof(double) * B * E) : 0);
    } else {
        d->logz = 0;
        d->extra = align_up(sizeof(float) * B);
    }
    return true;
}

ts_status hip_status(hipError_t e) {
    if (e == hipSuccess) return TS_OK;
    return fail(TS_ERR_HIP, std::string("HIP error: ") + hipGetErrorString(e));
}

// Workspace of a semi-Markov call: the expanded edges [B, N-1, KC, KC], the expanded
// marginals (marginals) or path [B, N] (Viterbi), then the chain plan over KC labels.
struct SemiPlan {
    int64_t KC = 0;
    size_t xpot = 0, xout = 0, chain = 0, total = 0;
    Plan base;
};

// Sizes only; returns the reason when the dimensions are out of range, else nullptr.
const char* plan_semi(int op, int64_t B, int64_t N, int64_t K, int64_t C, SemiPlan* q) {
    if (B < 1 || N < 1 || K < 1 || C < 1) return "B, N, K and C must all be >= 1";
    if (K > kMaxLabels || C > kMaxLabels || K * C > kMaxLabels)
        return "K * C exceeds ts_chain_max_labels()";
    int64_t bn;
    if (!mul_ok(B, N, &bn) || bn > kMaxGridItems)
        return "problem size overflows the supported range";
    q->KC = K * C;
    if (N == 1) return nullptr;   // one token per sequence: no edges, no workspace
    // finiteness masks only where the expansion has structural zeros (K > 1); with K = 1 the
    // expanded chain is the chain itself and takes the same kernels
    if (!make_plan(op, B, N, q->KC, nullptr, &q->base, /*masks=*/K > 1))
        return "problem size overflows the supported range";
    const size_t x = align_up(sizeof(float) * B * (N - 1) * q->KC * q->KC);
    q->xpot = 0;
    q->xout = x;
    q->chain = x + (op == TS_OP_MARGINALS ? x
                    : op == TS_OP_VITERBI ? align_up(sizeof(int32_t) * B * N) : 0);
    q->total = q->chain + q->base.bytes;
    return nullptr;
}

ts_status check_semi(const float* sp, int op, int64_t B, int64_t N, int64_t K, int64_t C,
                     void* ws, size_t ws_bytes, SemiPlan* q) {
    if (const char* why = plan_semi(op, B, N, K, C, q)) return fail(TS_ERR_BAD_DIM, why);
    if (N > 1 && !sp) return fail(TS_ERR_NULL_ARG, "sp is NULL");
    return check_ws(q->total, ws, ws_bytes);
}

}  // namespace
}  // namespace tsc

using namespace tsc;

extern "C" {

int ts_chain_max_labels(void) { return kMaxLabels; }

size_t ts_chain_workspace_bytes(int op, int64_t B, int64_t N, int64_t C) {
    if (op < TS_OP_LOGPARTITION || op > TS_OP_SAMPLE || B < 1 || N < 1 || C < 1 ||
        C > kMaxLabels)
        return 0;
    if (op >= TS_OP_ENTROPY) {
        Derived d;
        if (!plan_derived(op, B, N, C, &d)) return 0;
        return d.base.bytes + d.extra;
    }
    Plan p, q;
    if (op == TS_OP_MARGINALS_VITERBI) {
        // the marginals plan first, then the Viterbi plan at the next 256-byte boundary
        if (!make_plan(TS_OP_MARGINALS, B, N, C, nullptr, &p) ||
            !make_plan(TS_OP_VITERBI, B, N, C, nullptr, &q))
            return 0;
        return p.bytes + q.bytes;
    }
    if (!make_plan(op, B, N, C, nullptr, &p)) return 0;
    return p.bytes;
}

ts_status ts_chain_logpartition(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                                int64_t C, float* logZ, void* ws, size_t ws_bytes,
                                void* stream) {
    Plan p;
    ts_status st = check_common(pot, B, N, C, TS_OP_LOGPARTITION, ws, ws_bytes, &p);
    if (st != TS_OK) return st;
    if (!logZ) return fail(TS_ERR_NULL_ARG, "logZ is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1) return hip_status(launch_single_token(B, N, C, TS_OP_LOGPARTITION, logZ,
                                                      nullptr, nullptr, s));
    if (p.fused) return hip_status(launch_small_log(pot, lengths, B, N, C, logZ, nullptr, s));
    return hip_status(launch_logz_tree(p, pot, lengths, logZ, s));
}

ts_status ts_chain_marginals(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                             int64_t C, float* logZ, float* marg, void* ws, size_t ws_bytes,
                             void* stream) {
    Plan p;
    ts_status st = check_common(pot, B, N, C, TS_OP_MARGINALS, ws, ws_bytes, &p);
    if (st != TS_OK) return st;
    if (N > 1 && !marg) return fail(TS_ERR_NULL_ARG, "marg is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1) {
        if (!logZ) return TS_OK;
        return hip_status(launch_single_token(B, N, C, TS_OP_LOGPARTITION, logZ, nullptr,
                                              nullptr, s));
    }
    if (p.fused) return hip_status(launch_small_log(pot, lengths, B, N, C, logZ, marg, s));
    // up-sweep (and log Z when requested), then the outside sweep and the marginals
    hipError_t e = launch_logz_tree(p, pot, lengths, logZ, s);
    if (e != hipSuccess) return hip_status(e);
    return hip_status(launch_marginals_tree(p, pot, lengths, marg, s));
}

ts_status ts_chain_viterbi(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                           int64_t C, int32_t* path, float* score, void* ws, size_t ws_bytes,
                           void* stream) {
    Plan p;
    ts_status st = check_common(pot, B, N, C, TS_OP_VITERBI, ws, ws_bytes, &p);
    if (st != TS_OK) return st;
    if (!path || !score) return fail(TS_ERR_NULL_ARG, "path or score is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1)
        return hip_status(launch_single_token(B, N, C, TS_OP_VITERBI, nullptr, path, score, s));
    if (p.fused) return hip_status(launch_small_max(pot, lengths, B, N, C, path, score, s));
    return hip_status(launch_viterbi_tree(p, pot, lengths, path, score, s));
}

ts_status ts_chain_marginals_viterbi(const float* pot, const int32_t* lengths, int64_t B,
                                     int64_t N, int64_t C, float* logZ, float* marg,
                                     int32_t* path, float* score, void* ws, size_t ws_bytes,
                                     void* stream) {
    Plan pm, pv;
    ts_status st = check_dims(pot, B, N, C, TS_OP_MARGINALS, &pm);
    if (st != TS_OK) return st;
    // the Viterbi plan can fail where the marginals plan does not (its decode tables must
    // fit in LDS): report that before anything is launched, as ts_chain_viterbi does
    if (!make_plan(TS_OP_VITERBI, B, N, C, nullptr, &pv))
        return fail(TS_ERR_BAD_DIM, "problem size overflows the supported range");
    // the marginals plan first, then the Viterbi plan (both sizes are multiples of 256)
    if ((st = check_ws(pm.bytes + pv.bytes, ws, ws_bytes)) != TS_OK) return st;
    if (N > 1 && !marg) return fail(TS_ERR_NULL_ARG, "marg is NULL");
    if (!path || !score) return fail(TS_ERR_NULL_ARG, "path or score is NULL");
    if (pm.bytes > 0) make_plan(TS_OP_MARGINALS, B, N, C, ws, &pm);
    if (pv.bytes > 0) make_plan(TS_OP_VITERBI, B, N, C, static_cast<char*>(ws) + pm.bytes, &pv);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1) {
        if (logZ) {
            hipError_t e = launch_single_token(B, N, C, TS_OP_LOGPARTITION, logZ, nullptr,
                                               nullptr, s);
            if (e != hipSuccess) return hip_status(e);
        }
        return hip_status(launch_single_token(B, N, C, TS_OP_VITERBI, nullptr, path, score, s));
    }
    if (pm.fused && pv.fused)
        return hip_status(launch_small_both(pot, lengths, B, N, C, logZ, marg, path, score, s));
    // the two tree sequences share only read-only inputs and write disjoint outputs and
    // workspace halves: the Viterbi one runs on the side stream, forked from `stream` and
    // joined back into it, so the levels of one fill the compute units the other's small
    // levels leave idle
    Side* side = nullptr;
    hipError_t e = side_of_current_device(&side);
    if (e == hipSuccess) e = link(side->fork, s, side->stream);
    if (e == hipSuccess) e = launch_viterbi_tree(pv, pot, lengths, path, score, side->stream);
    if (e == hipSuccess) e = launch_logz_tree(pm, pot, lengths, logZ, s);
    if (e == hipSuccess) e = launch_marginals_tree(pm, pot, lengths, marg, s);
    if (e == hipSuccess) e = link(side->join, side->stream, s);
    return hip_status(e);
}

ts_status ts_chain_entropy(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                           int64_t C, float* entropy, void* ws, size_t ws_bytes, void* stream) {
    Derived d;
    ts_status st = check_dims(pot, B, N, C, TS_OP_MARGINALS, &d.base);
    if (st != TS_OK) return st;
    plan_derived(TS_OP_ENTROPY, B, N, C, &d);
    if ((st = check_ws(d.base.bytes + d.extra, ws, ws_bytes)) != TS_OK) return st;
    if (!entropy) return fail(TS_ERR_NULL_ARG, "entropy is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1) return hip_status(launch_entropy(nullptr, lengths, B, N, C, nullptr, entropy, s));
    char* extra = static_cast<char*>(ws) + d.base.bytes;
    float* mu = reinterpret_cast<float*>(extra + d.mu);
    double* part = reinterpret_cast<double*>(extra + d.part);
    hipError_t e;
    if (d.base.fused) {
        e = launch_small_log(pot, lengths, B, N, C, nullptr, mu, s);
    } else {
        make_plan(TS_OP_MARGINALS, B, N, C, ws, &d.base);
        e = launch_logz_tree(d.base, pot, lengths, nullptr, s);
        if (e == hipSuccess) e = launch_marginals_tree(d.base, pot, lengths, mu, s);
    }
    if (e == hipSuccess) e = launch_entropy(mu, lengths, B, N, C, part, entropy, s);
    return hip_status(e);
}

ts_status ts_chain_log_density(const float* pot, const int32_t* lengths, const int32_t* labels,
                               int64_t B, int64_t N, int64_t C, float* logp, void* ws,
                               size_t ws_bytes, void* stream) {
    Derived d;
    ts_status st = check_dims(pot, B, N, C, TS_OP_LOGPARTITION, &d.base);
    if (st != TS_OK) return st;
    plan_derived(TS_OP_LOG_DENSITY, B, N, C, &d);
    if ((st = check_ws(d.base.bytes + d.extra, ws, ws_bytes)) != TS_OK) return st;
    if (!labels || !logp) return fail(TS_ERR_NULL_ARG, "labels or logp is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if ((st = check_labels(labels, lengths, B, N, C, s)) != TS_OK) return st;
    float* logz = reinterpret_cast<float*>(static_cast<char*>(ws) + d.base.bytes + d.logz);
    hipError_t e;
    if (N == 1) {
        e = launch_single_token(B, N, C, TS_OP_LOGPARTITION, logz, nullptr, nullptr, s);
    } else if (d.base.fused) {
        e = launch_small_log(pot, lengths, B, N, C, logz, nullptr, s);
    } else {
        make_plan(TS_OP_LOGPARTITION, B, N, C, ws, &d.base);
        e = launch_logz_tree(d.base, pot, lengths, logz, s);
    }
    if (e == hipSuccess) e = launch_log_density(pot, lengths, labels, logz, B, N, C, logp, s);
    return hip_status(e);
}

ts_status ts_chain_sample(const float* pot, const int32_t* lengths, const float* uniforms,
                          int64_t S, int64_t B, int64_t N, int64_t C, int32_t* paths, void* ws,
                          size_t ws_bytes, void* stream) {
    Derived d;
    ts_status st = check_dims(pot, B, N, C, TS_OP_MARGINALS, &d.base);
    if (st != TS_OK) return st;
    if (S < 1) return fail(TS_ERR_BAD_DIM, "S must be >= 1");
    int64_t sbn;
    if (!mul_ok(S, B, &sbn) || sbn > ((int64_t)1 << 32) || !mul_ok(sbn, N, &sbn) ||
        sbn > ((int64_t)1 << 40))
        return fail(TS_ERR_BAD_DIM, "S * B * N overflows the supported range");
    plan_derived(TS_OP_SAMPLE, B, N, C, &d);
    if ((st = check_ws(d.base.bytes + d.extra, ws, ws_bytes)) != TS_OK) return st;
    if (!uniforms || !paths) return fail(TS_ERR_NULL_ARG, "uniforms or paths is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    float* mu = N > 1 ? reinterpret_cast<float*>(static_cast<char*>(ws) + d.base.bytes + d.mu)
                      : nullptr;
    hipError_t e = hipSuccess;
    if (N > 1) {
        if (d.base.fused) {
            e = launch_small_log(pot, lengths, B, N, C, nullptr, mu, s);
        } else {
            make_plan(TS_OP_MARGINALS, B, N, C, ws, &d.base);
            e = launch_logz_tree(d.base, pot, lengths, nullptr, s);
            if (e == hipSuccess) e = launch_marginals_tree(d.base, pot, lengths, mu, s);
        }
    }
    if (e == hipSuccess) e = launch_sample(mu, lengths, uniforms, S, B, N, C, paths, s);
    return hip_status(e);
}

ts_status ts_chain_logpartition_sequential(const float* pot, const int32_t* lengths, int64_t B,
                                           int64_t N, int64_t C, float* logZ, void* stream) {
    Plan p;
    ts_status st = check_dims(pot, B, N, C, TS_OP_LOGPARTITION, &p);
    if (st != TS_OK) return st;
    if (!logZ) return fail(TS_ERR_NULL_ARG, "logZ is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    return hip_status(launch_logz_sequential(pot, lengths, B, N, C, logZ, s));
}

size_t ts_semimarkov_workspace_bytes(int op, int64_t B, int64_t N, int64_t K, int64_t C) {
    if (op < TS_OP_LOGPARTITION || op > TS_OP_VITERBI) return 0;
    SemiPlan q;
    return plan_semi(op, B, N, K, C, &q) ? 0 : q.total;
}

ts_status ts_semimarkov_logpartition(const float* sp, const int32_t* lengths, int64_t B,
                                     int64_t N, int64_t K, int64_t C, float* logZ, void* ws,
                                     size_t ws_bytes, void* stream) {
    SemiPlan q;
    ts_status st = check_semi(sp, TS_OP_LOGPARTITION, B, N, K, C, ws, ws_bytes, &q);
    if (st != TS_OK) return st;
    if (!logZ) return fail(TS_ERR_NULL_ARG, "logZ is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1) return hip_status(launch_single_token(B, N, C, TS_OP_LOGPARTITION, logZ,
                                                      nullptr, nullptr, s));
    char* w = static_cast<char*>(ws);
    float* xp = reinterpret_cast<float*>(w + q.xpot);
    hipError_t e = launch_semi_expand(sp, lengths, B, N, K, C, xp, s);
    if (e == hipSuccess) {
        if (q.base.fused) {
            e = launch_small_log(xp, lengths, B, N, q.KC, logZ, nullptr, s);
        } else {
            make_plan(TS_OP_LOGPARTITION, B, N, q.KC, w + q.chain, &q.base, K > 1);
            e = launch_logz_tree(q.base, xp, lengths, logZ, s);
        }
    }
    if (e == hipSuccess) e = launch_semi_single(lengths, B, N, C, logZ, s);
    return hip_status(e);
}

ts_status ts_semimarkov_marginals(const float* sp, const int32_t* lengths, int64_t B,
                                  int64_t N, int64_t K, int64_t C, float* logZ, float* marg,
                                  void* ws, size_t ws_bytes, void* stream) {
    SemiPlan q;
    ts_status st = check_semi(sp, TS_OP_MARGINALS, B, N, K, C, ws, ws_bytes, &q);
    if (st != TS_OK) return st;
    if (N > 1 && !marg) return fail(TS_ERR_NULL_ARG, "marg is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1) {
        if (!logZ) return TS_OK;
        return hip_status(launch_single_token(B, N, C, TS_OP_LOGPARTITION, logZ, nullptr,
                                              nullptr, s));
    }
    char* w = static_cast<char*>(ws);
    float* xp = reinterpret_cast<float*>(w + q.xpot);
    float* xm = reinterpret_cast<float*>(w + q.xout);
    hipError_t e = launch_semi_expand(sp, lengths, B, N, K, C, xp, s);
    if (e == hipSuccess) {
        if (q.base.fused) {
            e = launch_small_log(xp, lengths, B, N, q.KC, logZ, xm, s);
        } else {
            make_plan(TS_OP_MARGINALS, B, N, q.KC, w + q.chain, &q.base, K > 1);
            e = launch_logz_tree(q.base, xp, lengths, logZ, s);
            if (e == hipSuccess) e = launch_marginals_tree(q.base, xp, lengths, xm, s);
        }
    }
    if (e == hipSuccess) e = launch_semi_gather(xm, B, N, K, C, marg, s);
    if (e == hipSuccess && logZ) e = launch_semi_single(lengths, B, N, C, logZ, s);
    return hip_status(e);
}

ts_status ts_semimarkov_viterbi(const float* sp, const int32_t* lengths, int64_t B, int64_t N,
                                int64_t K, int64_t C, int32_t* path, int32_t* seglen,
                                float* score, void* ws, size_t ws_bytes, void* stream) {
    SemiPlan q;
    ts_status st = check_semi(sp, TS_OP_VITERBI, B, N, K, C, ws, ws_bytes, &q);
    if (st != TS_OK) return st;
    if (!path || !score || (N > 1 && !seglen))
        return fail(TS_ERR_NULL_ARG, "path, seglen or score is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((st = check_lengths(lengths, B, N, s)) != TS_OK) return st;
    if (N == 1)
        return hip_status(launch_single_token(B, N, C, TS_OP_VITERBI, nullptr, path, score, s));
    char* w = static_cast<char*>(ws);
    float* xp = reinterpret_cast<float*>(w + q.xpot);
    int32_t* xs = reinterpret_cast<int32_t*>(w + q.xout);
    hipError_t e = launch_semi_expand(sp, lengths, B, N, K, C, xp, s);
    if (e == hipSuccess) {
        if (q.base.fused) {
            e = launch_small_max(xp, lengths, B, N, q.KC, xs, score, s);
        } else {
            make_plan(TS_OP_VITERBI, B, N, q.KC, w + q.chain, &q.base, K > 1);
            e = launch_viterbi_tree(q.base, xp, lengths, xs, score, s);
        }
    }
    if (e == hipSuccess) e = launch_semi_decode(xs, lengths, B, N, C, path, seglen, s);
    return hip_status(e);
}

const char* ts_last_error(void) { return g_err.c_str(); }

}  // extern "C"
