/*
 * ts_chain.h -- C ABI of the MI355X (gfx950) batched linear-chain CRF library.
 *
 * The library computes, for a batch of linear-chain CRFs (Torch-Struct, Rush 2020):
 *   - the log-partition  A(l) = log sum_z exp sum_t l[t, z_t, z_{t+1}]    (Sec. 5.1-5.2),
 *   - the edge marginals p(z_t = i, z_{t+1} = j) = dA/dl[t,i,j]          (Sec. 5.1),
 *   - the max score A*(l) and its argmax label sequence (Viterbi)        (Sec. 5.1-5.2,
 *     Table 2 "Max" semiring),
 * each as a balanced tree of C x C semiring matrix products over the edges of every
 * sequence, padded with the semiring identity (Sec. 6a, Fig. 3).  All arithmetic runs in
 * HIP kernels on the device; the host only validates arguments and enqueues work.
 *
 * Common arguments
 *   pot      device pointer, float32 [B, N-1, C, C], row-major and contiguous:
 *            pot[((b*(N-1) + t)*C + i)*C + j] is the log-potential of the labelled edge
 *            z_t = i -> z_{t+1} = j of sequence b (the earlier label is the row).  Finite
 *            values and -inf (the semiring zero) are allowed; +inf and NaN are not.
 *            May be NULL only when N == 1 (no edges).
 *   lengths  device pointer, int32 [B]: number of tokens of each sequence,
 *            1 <= lengths[b] <= N.  Edges t >= lengths[b]-1 are padding: they act as the
 *            identity and their values never affect any result (the multi-launch tree
 *            never reads them; the single-launch kernels for small label sets load whole
 *            sequences and discard them).  NULL means every length is N.  Values are not
 *            read on the host: out-of-range values are clamped to [1, N] by the kernels,
 *            unless the environment variable TS_CHECK=1 is set, in which case the call
 *            copies the lengths to the host synchronously and returns TS_ERR_LENGTHS.
 *   B, N, C  batch size, maximum number of tokens, number of labels:
 *            B >= 1, N >= 1, 1 <= C <= ts_chain_max_labels(), B * N <= 2^29 (one launch
 *            grid covers every edge); larger problems return TS_ERR_BAD_DIM.  The Viterbi
 *            calls also keep their backtrace tables in 64 KiB of LDS: with K the largest
 *            power of two <= 65536 / C, N - 1 <= K * floor(65536 / C) edges (C = 256:
 *            N <= 65537; C = 128: N <= 262145), else TS_ERR_BAD_DIM.
 *   ws       device workspace of at least ts_chain_workspace_bytes(op, B, N, C) bytes,
 *            aligned to 256 bytes (any hipMalloc / PyTorch CUDA allocation is).  May be
 *            NULL when that size is 0.  Its contents on entry are ignored.
 *   stream   the hipStream_t to enqueue on (NULL = the default stream), passed as void* so
 *            that this header needs no HIP header.
 *
 * Ownership and synchronisation: every pointer is owned by the caller.  The library
 * allocates no memory, keeps no pointer after returning, and enqueues its kernels on
 * `stream` (ts_chain_marginals_viterbi may fork part of its work onto a side stream and
 * joins it back, see there); results are ready once that stream is synchronised.  Calls with distinct
 * workspaces may run concurrently on different streams.  Results are bitwise
 * reproducible for identical inputs (no floating-point atomics).
 *
 * Errors: every call returns a ts_status.  On an error nothing has been enqueued
 * (TS_ERR_HIP aside, which reports a failed launch) and outputs are unspecified.
 * ts_last_error() returns a message for the last non-OK status of the calling thread.
 */
#ifndef TS_CHAIN_H
#define TS_CHAIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int ts_status;
#define TS_OK 0
#define TS_ERR_NULL_ARG -1  /* a required pointer is NULL */
#define TS_ERR_BAD_DIM -2   /* B, N or C out of range, or a size overflows */
#define TS_ERR_WORKSPACE -3 /* ws_bytes below ts_chain_workspace_bytes() */
#define TS_ERR_LENGTHS -4   /* TS_CHECK=1 and a length lies outside [1, N] */
#define TS_ERR_HIP -5       /* a HIP runtime call or kernel launch failed */
#define TS_ERR_LABELS -6    /* TS_CHECK=1 and a label lies outside [0, C) */

/* operation codes for ts_chain_workspace_bytes */
#define TS_OP_LOGPARTITION 0
#define TS_OP_MARGINALS 1
#define TS_OP_VITERBI 2
#define TS_OP_MARGINALS_VITERBI 3
#define TS_OP_ENTROPY 4
#define TS_OP_LOG_DENSITY 5
#define TS_OP_SAMPLE 6

/* Largest supported number of labels C. */
int ts_chain_max_labels(void);

/* Workspace bytes that operation `op` needs for (B, N, C); 0 for invalid arguments
 * (check with the call itself, which reports why). */
size_t ts_chain_workspace_bytes(int op, int64_t B, int64_t N, int64_t C);

/*
 * Log-partition (Sec. 5.1 A(l); Sec. 5.2 forward algorithm, evaluated as the tree of
 * log-semiring (logsumexp, +) matrix products of Sec. 6a).
 *   logZ  device float32 [B]: log Z of each sequence.  A sequence of one token has no
 *         edges and log Z = log C (its label is free: no start or end potentials).
 *         log Z = -inf when no label sequence has a finite score.
 */
ts_status ts_chain_logpartition(const float* pot, const int32_t* lengths, int64_t B,
                                int64_t N, int64_t C, float* logZ, void* ws, size_t ws_bytes,
                                void* stream);

/*
 * Edge marginals, the gradient of A (Sec. 5.1: p(z_p = 1) = dA/dl_p), computed by the
 * outside (down) sweep of the same tree followed by a per-edge local normaliser.
 *   logZ  device float32 [B] or NULL: as for ts_chain_logpartition.
 *   marg  device float32 [B, N-1, C, C], same layout as pot: p(z_t=i, z_{t+1}=j).
 *         Padding edges are written as exactly 0; every entry of a sequence whose
 *         log Z is -inf is 0.  May be NULL only when N == 1.
 */
ts_status ts_chain_marginals(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                             int64_t C, float* logZ, float* marg, void* ws, size_t ws_bytes,
                             void* stream);

/*
 * Viterbi: the (max, +) instance of the same tree (Sec. 5.1 A*; Sec. 5.2; Table 2 "Max"),
 * with float64 accumulation, followed by a lowest-index backtrace.
 *   path  device int32 [B, N]: the argmax label sequence; path[b*N + n] = -1 for
 *         n >= lengths[b].  Ties are broken by the lowest label index at each backtrace
 *         step: z_{L-1} is the lowest label of maximal forward score and
 *         z_t is the lowest i maximising delta_t(i) + l[t, i, z_{t+1}].
 *   score device float32 [B]: max_z sum_t l[t, z_t, z_{t+1}] (0 for a single token,
 *         -inf when no sequence is finite).
 */
ts_status ts_chain_viterbi(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                           int64_t C, int32_t* path, float* score, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * Marginals and Viterbi of the same potentials in one call: the outputs of
 * ts_chain_marginals (logZ nullable, marg) and of ts_chain_viterbi (path, score), with the
 * same meaning, layout and values.  For label sets small enough for the single-launch path
 * both passes run in one launch (one workgroup per sequence and pass, side by side);
 * otherwise the Viterbi kernel sequence runs on a side stream of the library's (one per
 * device, default priority, created by the first such call and kept until the process
 * ends), forked from `stream` and joined back into it with events, while the marginals
 * sequence runs on `stream`: the call stays ordered on `stream` as any other, and can be
 * captured into a HIP graph.  The workspace is
 * ts_chain_workspace_bytes(TS_OP_MARGINALS_VITERBI, ...): the marginals workspace followed
 * by the Viterbi workspace.  Errors as for the two separate calls.
 */
ts_status ts_chain_marginals_viterbi(const float* pot, const int32_t* lengths, int64_t B,
                                     int64_t N, int64_t C, float* logZ, float* marg,
                                     int32_t* path, float* score, void* ws, size_t ws_bytes,
                                     void* stream);

/*
 * Entropy H = -sum_z p(z) log p(z) of each sequence's label distribution (Sec. 5.1; the
 * quantity Table 2's "Entropy" semiring computes), from the edge marginals by the chain rule
 * of a Markov chain: H = H(z_0) + sum_t H(z_{t+1} | z_t), every term >= 0.
 *   entropy  device float32 [B].  One token: log C.  No finite path: 0.
 * The workspace, ts_chain_workspace_bytes(TS_OP_ENTROPY, ...), holds the marginals
 * workspace, the marginals themselves ([B, N-1, C, C] fp32) and per-edge partial sums.
 */
ts_status ts_chain_entropy(const float* pot, const int32_t* lengths, int64_t B, int64_t N,
                           int64_t C, float* entropy, void* ws, size_t ws_bytes, void* stream);

/*
 * Log-probability of given label sequences (Sec. 5.1: p(z) = exp(score(z) - A)):
 *   log p(z_b) = sum_{t < L_b - 1} l[b, t, z_b[t], z_b[t+1]] - log Z_b.
 *   labels   device int32 [B, N]; entries n >= lengths[b] are ignored.  Labels must lie in
 *            [0, C) (clamped on the device; TS_CHECK=1 validates them: TS_ERR_LABELS).
 *   logp     device float32 [B].
 * Workspace: ts_chain_workspace_bytes(TS_OP_LOG_DENSITY, ...) (the log-partition workspace
 * and log Z).
 */
ts_status ts_chain_log_density(const float* pot, const int32_t* lengths, const int32_t* labels,
                               int64_t B, int64_t N, int64_t C, float* logp, void* ws,
                               size_t ws_bytes, void* stream);

/*
 * S samples per sequence from p(z) = exp(score(z) - A) (Sec. 5.1; the distribution Table 2's
 * "Sample" semiring draws from) by forward filtering, backward sampling from the edge
 * marginals:  z_{L-1} ~ sum_i mu[L-2, i, .],  z_t | z_{t+1} = j ~ mu[t, ., j].
 *   uniforms device float32 [S, B, N] in [0, 1), supplied by the caller (the library draws no
 *            random numbers): u[s, b, t] draws token t of sample s of sequence b by inverse
 *            CDF -- the smallest label k whose inclusive prefix sum of the weights exceeds
 *            u * (their total).  One token: uniform over the C labels.
 *   paths    device int32 [S, B, N], -1 past each length.
 * Workspace: ts_chain_workspace_bytes(TS_OP_SAMPLE, ...) (the marginals workspace and the
 * marginals).  A sequence with no finite path draws label 0 everywhere.
 */
ts_status ts_chain_sample(const float* pot, const int32_t* lengths, const float* uniforms,
                          int64_t S, int64_t B, int64_t N, int64_t C, int32_t* paths, void* ws,
                          size_t ws_bytes, void* stream);

/*
 * Log-partition by the left-to-right forward algorithm (Sec. 5.2), the serial ordering that
 * Fig. 4a compares the parallel scan against: L - 1 dependent vector steps of C^2 work
 * instead of ceil(log2(L - 1)) tree levels of C^3 work per product.  Same output, layout
 * and errors as ts_chain_logpartition; needs no workspace.  Provided to measure the
 * depth-versus-work trade-off of the scan, not as the default path.
 */
ts_status ts_chain_logpartition_sequential(const float* pot, const int32_t* lengths, int64_t B,
                                           int64_t N, int64_t C, float* logZ, void* stream);

/*
 * Semi-Markov CRF (Table 1, "Semi-Markov": segment labels, parts N K C^2; Sec. 6a carries
 * the parallel scan over to it).  A sequence of L tokens has L-1 steps (the chain's edges),
 * covered by consecutive segments of lengths 1..K, each with a label; the first segment
 * follows a free initial label.
 *   sp       device float32 [B, N-1, K, C, C]: sp[(((b*(N-1) + t)*K + k-1)*C + i)*C + j]
 *            scores a segment of length k that starts at step t with label j after a
 *            segment labelled i.  Entries with t + k > L-1 are never used.
 *   K        maximum segment length, K >= 1 and K * C <= ts_chain_max_labels().
 *   lengths, B, N, C, ws, stream as above; ws is sized by ts_semimarkov_workspace_bytes.
 * The call runs the linear-chain scan over K*C expanded states (the label of the segment
 * in progress and the steps it has left), whose edges it builds in the workspace.
 * With K = 1 every result equals the linear chain's on sp[:, :, 0].
 */
size_t ts_semimarkov_workspace_bytes(int op /* TS_OP_LOGPARTITION, _MARGINALS or _VITERBI */,
                                     int64_t B, int64_t N, int64_t K, int64_t C);

/* log Z [B] (float32); one token gives log C.  Segmental forward algorithm. */
ts_status ts_semimarkov_logpartition(const float* sp, const int32_t* lengths, int64_t B,
                                     int64_t N, int64_t K, int64_t C, float* logZ, void* ws,
                                     size_t ws_bytes, void* stream);

/* Segment marginals marg [B, N-1, K, C, C] = dA/dsp (Sec. 5.1): the probability that a
 * segment of length k starts at step t with label j after label i; 0 for padding and for
 * segments that would overrun the sequence.  logZ [B] is optional (NULL skips it). */
ts_status ts_semimarkov_marginals(const float* sp, const int32_t* lengths, int64_t B,
                                  int64_t N, int64_t K, int64_t C, float* logZ, float* marg,
                                  void* ws, size_t ws_bytes, void* stream);

/* Best segmentation (Table 2 "Max" semiring):
 *   path   int32 [B, N]: path[b, 0] is the initial label, path[b, t+1] the label of the
 *          segment covering step t; -1 past the sequence;
 *   seglen int32 [B, N-1]: k where a segment of length k starts at step t, else 0; -1 past
 *          the last step (may be NULL when N == 1);
 *   score  float32 [B]: its score, accumulated in float64.
 * Ties: the lowest last label, then at every segment end (going back) the shortest segment,
 * then the lowest previous label. */
ts_status ts_semimarkov_viterbi(const float* sp, const int32_t* lengths, int64_t B, int64_t N,
                                int64_t K, int64_t C, int32_t* path, int32_t* seglen,
                                float* score, void* ws, size_t ws_bytes, void* stream);

/*
 * ts_chain_marginals without a workspace argument, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation.  Arguments, outputs, layout and errors are those of ts_chain_marginals without
 * ws / ws_bytes; the kernels and the results are the same.  The call allocates nothing: its
 * scratch is one array of ts_chain_noalloc_scratch_bytes() bytes (64 MiB) per GPU inside the
 * library, held from the first call on that GPU until the process ends.  A problem whose
 * ts_chain_workspace_bytes(TS_OP_MARGINALS, B, N, C) exceeds it returns TS_ERR_BAD_DIM
 * before any device call (the single-launch path for small label sets needs no scratch).
 * Every call on one GPU shares that GPU's array, which keeps the last call's contents (the
 * kernels need none of it cleared): calls that overlap on one GPU, from different streams
 * or threads, race on it and must be serialised by the caller.  TS_CHECK=1 copies the
 * lengths synchronously, which graph capture does not allow.
 */
size_t ts_chain_noalloc_scratch_bytes(void);
ts_status ts_chain_marginals_noalloc(const float* pot, const int32_t* lengths, int64_t B,
                                     int64_t N, int64_t C, float* logZ, float* marg,
                                     void* stream);

/* Message for the last non-OK status returned to the calling thread ("" if none). */
const char* ts_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TS_CHAIN_H */
