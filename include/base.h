/*
 * base.h -- C ABI of the balanced token-to-expert assignment path of BASE
 * layers (Lewis et al., "BASE Layers: Simplifying Training of Large, Sparse
 * Models", ICML 2021), built for AMD Instinct MI355X (gfx950).
 *
 * The path has three calls, in the order a BASE layer makes them during
 * training (Sec. 3, Fig. 2):
 *   base_affinity  token-expert scores S = H . W^T              (Sec. 3.1, Eq. 2)
 *   base_assign    balanced assignment maximising sum_t S[t,a_t],
 *                  every expert receiving exactly T/E tokens     (Sec. 3.2.1, Eq. 2)
 *   base_permute   rows routed into expert-contiguous order and back
 *                  (Fig. 2 caption; Sec. 3, third stage)
 *
 * Conventions shared by every entry point
 *   - Pointers marked [device] are HIP device pointers (hipMalloc / torch
 *     CUDA tensors); [host] pointers are ordinary host memory.
 *   - Matrices are dense, row-major, contiguous. Index ranges are half-open:
 *     tokens t in [0, T), experts e in [0, E).
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Work is enqueued on it and the call returns without waiting, except
 *     where a flag below asks for a synchronous result.
 *   - The caller owns every buffer. The library allocates no device memory
 *     in these calls and keeps no state between calls beyond the loaded
 *     kernels of each device.
 *   - Arguments are validated on the host before anything is enqueued; a
 *     call that returns an error has enqueued nothing, unless the error is
 *     BASE_ERR_HIP or one reported by a synchronous flag. Outputs are
 *     unspecified after an error.
 *   - Device buffers must be 16-byte aligned.
 *   - Calls on one stream are ordered; calls that share a workspace must not
 *     run concurrently on different streams.
 */
#ifndef BASE_MI355X_H
#define BASE_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every int-valued entry point. */
typedef enum {
    BASE_OK = 0,
    BASE_ERR_INVALID_ARG = -1,      /* null pointer, size <= 0, misaligned pointer, bad option */
    BASE_ERR_NOT_DIVISIBLE = -2,    /* T is not a multiple of E (Eq. 2 needs T/E tokens per expert) */
    BASE_ERR_UNSUPPORTED_DTYPE = -3,/* dtype not accepted by this entry point */
    BASE_ERR_NONFINITE = -4,        /* a score is NaN or infinite (only with BASE_ASSIGN_CHECK_FINITE) */
    BASE_ERR_NOT_CONVERGED = -5,    /* the round limit was reached before every expert was full */
    BASE_ERR_WORKSPACE = -6,        /* workspace missing or smaller than base_assign_workspace_size */
    BASE_ERR_HIP = -7,              /* a HIP runtime call failed */
    BASE_ERR_RANGE = -8,            /* a size or value outside what the kernels represent */
    BASE_ERR_INTERNAL = -9          /* a device-side consistency check failed (a bug, not bad input) */
} base_status;

/* Element types. BASE_I16 is accepted for scores only (the integer variant). */
typedef enum { BASE_F32 = 0, BASE_BF16 = 1, BASE_I16 = 2 } base_dtype;

/* Returns a static, human-readable name for a status code. Never NULL. */
const char *base_status_string(int status);

/* ------------------------------------------------------------------------ */
/* base_affinity: S[t, e] = sum_k H[t, k] * W[e, k]                          */
/* ------------------------------------------------------------------------ */
/*
 * Sec. 3.1 and Eq. 2: the score of token t for expert e is the dot product of
 * the token representation h_t and the expert embedding w_e. No sigmoid,
 * softmax or bias is applied (the sigmoid of Eq. 1 gates the expert output,
 * not the assignment).
 *
 *   H  [device] T x d, in_dtype (BASE_BF16 or BASE_F32), row-major
 *   W  [device] E x d, same dtype as H, row-major
 *   S  [device] T x E float32, row-major, written entirely
 *   T, E, d > 0; T, E <= 2^31 - 1; d % 8 == 0
 *
 * Arithmetic: BASE_BF16 multiplies bf16 values on the matrix cores and
 * accumulates in fp32; BASE_F32 multiplies and accumulates in fp32 (no
 * reduced-precision products). The summation order over k is unspecified.
 * Errors: BASE_ERR_INVALID_ARG (null/misaligned pointer, size <= 0,
 * d % 8 != 0), BASE_ERR_UNSUPPORTED_DTYPE, BASE_ERR_RANGE, BASE_ERR_HIP.
 */
int base_affinity(const void *H, const void *W, float *S, int64_t T, int64_t E, int64_t d,
                  int in_dtype, void *stream);

/*
 * base_affinity_gather - the same product with the rows of H taken through an
 * index: S[i, e] = H[rows[i], :] . W[e, :] for i in [0, N). Sec. 3.2.1
 * (Shuffling): before the assignment, tokens are sent to workers at random;
 * with rows = a random permutation of the B * T tokens, rows
 * [b T, (b + 1) T) of S are worker b's problem. The shuffled copy of H is
 * never materialised: the GEMM reads H through the index, and
 * base_permute_batched / base_gate_combine_batched take the same index.
 *
 *   H       [device] h_rows x d, in_dtype, row-major
 *   rows    [device] int32 [N], entries in [0, h_rows) (an entry outside
 *           that range gives a zero row of S; never read out of bounds)
 *   S       [device] N x E float32, row-major, written entirely
 *   N, h_rows <= 2^31 - 1; other arguments and arithmetic as base_affinity
 *   (bit-identical to base_affinity of the gathered rows).
 * Errors: as base_affinity; rows == NULL is BASE_ERR_INVALID_ARG.
 */
int base_affinity_gather(const void *H, int64_t h_rows, const int32_t *rows, const void *W,
                         float *S, int64_t N, int64_t E, int64_t d, int in_dtype, void *stream);

/* ------------------------------------------------------------------------ */
/* base_assign: balanced assignment of Eq. 2                                  */
/* ------------------------------------------------------------------------ */
/*
 * Sec. 3.2.1, Eq. 2: choose a_t in [0, E) maximising sum_t S[t, a_t] subject to
 * every expert receiving exactly C = T/E tokens. The paper solves it with an
 * auction algorithm (Sec. 3.2.1; appendix figure on the assignment algorithm).
 * This implementation is a forward auction with epsilon scaling in which
 * every expert is C identical objects: each round, every unassigned token
 * bids for its best expert (top-2 over the values S[t,e] - p[e]); each expert
 * keeps its C highest bids (ties: lower token index wins), evicts the rest,
 * and once full sets its price to its lowest held bid. A phase ends when
 * every expert holds C tokens; epsilon then shrinks by eps_factor (or
 * less, below) until eps_final. With the returned prices p the result satisfies
 *     sum_t max_e (S[t,e] - p[e]) + C * sum_e p[e] - sum_t S[t, a_t] <= T * eps_final
 * (up to fp32 rounding in float mode), i.e. the assignment is within
 * T * eps_final of the optimum: the left side is the duality gap, an upper
 * bound of optimum - objective. The last phase (epsilon = eps_final)
 * guarantees it by epsilon-complementary slackness. After every earlier
 * phase the device also measures the gap directly; when it already meets
 * the bound (with an allowance for fp32 rounding), the solve stops there
 * (stats.certified). When it misses by less than eps_factor, the next
 * epsilon shrinks only enough for the gap, taken as proportional to
 * epsilon, to reach half the bound. BASE_ASSIGN_FULL_SCHEDULE runs every
 * phase with the plain eps_factor steps instead.
 *
 * Integer mode (s_dtype == BASE_I16): scores are int16; the solve runs in
 * int64 on the scores scaled by K = 2^ceil(log2(T + 1)) with eps_final = 1
 * (one scaled unit, 1/K of a score unit), so T * eps_final < 1 score unit and
 * the assignment is an exact optimum of Eq. 2. Requires T < 2^21.
 *
 *   S          [device] T x E scores, s_dtype (BASE_F32 or BASE_I16), row-major
 *   T, E       T > 0, 0 < E <= 2048, T % E == 0, T < 2^24 (T < 2^21 in integer
 *              mode); other sizes return BASE_ERR_RANGE
 *   opts       [host] options, NULL for the defaults below
 *   assign     [device] int32 [T] out: a_t in [0, E)
 *   perm       [device] int32 [T] out: the sort vector of Fig. 2; perm[k] is
 *              the token placed at row k when tokens are grouped by expert in
 *              ascending expert order and ascending token order inside an
 *              expert, so rows [e*C, (e+1)*C) hold expert e's tokens
 *   prices     [device] out, may be NULL: E float32 (float mode) or E int64
 *              (integer mode, in scaled units); the dual prices certifying
 *              the bound above
 *   workspace  [device] at least base_assign_workspace_size(T, E) bytes,
 *              256-byte aligned; contents on entry are ignored
 *   stats      [host] out, may be NULL; filled only with BASE_ASSIGN_SYNC_STATS
 *
 * Errors: BASE_ERR_INVALID_ARG, BASE_ERR_NOT_DIVISIBLE, BASE_ERR_UNSUPPORTED_DTYPE,
 * BASE_ERR_WORKSPACE, BASE_ERR_RANGE, BASE_ERR_HIP; with BASE_ASSIGN_SYNC_STATS
 * also BASE_ERR_NOT_CONVERGED (max_rounds reached without the fallback flag)
 * and BASE_ERR_RANGE (a price left the representable range); with
 * BASE_ASSIGN_CHECK_FINITE also BASE_ERR_NONFINITE.
 */
enum {
    BASE_ASSIGN_GREEDY_FALLBACK = 1, /* when max_rounds is reached, fill the free slots
                                        with the still-unassigned tokens (balance kept,
                                        the epsilon bound void; stats.fell_back = 1) */
    BASE_ASSIGN_SYNC_STATS = 2,      /* wait for the solve, fill *stats, report
                                        NOT_CONVERGED / RANGE */
    BASE_ASSIGN_CHECK_FINITE = 4,    /* scan S first (synchronous); NaN/Inf -> BASE_ERR_NONFINITE */
    BASE_ASSIGN_WARM_PRICES = 8,     /* start from the prices in `prices` (then overwritten
                                        with the result) instead of 0, e.g. the prices of
                                        the previous batch; must be finite (float mode) or
                                        in scaled units (integer mode) */
    BASE_ASSIGN_FULL_SCHEDULE = 16   /* run every epsilon phase down to eps_final, without
                                        the duality check that may stop the solve earlier */
};

typedef struct {
    double eps_final;    /* float mode: final epsilon in score units; <= 0 -> 1e-4.
                            Ignored in integer mode (always 1 scaled unit). */
    double eps_initial;  /* first-phase epsilon in score units (also in integer mode,
                            where it is scaled by K); <= 0 -> (max S - min S) / 8
                            computed on the device */
    double eps_factor;   /* epsilon divisor between phases; <= 1 -> 32. After a duality
                            check that misses the bound, the step is smaller when the
                            measured gap asks for less (see above) */
    int32_t max_rounds;  /* bound on bidding rounds over all phases; <= 0 -> 4,000,000 */
    uint32_t flags;      /* BASE_ASSIGN_* */
} base_assign_opts;

typedef struct {
    /* The first six fields are the statistics of the problem statement's
     * boundary, in its order: a caller built against that layout reads them
     * at the same offsets (dual_gap at byte 32). The fields after them are
     * additions. */
    int32_t phases;      /* epsilon phases run */
    int32_t rounds;      /* bidding rounds over all phases */
    int64_t bids;        /* bids placed over all phases */
    double eps_final;    /* the bound per token, in score units: the assignment is within
                            T * eps_final of the optimum (eps_final as raised for fp32
                            resolution) */
    int32_t fell_back;   /* 1 if the greedy completion was used */
    double dual_gap;     /* D(p) - sum_t S[t, a_t] for the returned prices, in score
                            units: an upper bound of optimum - objective for a balanced
                            result (the certificate of the bound above; after the greedy
                            fallback it measures what the fallback gave up). Measured
                            only with BASE_ASSIGN_SYNC_STATS; NaN from base_assign_status */
    int32_t converged;   /* 1 if every expert holds exactly T/E tokens */
    int64_t engine_bids; /* the part of `bids` placed inside the single-workgroup
                            engine (the rounds with few active tokens) */
    double eps_last;     /* epsilon of the last phase run, in score units (above eps_final
                            when the solve stopped on the duality check) */
    int32_t certified;   /* problems whose solve stopped after an earlier phase because
                            the measured duality gap met T * eps_final */
    int32_t augmentations; /* shortest augmenting paths that finished phases (the
                            last few tokens of a phase), over all phases */
} base_assign_stats;

/* Bytes of device workspace base_assign needs for T tokens and E experts
 * (0 if T or E is not positive). */
size_t base_assign_workspace_size(int64_t T, int64_t E);

int base_assign(const void *S, int s_dtype, int64_t T, int64_t E, const base_assign_opts *opts,
                int32_t *assign, int32_t *perm, void *prices, void *workspace,
                size_t workspace_bytes, base_assign_stats *stats, void *stream);

/* ------------------------------------------------------------------------ */
/* base_assign_batched: many independent balanced assignments in one call   */
/* ------------------------------------------------------------------------ */
/*
 * Sec. 3.2.1 (Sharding): the assignment over all workers is split into
 * independent problems, one per worker, each of T tokens and E experts (the
 * paper's runs: T = 2 x 1024, E = 128, Sec. 4.1). This call solves B such
 * problems together on one device, every problem exactly as base_assign
 * would (same algorithm, same options, bit-identical results); the
 * single-workgroup parts of the solve run for all problems at once.
 * Sec. 3.2.1 (Shuffling) routes tokens to workers at random before the
 * solve: base_affinity_gather computes the scores of the shuffled rows, and
 * base_permute_batched / base_gate_combine_batched route them, all reading
 * the unshuffled H through the caller's random permutation.
 *
 *   S          [device] B x T x E scores, problem after problem (T * E * sizeof
 *              must be a multiple of 16 bytes when B > 1)
 *   assign     [device] int32 [B][T]: expert of token t of problem b
 *   perm       [device] int32 [B][T]: problem b's sort vector (token indices
 *              within the problem)
 *   prices     [device] may be NULL: [B][E] float32 (int64 in integer mode)
 *   workspace  [device] base_assign_batched_workspace_size(B, T, E) bytes,
 *              256-byte aligned
 *   stats      [host] aggregate over the problems: phases and rounds the
 *              largest, bids and engine_bids summed, eps_final the largest,
 *              fell_back if any problem fell back, converged if all did
 *   1 <= B <= 65535, B * T < 2^31; other arguments as for base_assign.
 * Errors: as base_assign; a status from SYNC_STATS reports the first kind of
 * failure found in any problem.
 */
size_t base_assign_batched_workspace_size(int64_t B, int64_t T, int64_t E);

int base_assign_batched(const void *S, int s_dtype, int64_t B, int64_t T, int64_t E,
                        const base_assign_opts *opts, int32_t *assign, int32_t *perm,
                        void *prices, void *workspace, size_t workspace_bytes,
                        base_assign_stats *stats, void *stream);

/*
 * base_assign_status - how the last solve enqueued on `workspace` ended,
 * read after the fact. base_assign and base_assign_batched return before
 * the solve has run (unless BASE_ASSIGN_SYNC_STATS asks them to wait), so
 * a device-side outcome -- the round limit reached without the greedy
 * completion, a price beyond the representable range, a failed internal
 * consistency check -- cannot be their return value. Each problem's control
 * block stays in its workspace until the workspace is used again; this call
 * waits for `stream` (the stream the solve was enqueued on), reads the B
 * control blocks and reports that outcome without re-running anything
 * (Sec. 3.2.1: the assignment must be balanced; the appendix figure's
 * caption: a solve may stop at its iteration bound).
 *
 *   workspace  [device] the workspace of the solve (B problems of T x E)
 *   B, T, E    as passed to that solve (B = 1 for base_assign)
 *   stats      [host] out, may be NULL: the statistics of base_assign_stats,
 *              aggregated over the problems as for SYNC_STATS, except
 *              dual_gap, which is NaN (it needs the scores and assignment)
 *   stream     the solve's stream (the call synchronises it)
 *
 * Returns BASE_OK when every problem ended balanced; otherwise the first
 * kind of failure found, in this order: BASE_ERR_INTERNAL (a device-side
 * check failed: the solve stopped there and its outputs are unspecified,
 * though every access stayed in bounds), BASE_ERR_RANGE (a price left the
 * representable range), BASE_ERR_NOT_CONVERGED (max_rounds reached without
 * BASE_ASSIGN_GREEDY_FALLBACK). BASE_ERR_INVALID_ARG for bad sizes or a
 * null or misaligned workspace; BASE_ERR_HIP if the read fails.
 */
int base_assign_status(const void *workspace, int64_t B, int64_t T, int64_t E,
                       base_assign_stats *stats, void *stream);

/*
 * base_assign_noalloc - base_assign with no workspace argument and no
 * allocation, for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. The solve's workspace is a library-owned device array of
 * BASE_ASSIGN_NOALLOC_MAX_WORKSPACE bytes (32 MiB; each device the library
 * runs on holds its own copy until the process ends). The call allocates
 * nothing, on the device or on the host. Same algorithm, options, outputs,
 * statistics and errors as base_assign (bit-identical results), plus:
 *   - BASE_ERR_RANGE when base_assign_workspace_size(T, E) exceeds the
 *     array (T = 32768 with E = 128, and T = 65536 with E = 256, fit);
 *   - BASE_ERR_HIP when the array's device address cannot be resolved.
 * Every call on one device shares that device's array, which keeps the
 * last solve's state (and base_assign_status cannot read it: the address
 * is not exported). Calls that overlap on one device -- on different
 * streams or threads without ordering between them -- race on it and give
 * unspecified results. The kernels run on `stream`'s device.
 */
#define BASE_ASSIGN_NOALLOC_MAX_WORKSPACE ((size_t)32 << 20)
int base_assign_noalloc(const void *S, int s_dtype, int64_t T, int64_t E,
                        const base_assign_opts *opts, int32_t *assign, int32_t *perm,
                        void *prices, base_assign_stats *stats, void *stream);

/* ------------------------------------------------------------------------ */
/* base_permute: route rows into expert-contiguous order, or back            */
/* ------------------------------------------------------------------------ */
/*
 * Fig. 2 caption: the assignment vector sorts tokens by expert so that row k
 * of the sorted features goes to expert floor(k E / T). Sec. 3: the expert
 * output returns to the token's original position afterwards.
 *
 *   in, out  [device] T x d rows of dtype (BASE_BF16 or BASE_F32); must not overlap
 *   perm     [device] int32 [T], a permutation of [0, T) (e.g. from base_assign)
 *   inverse  0: out[k, :] = in[perm[k], :]   (gather into expert order)
 *            1: out[perm[k], :] = in[k, :]   (scatter back to token order)
 *   T > 0, d > 0, d % 8 == 0
 *
 * Rows are copied bit for bit. An entry of perm outside [0, T) skips its row
 * (never read or written out of bounds); a repeated entry leaves rows of out
 * unwritten (gather) or written twice (scatter).
 * Errors: BASE_ERR_INVALID_ARG (also when in and out overlap),
 * BASE_ERR_UNSUPPORTED_DTYPE, BASE_ERR_RANGE, BASE_ERR_HIP.
 */
int base_permute(const void *in, const int32_t *perm, void *out, int64_t T, int64_t d, int dtype,
                 int inverse, void *stream);

/*
 * base_permute_batched - the permute of B independent problems of T tokens
 * (base_assign_batched's sort vectors) in one pass, optionally through the
 * shuffle index of base_affinity_gather (Sec. 3.2.1, Shuffling). Routed row
 * k = b T + j (problem b, position j) has the source row
 *     src(k) = shuffle[b T + perm[k]]   (shuffle given)
 *     src(k) = b T + perm[k]            (shuffle NULL)
 * and inverse 0: out[k] = in[src(k)];  inverse 1: out[src(k)] = in[k].
 * With the shuffle, inverse 0 reads the unshuffled H directly into each
 * worker's expert order, and inverse 1 returns expert rows straight to the
 * unshuffled token order.
 *
 *   in, out  [device] B T x d rows of dtype, must not overlap
 *   perm     [device] int32 [B][T], each row a permutation of [0, T)
 *   shuffle  [device] int32 [B T] or NULL, a permutation of [0, B T)
 *   1 <= B, T; B T <= 2^31 - 1; d % 8 == 0
 * Entries out of range skip their row, as in base_permute. B = 1 with no
 * shuffle is base_permute.
 * Errors: as base_permute.
 */
int base_permute_batched(const void *in, const int32_t *perm, const int32_t *shuffle, void *out,
                         int64_t B, int64_t T, int64_t d, int dtype, int inverse, void *stream);

/* ------------------------------------------------------------------------ */
/* Test-time routing and the gated residual                                  */
/* ------------------------------------------------------------------------ */
/*
 * base_greedy_assign - Sec. 3.2.2: at test time every token takes its
 * highest-scoring expert (lowest index on ties; a row of NaN/-inf takes
 * expert 0). No balance: expert loads are whatever the scores give.
 *   S         [device] T x E float32 scores, row-major, 16-byte aligned
 *   assign    [device] int32 [T] out
 *   perm      [device] int32 [T] out: the stable sort of assign (experts
 *             ascending, tokens ascending within an expert)
 *   offsets   [device] int32 [E + 1] out: expert e's rows of the routed order
 *             are [offsets[e], offsets[e + 1])
 *   workspace [device] base_greedy_workspace_size(T, E) bytes, 256-aligned;
 *             any contents at entry. Calls that overlap in time (other
 *             streams) need workspaces of their own.
 *   0 < T < 2^31, 0 < E <= 2048.
 * With E <= 512 the call is one launch whose blocks meet at a grid barrier;
 * it launches no more blocks than the device holds at once. Its waits are
 * bounded: should one give up (a block never scheduled, e.g. while another
 * stream's kernel holds every compute unit indefinitely), the tokens of the
 * blocks that gave up are left unplaced and get assign[t] = -1.
 * Errors: BASE_ERR_INVALID_ARG, BASE_ERR_RANGE, BASE_ERR_WORKSPACE, BASE_ERR_HIP.
 *
 * base_gate_combine - Sec. 3.1, Eq. 1, fused into the return to token order:
 *     out[t] = sigmoid(S[t, a_t]) * F[k] + H[t]   for t = perm[k],
 * where F [T x d] is the experts' output in routed order (row k belongs to
 * token perm[k]) and S[t, a_t] = h_t . w_{a_t} the affinity already computed.
 * fp32 arithmetic; BASE_BF16 rows are widened exactly and the result rounded
 * to nearest even. F, H, out: [device] T x d of dtype (BASE_BF16 or BASE_F32),
 * 16-byte aligned, out must not overlap F or H (BASE_ERR_INVALID_ARG);
 * d % 8 == 0. perm must be a permutation of [0, T) and assign[t] in [0, E)
 * (not checked; an entry out of range is treated as expert 0 / the row
 * skipped, never read out of bounds).
 *
 * base_gate_combine_batched - the same over B problems of T tokens routed
 * with base_assign_batched, optionally shuffled (base_affinity_gather): S
 * [B T x E], assign and perm [B][T] are in worker order, F [B T x d] in
 * routed order, H and out [B T x d] in the unshuffled token order. Routed
 * row k = b T + j belongs to worker token w = b T + perm[k] and to token
 * t = shuffle[w] (t = w if shuffle is NULL):
 *     out[t] = sigmoid(S[w, assign[w]]) * F[k] + H[t].
 * B T <= 2^31 - 1; shuffle a permutation of [0, B T) (entries out of range
 * skip their row). B = 1 with no shuffle is base_gate_combine.
 *
 * base_gate_backward - the gradient of Eq. 1's gate and residual with the
 * expert output held fixed (its own backward belongs to the expert network),
 * for an upstream gradient dY of the layer output:
 *     dS[t]  = g_t (1 - g_t) (dY[t] . f_t),   g_t = sigmoid(S[t, a_t])
 *     dH[t]  = dY[t] + dS[t] W[a_t]
 *     dF[k]  = g_t dY[t]                      (routed order, t = perm[k])
 *     dW[e]  = sum over t with a_t = e of dS[t] H[t]
 * dY, F, H, dH, dF: T x d of dtype; W: E x d of dtype (all 16-byte aligned);
 * dW: E x d float32, 16-byte aligned; dS: float32 [T]. offsets [E + 1]:
 * expert row ranges of the routed order (e * T/E for a balanced assignment;
 * base_greedy_assign's for a greedy one).
 * Accumulation in fp32 in a fixed order (deterministic).
 * Errors: BASE_ERR_INVALID_ARG, BASE_ERR_UNSUPPORTED_DTYPE, BASE_ERR_RANGE,
 * BASE_ERR_HIP.
 */
size_t base_greedy_workspace_size(int64_t T, int64_t E);
int base_greedy_assign(const float *S, int64_t T, int64_t E, int32_t *assign, int32_t *perm,
                       int32_t *offsets, void *workspace, size_t workspace_bytes, void *stream);
int base_gate_combine(const void *F, const void *H, const float *S, const int32_t *assign,
                      const int32_t *perm, void *out, int64_t T, int64_t E, int64_t d, int dtype,
                      void *stream);
int base_gate_combine_batched(const void *F, const void *H, const float *S,
                              const int32_t *assign, const int32_t *perm, const int32_t *shuffle,
                              void *out, int64_t B, int64_t T, int64_t E, int64_t d, int dtype,
                              void *stream);
int base_gate_backward(const void *dY, const void *F, const void *H, const void *W,
                       const float *S, const int32_t *assign, const int32_t *perm,
                       const int32_t *offsets, void *dH, void *dF, float *dW, float *dS,
                       int64_t T, int64_t E, int64_t d, int dtype, void *stream);

/* ------------------------------------------------------------------------ */
/* Measurement support                                                       */
/* ------------------------------------------------------------------------ */
/*
 * Not part of the path. While enabled, base_assign brackets every launch of
 * its single-workgroup engine kernel (the rounds of a phase with few active
 * tokens: most of a solve's time) with a pair of HIP events recorded on the
 * call's stream, so a tool can time that kernel over a stretch of ordinary
 * calls. At most `capacity` launches are recorded; later ones are not.
 *
 * base_timing_enable(capacity) creates 2 * capacity events on the current
 * device and clears the record; capacity <= 0 destroys them and disables the
 * timing. base_timing_read waits for the recorded launches, returns their
 * number and summed duration (milliseconds), and clears the record. One
 * process-wide record; not thread-safe.
 * Errors: BASE_ERR_INVALID_ARG (null pointer), BASE_ERR_HIP.
 */
int base_timing_enable(int32_t capacity);
int base_timing_read(int64_t *launches, double *total_ms);

#ifdef __cplusplus
}
#endif

#endif /* BASE_MI355X_H */
