// C ABI of the assignment path: argument validation on the host, then the
// HIP launchers. Nothing is enqueued when validation fails.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include "base.h"
#include "internal.hpp"

namespace {

constexpr int64_t kMaxTokens = (int64_t)1 << 24;      // token index field of a bid key
constexpr int64_t kMaxTokensInt = (int64_t)1 << 21;   // integer mode: scaled scores stay < 2^37
constexpr int64_t kMaxExperts = 2048;                 // per-expert tables staged in LDS
// Epsilon divisor between phases. Chosen from a sweep of the first-phase
// epsilon (score range / 4 ... / 16) and the divisor (16 ... 96) over twelve
// synthetic workloads (T from 2048 to 65536, E from 64 to 256, normal and
// clustered scores), with the duality check that ends a solve once its
// measured gap meets the bound and the gap-guided step after a check that
// misses it: range / 8 and 32 gave the lowest geometric-mean solve time.
// Without the check a solve runs 1 + ceil(log_32(range / (8 eps_final)))
// phases: 5 or fewer for ranges up to 8 * 32^4 * eps_final (about 840 at 1e-4).
constexpr double kDefaultEpsFactor = 32.0;
constexpr int64_t kMaxDim = (int64_t)1 << 30;
constexpr int64_t kMaxBatch = 65535;   // problems per batched call (grid y dimension)

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int hip_status(hipError_t e) { return e == hipSuccess ? BASE_OK : BASE_ERR_HIP; }

// [a, a + an) and [b, b + bn) share a byte.
bool overlap(const void *a, int64_t an, const void *b, int64_t bn) {
    const char *pa = static_cast<const char *>(a);
    const char *pb = static_cast<const char *>(b);
    return pa < pb + bn && pb < pa + an;
}

int affinity_impl(const void *H, int64_t h_rows, const int32_t *rows, const void *W, float *S,
                  int64_t T, int64_t E, int64_t d, int in_dtype, void *stream) {
    if (H == nullptr || W == nullptr || S == nullptr) return BASE_ERR_INVALID_ARG;
    if (T <= 0 || E <= 0 || d <= 0 || d % 8 != 0 || h_rows <= 0) return BASE_ERR_INVALID_ARG;
    if (!aligned(H, 16) || !aligned(W, 16) || !aligned(S, 16) || !aligned(rows, 4))
        return BASE_ERR_INVALID_ARG;
    if (in_dtype != BASE_BF16 && in_dtype != BASE_F32) return BASE_ERR_UNSUPPORTED_DTYPE;
    if (T > INT32_MAX || h_rows > INT32_MAX || E > 65535 * 128 || d > kMaxDim)
        return BASE_ERR_RANGE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (in_dtype == BASE_BF16)
        return hip_status(base::launch_affinity_bf16(static_cast<const uint16_t *>(H), rows, h_rows,
                                                     static_cast<const uint16_t *>(W), S, T, E, d,
                                                     s));
    return hip_status(base::launch_affinity_f32(static_cast<const float *>(H), rows, h_rows,
                                                static_cast<const float *>(W), S, T, E, d, s));
}

int permute_impl(const void *in, const int32_t *perm, const int32_t *shuffle, void *out,
                 int64_t B, int64_t T, int64_t d, int dtype, int inverse, void *stream) {
    if (in == nullptr || perm == nullptr || out == nullptr) return BASE_ERR_INVALID_ARG;
    if (B <= 0 || T <= 0 || d <= 0 || d % 8 != 0) return BASE_ERR_INVALID_ARG;
    if (inverse != 0 && inverse != 1) return BASE_ERR_INVALID_ARG;
    if (!aligned(in, 16) || !aligned(out, 16) || !aligned(perm, 4) || !aligned(shuffle, 4))
        return BASE_ERR_INVALID_ARG;
    if (dtype != BASE_BF16 && dtype != BASE_F32) return BASE_ERR_UNSUPPORTED_DTYPE;
    if (B > INT32_MAX || T > INT32_MAX || B * T > INT32_MAX || d > kMaxDim) return BASE_ERR_RANGE;
    const int64_t row_bytes = d * (dtype == BASE_BF16 ? 2 : 4);
    const int64_t bytes = B * T * row_bytes;
    if (overlap(in, bytes, out, bytes)) return BASE_ERR_INVALID_ARG;
    return hip_status(base::launch_permute(in, perm, shuffle, out, B, T, row_bytes, inverse,
                                           static_cast<hipStream_t>(stream)));
}

int gate_combine_impl(const void *F, const void *H, const float *S, const int32_t *assign,
                      const int32_t *perm, const int32_t *shuffle, void *out, int64_t B,
                      int64_t T, int64_t E, int64_t d, int dtype, void *stream) {
    if (F == nullptr || H == nullptr || S == nullptr || assign == nullptr || perm == nullptr ||
        out == nullptr)
        return BASE_ERR_INVALID_ARG;
    if (B <= 0 || T <= 0 || E <= 0 || d <= 0 || d % 8 != 0) return BASE_ERR_INVALID_ARG;
    if (dtype != BASE_BF16 && dtype != BASE_F32) return BASE_ERR_UNSUPPORTED_DTYPE;
    if (B > INT32_MAX || T > INT32_MAX || B * T > INT32_MAX || E > INT32_MAX || d > kMaxDim)
        return BASE_ERR_RANGE;
    if (!aligned(F, 16) || !aligned(H, 16) || !aligned(out, 16) || !aligned(S, 4) ||
        !aligned(assign, 4) || !aligned(perm, 4) || !aligned(shuffle, 4))
        return BASE_ERR_INVALID_ARG;
    const int64_t bytes = B * T * d * (dtype == BASE_BF16 ? 2 : 4);
    if (overlap(out, bytes, F, bytes) || overlap(out, bytes, H, bytes)) return BASE_ERR_INVALID_ARG;
    return hip_status(base::launch_gate_combine(F, H, S, assign, perm, shuffle, out, B, T, E, d,
                                                dtype == BASE_BF16 ? 1 : 0,
                                                static_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

const char *base_status_string(int status) {
    switch (status) {
        case BASE_OK: return "ok";
        case BASE_ERR_INVALID_ARG: return "invalid argument";
        case BASE_ERR_NOT_DIVISIBLE: return "T is not a multiple of E";
        case BASE_ERR_UNSUPPORTED_DTYPE: return "unsupported dtype";
        case BASE_ERR_NONFINITE: return "non-finite score";
        case BASE_ERR_NOT_CONVERGED: return "assignment did not converge within max_rounds";
        case BASE_ERR_WORKSPACE: return "workspace missing or too small";
        case BASE_ERR_HIP: return "HIP runtime error";
        case BASE_ERR_RANGE: return "size or value out of the supported range";
        case BASE_ERR_INTERNAL: return "device-side consistency check failed";
        default: return "unknown status";
    }
}

int base_affinity(const void *H, const void *W, float *S, int64_t T, int64_t E, int64_t d,
                  int in_dtype, void *stream) {
    return affinity_impl(H, T, nullptr, W, S, T, E, d, in_dtype, stream);
}

int base_affinity_gather(const void *H, int64_t h_rows, const int32_t *rows, const void *W,
                         float *S, int64_t N, int64_t E, int64_t d, int in_dtype, void *stream) {
    if (rows == nullptr) return BASE_ERR_INVALID_ARG;
    return affinity_impl(H, h_rows, rows, W, S, N, E, d, in_dtype, stream);
}

size_t base_assign_workspace_size(int64_t T, int64_t E) {
    if (T <= 0 || E <= 0 || T % E != 0 || T >= kMaxTokens || E > kMaxExperts) return 0;
    return base::assign_workspace_size(T, E);
}

}  // extern "C"


namespace base {

int aggregate_stats(const SolveCtrl *cs, int64_t B, int64_t E, bool with_gap, void *stats_out) {
    base_assign_stats agg{};
    agg.converged = 1;
    bool internal = false, overflow = false, not_converged = false;
    for (int64_t b = 0; b < B; ++b) {
        const SolveCtrl &c = cs[b];
        const double scale = c.integer ? (double)c.scale : 1.0;
        const int unconverged = c.unconverged_experts & ~(1 << 30);
        agg.phases = c.phase > agg.phases ? c.phase : agg.phases;
        agg.rounds = c.rounds > agg.rounds ? c.rounds : agg.rounds;
        agg.bids += (int64_t)c.bids;
        agg.engine_bids += (int64_t)c.engine_bids;
        agg.augmentations += c.augmentations;
        agg.dual_gap += c.dual_gap / scale;
        const double eps = c.eps / scale;
        agg.eps_last = eps > agg.eps_last ? eps : agg.eps_last;
        const double bound = c.eps_final_eff / scale;
        agg.eps_final = bound > agg.eps_final ? bound : agg.eps_final;
        agg.certified += c.certified != 0 ? 1 : 0;
        agg.fell_back |= c.fell_back;
        const bool conv = unconverged == 0 && (!c.not_converged || c.fell_back) &&
                          c.internal_error == 0;
        if (!conv) agg.converged = 0;
        internal |= c.internal_error != 0;
        overflow |= c.overflow != 0;
        not_converged |= unconverged != 0 || (c.not_converged && !c.fell_back);
    }
    if (!with_gap) agg.dual_gap = NAN;
    if (E == 1) {
        agg = base_assign_stats{};
        agg.converged = 1;
    }
    *static_cast<base_assign_stats *>(stats_out) = agg;
    if (E > 1) {
        if (internal) return BASE_ERR_INTERNAL;
        if (overflow) return BASE_ERR_RANGE;
        if (not_converged) return BASE_ERR_NOT_CONVERGED;
    }
    return BASE_OK;
}

}  // namespace base

namespace base {

// base_assign and base_assign_batched (and the allocation-free variant): B
// independent problems, each a T x E score matrix, solved by one sequence of
// launches (problem b in blockIdx.y of every solver kernel).
int assign_entry(const void *S, int s_dtype, int64_t B, int64_t T, int64_t E,
                 const base_assign_opts *opts, int32_t *assign, int32_t *perm, void *prices,
                 void *workspace, size_t workspace_bytes, base_assign_stats *stats, void *stream) {
    if (S == nullptr || assign == nullptr || perm == nullptr) return BASE_ERR_INVALID_ARG;
    if (T <= 0 || E <= 0 || B <= 0) return BASE_ERR_INVALID_ARG;
    if (s_dtype != BASE_F32 && s_dtype != BASE_I16) return BASE_ERR_UNSUPPORTED_DTYPE;
    if (T % E != 0) return BASE_ERR_NOT_DIVISIBLE;
    const bool integer = s_dtype == BASE_I16;
    if (T >= kMaxTokens || E > kMaxExperts || B > kMaxBatch || B * T > INT32_MAX)
        return BASE_ERR_RANGE;
    if (integer && T >= kMaxTokensInt) return BASE_ERR_RANGE;
    if (!aligned(S, 16) || !aligned(assign, 4) || !aligned(perm, 4)) return BASE_ERR_INVALID_ARG;
    if (B > 1 && ((T * E * (integer ? 2 : 4)) % 16) != 0) return BASE_ERR_INVALID_ARG;
    if (prices != nullptr && !aligned(prices, integer ? 8 : 4)) return BASE_ERR_INVALID_ARG;

    base_assign_opts o{1e-4, 0.0, kDefaultEpsFactor, 4000000, 0u};
    if (opts != nullptr) {
        o = *opts;
        if (isnan(o.eps_final) || isnan(o.eps_initial) || isnan(o.eps_factor) ||
            isinf(o.eps_final) || isinf(o.eps_initial) || isinf(o.eps_factor))
            return BASE_ERR_INVALID_ARG;
        if (!(o.eps_final > 0.0)) o.eps_final = 1e-4;
        if (!(o.eps_factor > 1.0)) o.eps_factor = kDefaultEpsFactor;
        if (o.max_rounds <= 0) o.max_rounds = kDefaultMaxRounds;
        const uint32_t known = BASE_ASSIGN_GREEDY_FALLBACK | BASE_ASSIGN_SYNC_STATS |
                               BASE_ASSIGN_CHECK_FINITE | BASE_ASSIGN_WARM_PRICES |
                               BASE_ASSIGN_FULL_SCHEDULE;
        if (o.flags & ~known) return BASE_ERR_INVALID_ARG;
        if ((o.flags & BASE_ASSIGN_WARM_PRICES) && prices == nullptr) return BASE_ERR_INVALID_ARG;
    }

    const size_t need = base::assign_workspace_size(T, E) * (size_t)B;
    if (workspace == nullptr || workspace_bytes < need || !aligned(workspace, 256))
        return BASE_ERR_WORKSPACE;

    hipStream_t s = static_cast<hipStream_t>(stream);
    base::AssignParams p{};
    p.T = T;
    p.E = E;
    p.C = T / E;
    p.integer = integer;
    p.scale = 1;
    if (integer) {
        int64_t K = 1;
        while (K < T + 1) K <<= 1;
        p.scale = K;
        p.eps_final = 1.0;
        p.eps_initial = o.eps_initial > 0.0 ? floor(o.eps_initial * (double)K) : 0.0;
    } else {
        p.eps_final = o.eps_final;
        p.eps_initial = o.eps_initial;
    }
    p.eps_factor = o.eps_factor;
    p.max_rounds = o.max_rounds;
    p.flags = o.flags;
    p.warm_prices = (o.flags & BASE_ASSIGN_WARM_PRICES) ? prices : nullptr;

    if ((o.flags & BASE_ASSIGN_CHECK_FINITE) && !integer) {
        int bad = 0;
        hipError_t e = base::check_scores_finite(static_cast<const float *>(S), B * T * E, T, E,
                                                 workspace, &bad, s);
        if (e != hipSuccess) return BASE_ERR_HIP;
        if (bad) return BASE_ERR_NONFINITE;
    }

    hipError_t e = base::launch_assign(S, p, B, assign, perm, prices, workspace, s);
    if (e != hipSuccess) return BASE_ERR_HIP;

    if (o.flags & BASE_ASSIGN_SYNC_STATS) {
        // One problem reads into a local control block (no host allocation).
        base::SolveCtrl one{};
        base::SolveCtrl *cs =
            B == 1 ? &one
                   : static_cast<base::SolveCtrl *>(calloc((size_t)B, sizeof(base::SolveCtrl)));
        if (cs == nullptr) return BASE_ERR_HIP;
        e = base::read_assign_stats(workspace, T, E, B, cs, s);
        if (e != hipSuccess) {
            if (cs != &one) free(cs);
            return BASE_ERR_HIP;
        }
        base_assign_stats agg{};
        const int st = base::aggregate_stats(cs, B, E, true, &agg);
        if (cs != &one) free(cs);
        if (stats != nullptr) *stats = agg;
        return st;
    }
    return BASE_OK;
}

}  // namespace base

extern "C" {

int base_assign(const void *S, int s_dtype, int64_t T, int64_t E, const base_assign_opts *opts,
                int32_t *assign, int32_t *perm, void *prices, void *workspace,
                size_t workspace_bytes, base_assign_stats *stats, void *stream) {
    return base::assign_entry(S, s_dtype, 1, T, E, opts, assign, perm, prices, workspace,
                              workspace_bytes, stats, stream);
}

size_t base_assign_batched_workspace_size(int64_t B, int64_t T, int64_t E) {
    if (B <= 0 || B > kMaxBatch) return 0;
    return base_assign_workspace_size(T, E) * (size_t)B;
}

int base_assign_batched(const void *S, int s_dtype, int64_t B, int64_t T, int64_t E,
                        const base_assign_opts *opts, int32_t *assign, int32_t *perm,
                        void *prices, void *workspace, size_t workspace_bytes,
                        base_assign_stats *stats, void *stream) {
    return base::assign_entry(S, s_dtype, B, T, E, opts, assign, perm, prices, workspace,
                              workspace_bytes, stats, stream);
}

int base_assign_status(const void *workspace, int64_t B, int64_t T, int64_t E,
                       base_assign_stats *stats, void *stream) {
    if (workspace == nullptr || !aligned(workspace, 256)) return BASE_ERR_INVALID_ARG;
    if (B <= 0 || T <= 0 || E <= 0 || T % E != 0 || B > kMaxBatch || T >= kMaxTokens ||
        E > kMaxExperts || B * T > INT32_MAX)
        return BASE_ERR_INVALID_ARG;
    base::SolveCtrl *cs = static_cast<base::SolveCtrl *>(calloc((size_t)B, sizeof(base::SolveCtrl)));
    if (cs == nullptr) return BASE_ERR_HIP;
    const hipError_t e =
        base::read_assign_stats(workspace, T, E, B, cs, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
        free(cs);
        return BASE_ERR_HIP;
    }
    base_assign_stats agg{};
    const int st = base::aggregate_stats(cs, B, E, false, &agg);
    free(cs);
    if (stats != nullptr) *stats = agg;
    return st;
}

size_t base_greedy_workspace_size(int64_t T, int64_t E) {
    if (T <= 0 || E <= 0 || T > INT32_MAX || E > kMaxExperts) return 0;
    return base::greedy_workspace_size(T, E);
}

int base_greedy_assign(const float *S, int64_t T, int64_t E, int32_t *assign, int32_t *perm,
                       int32_t *offsets, void *workspace, size_t workspace_bytes, void *stream) {
    if (S == nullptr || assign == nullptr || perm == nullptr || offsets == nullptr)
        return BASE_ERR_INVALID_ARG;
    if (T <= 0 || E <= 0) return BASE_ERR_INVALID_ARG;
    if (T > INT32_MAX || E > kMaxExperts) return BASE_ERR_RANGE;
    if (!aligned(S, 16) || !aligned(assign, 4) || !aligned(perm, 4) || !aligned(offsets, 4))
        return BASE_ERR_INVALID_ARG;
    if (workspace == nullptr || workspace_bytes < base::greedy_workspace_size(T, E) ||
        !aligned(workspace, 256))
        return BASE_ERR_WORKSPACE;
    return hip_status(base::launch_greedy(S, T, E, assign, perm, offsets, workspace,
                                          static_cast<hipStream_t>(stream)));
}

int base_gate_combine(const void *F, const void *H, const float *S, const int32_t *assign,
                      const int32_t *perm, void *out, int64_t T, int64_t E, int64_t d, int dtype,
                      void *stream) {
    return gate_combine_impl(F, H, S, assign, perm, nullptr, out, 1, T, E, d, dtype, stream);
}

int base_gate_combine_batched(const void *F, const void *H, const float *S,
                              const int32_t *assign, const int32_t *perm, const int32_t *shuffle,
                              void *out, int64_t B, int64_t T, int64_t E, int64_t d, int dtype,
                              void *stream) {
    return gate_combine_impl(F, H, S, assign, perm, shuffle, out, B, T, E, d, dtype, stream);
}

int base_gate_backward(const void *dY, const void *F, const void *H, const void *W,
                       const float *S, const int32_t *assign, const int32_t *perm,
                       const int32_t *offsets, void *dH, void *dF, float *dW, float *dS,
                       int64_t T, int64_t E, int64_t d, int dtype, void *stream) {
    if (dY == nullptr || F == nullptr || H == nullptr || W == nullptr || S == nullptr ||
        assign == nullptr || perm == nullptr || offsets == nullptr || dH == nullptr ||
        dF == nullptr || dW == nullptr || dS == nullptr)
        return BASE_ERR_INVALID_ARG;
    if (T <= 0 || E <= 0 || d <= 0 || d % 8 != 0) return BASE_ERR_INVALID_ARG;
    if (dtype != BASE_BF16 && dtype != BASE_F32) return BASE_ERR_UNSUPPORTED_DTYPE;
    if (T > INT32_MAX || E > 65535 || d > kMaxDim) return BASE_ERR_RANGE;
    if (!aligned(dY, 16) || !aligned(F, 16) || !aligned(H, 16) || !aligned(W, 16) ||
        !aligned(dH, 16) || !aligned(dF, 16) || !aligned(dW, 16) || !aligned(dS, 4) ||
        !aligned(S, 4) || !aligned(assign, 4) || !aligned(perm, 4) || !aligned(offsets, 4))
        return BASE_ERR_INVALID_ARG;
    return hip_status(base::launch_gate_backward(dY, F, H, W, S, assign, perm, offsets, dH, dF, dW,
                                                 dS, T, E, d, dtype == BASE_BF16 ? 1 : 0,
                                                 static_cast<hipStream_t>(stream)));
}

int base_timing_enable(int32_t capacity) {
    return hip_status(base::timing_enable(capacity));
}

int base_timing_read(int64_t *launches, double *total_ms) {
    if (launches == nullptr || total_ms == nullptr) return BASE_ERR_INVALID_ARG;
    return hip_status(base::timing_read(launches, total_ms));
}

int base_permute(const void *in, const int32_t *perm, void *out, int64_t T, int64_t d, int dtype,
                 int inverse, void *stream) {
    return permute_impl(in, perm, nullptr, out, 1, T, d, dtype, inverse, stream);
}

int base_permute_batched(const void *in, const int32_t *perm, const int32_t *shuffle, void *out,
                         int64_t B, int64_t T, int64_t d, int dtype, int inverse, void *stream) {
    return permute_impl(in, perm, shuffle, out, B, T, d, dtype, inverse, stream);
}

}  // extern "C"
