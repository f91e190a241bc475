// Balanced token-to-expert assignment (Sec. 3.2.1, Eq. 2) by a forward
// auction with epsilon scaling, every expert being C = T/E identical objects.
//
// State (all in the caller's workspace):
//   prices[E]          expert prices p_e (fp32, or int64 in integer mode)
//   holders[2][E][C]   each expert's held bid keys (two buffers, per-expert
//                      selector hsel[e]; hcount[e] valid entries)
//   bucket[E][cap]     the bids an expert received this round (bcount[e]);
//                      bids beyond `cap` go to one shared overflow list
//   active[2][T]       tokens without an expert (ping-pong between rounds)
//   ctrl               round/phase counters, epsilon, flags
//
// One round:
//   bid     every active token t finds its best and second-best values
//           v_e = S[t,e] - p_e over all experts and bids S[t,e1] - v2 + eps
//           for its best expert e1 (lowest index on ties).
//   update  every expert that received bids keeps the C highest keys among
//           its holders and the new bids (ties: lower token index), sends
//           the others back to the active list, and, once full, sets its
//           price to its lowest held bid.
// A phase ends when no token is active (every expert holds C); epsilon is
// then divided by eps_factor down to eps_final and all tokens bid again
// against the prices reached so far.
//
// Invariant behind the guarantee: a held token's bid was computed against
// prices no higher than the current ones and its expert's price never
// exceeds that bid, so S[t,a_t] - p[a_t] >= max_e (S[t,e] - p_e) - eps for
// every token; summed over tokens this bounds the distance to the optimum by
// T * eps.
//
// Execution: the first rounds of a phase (many active tokens) run as grid-wide
// bid and update kernels; the remaining rounds, which typically have a
// handful of active tokens each, run inside one workgroup that loops with
// block barriers instead of kernel launches.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

#include <map>
#include <mutex>
#include <tuple>

#include "common.hpp"
#include "internal.hpp"
#include "base.h"

namespace base {
namespace {

constexpr int kThreads = 256;
constexpr int kCandLds = 4096;   // candidates of one expert staged in LDS when they fit
constexpr int kRangeBlocks = 256;   // blocks of the score-range reduction
constexpr int kPrologueBlocks = 4096;   // largest grid of the prologue (one range partial each)
constexpr int kCountTile = 256;  // tokens per block in the permutation build
constexpr int kWideLoopRounds = 1024;  // rounds one launch of the round loop may run
constexpr int kCheckBlocks = 4096;     // largest grid of the phase check
// Experts the shortest-path finish serves: its exchange matrix then takes 16
// registers per thread (64 at E = 256 would leave too few for the rest of
// the kernel at 1024 threads).
constexpr int kSspMaxE = 256;

inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// Unassigned tokens of a phase below which the shortest-path finish takes
// over (0: never). Measured over seventeen workloads: 12 for T >= 8192 with
// E >= 64 (the mixture and normal T = 32768 shapes, T = 8192 with E = 64,
// T = 65536 with E = 256 all faster than at 8), 8 below (the worker shape
// T = 2048, E = 128 and the E = 16 shapes slower at 12). BASE_SSP_CAP
// overrides it (read at every solve; a tuning knob, not part of the
// interface).
inline int ssp_cap_setting(int64_t T, int64_t E) {
    const char *v = getenv("BASE_SSP_CAP");
    if (v == nullptr || *v == 0) return T >= 8192 && E >= 64 ? 12 : 8;
    return (int)strtol(v, nullptr, 10);
}

// Phases above the last end early (see end_round) once at most T / D
// tokens are left active (BASE_EARLY_END_DIV = D, 0: never; read at every
// solve, a tuning knob).
inline int early_end_tokens_setting(int64_t T) {
    const char *v = getenv("BASE_EARLY_END_DIV");
    const long d = (v == nullptr || *v == 0) ? 32 : strtol(v, nullptr, 10);
    return d > 0 ? (int)(T / d) : 0;
}

// Whether the single-workgroup rounds (small_solve_kernel) serve a shape
// that fits them: BASE_SMALL_PATH=1 always, =0 never (read at every solve;
// tests use it to cover both paths); unset, -1: the default rule.
inline int small_path_setting() {
    const char *v = getenv("BASE_SMALL_PATH");
    if (v == nullptr || *v == 0) return -1;
    return *v == '0' ? 0 : 1;
}

// BASE_TEST_SSP_FALLBACKS=1 (tests only) sends every step of the
// shortest-path finish through its fallback paths.
inline int ssp_fallbacks_setting() {
    const char *v = getenv("BASE_TEST_SSP_FALLBACKS");
    return (v != nullptr && *v == '1') ? 1 : 0;
}

// Polls a grid barrier's wait makes before it gives up. BASE_TEST_BARRIER_POLLS
// overrides the default (read at every solve): tests set it to 0 to force
// the give-up path from the host, so that every block still exits normally.
inline uint32_t barrier_polls() {
    const char *v = getenv("BASE_TEST_BARRIER_POLLS");
    if (v == nullptr || *v == 0) return 1u << 24;
    return (uint32_t)strtoul(v, nullptr, 10);
}

// With BASE_DEBUG set in the environment, notes why a launch path was taken
// or which HIP call failed, on stderr.
inline void debug_note(const char *what, hipError_t err) {
    static const bool on = getenv("BASE_DEBUG") != nullptr;
    if (on) fprintf(stderr, "[base] %s: %s\n", what, hipGetErrorString(err));
}

struct Layout {
    size_t ctrl, prices, hcount, hsel, bcount, holders, bucket, ovf_key, ovf_exp, active, blk,
        eck, ecs, ecn, sums, bar, rpart, gpart, sspm, sspa, sspt, total;
    int64_t cap, nblk;
};

Layout make_layout(int64_t T, int64_t E) {
    Layout L{};
    const int64_t C = T / E;
    L.cap = 16 * C + 4096;
    if (L.cap > T) L.cap = T;
    L.nblk = (T + kCountTile - 1) / kCountTile;
    size_t off = 0;
    L.ctrl = off;    off += align_up(sizeof(SolveCtrl));
    L.prices = off;  off += align_up((size_t)E * 8);
    L.hcount = off;  off += align_up((size_t)E * 4);
    L.hsel = off;    off += align_up((size_t)E * 4);
    L.bcount = off;  off += align_up((size_t)E * 4);
    L.holders = off; off += align_up((size_t)2 * T * 8);
    L.bucket = off;  off += align_up((size_t)E * L.cap * 8);
    L.ovf_key = off; off += align_up((size_t)T * 8);
    L.ovf_exp = off; off += align_up((size_t)T * 4);
    L.active = off;  off += align_up((size_t)2 * T * 4);
    L.blk = off;     off += align_up((size_t)L.nblk * E * 4);
    L.eck = off;     off += align_up((size_t)E * 64 * 8);   // engine entry lists (K <= 64)
    L.ecs = off;     off += align_up((size_t)E * 64 * 2);
    L.ecn = off;     off += align_up((size_t)E * 4);
    L.sums = off;    off += align_up((size_t)T * 64);          // per-token score summaries
    L.bar = off;     off += align_up(512);                      // grid barrier words
    L.rpart = off;   off += align_up((size_t)kPrologueBlocks * 12);   // score-range partials
    L.gpart = off;   off += align_up((size_t)kCheckBlocks * 8);    // phase-check partials
    // The exchange matrix of the shortest-path finish (E <= 256 only):
    // cheapest move from expert e to expert x and the slot of its token.
    const int64_t Es = E <= kSspMaxE ? E : 0;
    L.sspm = off;    off += align_up((size_t)Es * Es * 4);
    L.sspa = off;    off += align_up((size_t)Es * Es * 2);
    // Every expert's held tokens as uint16 in slot order (T <= 65536), in
    // the layout the finish keeps in LDS.
    L.sspt = off;    off += align_up(E <= kSspMaxE && T <= 65536 ? (size_t)T * 2 : 0);
    L.total = off;
    return L;
}

template <class M>
struct Ctx {
    using value_t = typename M::value_t;
    const typename M::score_t *S;
    int T, E, C, cap;
    int64_t scale;
    SolveCtrl *ctrl;
    value_t *prices;
    int *hcount, *hsel, *bcount;
    uint64_t *holders, *bucket, *ovf_key;
    int *ovf_exp, *active;
    int *ovf_count;   // lives in ctrl->pad0
    int engine_cap;   // > 0: rounds with at most this many active tokens go to the engine
    int eng_k;        // length of the engine's per-expert lists of lowest keys
    uint64_t *eng_ck; // the lists as built at the engine's entry
    uint16_t *eng_cs;
    int *eng_cn;
    uint32_t *sums;   // T x 16 words: each token's 8 best scores, their experts, a bound
    uint64_t *bar;    // grid barrier: arrivals at bar[0], release at bar[32] (own lines)
    double *gpart;    // per-block partial sums of the phase check
    int ssp_cap;      // > 0: a phase with at most this many active tokens left is finished
                      // by shortest augmenting paths
    int early_n;      // > 0: a phase above the last whose epsilon exceeds kEarlyRatio
                      // eps_final ends once at most early_n tokens are left active;
                      // < 0: every phase above the last ends at -early_n
    float *ssp_m;     // [E][E] min over tokens t of expert e of S[t,e] - S[t,x]
    uint16_t *ssp_a;  // [E][E] the holder slot of that token
    uint16_t *ssp_t;  // [E][C] the tokens of every expert's holder slots (0 past its count)
    int64_t ws_stride;   // bytes between the workspaces of consecutive problems of a batch

    // The view of problem b of a batch (blockIdx.y in every solver launch):
    // the workspace pointers move by b workspace strides, the scores by b
    // score matrices.
    template <class P>
    __host__ __device__ static P *shift(P *ptr, int64_t bytes) {
        return reinterpret_cast<P *>(reinterpret_cast<uintptr_t>(ptr) + bytes);
    }
    __host__ __device__ __attribute__((always_inline)) Ctx at(int b) const {
        Ctx r = *this;
        if (b == 0) return r;
        const int64_t w = (int64_t)b * ws_stride;
        r.S = S + (int64_t)b * T * E;
        r.ctrl = shift(ctrl, w);
        r.prices = shift(prices, w);
        r.hcount = shift(hcount, w);
        r.hsel = shift(hsel, w);
        r.bcount = shift(bcount, w);
        r.holders = shift(holders, w);
        r.bucket = shift(bucket, w);
        r.ovf_key = shift(ovf_key, w);
        r.ovf_exp = shift(ovf_exp, w);
        r.active = shift(active, w);
        r.ovf_count = shift(ovf_count, w);
        r.eng_ck = shift(eng_ck, w);
        r.eng_cs = shift(eng_cs, w);
        r.eng_cn = shift(eng_cn, w);
        r.sums = shift(sums, w);
        r.bar = shift(bar, w);
        r.gpart = shift(gpart, w);
        r.ssp_m = shift(ssp_m, w);
        r.ssp_a = shift(ssp_a, w);
        r.ssp_t = shift(ssp_t, w);
        return r;
    }
};

template <class M>
Ctx<M> make_ctx(const void *S, const AssignParams &p, char *ws) {
    const Layout L = make_layout(p.T, p.E);
    Ctx<M> c;
    c.S = static_cast<const typename M::score_t *>(S);
    c.T = (int)p.T;
    c.E = (int)p.E;
    c.C = (int)p.C;
    c.cap = (int)L.cap;
    c.scale = p.scale;
    c.ctrl = reinterpret_cast<SolveCtrl *>(ws + L.ctrl);
    c.prices = reinterpret_cast<typename M::value_t *>(ws + L.prices);
    c.hcount = reinterpret_cast<int *>(ws + L.hcount);
    c.hsel = reinterpret_cast<int *>(ws + L.hsel);
    c.bcount = reinterpret_cast<int *>(ws + L.bcount);
    c.holders = reinterpret_cast<uint64_t *>(ws + L.holders);
    c.bucket = reinterpret_cast<uint64_t *>(ws + L.bucket);
    c.ovf_key = reinterpret_cast<uint64_t *>(ws + L.ovf_key);
    c.ovf_exp = reinterpret_cast<int *>(ws + L.ovf_exp);
    c.active = reinterpret_cast<int *>(ws + L.active);
    c.ovf_count = &c.ctrl->pad0;
    c.engine_cap = 0;
    c.eng_k = 8;
    c.eng_ck = reinterpret_cast<uint64_t *>(ws + L.eck);
    c.eng_cs = reinterpret_cast<uint16_t *>(ws + L.ecs);
    c.eng_cn = reinterpret_cast<int *>(ws + L.ecn);
    c.sums = reinterpret_cast<uint32_t *>(ws + L.sums);
    c.bar = reinterpret_cast<uint64_t *>(ws + L.bar);
    c.gpart = reinterpret_cast<double *>(ws + L.gpart);
    c.ssp_cap = 0;
    c.ssp_m = reinterpret_cast<float *>(ws + L.sspm);
    c.ssp_a = reinterpret_cast<uint16_t *>(ws + L.sspa);
    c.ssp_t = reinterpret_cast<uint16_t *>(ws + L.sspt);
    c.ws_stride = (int64_t)L.total;
    c.early_n = 0;
    return c;
}

// ---------------------------------------------------------------- helpers --

__device__ inline int lane_id() { return threadIdx.x & 63; }

// Counters that other waves update with atomics are read with atomic loads so
// that no stale cached copy is used.
__device__ inline int ld_relaxed(const int *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Copies n16 16-byte words from global memory to LDS with kBlock threads,
// eight loads in flight per thread before any store (a plain loop waits for
// each load before the next).
template <int kBlock>
__device__ inline void copy16_to_lds(uint4 *dst, const uint4 *src, int n16) {
    constexpr int kU = 8;
    for (int i0 = threadIdx.x; i0 < n16; i0 += kU * kBlock) {
        uint4 v[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int i = i0 + u * kBlock;
            if (i < n16) v[u] = src[i];
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int i = i0 + u * kBlock;
            if (i < n16) dst[i] = v[u];
        }
    }
}

// A consistency check failed: the access is skipped and the call reports
// BASE_ERR_INTERNAL instead of touching memory outside the workspace. The
// solve also ends there: every later solver kernel sees `done` and returns
// at once, and the greedy completion does not run, so no kernel goes on
// from a half-finished round. The finalising kernels still run (every
// access in bounds); their outputs are unspecified.
__device__ inline void flag_internal(SolveCtrl *ctrl) {
    ctrl->internal_error = 1;
    ctrl->done = 1;
}

__device__ inline uint64_t lanemask_lt() {
    const int l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Appends `tok` to active list `which` for every lane with want == true.
// Must be reached by all lanes of the wave together.
template <class M>
__device__ inline void append_active(const Ctx<M> &c, int which, bool want, int tok) {
    const uint64_t mask = __ballot(want);
    if (mask == 0) return;
    const int leader = __ffsll((long long)mask) - 1;
    int base = 0;
    if (lane_id() == leader) base = atomicAdd(&c.ctrl->active_count[which], __popcll(mask));
    base = __shfl(base, leader);
    const int at = base + __popcll(mask & lanemask_lt());
    if (want) {
        if (at < c.T && tok >= 0 && tok < c.T) c.active[(int64_t)which * c.T + at] = tok;
        else flag_internal(c.ctrl);
    }
}

// -------------------------------------------------------------------- bid --

// One group of G lanes evaluates one token. VEC: rows are read as 16-byte
// vectors (E % 8 == 0 for int16, E % 4 == 0 for fp32).
// One group of G lanes evaluates one token: lane gl owns experts
// [8 gl, 8 gl + 8) of every chunk of 8 G experts and loads them with
// 16-byte vector reads issued before any comparison, so a row costs one
// memory latency. Ties keep the lowest expert index (ascending scan inside a
// lane, index comparison across lanes). s1 returns the score S[t, e1]
// itself, so the bid needs no second read.
template <class M>
__device__ inline void load8(const typename M::score_t *S, int64_t base, int e0, int E, int64_t scale,
                             typename M::value_t (&sv)[8]) {
    using score_t = typename M::score_t;
    constexpr int kVecElems = 16 / sizeof(score_t);   // 4 fp32 or 8 int16 per 16 bytes
    const bool vec = (e0 + 8 <= E) && ((base + e0) % kVecElems == 0);
    if (vec) {
        if constexpr (sizeof(score_t) == 4) {
            const float4 a = *reinterpret_cast<const float4 *>(S + base + e0);
            const float4 b = *reinterpret_cast<const float4 *>(S + base + e0 + 4);
            const float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
            for (int j = 0; j < 8; ++j) sv[j] = (typename M::value_t)f[j];
        } else {
            const uint4 a = *reinterpret_cast<const uint4 *>(S + base + e0);
            const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
            for (int j = 0; j < 8; ++j)
                sv[j] = (typename M::value_t)(int16_t)(uint16_t)(w[j >> 1] >> (16 * (j & 1))) * scale;
        }
    } else {
#pragma unroll
        for (int j = 0; j < 8; ++j)
            sv[j] = (e0 + j < E) ? M::load(S, base + e0 + j, scale) : (typename M::value_t)0;
    }
}

// Partner of a lane in step OFF (1, 2, 4, ...) of a butterfly reduction over
// aligned groups of lanes. Inside a row of 16 lanes the partner comes from a
// DPP move: swaps inside quads for OFF = 1, 2, then the mirror of the half
// row (OFF = 4) and of the row (OFF = 8). A mirror pairs each lane with one
// of the other half, which reduces as well as an xor once every half holds
// one value. Wider steps go through ds_bpermute.
template <int CTRL>
__device__ inline uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, CTRL, 0xf, 0xf, false);
}
template <int OFF, class T>
__device__ inline T grp_partner(T v) {
    constexpr int kCtrl = OFF == 1 ? 0xB1 : OFF == 2 ? 0x4E : OFF == 4 ? 0x141 : 0x140;
    if constexpr (OFF <= 8) {
        if constexpr (sizeof(T) == 8) {
            uint64_t u;
            __builtin_memcpy(&u, &v, 8);
            const uint64_t r = (uint64_t)dpp_u32<kCtrl>((uint32_t)u) |
                               ((uint64_t)dpp_u32<kCtrl>((uint32_t)(u >> 32)) << 32);
            T out;
            __builtin_memcpy(&out, &r, 8);
            return out;
        } else {
            uint32_t u;
            __builtin_memcpy(&u, &v, 4);
            const uint32_t r = dpp_u32<kCtrl>(u);
            T out;
            __builtin_memcpy(&out, &r, 4);
            return out;
        }
    } else {
        return __shfl_xor(v, OFF);
    }
}

// Merges the top-2 of the partner lane: (v1, e1) is the best value and its
// expert (ties to the lower expert), v2 the best value of any other expert,
// s1 the score of e1.
template <int OFF, class M>
__device__ inline void top2_step(typename M::value_t &v1, int &e1, typename M::value_t &v2,
                                 typename M::value_t &s1) {
    using value_t = typename M::value_t;
    const value_t ov1 = grp_partner<OFF>(v1);
    const int oe1 = grp_partner<OFF>(e1);
    const value_t ov2 = grp_partner<OFF>(v2);
    const value_t os1 = grp_partner<OFF>(s1);
    // Selects only (no branches: every lane takes the same instructions).
    const bool take = (ov1 > v1) | ((ov1 == v1) & (oe1 < e1));
    const value_t keep2 = v2 > ov1 ? v2 : ov1;
    const value_t take2 = v1 > ov2 ? v1 : ov2;
    v2 = take ? take2 : keep2;
    v1 = take ? ov1 : v1;
    e1 = take ? oe1 : e1;
    s1 = take ? os1 : s1;
}

// Top-2 over a group of G lanes; every lane of the group ends with the result.
template <class M, int G>
__device__ inline void top2_reduce(typename M::value_t &v1, int &e1, typename M::value_t &v2,
                                   typename M::value_t &s1) {
    if constexpr (G > 1) top2_step<1, M>(v1, e1, v2, s1);
    if constexpr (G > 2) top2_step<2, M>(v1, e1, v2, s1);
    if constexpr (G > 4) top2_step<4, M>(v1, e1, v2, s1);
    if constexpr (G > 8) top2_step<8, M>(v1, e1, v2, s1);
    if constexpr (G > 16) top2_step<16, M>(v1, e1, v2, s1);
    if constexpr (G > 32) top2_step<32, M>(v1, e1, v2, s1);
}

// Adds value v (expert e, score sc) to a lane's running top-2, with selects
// only. The first of equal values keeps the best place (experts arrive in
// ascending order).
template <class M>
__device__ __attribute__((always_inline)) inline void top2_push(
    typename M::value_t v, int e, typename M::value_t sc, typename M::value_t &v1, int &e1,
    typename M::value_t &v2, typename M::value_t &s1) {
    const bool gt1 = v > v1;
    const bool gt2 = v > v2;
    v2 = gt1 ? v1 : (gt2 ? v : v2);
    v1 = gt1 ? v : v1;
    e1 = gt1 ? e : e1;
    s1 = gt1 ? sc : s1;
}

// Top-2 of one token whose lane-local scores sv (experts e0 .. e0 + 7) are
// already in registers (rows that fit one chunk of 8 G experts).
template <class M, int G>
__device__ inline void top2_row(const typename M::value_t (&sv)[8], int e0, int E, bool valid,
                                const typename M::value_t *pr, typename M::value_t &v1, int &e1,
                                typename M::value_t &v2, typename M::value_t &s1) {
    using value_t = typename M::value_t;
    v1 = M::lowest();
    v2 = M::lowest();
    s1 = 0;
    e1 = 0x7fffffff;
    if (valid && e0 < E) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int e = e0 + j;
            const bool in = e < E;
            const value_t v = in ? sv[j] - pr[in ? e : 0] : M::lowest();
            top2_push<M>(v, e, sv[j], v1, e1, v2, s1);
        }
    }
    top2_reduce<M, G>(v1, e1, v2, s1);
}

template <class M, int G>
__device__ inline void top2_token(const Ctx<M> &c, int t, bool valid, const typename M::value_t *pr,
                                  typename M::value_t &v1, int &e1, typename M::value_t &v2,
                                  typename M::value_t &s1) {
    using value_t = typename M::value_t;
    const int gl = lane_id() & (G - 1);
    v1 = M::lowest();
    v2 = M::lowest();
    s1 = 0;
    e1 = 0x7fffffff;
    if (valid) {
        const int64_t row = (int64_t)t * c.E;
        for (int base = 0; base < c.E; base += 8 * G) {
            const int e0 = base + 8 * gl;
            if (e0 >= c.E) break;
            value_t sv[8];
            load8<M>(c.S, row, e0, c.E, c.scale, sv);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int e = e0 + j;
                const bool in = e < c.E;
                const value_t v = in ? sv[j] - pr[in ? e : 0] : M::lowest();
                top2_push<M>(v, e, sv[j], v1, e1, v2, s1);
            }
        }
    }
    top2_reduce<M, G>(v1, e1, v2, s1);
}

// ---------------------------------------------------------- score summaries --
//
// A token's summary is 64 bytes: its 8 highest scores (words 0..7, fp32 bits or
// the raw int16 score), their experts (words 8..11, two uint16 per word), the
// 9th highest score (word 12; the lowest value when E <= 8, where the 8 cover
// every expert) and the number of entries (word 13). Scores never change
// during a solve, so the summaries are built once. For prices p, every expert
// outside a summary has S[t,e] - p[e] <= bound - min_e p[e]; a top-2 taken
// over the summary is therefore the top-2 over all experts whenever its best
// value exceeds that limit and its second value reaches it.

constexpr int kSumWords = 16;
constexpr int kSumChunks = 4;   // chunks of 8 G experts per row: E <= 4 * 8 * 64 = 2048

template <class M>
__device__ inline uint32_t score_bits(typename M::value_t v, int64_t scale) {
    if constexpr (M::kInteger) return (uint32_t)(int32_t)(v / scale);
    else return __float_as_uint(v);
}
template <class M>
__device__ inline typename M::value_t bits_score(uint32_t w, int64_t scale) {
    if constexpr (M::kInteger) return (typename M::value_t)(int32_t)w * scale;
    else return __uint_as_float(w);
}

// Group maximum of (value, expert), ties to the lower expert, with selects
// only; every lane of the group ends with the result.
template <int OFF, class M>
__device__ __attribute__((always_inline)) inline void max_step(typename M::value_t &bv, int &be) {
    const typename M::value_t ov = grp_partner<OFF>(bv);
    const int oe = grp_partner<OFF>(be);
    const bool take = (ov > bv) | ((ov == bv) & (oe < be));
    bv = take ? ov : bv;
    be = take ? oe : be;
}
template <class M, int G>
__device__ __attribute__((always_inline)) inline void group_max(typename M::value_t &bv, int &be) {
    if constexpr (G > 1) max_step<1, M>(bv, be);
    if constexpr (G > 2) max_step<2, M>(bv, be);
    if constexpr (G > 4) max_step<4, M>(bv, be);
    if constexpr (G > 8) max_step<8, M>(bv, be);
    if constexpr (G > 16) max_step<16, M>(bv, be);
    if constexpr (G > 32) max_step<32, M>(bv, be);
}

// A fresh control block and the starting prices of problem b: 0, or the
// caller's (warm start: prices only rise from any starting point, which
// keeps every bid's complementary slackness argument intact). Called by one
// block; prices may be NULL (control block only).
__device__ inline void init_problem(SolveCtrl *ctrl, void *prices, int E, const AssignParams &p,
                                    int b) {
    if (threadIdx.x == 0) {
        SolveCtrl z{};
        z.smax_ord = 0u;
        z.smin_ord = 0xffffffffu;
        z.eps_final_eff = p.eps_final;
        z.scale = p.scale;
        z.integer = p.integer ? 1 : 0;
        *ctrl = z;
    }
    if (prices == nullptr) return;
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        if (p.warm_prices == nullptr) {
            reinterpret_cast<int64_t *>(prices)[e] = 0;
        } else if (p.integer) {
            reinterpret_cast<int64_t *>(prices)[e] =
                reinterpret_cast<const int64_t *>(p.warm_prices)[(int64_t)b * E + e];
        } else {
            reinterpret_cast<float *>(prices)[e] =
                reinterpret_cast<const float *>(p.warm_prices)[(int64_t)b * E + e];
        }
    }
}

// The first kernel of a solve, one group of G lanes per token:
//   - the token's score summary: 9 rounds of a group maximum (ties to the
//     lowest expert) over the lanes' 8 scores each;
//   - the score range and a non-finite flag over the same loaded scores, one
//     partial (max, min, bad) per block in rpart[3 * block] (start_kernel
//     combines them);
//   - assign[t] = -1 (the finalising kernels write every held token);
//   - in block 0, a fresh control block and the starting prices.
template <class M, int G>
__global__ __launch_bounds__(kThreads) void prologue_kernel(Ctx<M> c0, AssignParams p,
                                                            int32_t *assign, uint32_t *rpart) {
    const Ctx<M> c = c0.at(blockIdx.y);
    using value_t = typename M::value_t;
    if (blockIdx.x == 0) init_problem(c.ctrl, c.prices, c.E, p, blockIdx.y);
    assign += (int64_t)blockIdx.y * c.T;
    rpart = Ctx<M>::shift(rpart, (int64_t)blockIdx.y * c.ws_stride);
    uint32_t rmx = 0u, rmn = 0xffffffffu;
    int rbad = 0;
    const int lane = lane_id();
    const int gl = lane & (G - 1);
    const int per_block = kThreads / G;
    const int n_round = ((c.T + per_block * (int)gridDim.x - 1) / (per_block * (int)gridDim.x)) *
                        per_block * (int)gridDim.x;
    // Lane gl holds experts 8 gl .. 8 gl + 7 of each chunk of 8 G experts
    // (several chunks when E > 8 G, which happens only at G = 64).
    const int take = c.E < 8 ? c.E : 8;
    for (int t = blockIdx.x * per_block + threadIdx.x / G; t < n_round;
         t += per_block * gridDim.x) {
        const bool valid = t < c.T;
        value_t sv[kSumChunks][8];
#pragma unroll
        for (int ch = 0; ch < kSumChunks; ++ch) {
            const int e0 = ch * 8 * G + 8 * gl;
#pragma unroll
            for (int q = 0; q < 8; ++q) sv[ch][q] = M::lowest();
            if (valid && e0 < c.E) load8<M>(c.S, (int64_t)t * c.E, e0, c.E, c.scale, sv[ch]);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (e0 + q >= c.E) {
                    sv[ch][q] = M::lowest();
                } else if (valid) {
                    // range over order-preserving images; non-finite
                    // scores only raise the flag
                    bool fin = true;
                    uint32_t o;
                    if constexpr (M::kInteger) {
                        o = (uint32_t)(int32_t)(sv[ch][q] / c.scale) ^ 0x80000000u;
                    } else {
                        fin = isfinite(sv[ch][q]);
                        o = f32_ord(sv[ch][q]);
                    }
                    rbad |= !fin;
                    rmx = (fin && o > rmx) ? o : rmx;
                    rmn = (fin && o < rmn) ? o : rmn;
                }
            }
        }
        if (valid && gl == 0) assign[t] = -1;
        uint32_t *out = c.sums + (int64_t)(valid ? t : 0) * kSumWords;
        uint32_t pairs[4] = {0, 0, 0, 0};
        for (int r = 0; r <= take; ++r) {
            // Lane-local best, then the group's best (lowest expert on ties).
            value_t bv = M::lowest();
            int be = 0x7fffffff;
#pragma unroll
            for (int ch = 0; ch < kSumChunks; ++ch) {
                if (ch * 8 * G >= c.E) break;   // (uniform: chunks past the row)
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const int e = ch * 8 * G + 8 * gl + q;
                    const bool better = (e < c.E) & (sv[ch][q] > bv);
                    bv = better ? sv[ch][q] : bv;
                    be = better ? e : be;
                }
            }
            group_max<M, G>(bv, be);
            if (r < take) {
#pragma unroll
                for (int ch = 0; ch < kSumChunks; ++ch) {
                    if (ch * 8 * G >= c.E) break;
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        sv[ch][q] = ch * 8 * G + 8 * gl + q == be ? M::lowest() : sv[ch][q];
                }
                if (valid && gl == 0) out[r] = score_bits<M>(bv, c.scale);
                pairs[r >> 1] |= (uint32_t)(be & 0xffff) << (16 * (r & 1));
            } else if (valid && gl == 0) {
                // the 9th score bounds every expert outside the summary
                out[12] = (take < c.E) ? score_bits<M>(bv, c.scale)
                                       : (M::kInteger ? 0x80000000u : __float_as_uint(-INFINITY));
            }
        }
        if (valid && gl == 0) {
            for (int q = 0; q < 4; ++q) out[8 + q] = pairs[q];
            out[13] = (uint32_t)take;
        }
    }
    // The block's range partial.
    __shared__ uint32_t smx[kThreads / 64], smn[kThreads / 64];
    __shared__ int sbad[kThreads / 64];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t a = __shfl_xor(rmx, off), b = __shfl_xor(rmn, off);
        rmx = a > rmx ? a : rmx;
        rmn = b < rmn ? b : rmn;
        rbad |= __shfl_xor(rbad, off);
    }
    if (lane == 0) {
        smx[threadIdx.x >> 6] = rmx;
        smn[threadIdx.x >> 6] = rmn;
        sbad[threadIdx.x >> 6] = rbad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kThreads / 64; ++w) {
            rmx = smx[w] > rmx ? smx[w] : rmx;
            rmn = smn[w] < rmn ? smn[w] : rmn;
            rbad |= sbad[w];
        }
        rpart[3 * blockIdx.x] = rmx;
        rpart[3 * blockIdx.x + 1] = rmn;
        rpart[3 * blockIdx.x + 2] = (uint32_t)rbad;
    }
}

// Reads the summary table from `pf` blocks (a multiple of 8) spread over
// every XCD, so that the L2 of whichever XCD runs the one-workgroup engine
// holds it. Consecutive workgroups go to consecutive XCDs; block i of the
// pf covers chunk i / 8, so the blocks on any one XCD cover the whole table
// whatever XCD the first lands on.
__device__ inline void summary_prefill(const uint4 *sums, int64_t n16, int i, int pf,
                                       uint32_t *sink) {
    const int per_xcd = pf / 8;
    const int64_t chunk = (n16 + per_xcd - 1) / per_xcd;
    const int64_t lo = (int64_t)(i / 8) * chunk;
    const int64_t hi = lo + chunk < n16 ? lo + chunk : n16;
    uint32_t acc = 0;
    for (int64_t k = lo + threadIdx.x; k < hi; k += blockDim.x) {
        const uint4 v = sums[k];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u && threadIdx.x == 0) *sink = acc;   // keeps the loads
}

// Loads words of token t's summary into sw: lane gl of the group takes
// entry gl % 8 (score, expert half-word), the bound and the entry count.
__device__ inline void load_summary(const uint32_t *sums, int t, int gl, uint32_t (&sw)[4]) {
    const uint32_t *sm = sums + (int64_t)t * kSumWords;
    const int q = gl & 7;
    sw[0] = sm[q];
    sw[1] = sm[8 + (q >> 1)];
    const uint2 bc = *reinterpret_cast<const uint2 *>(sm + 12);
    sw[2] = bc.x;
    sw[3] = bc.y;
}

// Top-2 of token t from its summary words (called by the whole wave; groups
// with valid == false take part in the shuffles only). A token whose summary
// cannot decide (or any token when G < 8) reads its full row instead.
// pmin is a lower bound of every price.
//
// Exactness: every expert outside the summary has S[t,e] <= bound and
// p[e] >= pmin, so its value S[t,e] - p[e] <= bound - pmin (also after fp32
// rounding, which is monotone). A best value above that limit is therefore
// the best over all experts (with the same lowest-index tie rule, as no
// outside expert can tie it), and a second value reaching the limit is the
// second best over all experts.
template <class M, int G>
__device__ inline void top2_summary(const Ctx<M> &c, const uint32_t (&sw)[4], int t, bool valid,
                                    int gl, const typename M::value_t *pr,
                                    typename M::value_t pmin, typename M::value_t &v1, int &e1,
                                    typename M::value_t &v2, typename M::value_t &s1) {
    using value_t = typename M::value_t;
    const int cnt = (int)sw[3];
    v1 = M::lowest();
    v2 = M::lowest();
    s1 = 0;
    e1 = 0x7fffffff;
    if (valid && gl < 8 && gl < cnt) {
        const value_t sc = bits_score<M>(sw[0], c.scale);
        int ex = (int)((sw[1] >> (16 * (gl & 1))) & 0xffff);
        if (ex >= c.E) ex = 0;
        v1 = sc - pr[ex];
        e1 = ex;
        s1 = sc;
    }
    top2_reduce<M, G>(v1, e1, v2, s1);
    bool exact = cnt >= c.E;
    if (!exact) {
        const value_t lim = bits_score<M>(sw[2], c.scale) - pmin;
        exact = v1 > lim && v2 >= lim;
    }
    if (G < 8) exact = false;   // a group narrower than 8 lanes cannot hold the 8 entries
    const bool need = valid && !exact;
    if (__ballot(need)) {
        value_t w1, w2, ws1;
        int we1;
        top2_token<M, G>(c, t, need, pr, w1, we1, w2, ws1);
        if (need) {
            v1 = w1;
            v2 = w2;
            e1 = we1;
            s1 = ws1;
        }
    }
}

// Lowest of the E prices in LDS, for the whole block (every thread calls).
template <class M>
__device__ inline typename M::value_t block_min_price(const typename M::value_t *pr, int E) {
    using value_t = typename M::value_t;
    __shared__ value_t part[16];
    value_t m = pr[0];
    for (int e = threadIdx.x; e < E; e += blockDim.x) m = pr[e] < m ? pr[e] : m;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const value_t o = __shfl_xor(m, off);
        m = o < m ? o : m;
    }
    if (lane_id() == 0) part[threadIdx.x >> 6] = m;
    __syncthreads();
    m = part[0];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) m = part[w] < m ? part[w] : m;
    __syncthreads();
    return m;
}

// Bids of active tokens [i0, n) with stride `ngroups` groups, from the
// tokens' score summaries (rows only where a summary cannot decide; pmin is
// the lowest price). `touched` (LDS, may be null) collects experts receiving
// their first bid this round.
template <class M, int G>
__device__ void bid_range(const Ctx<M> &c, int n, bool all_active, const int *list,
                          typename M::value_t eps, const typename M::value_t *pr,
                          typename M::value_t pmin, int gid, int ngroups, int *touched,
                          int *ntouched) {
    using value_t = typename M::value_t;
    const int gl = lane_id() & (G - 1);
    const int n_round = ((n + ngroups - 1) / ngroups) * ngroups;
    for (int i = gid; i < n_round; i += ngroups) {
        int t = (i < n) ? (all_active ? i : list[i]) : 0;
        if (t < 0 || t >= c.T) {
            if (i < n && gl == 0) flag_internal(c.ctrl);
            t = 0;
        }
        const bool valid = i < n && t >= 0;
        value_t v1, v2, s1;
        int e1;
        uint32_t sw[4] = {0, 0, 0, 0};
        if (valid) load_summary(c.sums, t, gl, sw);
        top2_summary<M, G>(c, sw, t, valid, gl, pr, pmin, v1, e1, v2, s1);
        if (valid && gl == 0) {
            if (e1 >= c.E) {   // every value non-finite: any expert, the bid overflows
                e1 = 0;
                s1 = 0;   // with v2 = -inf the bid is +inf: overflow is flagged
            }
            const value_t bid = (c.E > 1) ? (value_t)((s1 - v2) + eps) : (value_t)(s1 + eps);
            int overflow = 0;
            const uint64_t key = M::make_key(bid, t, &overflow);
            if (overflow) c.ctrl->overflow = 1;
            const int pos = atomicAdd(&c.bcount[e1], 1);
            if (pos < c.cap) {
                c.bucket[(int64_t)e1 * c.cap + pos] = key;
            } else {
                const int q = atomicAdd(c.ovf_count, 1);
                if (q < c.T) {
                    c.ovf_key[q] = key;
                    c.ovf_exp[q] = e1;
                } else {
                    flag_internal(c.ctrl);
                }
            }
            if (touched != nullptr && pos == 0) {
                const int at = atomicAdd(ntouched, 1);
                if (at < c.E) touched[at] = e1;
                else flag_internal(c.ctrl);
            }
        }
    }
}

// Bids of the active tokens with list index in [i0, i1) (i1 - i0 <=
// kBidTile), by one block (every thread calls): each group of G lanes bids
// for tokens strided by the block's group count, four summaries in flight.
// The bids collect in LDS with a per-expert rank (an LDS atomic); then one
// global atomic per expert the block touched reserves the bucket slots, and
// the keys are written. (One global atomic per bid serialised on the few
// experts that most tokens prefer.)
//   lcnt  LDS [E], zero on entry and on return
//   lkey, lexp, lrank  LDS [kBidTile]
constexpr int kBidTile = 64;
constexpr int kBidRows = 4;

template <class M, int G>
__device__ void bid_block(const Ctx<M> &c, int i0, int i1, bool all_active, const int *list,
                          typename M::value_t eps, const typename M::value_t *pr,
                          typename M::value_t pmin, int *lcnt, uint64_t *lkey, int *lexp,
                          int *lrank) {
    using value_t = typename M::value_t;
    const int tid = threadIdx.x;
    const int gl = lane_id() & (G - 1);
    const int per_block = (int)blockDim.x / G;
    const int m = i1 - i0;
    const int stride = per_block * kBidRows;
    const int m_round = ((m + stride - 1) / stride) * stride;
    for (int j0 = tid / G; j0 < m_round; j0 += stride) {
        uint32_t sw[kBidRows][4];
        int toks[kBidRows];
#pragma unroll
        for (int u = 0; u < kBidRows; ++u) {
            const int j = j0 + u * per_block;
            int t = 0;
            if (j < m) {
                t = all_active ? i0 + j : list[i0 + j];
                if (t < 0 || t >= c.T) {
                    if (gl == 0) flag_internal(c.ctrl);
                    t = 0;
                }
            }
            toks[u] = t;
            sw[u][0] = sw[u][1] = sw[u][2] = sw[u][3] = 0;
            if (j < m) load_summary(c.sums, t, gl, sw[u]);
        }
#pragma unroll
        for (int u = 0; u < kBidRows; ++u) {
            const int j = j0 + u * per_block;
            const bool valid = j < m;
            if (__ballot(valid) == 0) break;
            const int t = toks[u];
            value_t v1, v2, s1;
            int e1;
            top2_summary<M, G>(c, sw[u], t, valid, gl, pr, pmin, v1, e1, v2, s1);
            if (valid && gl == 0) {
                if (e1 >= c.E) {   // every value non-finite: any expert, the bid overflows
                    e1 = 0;
                    s1 = 0;   // with v2 = -inf the bid is +inf: overflow is flagged
                }
                const value_t bid = (c.E > 1) ? (value_t)((s1 - v2) + eps) : (value_t)(s1 + eps);
                int overflow = 0;
                lkey[j] = M::make_key(bid, t, &overflow);
                if (overflow) c.ctrl->overflow = 1;
                lexp[j] = e1;
                lrank[j] = atomicAdd(&lcnt[e1], 1);
            }
        }
    }
    __syncthreads();
    for (int e = tid; e < c.E; e += blockDim.x) {
        const int k = lcnt[e];
        if (k > 0) lcnt[e] = atomicAdd(&c.bcount[e], k);   // now the base of the block's slots
    }
    __syncthreads();
    for (int j = tid; j < m; j += blockDim.x) {
        const int e = lexp[j];
        const int pos = lcnt[e] + lrank[j];
        if (pos < c.cap) {
            c.bucket[(int64_t)e * c.cap + pos] = lkey[j];
        } else {
            const int q = atomicAdd(c.ovf_count, 1);
            if (q < c.T) {
                c.ovf_key[q] = lkey[j];
                c.ovf_exp[q] = e;
            } else {
                flag_internal(c.ctrl);
            }
        }
    }
    __syncthreads();
    for (int e = tid; e < c.E; e += blockDim.x) lcnt[e] = 0;
    __syncthreads();
}

// Dynamic LDS of a kernel that bids with bid_block: prices, then lcnt [E],
// then lkey / lexp / lrank [kBidTile].
struct BidSmem {
    size_t lcnt, lkey, lexp, lrank, total;
};
__host__ __device__ inline BidSmem bid_smem(int E, int value_bytes) {
    BidSmem L{};
    size_t off = ((size_t)E * value_bytes + 15) & ~size_t(15);
    L.lcnt = off;  off = (off + (size_t)E * 4 + 15) & ~size_t(15);
    L.lkey = off;  off += (size_t)kBidTile * 8;
    L.lexp = off;  off += (size_t)kBidTile * 4;
    L.lrank = off; off += (size_t)kBidTile * 4;
    L.total = off;
    return L;
}

// ----------------------------------------------------------------- update --

struct UpdateSmem {
    uint64_t cand[kCandLds];
    uint32_t hist[256];
    uint64_t minkey, kmin, kmax;
    int sel_digit, sel_count, need, kept, pos;
};

// Calls fn(key) for every candidate of expert e (holders, bucket, overflow)
// with a wave-uniform trip count: fn(key, valid) is called by all lanes.
template <class M, class F>
__device__ inline void for_each_candidate(const Ctx<M> &c, int e, const uint64_t *hold, int h,
                                          int nb, int novf, F fn) {
    for (int b = 0; b < h; b += blockDim.x) {
        const int i = b + threadIdx.x;
        const bool v = i < h;
        fn(v ? hold[i] : 0ull, v);
    }
    const uint64_t *bk = c.bucket + (int64_t)e * c.cap;
    for (int b = 0; b < nb; b += blockDim.x) {
        const int i = b + threadIdx.x;
        const bool v = i < nb;
        fn(v ? bk[i] : 0ull, v);
    }
    for (int b = 0; b < novf; b += blockDim.x) {
        const int i = b + threadIdx.x;
        const bool v = i < novf && c.ovf_exp[i] == e;
        fn(v ? c.ovf_key[i] : 0ull, v);
    }
}

// Suffix scan of sm.hist by wave 0: finds the digit holding the need-th
// largest candidate; stores it in sm.sel_digit and the remaining rank in sm.need.
__device__ inline void pick_digit(UpdateSmem &sm, int need) {
    if (threadIdx.x < 64) {
        const int l = threadIdx.x;
        // Lane l owns digits 255-4l .. 252-4l (descending).
        uint32_t h[4];
        uint32_t s = 0;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            h[j] = sm.hist[255 - 4 * l - j];
            s += h[j];
        }
        // Exclusive prefix (over lanes below l) of the per-lane sums.
        uint32_t incl = s;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t o = __shfl_up(incl, off);
            if (l >= off) incl += o;
        }
        uint32_t before = incl - s;
        if ((int)before < need && (int)incl >= need) {
            uint32_t cum = before;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if ((int)(cum + h[j]) >= need) {
                    sm.sel_digit = 255 - 4 * l - j;
                    sm.sel_count = (int)h[j];
                    sm.need = need - (int)cum;
                    break;
                }
                cum += h[j];
            }
        }
    }
}

// Merges the new bids of expert e into its holder table. Executed by a whole
// block; `next` is the active list that receives evicted tokens.
template <class M>
__device__ void update_expert(const Ctx<M> &c, int e, int next, int novf, UpdateSmem &sm) {
    if (e < 0 || e >= c.E) {
        if (threadIdx.x == 0) flag_internal(c.ctrl);
        return;
    }
    int n = ld_relaxed(&c.bcount[e]);
    if (n == 0) return;
    int h = ld_relaxed(&c.hcount[e]);
    int sel = ld_relaxed(&c.hsel[e]);
    if (n < 0 || n > c.T || h < 0 || h > c.C || (sel & ~1)) {
        if (threadIdx.x == 0) flag_internal(c.ctrl);
        n = n < 0 ? 0 : (n > c.T ? c.T : n);
        h = h < 0 ? 0 : (h > c.C ? c.C : h);
        sel &= 1;
        if (n == 0) return;
    }
    uint64_t *hold = c.holders + (int64_t)sel * c.T + (int64_t)e * c.C;
    const int nb = n < c.cap ? n : c.cap;
    const int novf_e = (n > c.cap) ? novf : 0;
    const int total = h + n;
    const int tid = threadIdx.x;

    if (total <= c.C) {
        // Room for every bid: append them after the current holders.
        if (tid == 0) {
            sm.pos = h;
            sm.minkey = ~0ull;
        }
        __syncthreads();
        const uint64_t *bk = c.bucket + (int64_t)e * c.cap;
        for (int i = tid; i < nb; i += blockDim.x) hold[h + i] = bk[i];
        if (tid == 0) sm.pos = h + nb;
        __syncthreads();
        if (novf_e) {
            for (int i = tid; i < novf_e; i += blockDim.x)
                if (c.ovf_exp[i] == e) {
                    const int at = atomicAdd(&sm.pos, 1);
                    if (at < c.C) hold[at] = c.ovf_key[i];
                }
        }
        __syncthreads();
        if (total == c.C) {
            // Full now: the price becomes the lowest held bid.
            uint64_t m = ~0ull;
            for (int i = tid; i < c.C; i += blockDim.x) {
                const uint64_t k = hold[i];
                m = k < m ? k : m;
            }
            atomicMin(reinterpret_cast<unsigned long long *>(&sm.minkey), (unsigned long long)m);
            __syncthreads();
            if (tid == 0) c.prices[e] = M::key_bid(sm.minkey);
        }
        if (tid == 0) {
            c.hcount[e] = total;
            c.bcount[e] = 0;
        }
        __syncthreads();
        return;
    }

    // More candidates than slots: find the C-th largest key by MSD radix
    // select (8 bits per pass), keep keys >= it, evict the rest. The passes
    // start below the leading bytes every candidate shares (from their
    // smallest and largest key) and stop once the chosen digit's keys are
    // exactly the ones still needed: the C-th largest is then their minimum.
    const bool staged = total <= kCandLds;
    if (tid == 0) {
        sm.pos = 0;
        sm.kmin = ~0ull;
        sm.kmax = 0;
    }
    __syncthreads();
    // Smallest and largest candidate: per thread, then per wave, then one
    // LDS atomic per wave (one per candidate would serialise on two words).
    uint64_t tmin = ~0ull, tmax = 0;
    auto range = [&](uint64_t k, bool v) {
        if (v) {
            tmin = k < tmin ? k : tmin;
            tmax = k > tmax ? k : tmax;
        }
    };
    auto range_done = [&]() {
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const uint64_t a = __shfl_xor(tmin, off), b = __shfl_xor(tmax, off);
            tmin = a < tmin ? a : tmin;
            tmax = b > tmax ? b : tmax;
        }
        if (lane_id() == 0) {
            atomicMin(reinterpret_cast<unsigned long long *>(&sm.kmin), (unsigned long long)tmin);
            atomicMax(reinterpret_cast<unsigned long long *>(&sm.kmax), (unsigned long long)tmax);
        }
    };
    if (staged) {
        for_each_candidate<M>(c, e, hold, h, nb, novf_e, [&](uint64_t k, bool v) {
            range(k, v);
            const uint64_t m = __ballot(v);
            if (m == 0) return;
            const int leader = __ffsll((long long)m) - 1;
            int base = 0;
            if (lane_id() == leader) base = atomicAdd(&sm.pos, __popcll(m));
            base = __shfl(base, leader);
            const int at = base + __popcll(m & lanemask_lt());
            if (v && at < kCandLds) sm.cand[at] = k;
        });
    } else {
        for_each_candidate<M>(c, e, hold, h, nb, novf_e, range);
    }
    range_done();
    __syncthreads();
    const uint64_t kdiff = sm.kmin ^ sm.kmax;   // non-zero: more than C distinct keys
    const int first = kdiff ? ((63 - __clzll((long long)kdiff)) / 8) * 8 : 0;
    uint64_t pmask = first >= 56 ? 0ull : ~0ull << (first + 8);
    uint64_t prefix = sm.kmin & pmask;
    int need = c.C;
    bool at_min = false;
    for (int shift = first; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += blockDim.x) sm.hist[i] = 0;
        __syncthreads();
        auto count = [&](uint64_t k, bool v) {
            if (v && (k & pmask) == prefix) atomicAdd(&sm.hist[(k >> shift) & 255], 1u);
        };
        if (staged) {
            for (int i = tid; i < total; i += blockDim.x) count(sm.cand[i], true);
        } else {
            for_each_candidate<M>(c, e, hold, h, nb, novf_e, count);
        }
        __syncthreads();
        pick_digit(sm, need);
        __syncthreads();
        prefix |= (uint64_t)sm.sel_digit << shift;
        pmask |= 255ull << shift;
        need = sm.need;
        const bool whole = sm.sel_count == need;
        __syncthreads();
        if (whole && shift > 0) {
            at_min = true;
            break;
        }
    }
    if (at_min) {
        if (tid == 0) sm.kmin = ~0ull;
        __syncthreads();
        tmin = ~0ull;
        tmax = 0;
        auto low = [&](uint64_t k, bool v) { range(k, v && (k & pmask) == prefix); };
        if (staged) {
            for (int i = tid; i < total; i += blockDim.x) low(sm.cand[i], true);
        } else {
            for_each_candidate<M>(c, e, hold, h, nb, novf_e, low);
        }
        range_done();
        __syncthreads();
    }
    const uint64_t kstar = at_min ? sm.kmin : prefix;   // keys are unique: a key

    uint64_t *alt = c.holders + (int64_t)(sel ^ 1) * c.T + (int64_t)e * c.C;
    if (tid == 0) sm.kept = 0;
    __syncthreads();
    auto split = [&](uint64_t k, bool v) {
        const bool keep = v && k >= kstar;
        const uint64_t m = __ballot(keep);
        if (m) {
            const int leader = __ffsll((long long)m) - 1;
            int base = 0;
            if (lane_id() == leader) base = atomicAdd(&sm.kept, __popcll(m));
            base = __shfl(base, leader);
            const int at = base + __popcll(m & lanemask_lt());
            if (keep && at < c.C) alt[at] = k;
        }
        append_active<M>(c, next, v && k < kstar, key_token(k));
    };
    if (staged) {
        const int trips = ((total + blockDim.x - 1) / blockDim.x) * blockDim.x;
        for (int i = tid; i < trips; i += blockDim.x) {
            const bool v = i < total;
            split(v ? sm.cand[i] : 0ull, v);
        }
    } else {
        for_each_candidate<M>(c, e, hold, h, nb, novf_e, split);
    }
    __syncthreads();
    if (tid == 0) {
        c.hsel[e] = sel ^ 1;
        c.hcount[e] = c.C;
        c.prices[e] = M::key_bid(kstar);
        c.bcount[e] = 0;
    }
    __syncthreads();
}

// ------------------------------------------------------- round bookkeeping --

// Called by one thread once a round's updates are complete and visible.
//
// A phase above the last whose epsilon exceeds kEarlyRatio eps_final ends
// as soon as at most early_n tokens are left active: its assignment is only ever used by
// the duality check, whose gap at such an epsilon could neither certify the
// solve nor guide the next step (the measured gap stays far above both
// T eps_final and the guided step's reach), so placing its last tokens
// would be wasted rounds. Its prices start the next phase, as any prices
// may: the auction's guarantee for a phase holds from every starting price.
constexpr double kEarlyRatio = 4096.0;
template <class M>
__device__ inline void end_round(const Ctx<M> &c) {
    SolveCtrl *ctrl = c.ctrl;
    const int old = ctrl->cur;
    const int nw = old ^ 1;
    const int n = ctrl->all_active ? c.T : ld_relaxed(&ctrl->active_count[old]);
    if (n == 0) return;
    ctrl->bids += (unsigned long long)n;
    ctrl->rounds += 1;
    ctrl->active_count[old] = 0;
    ctrl->cur = nw;
    ctrl->all_active = 0;
    ctrl->pad0 = 0;   // overflow list count
    const int left = ld_relaxed(&ctrl->active_count[nw]);
    if (left == 0) {
        if (ctrl->last_phase) ctrl->done = 1;
    } else if (c.early_n != 0 && !ctrl->last_phase &&
               left <= (c.early_n > 0 ? c.early_n : -c.early_n) &&
               (c.early_n < 0 || ctrl->early_ok)) {
        ctrl->active_count[nw] = 0;
        ctrl->skip_check = 1;
    }
}

// Starts the next epsilon phase (one thread). Returns false if the solve is done.
__device__ inline void begin_phase_scalar(SolveCtrl *ctrl, const AssignParams &p, int T) {
    double eps;
    if (ctrl->phase == 0) {
        eps = p.eps_initial;
        if (!(eps > 0.0)) {
            double range;
            if (p.integer)
                range = ((double)(int32_t)(ctrl->smax_ord ^ 0x80000000u) -
                         (double)(int32_t)(ctrl->smin_ord ^ 0x80000000u)) *
                        (double)p.scale;
            else
                range = (double)f32_unord(ctrl->smax_ord) - (double)f32_unord(ctrl->smin_ord);
            eps = range / 8.0;
        }
    } else {
        eps = ctrl->eps / p.eps_factor;
        // A gap measured after the previous phase that misses T eps_final by
        // less than the divisor asks for a smaller step: epsilon shrinks just
        // enough for the gap, taken as proportional to epsilon, to fall to
        // half the bound.
        const double gap = ctrl->check_gap;
        if (gap > 0.0) {
            const double guided = ctrl->eps * 0.5 * (double)T * ctrl->eps_final_eff / gap;
            if (guided > eps) eps = guided;
        }
    }
    ctrl->check_gap = 0.0;
    if (p.integer) eps = floor(eps);
    if (!(eps > ctrl->eps_final_eff)) eps = ctrl->eps_final_eff;
    ctrl->eps = eps;
    ctrl->last_phase = eps <= ctrl->eps_final_eff ? 1 : 0;
    ctrl->phase += 1;
    ctrl->all_active = 1;
    ctrl->active_count[ctrl->cur] = 0;
    ctrl->active_count[ctrl->cur ^ 1] = 0;
    ctrl->pad0 = 0;
}

// The early-end state of a phase just begun by begin_phase_scalar (kept out
// of it: the single-workgroup solver, which inlines it, never ends a phase
// early).
__device__ inline void begin_phase_early(SolveCtrl *ctrl) {
    ctrl->skip_check = 0;
    ctrl->early_ok = ctrl->eps > kEarlyRatio * ctrl->eps_final_eff ? 1 : 0;
}

// ---------------------------------------------------------------- kernels --

__global__ void init_kernel(SolveCtrl *ctrl, void *prices, int E, AssignParams p,
                            int64_t ws_stride) {
    ctrl = Ctx<FloatMode>::shift(ctrl, (int64_t)blockIdx.y * ws_stride);
    if (prices != nullptr) prices = Ctx<FloatMode>::shift(prices, (int64_t)blockIdx.y * ws_stride);
    init_problem(ctrl, prices, E, p, blockIdx.y);
}

// Score range (order-preserving images) and a non-finite flag: each block
// reduces its share of S (16-byte loads) and writes one partial (max, min,
// bad) to part[3 * block]; range_finish_kernel combines them. (One atomic
// per wave on a single address took 99 us at T x E = 4M.)

template <class M>
__device__ inline void range_take(typename M::score_t x, uint32_t &mx, uint32_t &mn, int &bad) {
    uint32_t o;
    if constexpr (M::kInteger) {
        o = (uint32_t)((int32_t)x) ^ 0x80000000u;
    } else {
        if (!isfinite(x)) {
            bad = 1;
            return;
        }
        o = f32_ord(x);
    }
    mx = o > mx ? o : mx;
    mn = o < mn ? o : mn;
}

template <class M>
__global__ __launch_bounds__(256) void range_kernel(const typename M::score_t *S, int64_t n,
                                                    uint32_t *part, int64_t ws_stride) {
    S += (int64_t)blockIdx.y * n;
    part = Ctx<FloatMode>::shift(part, (int64_t)blockIdx.y * ws_stride);
    using score_t = typename M::score_t;
    constexpr int kVec = 16 / sizeof(score_t);
    __shared__ uint32_t smx[4], smn[4];
    __shared__ int sbad[4];
    uint32_t mx = 0u, mn = 0xffffffffu;
    int bad = 0;
    const int64_t nvec = n / kVec;   // S is 16-byte aligned
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nvec; i += stride) {
        const uint4 v = reinterpret_cast<const uint4 *>(S)[i];
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int j = 0; j < kVec; ++j) {
            score_t x;
            if constexpr (sizeof(score_t) == 4) x = __uint_as_float(w[j]);
            else x = (score_t)(int16_t)(uint16_t)(w[j >> 1] >> (16 * (j & 1)));
            range_take<M>(x, mx, mn, bad);
        }
    }
    for (int64_t i = nvec * kVec + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        range_take<M>(S[i], mx, mn, bad);
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t a = __shfl_xor(mx, off), b = __shfl_xor(mn, off);
        mx = a > mx ? a : mx;
        mn = b < mn ? b : mn;
        bad |= __shfl_xor(bad, off);
    }
    const int wave = threadIdx.x >> 6;
    if (lane_id() == 0) {
        smx[wave] = mx;
        smn[wave] = mn;
        sbad[wave] = bad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < (int)(blockDim.x >> 6); ++w) {
            mx = smx[w] > mx ? smx[w] : mx;
            mn = smn[w] < mn ? smn[w] : mn;
            bad |= sbad[w];
        }
        part[3 * blockIdx.x] = mx;
        part[3 * blockIdx.x + 1] = mn;
        part[3 * blockIdx.x + 2] = (uint32_t)bad;
    }
}

// Combines the range partials into the control block (one block).
__global__ __launch_bounds__(256) void range_finish_kernel(SolveCtrl *ctrl, const uint32_t *part,
                                                           int nparts, int64_t ws_stride) {
    ctrl = Ctx<FloatMode>::shift(ctrl, (int64_t)blockIdx.y * ws_stride);
    part = Ctx<FloatMode>::shift(part, (int64_t)blockIdx.y * ws_stride);
    __shared__ uint32_t smx[4], smn[4], sbad[4];
    uint32_t mx = 0u, mn = 0xffffffffu, bad = 0u;
    for (int i = threadIdx.x; i < nparts; i += blockDim.x) {
        mx = part[3 * i] > mx ? part[3 * i] : mx;
        mn = part[3 * i + 1] < mn ? part[3 * i + 1] : mn;
        bad |= part[3 * i + 2];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t a = __shfl_xor(mx, off), b = __shfl_xor(mn, off);
        mx = a > mx ? a : mx;
        mn = b < mn ? b : mn;
        bad |= __shfl_xor(bad, off);
    }
    const int wave = threadIdx.x >> 6;
    if (lane_id() == 0) {
        smx[wave] = mx;
        smn[wave] = mn;
        sbad[wave] = bad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < (int)(blockDim.x >> 6); ++w) {
            mx = smx[w] > mx ? smx[w] : mx;
            mn = smn[w] < mn ? smn[w] : mn;
            bad |= sbad[w];
        }
        ctrl->smax_ord = mx > ctrl->smax_ord ? mx : ctrl->smax_ord;
        ctrl->smin_ord = mn < ctrl->smin_ord ? mn : ctrl->smin_ord;
        if (bad) ctrl->unconverged_experts |= 1 << 30;
    }
}

// ------------------------------------------------------------ phase check --
//
// The duality certificate after a phase that is not the last. With every
// expert holding C tokens, D(p) - objective equals
//     sum over held tokens t of [max_e (S[t,e] - p[e]) - (S[t,a_t] - p[a_t])],
// a sum of nonnegative per-token slacks (no cancellation between two large
// sums). By weak duality it bounds optimum - objective. When it is at most
// T eps_final, less an allowance for the rounding of the per-token maxima
// in the solve's arithmetic, the assignment already meets the bound the
// last phase would guarantee, and the solve stops here. Groups of G lanes
// take holder slots in expert order and read each token's maximum from its
// score summary (its row when the summary cannot decide); each block writes
// one partial sum, and the next slot's phase_begin_kernel decides.
template <class M, int G>
__global__ __launch_bounds__(kThreads) void phase_check_kernel(Ctx<M> c0) {
    using value_t = typename M::value_t;
    const Ctx<M> c = c0.at(blockIdx.y);
    SolveCtrl *ctrl = c.ctrl;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    value_t *pr = reinterpret_cast<value_t *>(smem_raw);
    __shared__ double part[kThreads / 64];
    __shared__ int go;
    if (threadIdx.x == 0) {
        go = !ctrl->done && !ctrl->last_phase && ctrl->phase > 0 && !ctrl->all_active &&
             !ctrl->skip_check && ld_relaxed(&ctrl->active_count[ctrl->cur]) == 0;
    }
    __syncthreads();
    if (!go) return;
    // The holder-table selectors, as the previous kernels left them.
    int *sel = reinterpret_cast<int *>(smem_raw + (((size_t)c.E * sizeof(value_t) + 15) & ~size_t(15)));
    for (int e = threadIdx.x; e < c.E; e += kThreads) {
        pr[e] = c.prices[e];
        sel[e] = c.hsel[e] & 1;
    }
    __syncthreads();
    const value_t pmin = block_min_price<M>(pr, c.E);
    const int gl = lane_id() & (G - 1);
    const int per_block = kThreads / G;
    const int ngroups = per_block * gridDim.x;
    const int n_round = ((c.T + ngroups - 1) / ngroups) * ngroups;
    double acc = 0.0;
    for (int i = blockIdx.x * per_block + threadIdx.x / G; i < n_round; i += ngroups) {
        bool valid = i < c.T;
        const int e = valid ? i / c.C : 0;
        int t = 0;
        if (valid) {
            const uint64_t *hold = c.holders + (int64_t)sel[e] * c.T + (int64_t)e * c.C;
            t = key_token(hold[i - e * c.C]);
            if (t < 0 || t >= c.T) {
                if (gl == 0) flag_internal(ctrl);
                valid = false;
                t = 0;
            }
        }
        uint32_t sw[4] = {0, 0, 0, 0};
        if (valid) load_summary(c.sums, t, gl, sw);
        value_t v1, v2, s1;
        int e1;
        top2_summary<M, G>(c, sw, t, valid, gl, pr, pmin, v1, e1, v2, s1);
        if (valid && gl == 0)
            acc += (double)v1 -
                   ((double)M::load(c.S, (int64_t)t * c.E + e, c.scale) - (double)pr[e]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane_id() == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double sum = 0.0;
        for (int w = 0; w < kThreads / 64; ++w) sum += part[w];
        c.gpart[blockIdx.x] = sum;
    }
}

// The decision on the gap phase_check_kernel measured, by one block: the
// partials added in a fixed order (thread i takes blocks i, i + blockDim,
// ...; then the waves' shuffle trees and the waves in order), so it does not
// depend on scheduling. (A last-block counter in the check kernel instead
// cost about 70 us: a thousand device-scope atomics on one address.)
template <class M>
__device__ void phase_check_decide(const Ctx<M> &c, int nparts) {
    SolveCtrl *ctrl = c.ctrl;
    __shared__ double part[16], pbig[16];
    double g = 0.0, pm = 0.0;
    for (int b = threadIdx.x; b < nparts; b += blockDim.x) g += c.gpart[b];
    for (int e = threadIdx.x; e < c.E; e += blockDim.x) pm = fmax(pm, fabs((double)c.prices[e]));
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        g += __shfl_xor(g, off);
        pm = fmax(pm, __shfl_xor(pm, off));
    }
    if (lane_id() == 0) {
        part[threadIdx.x >> 6] = g;
        pbig[threadIdx.x >> 6] = pm;
    }
    __syncthreads();
    if (threadIdx.x != 0) return;
    double gap = 0.0, pmax = 0.0;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
        gap += part[w];
        pmax = fmax(pmax, pbig[w]);
    }
    double allowance = 0.0;
    if (!M::kInteger) {
        // Each maximum is one fp32 subtraction of values below max|S| + max|p|:
        // at most half an ulp, 2^-24 of that magnitude; four times that per token.
        const double smax = fmax(fabs((double)f32_unord(ctrl->smax_ord)),
                                 fabs((double)f32_unord(ctrl->smin_ord)));
        allowance = (double)c.T * ldexp(smax + pmax, -22);
    }
    if (gap + allowance <= (double)c.T * ctrl->eps_final_eff) {
        ctrl->certified = 1;
        ctrl->done = 1;
    } else {
        ctrl->check_gap = gap + allowance;
    }
}

// Blocks of phase_check_kernel for T tokens (the partials the next slot's
// phase_begin_kernel adds).
inline int phase_check_blocks(int T, int G) {
    const int per_block = kThreads / G;
    const int blocks = (T + 2 * per_block - 1) / (2 * per_block);
    return blocks < kCheckBlocks ? blocks : kCheckBlocks;
}

template <class M, int G>
hipError_t launch_phase_check(const Ctx<M> &c, int B, hipStream_t s) {
    const size_t pr_bytes = (((size_t)c.E * sizeof(typename M::value_t) + 15) & ~size_t(15)) +
                            (size_t)c.E * sizeof(int);
    const int blocks = phase_check_blocks(c.T, G);
    hipLaunchKernelGGL((phase_check_kernel<M, G>), dim3(blocks, B), dim3(kThreads), pr_bytes, s,
                       c);
    return hipGetLastError();
}

// Starts a phase slot (one block per problem): first the decision on the
// duality gap the previous slot measured (nparts partials; 0 when no check
// ran), then the next epsilon phase, unless the solve is done or the
// current phase still has active tokens (its rounds then go on in this slot).
template <class M>
__global__ void phase_begin_kernel(Ctx<M> c0, AssignParams p, int nparts) {
    const Ctx<M> c = c0.at(blockIdx.y);
    SolveCtrl *ctrl = c.ctrl;
    __shared__ int check, begin;
    if (threadIdx.x == 0) {
        const bool finished = ctrl->phase > 0 && !ctrl->all_active &&
                              ld_relaxed(&ctrl->active_count[ctrl->cur]) == 0;
        check = nparts > 0 && !ctrl->done && !ctrl->last_phase && finished && !ctrl->skip_check;
        c.bar[0] = 0;    // the round loop's barrier counts from zero in every launch
        c.bar[32] = 0;
    }
    __syncthreads();
    if (check) phase_check_decide<M>(c, nparts);
    __syncthreads();
    if (threadIdx.x == 0) {
        begin = 0;
        if (!ctrl->done) {
            const bool in_progress =
                ctrl->phase > 0 &&
                (ctrl->all_active || ld_relaxed(&ctrl->active_count[ctrl->cur]) > 0);
            if (!in_progress) {
                begin_phase_scalar(ctrl, p, c.T);
                begin_phase_early(ctrl);
                begin = 1;
            }
        }
    }
    __syncthreads();
    if (!begin) return;
    for (int e = threadIdx.x; e < c.E; e += blockDim.x) {
        c.hcount[e] = 0;
        c.hsel[e] = 0;
        c.bcount[e] = 0;
    }
}

// The second kernel of a solve (one block per problem): the score range from
// the prologue's nparts partials (and the non-finite flag), the floor of
// eps_final in float mode, and the first epsilon phase.
template <class M>
__global__ __launch_bounds__(256) void start_kernel(Ctx<M> c0, AssignParams p, const uint32_t *rpart,
                                                    int nparts) {
    const Ctx<M> c = c0.at(blockIdx.y);
    SolveCtrl *ctrl = c.ctrl;
    rpart = Ctx<M>::shift(rpart, (int64_t)blockIdx.y * c.ws_stride);
    __shared__ uint32_t smx[4], smn[4], sbad[4];
    uint32_t mx = 0u, mn = 0xffffffffu, bad = 0u;
    for (int i = threadIdx.x; i < nparts; i += blockDim.x) {
        mx = rpart[3 * i] > mx ? rpart[3 * i] : mx;
        mn = rpart[3 * i + 1] < mn ? rpart[3 * i + 1] : mn;
        bad |= rpart[3 * i + 2];
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t a = __shfl_xor(mx, off), b = __shfl_xor(mn, off);
        mx = a > mx ? a : mx;
        mn = b < mn ? b : mn;
        bad |= __shfl_xor(bad, off);
    }
    const int wave = threadIdx.x >> 6;
    if (lane_id() == 0) {
        smx[wave] = mx;
        smn[wave] = mn;
        sbad[wave] = bad;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < (int)(blockDim.x >> 6); ++w) {
            mx = smx[w] > mx ? smx[w] : mx;
            mn = smn[w] < mn ? smn[w] : mn;
            bad |= sbad[w];
        }
        ctrl->smax_ord = mx;
        ctrl->smin_ord = mn;
        if (bad) ctrl->unconverged_experts |= 1 << 30;
        if (M::kInteger) {
            ctrl->eps_final_eff = 1.0;
        } else {
            // Raise eps_final so that it stays far above fp32 rounding at the
            // magnitude prices and bids reach (scores plus a few score ranges).
            const double smax = (double)f32_unord(mx);
            const double smin = (double)f32_unord(mn);
            const double mag = fmax(fabs(smax), fabs(smin)) + 3.0 * (smax - smin) + 1e-30;
            const double floor_eps = ldexp(mag, -20);
            if (ctrl->eps_final_eff < floor_eps) ctrl->eps_final_eff = floor_eps;
        }
        c.bar[0] = 0;    // the round loop's barrier counts from zero in every launch
        c.bar[32] = 0;
        begin_phase_scalar(ctrl, p, c.T);
        begin_phase_early(ctrl);
    }
    for (int e = threadIdx.x; e < c.E; e += blockDim.x) {
        c.hcount[e] = 0;
        c.hsel[e] = 0;
        c.bcount[e] = 0;
    }
}

template <class M, int G>
__global__ __launch_bounds__(kThreads) void bid_wide_kernel(Ctx<M> c0) {
    const Ctx<M> c = c0.at(blockIdx.y);
    using value_t = typename M::value_t;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    value_t *pr = reinterpret_cast<value_t *>(smem_raw);
    SolveCtrl *ctrl = c.ctrl;
    if (ctrl->done) return;
    const int cur = ctrl->cur;
    const bool all = ctrl->all_active != 0;
    const int n = all ? c.T : ld_relaxed(&ctrl->active_count[cur]);
    if (n == 0) return;
    if (!all && n <= c.engine_cap) return;   // left to the tail engine
    const int i0 = blockIdx.x * kBidTile;
    if (i0 >= n) return;
    const BidSmem B = bid_smem(c.E, (int)sizeof(value_t));
    int *lcnt = reinterpret_cast<int *>(smem_raw + B.lcnt);
    for (int e = threadIdx.x; e < c.E; e += blockDim.x) {
        pr[e] = c.prices[e];
        lcnt[e] = 0;
    }
    __syncthreads();
    const value_t eps = (value_t)ctrl->eps;
    const value_t pmin = block_min_price<M>(pr, c.E);
    bid_block<M, G>(c, i0, i0 + kBidTile < n ? i0 + kBidTile : n, all,
                    c.active + (int64_t)cur * c.T, eps, pr, pmin, lcnt,
                    reinterpret_cast<uint64_t *>(smem_raw + B.lkey),
                    reinterpret_cast<int *>(smem_raw + B.lexp),
                    reinterpret_cast<int *>(smem_raw + B.lrank));
}

template <class M>
__global__ __launch_bounds__(kThreads) void update_wide_kernel(Ctx<M> c0) {
    const Ctx<M> c = c0.at(blockIdx.y);
    __shared__ UpdateSmem sm;
    __shared__ int last;
    SolveCtrl *ctrl = c.ctrl;
    if (ctrl->done) return;
    const int cur = ctrl->cur;
    {
        const bool all = ctrl->all_active != 0;
        const int n = all ? c.T : ld_relaxed(&ctrl->active_count[cur]);
        if (!all && n <= c.engine_cap) return;   // the bid kernel skipped this round too
    }
    const int novf = min(ld_relaxed(c.ovf_count), c.T);
    for (int e = blockIdx.x; e < c.E; e += gridDim.x) update_expert<M>(c, e, cur ^ 1, novf, sm);
    // The last block to finish closes the round.
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) last = atomicAdd(&ctrl->blocks_done, 1) == (int)gridDim.x - 1;
    __syncthreads();
    if (last && threadIdx.x == 0) {
        __threadfence();
        ctrl->blocks_done = 0;
        end_round<M>(c);
    }
}

// ------------------------------------------------------ wide round loop --
//
// Rounds that still have more active tokens than the engine takes after
// the fixed wide launches: one block per compute unit runs them back to
// back with a grid barrier between the bids and the updates and after the
// updates (the last block to finish closes the round). The launch follows
// the stream's previous kernels, so on the idle device every block is
// resident at once (each compute unit holds at least one; the host checks
// the occupancy). A cooperative launch would guarantee that too, but costs
// 20-40 us per launch here against about 2.5 us for a plain one, and this
// kernel is launched once per phase slot. The barrier's wait is bounded,
// so a block that never got scheduled ends the loop with an internal
// error, not a hang. All blocks read the same control words after a barrier and take
// the same exit. The launch returns at once when there is nothing to do.

// Barrier k of a launch completes when bar[0] reaches k * gridDim.x. Every
// thread waits for its own stores first; one thread per block then writes
// back its L2 (device-scope release), arrives, waits for the release word
// (on its own line, stored by the last arrival) and invalidates its caches
// (acquire). The wait gives up after `poll_limit` polls (2^24 by default,
// about a second): the block flags an internal error and returns false.
__device__ inline bool grid_barrier(uint64_t *bar, uint64_t target, SolveCtrl *ctrl,
                                    uint32_t poll_limit) {
    __shared__ int ok;
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this thread's stores are done
    __syncthreads();
    if (threadIdx.x == 0) {
        ok = 1;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const uint64_t arrived =
            __hip_atomic_fetch_add(bar, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1;
        if (arrived == target) {
            __hip_atomic_store(bar + 32, target, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            uint32_t polls = 0;
            while (__hip_atomic_load(bar + 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
                if (polls >= poll_limit) {
                    flag_internal(ctrl);
                    ok = 0;
                    break;
                }
                ++polls;
                __builtin_amdgcn_s_sleep(2);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    return ok != 0;
}

// As grid_barrier, and the block that arrives last runs on_last() (thread 0,
// after an acquire: every block's writes before its arrival are visible)
// before it releases the others, which then see its writes. This folds a
// round's closing step into the barrier that ends the round instead of a
// separate last-block counter (one fewer chain of device atomics on one
// address per round).
template <class F>
__device__ inline bool grid_barrier_last(uint64_t *bar, uint64_t target, SolveCtrl *ctrl,
                                         uint32_t poll_limit, F on_last) {
    __shared__ int ok;
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this thread's stores are done
    __syncthreads();
    if (threadIdx.x == 0) {
        ok = 1;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        const uint64_t arrived =
            __hip_atomic_fetch_add(bar, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1;
        if (arrived == target) {
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            on_last();
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
            __hip_atomic_store(bar + 32, target, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
            uint32_t polls = 0;
            while (__hip_atomic_load(bar + 32, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
                if (polls >= poll_limit) {
                    flag_internal(ctrl);
                    ok = 0;
                    break;
                }
                ++polls;
                __builtin_amdgcn_s_sleep(2);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    }
    __syncthreads();
    return ok != 0;
}

template <class M, int G>
__global__ __launch_bounds__(kThreads) void wide_loop_kernel(Ctx<M> c0, int max_wide,
                                                             int32_t max_rounds,
                                                             uint32_t poll_limit) {
    const Ctx<M> c = c0.at(blockIdx.y);
    using value_t = typename M::value_t;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    value_t *pr = reinterpret_cast<value_t *>(smem_raw);
    __shared__ UpdateSmem sm;
    __shared__ int st_go, st_cur, st_all, st_n;
    SolveCtrl *ctrl = c.ctrl;
    const int tid = threadIdx.x;
    const BidSmem B = bid_smem(c.E, (int)sizeof(value_t));
    int *lcnt = reinterpret_cast<int *>(smem_raw + B.lcnt);
    for (int e = tid; e < c.E; e += kThreads) lcnt[e] = 0;
    uint64_t target = 0;
    for (int r = 0; r < max_wide; ++r) {
        if (tid == 0) {
            const int done = ld_relaxed(&ctrl->done);
            const int cur = ld_relaxed(&ctrl->cur) & 1;
            const int all = ld_relaxed(&ctrl->all_active);
            const int n = all ? c.T : ld_relaxed(&ctrl->active_count[cur]);
            st_go = !done && n > 0 && (all || n > c.engine_cap) &&
                    ld_relaxed(&ctrl->rounds) < max_rounds && !ld_relaxed(&ctrl->internal_error);
            st_cur = cur;
            st_all = all;
            st_n = n;
        }
        __syncthreads();
        if (!st_go) break;
        for (int e = tid; e < c.E; e += kThreads) pr[e] = c.prices[e];
        __syncthreads();
        const value_t eps = (value_t)ctrl->eps;
        const value_t pmin = block_min_price<M>(pr, c.E);
        for (int i0 = blockIdx.x * kBidTile; i0 < st_n; i0 += gridDim.x * kBidTile)
            bid_block<M, G>(c, i0, i0 + kBidTile < st_n ? i0 + kBidTile : st_n, st_all != 0,
                            c.active + (int64_t)st_cur * c.T, eps, pr, pmin, lcnt,
                            reinterpret_cast<uint64_t *>(smem_raw + B.lkey),
                            reinterpret_cast<int *>(smem_raw + B.lexp),
                            reinterpret_cast<int *>(smem_raw + B.lrank));
        target += gridDim.x;
        if (!grid_barrier(c.bar, target, ctrl, poll_limit)) return;
        const int novf = min(ld_relaxed(c.ovf_count), c.T);
        for (int e = blockIdx.x; e < c.E; e += gridDim.x) update_expert<M>(c, e, st_cur ^ 1, novf, sm);
        target += gridDim.x;
        if (!grid_barrier_last(c.bar, target, ctrl, poll_limit, [&]() { end_round<M>(c); }))
            return;
    }
}

// Remaining rounds of the current phase inside one workgroup. With
// `continue_phases` the block also runs every later phase to the end.
template <class M, int G>
__global__ __launch_bounds__(kThreads) void tail_kernel(Ctx<M> c0, AssignParams p,
                                                        int continue_phases) {
    const Ctx<M> c = c0.at(blockIdx.y);
    using value_t = typename M::value_t;
    __shared__ UpdateSmem sm;
    __shared__ int st_n, st_cur, st_all, st_stop, st_begin, ntouched;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    value_t *pr = reinterpret_cast<value_t *>(smem_raw);
    int *touched = reinterpret_cast<int *>(pr + c.E);
    SolveCtrl *ctrl = c.ctrl;
    const int tid = threadIdx.x;
    for (;;) {
        if (tid == 0) {
            st_stop = 0;
            st_begin = 0;
            if (ctrl->done) {
                st_stop = 1;
            } else {
                st_cur = ctrl->cur;
                st_all = ctrl->all_active;
                st_n = st_all ? c.T : ld_relaxed(&ctrl->active_count[st_cur]);
                if (st_n == 0) {
                    if (ctrl->last_phase) {
                        ctrl->done = 1;
                        st_stop = 1;
                    } else if (!continue_phases) {
                        st_stop = 1;
                    } else {
                        begin_phase_scalar(ctrl, p, c.T);
                        begin_phase_early(ctrl);
                        st_begin = 1;
                    }
                } else if (ctrl->rounds >= p.max_rounds) {
                    ctrl->not_converged = 1;
                    ctrl->done = 1;
                    st_stop = 1;
                }
            }
            ntouched = 0;
        }
        __syncthreads();
        if (st_stop) break;
        if (st_begin) {
            for (int e = tid; e < c.E; e += blockDim.x) {
                c.hcount[e] = 0;
                c.hsel[e] = 0;
                c.bcount[e] = 0;
            }
            __threadfence_block();
            __syncthreads();
            continue;
        }
        for (int e = tid; e < c.E; e += blockDim.x) pr[e] = c.prices[e];
        __syncthreads();
        const value_t eps = (value_t)ctrl->eps;
        const value_t pmin = block_min_price<M>(pr, c.E);
        bid_range<M, G>(c, st_n, st_all != 0, c.active + (int64_t)st_cur * c.T, eps, pr, pmin,
                        tid / G, kThreads / G, touched, &ntouched);
        __threadfence_block();
        __syncthreads();
        const int novf = min(ld_relaxed(c.ovf_count), c.T);
        const int nt = ntouched < c.E ? ntouched : c.E;
        for (int i = 0; i < nt; ++i) update_expert<M>(c, touched[i], st_cur ^ 1, novf, sm);
        __threadfence_block();
        __syncthreads();
        if (tid == 0) end_round<M>(c);
        __threadfence_block();
        __syncthreads();
    }
}

// ------------------------------------------------------------ tail engine --
//
// The rounds left once at most kEngCap tokens are active run inside one
// workgroup with all mutable state in LDS:
//   prices and holder counts of every expert,
//   the K lowest held keys of every expert (sorted ascending) with the slot
//   each occupies in the expert's holder table in global memory,
//   the active tokens and the round's bids grouped by expert.
// Bids are computed against the prices at the start of the round (Jacobi),
// then one wave per touched expert streams that expert's bids through the
// rule "a new key replaces the lowest held key when it is larger"; for any
// arrival order this leaves the C largest keys of holders and bids, i.e. the
// same result as a selection. The lowest held key is the expert's price once
// it is full. A cached list that runs empty is refilled from the holder table.

// Workgroup barrier that orders LDS only: in-flight global stores are not
// waited for (the engine's one full barrier per round, after the bids, covers
// the holder-table stores before any later refill reads them).
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

constexpr int kEngThreads = 1024;
constexpr int kEngWaves = kEngThreads / 64;
constexpr int kEngCap = 256;
constexpr int kEngDirect = 64;   // rounds with at most this many bids skip the grouping
constexpr int kEngMaxE = 512;
constexpr int kEngMaxC = 512;    // holder tables a wave holds in registers (8 keys per lane)
constexpr int kEngMaxK = 64;     // longest per-expert list of lowest keys
constexpr int kEngRows = 4;      // score rows a bidding group keeps in flight

struct EngLayout {
    size_t pr, cnt, cn, sel, bcnt, boff, bfill, tch, ck, cs, bkey, bexp, bsort, actA, actB, skey,
        sslot, total;
};

__host__ __device__ inline size_t eng_align(size_t x) { return (x + 15) & ~size_t(15); }

__host__ __device__ inline EngLayout eng_layout(int E, int value_bytes, int K) {
    EngLayout L{};
    size_t off = 0;
    L.pr = off;    off = eng_align(off + (size_t)E * value_bytes);
    L.cnt = off;   off = eng_align(off + (size_t)E * 4);
    L.cn = off;    off = eng_align(off + (size_t)E * 4);
    L.sel = off;   off = eng_align(off + (size_t)E * 4);
    L.bcnt = off;  off = eng_align(off + (size_t)2 * E * 4);   // two rounds' worth
    L.boff = off;  off = eng_align(off + (size_t)E * 4);
    L.bfill = off; off = eng_align(off + (size_t)E * 4);
    L.tch = off;   off = eng_align(off + (size_t)2 * E * 4);
    L.ck = off;    off = eng_align(off + (size_t)E * K * 8);
    L.cs = off;    off = eng_align(off + (size_t)E * K * 2);
    L.bkey = off;  off = eng_align(off + (size_t)kEngCap * 8);
    L.bexp = off;  off = eng_align(off + (size_t)kEngCap * 4);
    L.bsort = off; off = eng_align(off + (size_t)kEngCap * 8);
    L.actA = off;  off = eng_align(off + (size_t)kEngCap * 4);
    L.actB = off;  off = eng_align(off + (size_t)kEngCap * 4);
    L.skey = off;  off = eng_align(off + (size_t)kEngWaves * 64 * 8);   // per-wave scratch
    L.sslot = off; off = eng_align(off + (size_t)kEngWaves * 64 * 4);
    L.total = off;
    return L;
}

template <class M>
struct Eng {
    typename M::value_t *pr;
    int *cnt, *cn, *sel, *boff, *bfill;
    int *bcnt, *tch;   // [2][E]: consecutive rounds alternate halves
    uint64_t *ck;
    uint16_t *cs;
    uint64_t *bkey, *bsort;
    int *bexp;
    uint64_t *scr_key;
    int *scr_slot;
    int K;
};

// Cross-lane moves inside the engine's update, on the VALU instead of the
// LDS crossbar: readlane broadcasts the value of one (uniform) lane; the DPP
// wavefront shifts move every lane's value one lane up (lane i receives lane
// i-1) or down (lane i receives lane i+1).
__device__ inline int rl32(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }
__device__ inline uint64_t rl64(uint64_t v, int lane) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
    return ((uint64_t)hi << 32) | lo;
}
constexpr int kDppWaveShr1 = 0x138;
constexpr int kDppWaveShl1 = 0x130;
__device__ inline int up1_i32(int v) { return __builtin_amdgcn_update_dpp(v, v, kDppWaveShr1, 0xf, 0xf, false); }
__device__ inline int down1_i32(int v) { return __builtin_amdgcn_update_dpp(v, v, kDppWaveShl1, 0xf, 0xf, false); }
__device__ inline uint64_t up1_u64(uint64_t v) {
    const uint32_t lo = (uint32_t)up1_i32((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)up1_i32((int)(uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t down1_u64(uint64_t v) {
    const uint32_t lo = (uint32_t)down1_i32((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)down1_i32((int)(uint32_t)(v >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// Expert state while one wave updates it, held in registers: lane q owns
// entry q of the sorted list of lowest keys (key, slot), and lane q also
// owns pending holder-table store q. Every lane keeps identical copies of
// the scalar fields, and every exchange between lanes is a shuffle, so no
// lane ever depends on an LDS word another lane wrote.
template <class M>
struct ExpertRegs {
    uint64_t key;    // this lane's list entry (~0 when unused)
    int slot;
    int cn;          // list length (uniform)
    int cnt;         // holders (uniform)
    uint64_t pkey;   // this lane's pending store
    int pslot;
    int np;          // pending stores (uniform)
    typename M::value_t price;
};

template <class M>
__device__ inline void er_flush(const Ctx<M> &c, uint64_t *hold, ExpertRegs<M> &r) {
    if (lane_id() < r.np) {
        if (r.pslot >= 0 && r.pslot < c.C) hold[r.pslot] = r.pkey;
        else flag_internal(c.ctrl);
    }
    r.np = 0;
}

// Records hold[slot] = key (stored by er_flush). A slot written again
// before the flush keeps a single pending entry with the latest key: the
// lanes of one store instruction reach memory in no defined order, so two
// entries for one slot could leave the older key in the table (its token
// then held twice, the newer one lost).
template <class M>
__device__ inline void er_write(const Ctx<M> &c, uint64_t *hold, ExpertRegs<M> &r, int slot,
                                uint64_t key) {
    const uint64_t same = __ballot(lane_id() < r.np && r.pslot == slot);
    if (same != 0) {
        if (lane_id() == __ffsll((long long)same) - 1) r.pkey = key;
        return;
    }
    if (r.np == 64) er_flush<M>(c, hold, r);
    if (lane_id() == r.np) {
        r.pslot = slot;
        r.pkey = key;
    }
    r.np += 1;
}

// Rank of `key` among keys[0, n) in the wave's LDS scratch (keys
// distinct): every lane reads the same word at a time (broadcast loads,
// several in flight).
__device__ inline int lds_rank(const uint64_t *keys, int n, uint64_t key) {
    int r = 0;
#pragma unroll 8
    for (int j = 0; j < n; ++j) r += keys[j] < key ? 1 : 0;
    return r;
}

// The K lowest keys of the expert's holder table, sorted, into the lanes.
// The table is read from global memory and patched with the pending stores;
// the K-th smallest key is found by a bitwise search on ballot counts, the
// keys up to it are compacted through the wave's LDS scratch, and a 64-lane
// bitonic network sorts them.
template <class M>
__device__ void er_refill(const Ctx<M> &c, const uint64_t *hold, int K, ExpertRegs<M> &r,
                          uint64_t *scr_key, int *scr_slot) {
    const int lane = lane_id();
    uint64_t kk[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const int idx = lane + 64 * q;
        kk[q] = idx < r.cnt ? hold[idx] : ~0ull;
    }
    for (int j = 0; j < r.np; ++j) {
        const int slot = rl32(r.pslot, j);
        const uint64_t key = rl64(r.pkey, j);
        if ((slot & 63) == lane) {
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if ((slot >> 6) == q) kk[q] = key;
        }
    }
    const int take = r.cnt < K ? r.cnt : K;
    r.cn = take;
    r.key = ~0ull;
    r.slot = 0;
    if (take == 0) return;
    // thr: the largest value with fewer than `take` keys below it, i.e. the
    // take-th smallest key (keys are distinct). The bits above the highest
    // one where the smallest and largest key differ are common to every key
    // (and to thr): the search starts below them.
    uint64_t kmin = ~0ull, kmax = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        if (kk[q] != ~0ull) {
            kmin = kk[q] < kmin ? kk[q] : kmin;
            kmax = kk[q] > kmax ? kk[q] : kmax;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint64_t a = __shfl_xor(kmin, off), b = __shfl_xor(kmax, off);
        kmin = a < kmin ? a : kmin;
        kmax = b > kmax ? b : kmax;
    }
    const uint64_t kdiff = kmin ^ kmax;
    const int top = kdiff ? 63 - __clzll((long long)kdiff) : 0;
    uint64_t thr = top >= 63 ? 0ull : kmin & (~0ull << (top + 1));
    // Bit by bit over the top 12 differing bits; then, when at most 64 keys
    // share the prefix found, the take-th smallest is among them (the keys
    // below the prefix are fewer than take, those up to its end at least
    // take): ranking them finishes the search. Otherwise the bits go on.
    const int lo = top >= 12 ? top - 11 : 0;
    int bit = top;
    for (; bit >= lo; --bit) {
        const uint64_t trial = thr | (1ull << bit);
        int below = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) below += __popcll(__ballot(kk[q] < trial));
        if (below < take) thr = trial;
    }
    if (lo > 0) {
        const uint64_t hi = thr >> lo;
        int below = 0, inb = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            below += __popcll(__ballot((kk[q] >> lo) < hi));
            inb += __popcll(__ballot((kk[q] >> lo) == hi));
        }
        if (inb <= 64) {
            int at = 0;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const bool in = (kk[q] >> lo) == hi;
                const uint64_t m = __ballot(in);
                if (in) scr_key[at + __popcll(m & lanemask_lt())] = kk[q];
                at += __popcll(m);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const uint64_t bk = lane < inb ? scr_key[lane] : ~0ull;
            const int need = take - below;   // in [1, inb]
            const uint64_t hit = __ballot(lane < inb && lds_rank(scr_key, inb, bk) == need - 1);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (hit != 0) thr = rl64(bk, __ffsll((long long)hit) - 1);
            else flag_internal(c.ctrl);
            bit = -1;
        }
    }
    for (; bit >= 0; --bit) {
        const uint64_t trial = thr | (1ull << bit);
        int below = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) below += __popcll(__ballot(kk[q] < trial));
        if (below < take) thr = trial;
    }
    int base = 0;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const bool sel = kk[q] <= thr;
        const uint64_t m = __ballot(sel);
        if (sel) {
            const int at = base + __popcll(m & lanemask_lt());
            if (at < 64) {
                scr_key[at] = kk[q];
                scr_slot[at] = lane + 64 * q;
            }
        }
        base += __popcll(m);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // The take selected keys in ascending order: each goes to its rank.
    const uint64_t sk = lane < take ? scr_key[lane] : ~0ull;
    const int ss = lane < take ? scr_slot[lane] : 0;
    const int rk = lds_rank(scr_key, take, sk);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < take && rk < 64) {
        scr_key[rk] = sk;
        scr_slot[rk] = ss;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (lane < take) {
        r.key = scr_key[lane];
        r.slot = scr_slot[lane];
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Loads expert e's state into the wave's registers.
template <class M>
__device__ inline void er_load(const Eng<M> &s, int e, ExpertRegs<M> &r) {
    const int lane = lane_id();
    const int K = s.K;
    // The list words are read for every lane below K (no wait for cn) and
    // masked afterwards.
    const uint64_t kv = lane < K ? s.ck[e * K + lane] : ~0ull;
    const int sv = lane < K ? (int)s.cs[e * K + lane] : 0;
    r.cn = s.cn[e];
    r.cnt = s.cnt[e];
    r.key = lane < r.cn ? kv : ~0ull;
    r.slot = lane < r.cn ? sv : 0;
    r.price = s.pr[e];
    r.np = 0;
    r.pkey = 0;
    r.pslot = 0;
}

// Stores the pending holder-table entries and expert e's state back.
template <class M>
__device__ inline void er_store(const Ctx<M> &c, const Eng<M> &s, int e, uint64_t *hold,
                                ExpertRegs<M> &r) {
    const int lane = lane_id();
    const int K = s.K;
    er_flush<M>(c, hold, r);
    if (lane < r.cn) {
        s.ck[e * K + lane] = r.key;
        s.cs[e * K + lane] = (uint16_t)r.slot;
    }
    if (r.cnt == c.C) r.price = M::key_bid(rl64(r.key, 0));   // full: the lowest held bid
    if (lane == 0) {
        s.cn[e] = r.cn;
        s.cnt[e] = r.cnt;
        s.pr[e] = r.price;
    }
}

// Streams one bid key b into the expert held in r: a free slot takes it;
// otherwise it replaces the lowest held key when larger. Returns the token
// that leaves (the displaced holder or the bidder itself), or -1.
// The list update is one ballot (b's rank among the listed keys) and one
// one-lane shift: up for an insertion, down for a replacement of the head
// (the head leaves and b enters at its rank among the rest). A key above
// every listed one enters only when the list holds every holder. A full
// expert leaves with a non-empty list (refilled in one place, at the end);
// its price is taken from the list head when the state is stored.
template <class M>
__device__ __attribute__((always_inline)) inline int er_bid(const Ctx<M> &c, uint64_t *hold,
                                                            int K, ExpertRegs<M> &r, uint64_t b,
                                                            uint64_t *scr_key, int *scr_slot) {
    const int lane = lane_id();
    int out_tok = -1;
    if (r.cnt < c.C) {
        const int slot = r.cnt;
        const bool complete = r.cn == r.cnt;
        er_write<M>(c, hold, r, slot, b);
        r.cnt += 1;
        const int pos = __popcll(__ballot(lane < r.cn && r.key < b));
        if ((pos < r.cn || complete) && pos < K) {
            const uint64_t kprev = up1_u64(r.key);
            const int sprev = up1_i32(r.slot);
            const int nn = r.cn + 1 < K ? r.cn + 1 : K;
            if (lane >= pos && lane < nn) {
                r.key = lane == pos ? b : kprev;
                r.slot = lane == pos ? slot : sprev;
            }
            r.cn = nn;
        }
    } else {
        // (an empty list here only follows a flagged inconsistency: every
        // bid is then refused)
        const uint64_t head = r.cn > 0 ? rl64(r.key, 0) : ~0ull;
        if (b > head) {
            const int slot = rl32(r.slot, 0);
            out_tok = key_token(head);
            er_write<M>(c, hold, r, slot, b);
            const bool complete = r.cn == r.cnt;
            const int pos = __popcll(__ballot(lane >= 1 && lane < r.cn && r.key < b)) ;
            const bool keep = pos < r.cn - 1 || complete;
            const uint64_t knext = down1_u64(r.key);
            const int snext = down1_i32(r.slot);
            if (lane < pos) {
                r.key = knext;
                r.slot = snext;
            } else if (lane == pos) {
                r.key = keep ? b : ~0ull;
                r.slot = keep ? slot : 0;
            }
            if (!keep) r.cn -= 1;
        } else {
            out_tok = key_token(b);
        }
    }
    if (r.cnt == c.C && r.cn == 0) er_refill<M>(c, hold, K, r, scr_key, scr_slot);
    return out_tok;
}

template <class M>
__device__ inline uint64_t *expert_holders(const Ctx<M> &c, const Eng<M> &s, int e) {
    return c.holders + (int64_t)(s.sel[e] & 1) * c.T + (int64_t)e * c.C;
}

// One wave: streams expert e's bids of this round into its holders. Bids are
// bids[0..nb), or, with `exps`, the entries of bids[0..nb) whose expert is e
// (picked out by a ballot, 64 entries per step).
// Tokens that leave, collected by one wave in lane order (lane k holds
// the k-th) over the experts it updates in a round, and appended to the
// next active list 64 at a time (one LDS atomic per append).
struct OutQueue {
    int n = 0;
    int tok = 0;
};

template <class M>
__device__ inline void flush_outs(const Ctx<M> &c, OutQueue &q, int *nxt, int *nnext) {
    const int lane = lane_id();
    if (q.n == 0) return;
    int base = 0;
    if (lane == 0) base = atomicAdd(nnext, q.n);
    base = __builtin_amdgcn_readfirstlane(base);
    if (lane < q.n) {
        const int at = base + lane;
        if (at < kEngCap && q.tok >= 0 && q.tok < c.T) nxt[at] = q.tok;
        else flag_internal(c.ctrl);
    }
    q.n = 0;
}

template <class M>
__device__ __attribute__((always_inline)) void eng_update(const Ctx<M> &c, const Eng<M> &s, int e, const uint64_t *bids,
                           const int *exps, int nb, int *nxt, int *nnext, OutQueue &q) {
    const int lane = lane_id();
    uint64_t *hold = expert_holders<M>(c, s, e);
    uint64_t *scr_key = s.scr_key + (threadIdx.x >> 6) * 64;
    int *scr_slot = s.scr_slot + (threadIdx.x >> 6) * 64;
    ExpertRegs<M> r;
    er_load<M>(s, e, r);
    // Bids are read 64 at a time, one per lane, and taken in lane order.
    for (int j0 = 0; j0 < nb; j0 += 64) {
        const int j = j0 + lane;
        const bool mine = j < nb && (exps == nullptr || exps[j] == e);
        const uint64_t mykey = j < nb ? bids[j] : 0ull;
        uint64_t mask = __ballot(mine);
        while (mask) {
            const int src = __ffsll((long long)mask) - 1;
            mask &= mask - 1;
            const int out_tok = er_bid<M>(c, hold, s.K, r, rl64(mykey, src), scr_key, scr_slot);
            if (out_tok >= 0) {
                if (lane == q.n) q.tok = out_tok;
                if (++q.n == 64) flush_outs<M>(c, q, nxt, nnext);
            }
        }
    }
    er_store<M>(c, s, e, hold, r);
}

// Orders one wave's LDS (and global) accesses for the compiler: values one
// lane stored are seen by every lane after it (the hardware keeps a wave's
// accesses in order).
__device__ inline void wave_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One bid b for expert e in the common case of the solo rounds: e is full
// and its list holds at least two keys. The list words, count and length
// are read in one LDS round trip; a refused bid changes nothing (the price
// already is the lowest held bid); an accepted one replaces the head in the
// list (one ballot and one DPP shift), stores b into the head's slot of the
// holder table and sets the price from the new head. Returns the leaving
// token, or -2 when the case does not apply (nothing changed then). The
// holder-table store is left to the caller (*store_slot >= 0: store b
// there), so that loads the caller issues first do not wait behind it.
template <class M>
__device__ __attribute__((always_inline)) inline int solo_replace_head(const Ctx<M> &c,
                                                                       const Eng<M> &s, int e,
                                                                       uint64_t b,
                                                                       int *store_slot) {
    *store_slot = -1;
    const int lane = lane_id();
    const int K = s.K;
    const uint64_t kv = lane < K ? s.ck[e * K + lane] : ~0ull;
    const int sv = lane < K ? (int)s.cs[e * K + lane] : 0;
    const int cn = s.cn[e];
    const int cnt = s.cnt[e];
    if (cnt != c.C || cn < 2) return -2;
    const uint64_t key = lane < cn ? kv : ~0ull;
    const uint64_t head = rl64(key, 0);
    if (b <= head) return key_token(b);
    const int slot0 = rl32(sv, 0);
    const bool complete = cn == cnt;
    const int pos = __popcll(__ballot(lane >= 1 && lane < cn && key < b));
    const bool keep = pos < cn - 1 || complete;
    const uint64_t knext = down1_u64(key);
    const int snext = down1_i32(sv);
    uint64_t nk = key;
    int ns = sv;
    if (lane < pos) {
        nk = knext;
        ns = snext;
    } else if (lane == pos) {
        nk = keep ? b : ~0ull;
        ns = keep ? slot0 : 0;
    }
    if (lane <= pos && lane < K) {
        s.ck[e * K + lane] = nk;
        s.cs[e * K + lane] = (uint16_t)ns;
    }
    const uint64_t nhead = rl64(nk, 0);
    if (lane == 0) {
        if (!keep) s.cn[e] = cn - 1;
        s.pr[e] = M::key_bid(nhead);
    }
    *store_slot = slot0;
    return key_token(head);
}

// Tokens one wave bids for at once: one group of G lanes each, at most 8.
template <int G>
constexpr int solo_tokens() { return (64 / G) < 8 ? (64 / G) : 8; }

// Rounds with at most solo_tokens<G>() active tokens, run by one wave with
// no workgroup barrier: each group bids for one token (same prices for all,
// as in every round), then the wave streams the bids into their experts one
// after another. A bid leaves at most one token active, so once a round fits
// every later round of the phase fits as well; the loop runs until no token
// is active or the round limit is reached. The other waves wait at the
// caller's next barrier.
template <class M, int G>
__device__ __attribute__((always_inline)) void engine_solo(const Ctx<M> &c, const Eng<M> &s, int *act, typename M::value_t eps,
                            typename M::value_t pmin, int max_rounds_left, int n, int rounds,
                            int *s_n, int *s_rounds, unsigned long long *s_bids) {
    using value_t = typename M::value_t;
    const int lane = lane_id();
    const int gl = lane & (G - 1);
    const int g = lane / G;
    unsigned long long bids = 0;
    int tokv = lane < n ? act[lane] : 0;   // lane k holds active token k
    int overflow = 0;
    // Holder-table stores of the head replacements wait in a register queue
    // (lane j: address and key of store j; one entry per address) and go out
    // 64 at a time, before any update that reads the tables, and at the end:
    // a store in the round's path would make the next round's first load
    // wait for it.
    uint64_t *q_addr = nullptr;
    uint64_t q_key = 0;
    int qn = 0;
    auto q_flush = [&]() {
        if (lane < qn) *q_addr = q_key;
        qn = 0;
    };
    // Group g bids for token g; its summary for the coming round is loaded
    // as soon as the token is known (for the next round: right after the
    // update that makes it leave, ahead of that update's table stores).
    int t = 0;
    for (int k = 0; k < n; ++k) {
        const int tk = rl32(tokv, k);
        if (g == k) t = tk;
    }
    uint32_t sw[4] = {0, 0, 0, 0};
    if (g < n) load_summary(c.sums, t, gl, sw);
    while (n > 0 && rounds < max_rounds_left) {
        const bool valid = g < n;
        value_t v1, v2, s1;
        int e1;
        top2_summary<M, G>(c, sw, t, valid, gl, s.pr, pmin, v1, e1, v2, s1);
        uint64_t key = 0;
        int ex = 0;
        if (valid && gl == 0) {
            if (e1 >= c.E) {
                e1 = 0;
                s1 = 0;   // with v2 = -inf the bid is +inf: overflow is flagged
            }
            const value_t bid = (value_t)((s1 - v2) + eps);
            key = M::make_key(bid, t, &overflow);
            ex = e1;
        }
        int nn = 0, nxt_tok = 0, t_next = 0;
        uint32_t sw_next[4] = {0, 0, 0, 0};
        for (int k = 0; k < n; ++k) {
            const int e = rl32(ex, k * G);
            const uint64_t b = rl64(key, k * G);
            int store_slot = -1;
            int out = solo_replace_head<M>(c, s, e, b, &store_slot);
            if (out == -2) {
                q_flush();
                uint64_t *hold = expert_holders<M>(c, s, e);
                ExpertRegs<M> r;
                er_load<M>(s, e, r);
                out = er_bid<M>(c, hold, s.K, r, b, s.scr_key, s.scr_slot);
                er_store<M>(c, s, e, hold, r);
            }
            if (out >= c.T) {
                flag_internal(c.ctrl);
                out = 0;
            }
            if (out >= 0) {
                if (lane == nn) nxt_tok = out;
                if (g == nn) {
                    t_next = out;
                    load_summary(c.sums, out, gl, sw_next);
                }
                ++nn;
            }
            if (store_slot >= c.C) {
                flag_internal(c.ctrl);
            } else if (store_slot >= 0) {
                uint64_t *addr = expert_holders<M>(c, s, e) + store_slot;
                const uint64_t same = __ballot(lane < qn && q_addr == addr);
                if (same != 0) {
                    if (lane == __ffsll((long long)same) - 1) q_key = b;
                } else {
                    if (qn == 64) q_flush();
                    if (lane == qn) {
                        q_addr = addr;
                        q_key = b;
                    }
                    ++qn;
                }
            }
            wave_sync();
        }
        rounds += 1;
        bids += (unsigned long long)n;
        tokv = nxt_tok;
        n = nn;
        t = t_next;
#pragma unroll
        for (int q = 0; q < 4; ++q) sw[q] = sw_next[q];
    }
    q_flush();
    if (lane < n) act[lane] = tokv;
    if (__ballot(overflow != 0) && lane == 0) c.ctrl->overflow = 1;
    if (lane == 0) {
        *s_n = n;
        *s_rounds = rounds;
        *s_bids += bids;
    }
}

// The engine's phase entry, one launch: blocks [0, E) sort expert e's
// holder table and store its K lowest keys (with slots) for the engine to
// load; the `pf` blocks after them pull the score summaries into every L2.
template <class M>
__global__ __launch_bounds__(256) void engine_entry_kernel(Ctx<M> c0, int pf) {
    const Ctx<M> c = c0.at(blockIdx.y);
    __shared__ uint64_t keys[kEngMaxC];
    __shared__ uint16_t slots[kEngMaxC];
    __shared__ int go;
    SolveCtrl *ctrl = c.ctrl;
    if (threadIdx.x == 0) {
        go = 0;
        if (!ctrl->done && !ctrl->all_active) {
            const int n = ld_relaxed(&ctrl->active_count[ctrl->cur]);
            if (n > c.ssp_cap && n <= c.engine_cap) go = 1;
        }
    }
    __syncthreads();
    if (!go) return;
    if ((int)blockIdx.x >= c.E) {
        summary_prefill(reinterpret_cast<const uint4 *>(c.sums), (int64_t)c.T * 4,
                        (int)blockIdx.x - c.E, pf, reinterpret_cast<uint32_t *>(&ctrl->pad2));
        return;
    }
    const int e = blockIdx.x;
    int cnt = ld_relaxed(&c.hcount[e]);
    if (cnt < 0 || cnt > c.C) {
        if (threadIdx.x == 0) flag_internal(ctrl);
        cnt = cnt < 0 ? 0 : c.C;
    }
    const uint64_t *hold = c.holders + (int64_t)(ld_relaxed(&c.hsel[e]) & 1) * c.T + (int64_t)e * c.C;
    int P = 1;
    while (P < cnt) P <<= 1;
    for (int i = threadIdx.x; i < P; i += blockDim.x) {
        keys[i] = i < cnt ? hold[i] : ~0ull;
        slots[i] = (uint16_t)i;
    }
    __syncthreads();
    for (int k = 2; k <= P; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = threadIdx.x; i < P; i += blockDim.x) {
                const int ixj = i ^ j;
                if (ixj > i) {
                    const bool up = (i & k) == 0;
                    const uint64_t a = keys[i], b = keys[ixj];
                    if ((a > b) == up) {
                        keys[i] = b;
                        keys[ixj] = a;
                        const uint16_t t = slots[i];
                        slots[i] = slots[ixj];
                        slots[ixj] = t;
                    }
                }
            }
            __syncthreads();
        }
    }
    const int take = cnt < c.eng_k ? cnt : c.eng_k;
    for (int q = threadIdx.x; q < take; q += blockDim.x) {
        c.eng_ck[(int64_t)e * c.eng_k + q] = keys[q];
        c.eng_cs[(int64_t)e * c.eng_k + q] = slots[q];
    }
    if (threadIdx.x == 0) c.eng_cn[e] = take;
}

template <class M, int G>
__global__ __launch_bounds__(kEngThreads) void engine_kernel(Ctx<M> c0, AssignParams p) {
    const Ctx<M> c = c0.at(blockIdx.y);
    using value_t = typename M::value_t;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int K = c.eng_k;
    const EngLayout L = eng_layout(c.E, (int)sizeof(value_t), K);
    Eng<M> s;
    s.K = K;
    s.pr = reinterpret_cast<value_t *>(smem_raw + L.pr);
    s.cnt = reinterpret_cast<int *>(smem_raw + L.cnt);
    s.cn = reinterpret_cast<int *>(smem_raw + L.cn);
    s.sel = reinterpret_cast<int *>(smem_raw + L.sel);
    s.bcnt = reinterpret_cast<int *>(smem_raw + L.bcnt);
    s.boff = reinterpret_cast<int *>(smem_raw + L.boff);
    s.bfill = reinterpret_cast<int *>(smem_raw + L.bfill);
    s.tch = reinterpret_cast<int *>(smem_raw + L.tch);
    s.ck = reinterpret_cast<uint64_t *>(smem_raw + L.ck);
    s.cs = reinterpret_cast<uint16_t *>(smem_raw + L.cs);
    s.bkey = reinterpret_cast<uint64_t *>(smem_raw + L.bkey);
    s.bexp = reinterpret_cast<int *>(smem_raw + L.bexp);
    s.bsort = reinterpret_cast<uint64_t *>(smem_raw + L.bsort);
    s.scr_key = reinterpret_cast<uint64_t *>(smem_raw + L.skey);
    s.scr_slot = reinterpret_cast<int *>(smem_raw + L.sslot);
    int *act = reinterpret_cast<int *>(smem_raw + L.actA);
    int *nxt = reinterpret_cast<int *>(smem_raw + L.actB);
    __shared__ int s_go, s_cur, s_n, s_nnext[2], s_ntouched[2], s_grab[2], s_rounds, s_stop;
    __shared__ unsigned long long s_bids;

    SolveCtrl *ctrl = c.ctrl;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if (tid == 0) {
        s_go = 0;
        if (!ctrl->done && !ctrl->all_active) {
            s_cur = ctrl->cur;
            const int n = ld_relaxed(&ctrl->active_count[s_cur]);
            if (n > 0 && n > c.ssp_cap && n <= kEngCap) {
                s_go = 1;
                s_n = n;
            }
        }
        s_nnext[0] = s_nnext[1] = 0;
        s_ntouched[0] = s_ntouched[1] = 0;
        s_grab[0] = s_grab[1] = 0;
        s_rounds = 0;
        s_stop = 0;
        s_bids = 0;
    }
    __syncthreads();
    if (!s_go) return;
    const int max_rounds_left = p.max_rounds - ctrl->rounds;
    const value_t eps = (value_t)ctrl->eps;
    for (int e = tid; e < c.E; e += kEngThreads) {
        s.pr[e] = c.prices[e];
        int cnt = ld_relaxed(&c.hcount[e]);
        int cn = c.eng_cn[e];
        if (cnt < 0 || cnt > c.C || cn < 0 || cn > K || cn > cnt) {
            flag_internal(ctrl);
            cnt = cnt < 0 ? 0 : (cnt > c.C ? c.C : cnt);
            cn = 0;
        }
        s.cnt[e] = cnt;
        s.cn[e] = cn;
        s.sel[e] = ld_relaxed(&c.hsel[e]) & 1;
        s.bcnt[e] = 0;
        s.bcnt[c.E + e] = 0;
        s.bfill[e] = 0;
    }
    // The entry lists (every expert's K slots, used or not).
    copy16_to_lds<kEngThreads>(reinterpret_cast<uint4 *>(s.ck),
                               reinterpret_cast<const uint4 *>(c.eng_ck), c.E * K / 2);
    copy16_to_lds<kEngThreads>(reinterpret_cast<uint4 *>(s.cs),
                               reinterpret_cast<const uint4 *>(c.eng_cs), c.E * K / 8);
    for (int i = tid; i < s_n; i += kEngThreads) {
        const int t = c.active[(int64_t)s_cur * c.T + i];
        act[i] = (t >= 0 && t < c.T) ? t : 0;
        if (t < 0 || t >= c.T) flag_internal(ctrl);
    }
    __syncthreads();
    // Lowest price at entry: prices only rise, so it stays a lower bound of
    // every price for the whole run (used by the summary test).
    __shared__ value_t s_pmin;
    if (wave == 0) {
        value_t m = s.pr[0];
        for (int e = lane; e < c.E; e += 64) m = s.pr[e] < m ? s.pr[e] : m;
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            const value_t o = __shfl_xor(m, off);
            m = o < m ? o : m;
        }
        if (lane == 0) s_pmin = m;
    }
    __syncthreads();
    const value_t pmin = s_pmin;

    const int per_pass = kEngThreads / G;
    const int gid = tid / G;
    const int gl = lane & (G - 1);
    // Round bookkeeping: every thread keeps the active count and the round
    // number in registers. The per-expert bid counts, the touched-expert
    // list and the LDS counters (next list length, touched experts, experts
    // taken) alternate halves between consecutive rounds (parity h): a round
    // clears what the round before used while it bids, so a round needs two
    // workgroup barriers (four when it groups its bids) and no separate
    // clearing step.
    int n = s_n;
    int rounds = 0;
    int h = 0;
    int nt_prev = 0;
    for (;;) {
        if (n == 0) break;
        if (n <= c.ssp_cap) break;   // the shortest-path finish takes the last tokens
        if (rounds >= max_rounds_left) {
            if (tid == 0) s_stop = 1;
            break;
        }
        if (n <= solo_tokens<G>()) {
            // Runs the rest of the phase (see engine_solo): the loop ends next.
            if (wave == 0)
                engine_solo<M, G>(c, s, act, eps, pmin, max_rounds_left, n, rounds, &s_n,
                                  &s_rounds, &s_bids);
            __syncthreads();
            n = s_n;
            rounds = s_rounds;
            continue;
        }
        int *const bcnt = s.bcnt + h * c.E;
        int *const tch = s.tch + h * c.E;
        {
            // The previous round's counts and fill counters back to zero
            // (read last before the barrier that ended it).
            const int *tch_prev = s.tch + (h ^ 1) * c.E;
            int *bcnt_prev = s.bcnt + (h ^ 1) * c.E;
            for (int j = tid; j < nt_prev; j += kEngThreads) {
                const int e = tch_prev[j];
                bcnt_prev[e] = 0;
                s.bfill[e] = 0;
            }
            if (tid == 0) {
                s_ntouched[h ^ 1] = 0;
                s_grab[h ^ 1] = 0;
            }
        }
        // Bids against the prices at the start of the round.
        // Each group keeps kEngRows score rows in flight: all loads first,
        // then the reductions. With E <= kEngMaxE = 8 * 64 a row is one chunk
        // of 8 experts per lane (lanes_per_token picks G >= E / 8).
        // Summaries first (one 64-byte line per token, held in L2); a token
        // whose summary cannot decide its top-2 reads its whole row.
        const int stride = per_pass * kEngRows;
        const int n_round = ((n + stride - 1) / stride) * stride;
        for (int i0 = gid; i0 < n_round; i0 += stride) {
          uint32_t sw[kEngRows][4];   // entry gl % 8 of the summary, bound, count
          int toks[kEngRows];
#pragma unroll
          for (int u = 0; u < kEngRows; ++u) {
              const int i = i0 + u * per_pass;
              toks[u] = i < n ? act[i] : 0;
              sw[u][0] = sw[u][1] = sw[u][2] = sw[u][3] = 0;
              if (i < n) load_summary(c.sums, toks[u], gl, sw[u]);
          }
#pragma unroll
          for (int u = 0; u < kEngRows; ++u) {
            const int i = i0 + u * per_pass;
            const bool valid = i < n;
            if (__ballot(valid) == 0) break;   // no token of this slot in the wave
            const int t = toks[u];
            value_t v1, v2, s1;
            int e1;
            top2_summary<M, G>(c, sw[u], t, valid, gl, s.pr, pmin, v1, e1, v2, s1);
            if (valid && gl == 0) {
                if (e1 >= c.E) {
                    e1 = 0;
                    s1 = 0;   // with v2 = -inf the bid is +inf: overflow is flagged
                }
                const value_t bid = (value_t)((s1 - v2) + eps);
                int overflow = 0;
                const uint64_t key = M::make_key(bid, t, &overflow);
                if (overflow) ctrl->overflow = 1;
                s.bkey[i] = key;
                s.bexp[i] = e1;
                if (atomicAdd(&bcnt[e1], 1) == 0) {
                    const int at = atomicAdd(&s_ntouched[h], 1);
                    if (at < c.E) tch[at] = e1;
                }
            }
          }
        }
        __syncthreads();   // also completes the previous round's holder-table stores
        const int nt = s_ntouched[h] < c.E ? s_ntouched[h] : c.E;
        int *const nnext = &s_nnext[h];
        if (tid == 0) s_nnext[h ^ 1] = 0;   // read last right after the previous round
        if (n <= kEngDirect) {
            // Few bids: every wave reads them all and keeps its experts' ones.
            OutQueue q;
            for (int j = wave; j < nt; j += kEngWaves)
                eng_update<M>(c, s, tch[j], s.bkey, s.bexp, n, nxt, nnext, q);
            flush_outs<M>(c, q, nxt, nnext);
        } else {
            if (wave == 0) {
                int base = 0;
                for (int j0 = 0; j0 < nt; j0 += 64) {
                    const int j = j0 + lane;
                    const int cj = j < nt ? bcnt[tch[j]] : 0;
                    int incl = cj;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const int o = __shfl_up(incl, off);
                        if (lane >= off) incl += o;
                    }
                    if (j < nt) s.boff[tch[j]] = base + incl - cj;
                    base += __shfl(incl, 63);
                }
            }
            lds_barrier();
            for (int i = tid; i < n; i += kEngThreads) {
                const int e = s.bexp[i];
                const int pos = s.boff[e] + atomicAdd(&s.bfill[e], 1);
                if (pos < kEngCap) s.bsort[pos] = s.bkey[i];
                else flag_internal(ctrl);
            }
            lds_barrier();
            // Waves take the touched experts one at a time from a shared
            // counter (their bid counts differ widely).
            OutQueue q;
            for (;;) {
                int j = 0;
                if (lane == 0) j = atomicAdd(&s_grab[h], 1);
                j = __builtin_amdgcn_readfirstlane(j);
                if (j >= nt) break;
                const int e = tch[j];
                int nb = bcnt[e];
                const int off = s.boff[e];
                if (off + nb > kEngCap) {
                    if (lane == 0) flag_internal(ctrl);
                    nb = kEngCap - off;
                }
                eng_update<M>(c, s, e, s.bsort + off, nullptr, nb, nxt, nnext, q);
            }
            flush_outs<M>(c, q, nxt, nnext);
        }
        lds_barrier();
        rounds += 1;
        if (tid == 0) s_bids += (unsigned long long)n;
        n = *nnext < kEngCap ? *nnext : kEngCap;
        nt_prev = nt;
        h ^= 1;
        int *tmp = act;
        act = nxt;
        nxt = tmp;
    }

    // Hand the state back.
    for (int e = tid; e < c.E; e += kEngThreads) {
        c.prices[e] = s.pr[e];
        c.hcount[e] = s.cnt[e];
        c.bcount[e] = 0;
    }
    for (int i = tid; i < n; i += kEngThreads) c.active[(int64_t)s_cur * c.T + i] = act[i];
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        ctrl->rounds += rounds;
        ctrl->bids += s_bids;
        ctrl->engine_bids += s_bids;
        ctrl->active_count[s_cur] = n;
        ctrl->active_count[s_cur ^ 1] = 0;
        ctrl->pad0 = 0;
        if (s_stop) {
            ctrl->not_converged = 1;
            ctrl->done = 1;
        } else if (n == 0 && ctrl->last_phase) {
            ctrl->done = 1;
        }
    }
}

// ------------------------------------------------- shortest-path finish --
//
// The last few tokens of a phase (at most ssp_cap, float mode, E <= 256)
// are not left to the auction's rounds: each would wander through many
// experts, one eviction per round, until it meets a free slot. Instead each
// is placed by one shortest augmenting path over the E experts, as in the
// successive-shortest-path method for the transportation problem, starting
// from the auction's epsilon-complementary-slack state:
//
//   arc e -> x   moving the cheapest token t of expert e to expert x costs
//                w(e,x) = min_t [(S[t,e] - p_e) - (S[t,x] - p_x)]
//                       = M(e,x) - p_e + p_x,  M(e,x) = min_t S[t,e] - S[t,x].
//                Epsilon-CS says w >= -eps; the search uses w+ = max(w, 0).
//   sources      every unassigned token u reaches expert x at
//                dist0(x) = max_y (S[u,y] - p_y) - (S[u,x] - p_x) >= 0.
//   target       the expert with a free slot at the least distance D.
//
// Bellman-Ford over the dense E x E arcs (all arcs relaxed in parallel, a
// few iterations: shortest paths have few hops) gives dist(); the path is
// applied (each expert on it hands its cheapest token to the next, the free
// expert gains one) and every price rises by max(0, D - dist(x)). With
// dist(x') <= dist(x) + w+(x,x') <= dist(x) + w(x,x') + eps, every arc keeps
// w >= -eps after the rise, the moved tokens' arcs included, and the placed
// token ends at its best value: epsilon-CS holds for every assigned token,
// so the finished phase carries the auction's own guarantee (T * eps). Free
// experts keep their prices (their distance is at least D).
//
// ssp_build_kernel computes M and the slot of its token for every expert
// (one block per expert, reading its tokens' score rows); ssp_kernel keeps
// M in registers (thread (x, part) holds rows [part R, part R + R) of
// column x), the slots in LDS, and updates both after each path: an expert
// that received a token takes the minimum with that token's row; a column
// whose cheapest token left is recomputed over the expert's slots.

constexpr int kSspThreads = 1024;
constexpr int kSspMaxCap = 32;   // most unassigned tokens a phase hands over
constexpr int kSspMinCap = 8;
constexpr int kSspRc = 256;      // column recomputes taken per pass
constexpr int kSspMnew = 8;      // path experts whose received rows go through LDS
// (sixteen with 256 experts, whose paths run longer)
template <int Ep>
constexpr int ssp_mnew() { return Ep > 128 ? 2 * kSspMnew : kSspMnew; }


// Whether problem c's current phase waits for the shortest-path finish.
template <class M>
__device__ inline bool ssp_pending(const Ctx<M> &c, int *n_out) {
    const SolveCtrl *ctrl = c.ctrl;
    if (c.ssp_cap <= 0 || ctrl->done || ctrl->all_active) return false;
    const int n = ld_relaxed(&ctrl->active_count[ctrl->cur]);
    *n_out = n;
    return n > 0 && n <= c.ssp_cap;
}

// Threads of a build block: a quarter for experts of at most 64 tokens in
// grids of more than 1024 blocks (a batch of 256 worker-shape problems
// launches 32768, and four times as many fit on a compute unit at once:
// 117 -> 134 M tokens/s through the batch); a single problem keeps full
// blocks (its 128 blocks at a quarter of the threads were slower).
inline int ssp_build_threads(int64_t C, int64_t blocks) {
    return C <= 64 && blocks > 1024 ? kSspThreads / 4 : kSspThreads;
}

template <class M>
__global__ __launch_bounds__(kSspThreads) void ssp_build_kernel(Ctx<M> c0) {
    const Ctx<M> c = c0.at(blockIdx.y);
    __shared__ int go;
    __shared__ int tok[kEngMaxC];
    __shared__ float se[kEngMaxC];
    __shared__ float rv[kSspThreads];
    __shared__ int rs[kSspThreads];
    const int tid = threadIdx.x;
    if (tid == 0) {
        int n = 0;
        go = ssp_pending<M>(c, &n) ? 1 : 0;
    }
    __syncthreads();
    if (!go) return;
    const int e = blockIdx.x;
    int cnt = ld_relaxed(&c.hcount[e]);
    if (cnt < 0 || cnt > c.C) {
        if (tid == 0) flag_internal(c.ctrl);
        cnt = 0;
    }
    const uint64_t *hold = c.holders + (int64_t)(ld_relaxed(&c.hsel[e]) & 1) * c.T + (int64_t)e * c.C;
    const int nth = blockDim.x;   // a multiple of Ep (kSspThreads or a quarter of it)
    for (int q = tid; q < cnt; q += nth) {
        int t = key_token(hold[q]);
        if (t < 0 || t >= c.T) {
            flag_internal(c.ctrl);
            t = 0;
        }
        tok[q] = t;
        se[q] = c.S[(int64_t)t * c.E + e];
    }
    __syncthreads();
    // The expert's tokens for the finish's LDS copy (uint16: T <= 65536).
    for (int q = tid; q < c.C; q += nth)
        c.ssp_t[(int64_t)e * c.C + q] = (uint16_t)(q < cnt ? tok[q] : 0);
    int Ep = 1;
    while (Ep < c.E) Ep <<= 1;
    const int subs = nth / Ep;
    const int x = tid % Ep, sub = tid / Ep;
    float best = INFINITY;
    int bs = 0xffff;
    if (x < c.E) {
#pragma unroll 8
        for (int q = sub; q < cnt; q += subs) {
            const float v = se[q] - c.S[(int64_t)tok[q] * c.E + x];
            if (v < best) {
                best = v;
                bs = q;
            }
        }
    }
    rv[tid] = best;
    rs[tid] = bs;
    __syncthreads();
    if (sub == 0 && x < c.E) {
        for (int j = 1; j < subs; ++j) {
            const float v = rv[j * Ep + x];
            const int q = rs[j * Ep + x];
            if (v < best || (v == best && q < bs)) {
                best = v;
                bs = q;
            }
        }
        c.ssp_m[(int64_t)e * c.E + x] = best;
        c.ssp_a[(int64_t)e * c.E + x] = (uint16_t)bs;
    }
}

// LDS of ssp_kernel for Ep padded experts: fixed-size arrays at offsets
// known at compile time, then the slot matrix [E][E] (u16), the rows of the
// unassigned tokens transposed [E][K + 1] (fp32; the odd stride keeps the
// lanes of a wave on distinct banks both ways) and every expert's holder
// slots [E][C] as u16 tokens (T <= 65536).
template <int Ep>
struct SspLds {
    // Ep = 256: the slot matrix and the token lists stay in global memory
    // (the workspace tables the build kernel wrote); they would not fit.
    static constexpr bool kGlobal = Ep > 128;
    static constexpr size_t distp = 0;                       // u64 [3][Ep]
    static constexpr size_t rckey = distp + 3 * Ep * 8;      // u64 [ssp_mnew][Ep]
    static constexpr size_t pr = rckey + ssp_mnew<Ep>() * Ep * 8;  // f32 [Ep]
    static constexpr size_t cnt = pr + Ep * 4;               // i32 [Ep]
    static constexpr size_t sel = cnt + Ep * 4;
    static constexpr size_t path = sel + Ep * 4;             // i32 [Ep + 4]
    static constexpr size_t hslot = path + (Ep + 4) * 4;
    static constexpr size_t htok = hslot + Ep * 4;
    static constexpr size_t urow = htok + Ep * 4;
    static constexpr size_t rcj = urow + Ep * 4;             // [kSspRc]
    static constexpr size_t rcx = rcj + kSspRc * 4;
    static constexpr size_t act = rcx + kSspRc * 4;          // [kSspMaxCap]
    static constexpr size_t vstar = act + kSspMaxCap * 4;
    static constexpr size_t mnew = vstar + kSspMaxCap * 4;   // f32 [ssp_mnew][Ep]
    static constexpr size_t am = mnew + ssp_mnew<Ep>() * Ep * 4;   // u16 [Ep][Ep]
    static constexpr size_t rows = am + (kGlobal ? 0 : (size_t)Ep * Ep * 2); // f32 [E][K + 1]
    __host__ __device__ static size_t toks(int E, int K) {
        return (rows + (size_t)E * (K + 1) * 4 + 15) & ~size_t(15);
    }
    __host__ __device__ static size_t total(int E, int K, int C) {
        return toks(E, K) + (kGlobal ? 0 : (size_t)E * C * 2);
    }
};

inline int ssp_pad(int E) {
    int Ep = 32;
    while (Ep < E) Ep <<= 1;
    return Ep;
}

inline size_t ssp_lds_bytes(int E, int K, int C) {
    switch (ssp_pad(E)) {
        case 32: return SspLds<32>::total(E, K, C);
        case 64: return SspLds<64>::total(E, K, C);
        case 128: return SspLds<128>::total(E, K, C);
        default: return SspLds<256>::total(E, K, C);
    }
}

// Packed distance label: the (non-negative) distance's bits above, the
// predecessor below (an expert, or kSspSrc + i for unassigned token i), so
// that one 64-bit minimum keeps a distance with its predecessor.
constexpr uint32_t kSspSrc = 0x10000u;
__device__ inline uint64_t ssp_pack(float d, uint32_t lab) {
    return ((uint64_t)__float_as_uint(d) << 32) | lab;
}
__device__ inline float ssp_dist(uint64_t v) { return __uint_as_float((uint32_t)(v >> 32)); }
// An exchange-matrix entry with the slot of its token, ordered by value.
__device__ inline uint64_t ssp_entry(float v, int q) {
    return ((uint64_t)f32_ord(v) << 32) | (uint32_t)q;
}

// Sixteen waves (four per SIMD) for every Ep: wave w owns rows
// [w RW, w RW + RW) of the exchange matrix (RW = Ep / 16), lane l its
// columns l + 64 j. A Bellman-Ford step costs each wave one uniform test
// per row it owns, relaxed or not, and a wave issues one instruction at a
// time: few rows per wave, with four waves interleaved on each SIMD, keep
// the steps short (with four waves of 32 rows a step took about 3000
// cycles, most of them in the test chain). For Ep = 256 the arcs'
// M(e,x) + p_x are formed where they are used instead of kept in a second
// array (registers).
constexpr int kSspBlock = 1024;
template <int Ep>
constexpr int ssp_block() { return kSspBlock; }

// small != 0 (tests only) routes every step through the fallbacks: no
// recompute list (whole rows instead) and received rows read by the owners.
template <class M, int Ep>
__global__ __launch_bounds__(ssp_block<Ep>()) void ssp_kernel(Ctx<M> c0, int K, int small) {
    static_assert(!M::kInteger, "the shortest-path finish runs in float mode");
    constexpr int kBlk = ssp_block<Ep>();
    constexpr int kW = kBlk / 64;
    constexpr int RW = Ep / kW;                  // rows per wave
    constexpr int CL = Ep >= 64 ? Ep / 64 : 1;   // columns per lane
    constexpr bool kG = SspLds<Ep>::kGlobal;
    const Ctx<M> c = c0.at(blockIdx.y);
    SolveCtrl *ctrl = c.ctrl;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    using LY = SspLds<Ep>;
    uint64_t *distp = reinterpret_cast<uint64_t *>(smem_raw + LY::distp);
    uint64_t *rckey = reinterpret_cast<uint64_t *>(smem_raw + LY::rckey);
    float *pr = reinterpret_cast<float *>(smem_raw + LY::pr);
    int *cnt = reinterpret_cast<int *>(smem_raw + LY::cnt);
    int *sel = reinterpret_cast<int *>(smem_raw + LY::sel);
    int *path = reinterpret_cast<int *>(smem_raw + LY::path);
    int *hslot = reinterpret_cast<int *>(smem_raw + LY::hslot);
    int *htok = reinterpret_cast<int *>(smem_raw + LY::htok);
    float *urow = reinterpret_cast<float *>(smem_raw + LY::urow);
    int *rcj = reinterpret_cast<int *>(smem_raw + LY::rcj);
    int *rcx = reinterpret_cast<int *>(smem_raw + LY::rcx);
    int *act = reinterpret_cast<int *>(smem_raw + LY::act);
    float *vstar = reinterpret_cast<float *>(smem_raw + LY::vstar);
    float *mnew = reinterpret_cast<float *>(smem_raw + LY::mnew);
    uint16_t *am = kG ? c.ssp_a : reinterpret_cast<uint16_t *>(smem_raw + LY::am);
    float *rowsT = reinterpret_cast<float *>(smem_raw + LY::rows);
    __shared__ int s_go, s_n, s_cur, s_flag[3], s_L, s_i, s_u, s_err, s_nrc, s_full;
    // The nearest expert with room at each step's labels, as a 64-bit
    // minimum of (distance, expert) beside the label buffers: the waves read
    // it instead of each reducing the labels of every expert.
    __shared__ uint64_t s_rkey[3];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int E = c.E, C = c.C, T = c.T;
    const int KS = K + 1;   // stride of the transposed rows
    uint16_t *toks = kG ? c.ssp_t : reinterpret_cast<uint16_t *>(smem_raw + LY::toks(E, K));
    const int e0 = wave * RW;   // this wave's rows
    const int rc_cap = small ? 0 : kSspRc;
    const int mn_cap = small ? 1 : ssp_mnew<Ep>();
    if (tid == 0) {
        int n = 0;
        s_go = ssp_pending<M>(c, &n) && n <= K && T <= 65536 ? 1 : 0;
        s_n = n;
        s_cur = ctrl->cur;
        s_err = 0;
        s_nrc = 0;
        s_full = 0;
        s_flag[0] = s_flag[1] = s_flag[2] = 0;
    }
    __syncthreads();
    if (!s_go) return;
    // State into LDS and registers: prices, counts, holder selectors, every
    // expert's held tokens, the slot matrix, the unassigned tokens' rows.
    for (int e = tid; e < Ep; e += kBlk) {
        const bool real = e < E;
        pr[e] = real ? c.prices[e] : 0.0f;
        int h = real ? ld_relaxed(&c.hcount[e]) : C;
        if (h < 0 || h > C) {
            flag_internal(ctrl);
            s_err = 1;
            h = C;
        }
        cnt[e] = h;
        sel[e] = real ? (ld_relaxed(&c.hsel[e]) & 1) : 0;
    }
    __syncthreads();
    // The token table and the slot matrix as the build kernel wrote them:
    // 16-byte loads, all in flight together (one element at a time, the
    // setup took 65 us of dependent loads at T = 32768).
    if constexpr (!kG) {
        const int nt16 = (E * C * 2) / 16;
        copy16_to_lds<kBlk>(reinterpret_cast<uint4 *>(toks),
                            reinterpret_cast<const uint4 *>(c.ssp_t), nt16);
        for (int i = nt16 * 8 + tid; i < E * C; i += kBlk) toks[i] = c.ssp_t[i];
        const int na16 = (E * E * 2) / 16;
        copy16_to_lds<kBlk>(reinterpret_cast<uint4 *>(am),
                            reinterpret_cast<const uint4 *>(c.ssp_a), na16);
        for (int i = na16 * 8 + tid; i < E * E; i += kBlk) am[i] = c.ssp_a[i];
    }
    if (tid < s_n) {
        int t = c.active[(int64_t)s_cur * T + tid];
        if (t < 0 || t >= T) {
            flag_internal(ctrl);
            s_err = 1;
            t = 0;
        }
        act[tid] = t;
    }
    __syncthreads();
    // The unassigned tokens' rows, transposed (all loads of the pass in flight).
    for (int q = tid; q < s_n * E; q += kBlk) {
        const int i = q / E, y = q - i * E;
        rowsT[y * KS + i] = c.S[(int64_t)act[i] * E + y];
    }
    float mreg[RW][CL];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int j = 0; j < CL; ++j) {
            const int x = lane + 64 * j;
            mreg[r][j] = (x < E && e0 + r < E) ? c.ssp_m[(int64_t)(e0 + r) * E + x] : INFINITY;
        }
    __syncthreads();
    int k = s_n;
    int augs = 0;
    while (k > 0 && !s_err) {
        // (1) Every unassigned token's best value (eight lanes per token),
        // then the sources' distances (a thread per expert).
        {
            const int i = tid >> 3, part = tid & 7;
            float m = -INFINITY;
            if (i < k)
                for (int y = part; y < E; y += 8) m = fmaxf(m, rowsT[y * KS + i] - pr[y]);
            m = fmaxf(m, grp_partner<1>(m));
            m = fmaxf(m, grp_partner<2>(m));
            m = fmaxf(m, grp_partner<4>(m));
            if (i < k && part == 0) vstar[i] = m;
        }
        if (tid == 0) {
            s_flag[0] = s_flag[1] = s_flag[2] = 0;
            s_rkey[0] = s_rkey[1] = s_rkey[2] = ~0ull;
        }
        __syncthreads();
        if (tid < Ep) {
            // Ties between tokens go to the lower token index: the list's
            // order comes from atomics and is not reproducible.
            const int x = tid;
            float best = INFINITY;
            int bi = 0, bt = 0x7fffffff;
            if (x < E) {
                const float px = pr[x];
                for (int i = 0; i < k; ++i) {
                    const float v = vstar[i] - (rowsT[x * KS + i] - px);
                    const int ti = act[i];
                    const bool t = (v < best) | ((v == best) & (ti < bt));
                    best = t ? v : best;
                    bi = t ? i : bi;
                    bt = t ? ti : bt;
                }
            }
            distp[x] = ssp_pack(best, kSspSrc + (uint32_t)bi);
            distp[Ep + x] = ~0ull;
            if (x < E && cnt[x] < C)
                atomicMin(reinterpret_cast<unsigned long long *>(&s_rkey[0]),
                          (unsigned long long)ssp_pack(best, (uint32_t)x));
        }
        // The arcs at the current prices: M(e,x) + p_x, and -p_e per row;
        // which of this lane's experts have room.
        float mp[kG ? 1 : RW][CL];
        float pxl[CL];
        bool room[CL];
#pragma unroll
        for (int j = 0; j < CL; ++j) {
            const int x = lane + 64 * j;
            const float px = x < E ? pr[x] : 0.0f;
            pxl[j] = px;
            room[j] = x < E && cnt[x] < C;
            if constexpr (!kG) {
#pragma unroll
                for (int r = 0; r < RW; ++r) mp[r][j] = mreg[r][j] + px;
            }
        }
        const float prow = lane < RW ? pr[e0 + lane] : 0.0f;   // lane r: price of row r
        float dused = INFINITY;                                 // lane r: dist row r was relaxed at
        __syncthreads();
        // (2) Bellman-Ford, one synchronous step per iteration: step `it`
        // reads buffer it % 3 and writes the next one (cleared a step
        // ahead), into which the owners fold the current labels and the
        // waves their strict improvements, as 64-bit minima of (distance,
        // predecessor): equal distances keep the lower expert, whatever
        // the order of the atomics, so the result does not depend on
        // scheduling. Only experts nearer than the nearest expert with room
        // (dcur, which every wave takes from the labels it reads) can lie on
        // the path or gain a price: a wave relaxes only those of its rows,
        // and only when their distance fell since it last relaxed them.
        int fin = 0;     // the buffer with the converged labels
        float D = INFINITY;
        int f = 0x7fffffff;   // the nearest expert with room
        for (int it = 0;; ++it) {
            const uint64_t *cur = distp + (it % 3) * Ep;
            uint64_t *nxt = distp + ((it + 1) % 3) * Ep;
            if (tid < Ep) {
                atomicMin(reinterpret_cast<unsigned long long *>(&nxt[tid]),
                          (unsigned long long)cur[tid]);
                distp[((it + 2) % 3) * Ep + tid] = ~0ull;
            }
            if (tid == 0) {
                atomicMin(reinterpret_cast<unsigned long long *>(&s_rkey[(it + 1) % 3]),
                          (unsigned long long)s_rkey[it % 3]);
                s_rkey[(it + 2) % 3] = ~0ull;
            }
            const float dnow = lane < RW ? ssp_dist(cur[e0 + lane]) : INFINITY;
            float dcol[CL];
#pragma unroll
            for (int j = 0; j < CL; ++j) {
                const int x = lane + 64 * j;
                dcol[j] = x < E ? ssp_dist(cur[x]) : -INFINITY;
            }
            const uint64_t rk = s_rkey[it % 3];
            const float dcur = rk == ~0ull ? INFINITY : ssp_dist(rk);
            const int fcur = rk == ~0ull ? 0x7fffffff : (int)(uint32_t)rk;
            const bool relax = lane < RW && dnow < dused && dnow < dcur;
            const uint64_t todo = __ballot(relax);
            dused = relax ? dnow : dused;
            float best[CL];
            int bj[CL];
#pragma unroll
            for (int j = 0; j < CL; ++j) {
                best[j] = INFINITY;
                bj[j] = 0;
            }
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                if (!((todo >> r) & 1)) continue;   // uniform
                const float de = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(dnow), r));
                const float q = de - __int_as_float(__builtin_amdgcn_readlane(__float_as_int(prow), r));
#pragma unroll
                for (int j = 0; j < CL; ++j) {
                    const float mpv = kG ? mreg[r][j] + pxl[j] : mp[kG ? 0 : r][j];
                    const float cand = fmaxf(q + mpv, de);
                    const bool t = cand < best[j];
                    best[j] = t ? cand : best[j];
                    bj[j] = t ? e0 + r : bj[j];
                }
            }
            bool imp = false;
#pragma unroll
            for (int j = 0; j < CL; ++j) {
                const int x = lane + 64 * j;
                if (best[j] < fminf(dcol[j], dcur)) {   // strict improvement (x < E)
                    atomicMin(reinterpret_cast<unsigned long long *>(&nxt[x]),
                              (unsigned long long)ssp_pack(best[j], (uint32_t)bj[j]));
                    if (room[j])
                        atomicMin(reinterpret_cast<unsigned long long *>(&s_rkey[(it + 1) % 3]),
                                  (unsigned long long)ssp_pack(best[j], (uint32_t)x));
                    imp = true;
                }
            }
            const int slot = it % 3;
            if (__ballot(imp) != 0 && lane == 0) s_flag[slot] = 1;
            if (tid == 0) s_flag[(it + 1) % 3] = 0;
            __syncthreads();
            if (!s_flag[slot]) {   // converged: cur holds the labels
                fin = it % 3;
                D = dcur;
                f = fcur;
                break;
            }
            if (it > Ep + 2) {   // shortest paths have at most E - 1 hops
                if (tid == 0) {
                    flag_internal(ctrl);
                    s_err = 1;
                }
                break;
            }
        }
        __syncthreads();
        if (s_err) break;
        const uint64_t *dfin = distp + fin * Ep;
        // (3) The path to the nearest expert with room (one lane).
        if (tid == 0) {
            int L = 0;
            bool ok = f < E && D < INFINITY;
            if (ok) {
                for (uint32_t lab = (uint32_t)dfin[f]; lab < kSspSrc; lab = (uint32_t)dfin[lab]) {
                    if (lab >= (uint32_t)E || ++L > E) {
                        ok = false;
                        break;
                    }
                }
            }
            if (ok) {
                int y = f;
                for (int j = L; j > 0; --j) {
                    path[j] = y;
                    y = (int)(uint32_t)dfin[y];
                }
                path[0] = y;
                const uint32_t i = (uint32_t)dfin[y] - kSspSrc;
                ok = i < (uint32_t)k;
                s_i = ok ? (int)i : 0;
                s_u = ok ? act[s_i] : 0;
            }
            if (!ok) {
                flag_internal(ctrl);
                s_err = 1;
            }
            s_L = L;
        }
        __syncthreads();
        if (s_err) break;
        const int L = s_L, u = s_u, iu = s_i;
        const int nmn = L + 1 < mn_cap ? L + 1 : mn_cap;   // path experts through LDS
        // (A) New prices; the slot each expert on the path hands on and its
        // token; the columns whose cheapest token leaves (queued for a
        // recompute); the placed token's row.
        for (int y = tid; y < E; y += kBlk) {
            pr[y] = pr[y] + fmaxf(D - ssp_dist(dfin[y]), 0.0f);
            urow[y] = rowsT[y * KS + iu];
        }
        for (int j = tid; j < L; j += kBlk) {
            const int e = path[j];
            const int q = am[e * E + path[j + 1]];
            hslot[j] = q;
            htok[j] = q < cnt[e] ? (int)toks[e * C + q] : 0;
            if (q >= cnt[e]) {
                flag_internal(ctrl);
                s_err = 1;
            }
        }
        for (int i = tid; i < L * E; i += kBlk) {
            const int j = i / E, x = i - j * E;
            const int e = path[j];
            if (am[e * E + x] == am[e * E + path[j + 1]]) {
                const int at = j < mn_cap ? atomicAdd(&s_nrc, 1) : rc_cap;
                if (at < rc_cap) {
                    rcj[at] = j;
                    rcx[at] = x;
                    rckey[j * Ep + x] = ~0ull;
                } else {
                    s_full = 1;   // the path's rows are recomputed whole
                }
            }
        }
        __syncthreads();
        if (s_err) break;
        // (B) Apply the path in the holder tables; one flat pass over every
        // global read of the step, so that they are all in flight together:
        // the received tokens' rows of the first kSspMnew path experts (into
        // LDS), and each queued column's entries over its expert's slots
        // (into a 64-bit minimum of (order-preserving value, slot)).
        const int nrc = s_nrc < rc_cap ? s_nrc : rc_cap;
        const int full = s_full;
        auto token_in = [&](int j) -> int { return j == 0 ? u : htok[j - 1]; };
        for (int j = tid; j <= L; j += kBlk) {
            const int e = path[j];
            const int q = j < L ? hslot[j] : cnt[e];
            if (q < C) {
                int overflow = 0;
                uint64_t *hold = c.holders + (int64_t)sel[e] * T + (int64_t)e * C;
                hold[q] = M::make_key(pr[e], token_in(j), &overflow);
                if (overflow) ctrl->overflow = 1;
            } else {
                flag_internal(ctrl);
                s_err = 1;
            }
        }
        {
            const int nm = nmn * E;
            const int nitems = nm + nrc * C;
#pragma unroll 4
            for (int i = tid; i < nitems; i += kBlk) {
                if (i < nm) {
                    const int j = i / E, x = i - j * E;
                    const int e = path[j];
                    float v;
                    if (j == 0) {
                        v = urow[e] - urow[x];
                    } else {
                        const int tin = htok[j - 1];
                        v = c.S[(int64_t)tin * E + e] - c.S[(int64_t)tin * E + x];
                    }
                    mnew[j * Ep + x] = v;
                } else {
                    const int i2 = i - nm;
                    const int p = i2 / C, q = i2 - p * C;
                    const int j = rcj[p], y = rcx[p];
                    const int e = path[j];
                    if (q < cnt[e]) {
                        const int t = q == hslot[j] ? token_in(j) : (int)toks[e * C + q];
                        const float v = c.S[(int64_t)t * E + e] - c.S[(int64_t)t * E + y];
                        atomicMin(reinterpret_cast<unsigned long long *>(&rckey[j * Ep + y]),
                                  (unsigned long long)ssp_entry(v, q));
                    }
                }
            }
        }
        // Path experts beyond the LDS rows: their owners read directly.
        for (int j = mn_cap; j <= L; ++j) {
            const int e = path[j];
            if (e < e0 || e >= e0 + RW) continue;   // uniform: rows are the wave's
            const int rr = e - e0;
            const int tin = token_in(j);
            const int qin = j < L ? hslot[j] : cnt[e];
            const float se = c.S[(int64_t)tin * E + e];
#pragma unroll
            for (int jj = 0; jj < CL; ++jj) {
                const int x = lane + 64 * jj;
                if (x >= E) continue;
                if (j < L && am[e * E + x] == hslot[j]) continue;   // recomputed whole
                const float v = se - c.S[(int64_t)tin * E + x];
                float cv = 0.0f;
#pragma unroll
                for (int r = 0; r < RW; ++r) cv = r == rr ? mreg[r][jj] : cv;
                if (v < cv) {
#pragma unroll
                    for (int r = 0; r < RW; ++r) mreg[r][jj] = r == rr ? v : mreg[r][jj];
                    am[e * E + x] = (uint16_t)qin;
                }
            }
        }
        __syncthreads();
        if (s_err) break;
        // (C) Owners take, for each path expert they own, the recomputed
        // columns and the minimum with the received row elsewhere.
        for (int j = 0; j < nmn; ++j) {
            const int e = path[j];
            if (e < e0 || e >= e0 + RW) continue;   // uniform
            const int rr = e - e0;
            const int qin = j < L ? hslot[j] : cnt[e];
#pragma unroll
            for (int jj = 0; jj < CL; ++jj) {
                const int x = lane + 64 * jj;
                if (x >= E) continue;
                float v;
                int q;
                if (j < L && am[e * E + x] == hslot[j]) {
                    const uint64_t key = rckey[j * Ep + x];
                    v = f32_unord((uint32_t)(key >> 32));
                    q = (int)(uint32_t)key;
                } else {
                    v = mnew[j * Ep + x];
                    q = qin;
                    float cv = 0.0f;
#pragma unroll
                    for (int r = 0; r < RW; ++r) cv = r == rr ? mreg[r][jj] : cv;
                    if (!(v < cv)) continue;
                }
#pragma unroll
                for (int r = 0; r < RW; ++r) mreg[r][jj] = r == rr ? v : mreg[r][jj];
                am[e * E + x] = (uint16_t)q;
            }
        }
        if (full) {
            // More recomputes than the list holds (or a path longer than the
            // LDS rows): every row of the path's experts that hand on a
            // token is recomputed, all threads splitting the slots, with one
            // 64-bit minimum per column (distp is free until the next search).
            for (int j = 0; j < L; ++j) {
                const int e = path[j];
                const int q_out = hslot[j];
                const int t_in = token_in(j);
                __syncthreads();
                if (tid < E) distp[tid] = ~0ull;
                __syncthreads();
#pragma unroll
                for (int jj = 0; jj < CL; ++jj) {
                    const int x = lane + 64 * jj;
                    if (x >= E) continue;
                    uint64_t bk = ~0ull;
                    for (int q = wave; q < cnt[e]; q += kW) {
                        const int t = q == q_out ? t_in : (int)toks[e * C + q];
                        const float v = c.S[(int64_t)t * E + e] - c.S[(int64_t)t * E + x];
                        const uint64_t key = ssp_entry(v, q);
                        bk = key < bk ? key : bk;
                    }
                    atomicMin(reinterpret_cast<unsigned long long *>(&distp[x]),
                              (unsigned long long)bk);
                }
                __syncthreads();
                if (e >= e0 && e < e0 + RW) {
                    const int rr = e - e0;
#pragma unroll
                    for (int jj = 0; jj < CL; ++jj) {
                        const int x = lane + 64 * jj;
                        if (x >= E) continue;
                        const uint64_t bk = distp[x];
                        const float v = f32_unord((uint32_t)(bk >> 32));
#pragma unroll
                        for (int r = 0; r < RW; ++r) mreg[r][jj] = r == rr ? v : mreg[r][jj];
                        am[e * E + x] = (uint16_t)(uint32_t)bk;
                    }
                }
            }
        }
        // The token lists, the unassigned list and the free expert's count
        // follow the path.
        for (int j = tid; j <= L; j += kBlk) {
            const int e = path[j];
            const int q = j < L ? hslot[j] : cnt[e];
            if (q < C) toks[e * C + q] = (uint16_t)token_in(j);
        }
        for (int y = tid; y < E; y += kBlk) rowsT[y * KS + iu] = rowsT[y * KS + k - 1];
        if (tid == 0) {
            act[iu] = act[k - 1];
            s_nrc = 0;
            s_full = 0;
        }
        __syncthreads();
        if (tid == 0) cnt[f] += 1;
        ++augs;
        --k;
    }
    __syncthreads();
    // Hand the state back: the phase is complete (or flagged).
    for (int e = tid; e < E; e += kBlk) {
        c.prices[e] = pr[e];
        c.hcount[e] = cnt[e];
    }
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        ctrl->augmentations += augs;
        if (!s_err) {
            ctrl->active_count[s_cur] = 0;
            ctrl->active_count[s_cur ^ 1] = 0;
            if (ctrl->last_phase) ctrl->done = 1;
        }
    }
}

// Wave-wide maximum of (v, i), ties to the lower i; every lane ends with it.
template <class V>
__device__ inline V readlane_v(V v, int l) {
    if constexpr (sizeof(V) == 8) {
        uint64_t u;
        __builtin_memcpy(&u, &v, 8);
        const uint64_t r = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l) |
                           ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l)
                            << 32);
        V out;
        __builtin_memcpy(&out, &r, 8);
        return out;
    } else {
        uint32_t u;
        __builtin_memcpy(&u, &v, 4);
        const uint32_t r = (uint32_t)__builtin_amdgcn_readlane((int)u, l);
        V out;
        __builtin_memcpy(&out, &r, 4);
        return out;
    }
}
template <int OFF, class V>
__device__ __attribute__((always_inline)) inline void max_pair_step(V &v, int &i) {
    const V ov = grp_partner<OFF>(v);
    const int oi = grp_partner<OFF>(i);
    const bool t = (ov > v) | ((ov == v) & (oi < i));
    v = t ? ov : v;
    i = t ? oi : i;
}
template <class V>
__device__ inline void wave_max_pair(V &v, int &i) {
    max_pair_step<1>(v, i);
    max_pair_step<2>(v, i);
    max_pair_step<4>(v, i);
    max_pair_step<8>(v, i);
    V rv = readlane_v(v, 0);
    int ri = __builtin_amdgcn_readlane(i, 0);
#pragma unroll
    for (int q = 1; q < 4; ++q) {
        const V ov = readlane_v(v, 16 * q);
        const int oi = __builtin_amdgcn_readlane(i, 16 * q);
        const bool t = (ov > rv) | ((ov == rv) & (oi < ri));
        rv = t ? ov : rv;
        ri = t ? oi : ri;
    }
    v = rv;
    i = ri;
}

// ------------------------------------------------- single-workgroup solve --
//
// A problem of at most kSmallT tokens and kSmallE experts is solved whole by
// one workgroup (one per problem of a batch, all in one launch), with every
// piece of mutable state in LDS: the prices, each expert's C held keys with
// the lowest of them and its slot, the active tokens and the round's bids
// grouped by expert. It follows the same rules as the multi-kernel path:
// Jacobi bids from the score summaries against the prices at the start of
// the round; an expert keeps the C largest keys of its holders and its bids
// (streamed through "a larger key replaces the lowest held key", which gives
// the same set for any arrival order); the lowest held key is the expert's
// price once it is full; epsilon phases begun by begin_phase_scalar, and the
// duality check between phases with the same allowance and decision. The
// result is therefore deterministic and carries the same guarantee.
constexpr int kSmallThreads = 1024;
constexpr int kSmallWaves = kSmallThreads / 64;
constexpr int kSmallT = 2048;
constexpr int kSmallE = 256;
constexpr int kSmallRows = 4;   // tokens a bidding group handles per pass (loads first)
constexpr int kSmallBatch = 8;  // batches from this size take the single-workgroup rounds
constexpr int kSmallSoloT = 512;   // and single problems up to this many tokens

struct SmallLds {
    size_t pr, cnt, mk, ms, bcnt, boff, bfill, tch, hk, actA, actB, bkey, bexp, bsort, total;
};
__host__ __device__ inline SmallLds small_lds(int T, int E, int vbytes) {
    SmallLds L{};
    size_t off = 0;
    L.pr = off;    off = eng_align(off + (size_t)E * vbytes);
    L.cnt = off;   off = eng_align(off + (size_t)E * 4);
    L.mk = off;    off = eng_align(off + (size_t)E * 8);
    L.ms = off;    off = eng_align(off + (size_t)E * 4);
    L.bcnt = off;  off = eng_align(off + (size_t)E * 4);
    L.boff = off;  off = eng_align(off + (size_t)E * 4);
    L.bfill = off; off = eng_align(off + (size_t)E * 4);
    L.tch = off;   off = eng_align(off + (size_t)E * 4);
    L.hk = off;    off = eng_align(off + (size_t)T * 8);
    L.actA = off;  off = eng_align(off + (size_t)T * 4);
    L.actB = off;  off = eng_align(off + (size_t)T * 4);
    L.bkey = off;  off = eng_align(off + (size_t)T * 8);
    L.bexp = off;  off = eng_align(off + (size_t)T * 4);
    L.bsort = off; off = eng_align(off + (size_t)T * 8);
    L.total = off;
    return L;
}

// Wave-wide minimum of (key, slot); every lane ends with it.
__device__ inline void wave_min_key(uint64_t &k, int &q) {
#define BASE_KMIN_STEP(OFF)                                  \
    {                                                        \
        const uint64_t ok = grp_partner<OFF>(k);             \
        const int oq = grp_partner<OFF>(q);                  \
        const bool t = ok < k;                               \
        k = t ? ok : k;                                      \
        q = t ? oq : q;                                      \
    }
    BASE_KMIN_STEP(1)
    BASE_KMIN_STEP(2)
    BASE_KMIN_STEP(4)
    BASE_KMIN_STEP(8)
#undef BASE_KMIN_STEP
    uint64_t rk = readlane_v(k, 0);
    int rq = __builtin_amdgcn_readlane(q, 0);
#pragma unroll
    for (int l = 1; l < 4; ++l) {
        const uint64_t ok = readlane_v(k, 16 * l);
        const int oq = __builtin_amdgcn_readlane(q, 16 * l);
        const bool t = ok < rk;
        rk = t ? ok : rk;
        rq = t ? oq : rq;
    }
    k = rk;
    q = rq;
}

// Top-2 of tokens tk[u] (valid where ok[u]) from their summaries, against
// prices pr (the whole block calls; the summary loads go first).
template <class M, int G>
__device__ inline void small_top2(const Ctx<M> &c, const int (&tk)[kSmallRows],
                                  const bool (&ok)[kSmallRows], int gl,
                                  const typename M::value_t *pr, typename M::value_t pmin,
                                  typename M::value_t (&v1)[kSmallRows], int (&e1)[kSmallRows],
                                  typename M::value_t (&v2)[kSmallRows],
                                  typename M::value_t (&s1)[kSmallRows]) {
    uint32_t sw[kSmallRows][4];
#pragma unroll
    for (int u = 0; u < kSmallRows; ++u) {
        sw[u][0] = sw[u][1] = sw[u][2] = sw[u][3] = 0;
        if (ok[u]) load_summary(c.sums, tk[u], gl, sw[u]);
    }
#pragma unroll
    for (int u = 0; u < kSmallRows; ++u)
        top2_summary<M, G>(c, sw[u], tk[u], ok[u], gl, pr, pmin, v1[u], e1[u], v2[u], s1[u]);
}

// One launch runs from the state the control block and the holder tables
// describe (a phase just begun, a phase the shortest-path finish completed,
// or one in progress) through as many rounds and phases as it can: it stops
// when the solve is done, when the round bound is reached, or when at most
// `cap` tokens of a phase are left (cap > 0: the shortest-path finish takes
// them; the next launch continues after it), handing the state back in the
// multi-kernel path's layout (holder table 0, active list 0).
template <class M, int G>
__global__ __launch_bounds__(kSmallThreads) void small_solve_kernel(Ctx<M> c0, AssignParams p,
                                                                    int cap) {
    using value_t = typename M::value_t;
    const Ctx<M> c = c0.at(blockIdx.y);
    SolveCtrl *ctrl = c.ctrl;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int E = c.E, C = c.C, T = c.T;
    const SmallLds L = small_lds(T, E, (int)sizeof(value_t));
    value_t *pr = reinterpret_cast<value_t *>(smem_raw + L.pr);
    int *cnt = reinterpret_cast<int *>(smem_raw + L.cnt);
    uint64_t *mk = reinterpret_cast<uint64_t *>(smem_raw + L.mk);
    int *ms = reinterpret_cast<int *>(smem_raw + L.ms);
    int *bcnt = reinterpret_cast<int *>(smem_raw + L.bcnt);
    int *boff = reinterpret_cast<int *>(smem_raw + L.boff);
    int *bfill = reinterpret_cast<int *>(smem_raw + L.bfill);
    int *tch = reinterpret_cast<int *>(smem_raw + L.tch);
    uint64_t *hk = reinterpret_cast<uint64_t *>(smem_raw + L.hk);
    int *act = reinterpret_cast<int *>(smem_raw + L.actA);
    int *nxt = reinterpret_cast<int *>(smem_raw + L.actB);
    uint64_t *bkey = reinterpret_cast<uint64_t *>(smem_raw + L.bkey);
    int *bexp = reinterpret_cast<int *>(smem_raw + L.bexp);
    uint64_t *bsort = reinterpret_cast<uint64_t *>(smem_raw + L.bsort);
    __shared__ int s_n, s_nnext, s_ntch, s_stop, s_last;
    __shared__ value_t s_eps, s_early_eps;
    __shared__ double s_part[kSmallWaves], s_pmax[kSmallWaves];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int per = kSmallThreads / G;
    const int gid = tid / G;
    const int gl = lane & (G - 1);
    const bool checks = !(p.flags & BASE_ASSIGN_FULL_SCHEDULE);

    __shared__ int s_all, s_cur;
    if (tid == 0) {
        s_stop = ctrl->done || ctrl->internal_error;
        s_all = ctrl->all_active;
        s_cur = ctrl->cur & 1;
        s_n = s_all ? T : ld_relaxed(&ctrl->active_count[s_cur]);
        if (s_n < 0 || s_n > T) {
            flag_internal(ctrl);
            s_stop = 1;
        }
        s_ntch = 0;
        s_eps = (value_t)ctrl->eps;
        s_last = ctrl->last_phase;
        // Phases with epsilon above this end early (see end_round).
        s_early_eps = c.early_n < 0 ? (value_t)0 : (value_t)(kEarlyRatio * ctrl->eps_final_eff);
    }
    __syncthreads();
    if (s_stop) return;
    // The state: prices, every expert's holders (with the lowest key and its
    // slot), the active tokens.
    for (int e = tid; e < E; e += kSmallThreads) {
        pr[e] = c.prices[e];
        int h = s_all ? 0 : ld_relaxed(&c.hcount[e]);
        if (h < 0 || h > C) {
            flag_internal(ctrl);
            h = 0;
        }
        cnt[e] = h;
        bcnt[e] = 0;
        bfill[e] = 0;
    }
    __syncthreads();
    for (int i = tid; i < T; i += kSmallThreads) {
        const int e = i / C, q = i - e * C;
        hk[i] = q < cnt[e] ? c.holders[(int64_t)(c.hsel[e] & 1) * T + i] : ~0ull;
        if (s_all) act[i] = i;
        else if (i < s_n) {
            const int t = c.active[(int64_t)s_cur * T + i];
            act[i] = (t >= 0 && t < T) ? t : 0;
        }
    }
    __syncthreads();
    for (int e = wave; e < E; e += kSmallWaves) {
        uint64_t m = ~0ull;
        int mq = 0;
        for (int q = lane; q < cnt[e]; q += 64) {
            const uint64_t v = hk[(size_t)e * C + q];
            if (v < m) {
                m = v;
                mq = q;
            }
        }
        wave_min_key(m, mq);
        if (lane == 0) {
            mk[e] = m;
            ms[e] = mq;
        }
    }
    __syncthreads();
    // Prices only rise: their lowest value now bounds them for the whole solve.
    const value_t pmin = block_min_price<M>(pr, E);
    const int ctrl_rounds0 = ctrl->rounds;
    int rounds = 0;
    unsigned long long bids = 0;
    const int early_lim = c.early_n > 0 ? c.early_n : -c.early_n;
    while (!s_stop) {
        const int n = s_n;
        // A large-epsilon phase above the last ends early, unchecked (see end_round).
        const bool early = n > 0 && n <= early_lim && !s_last && s_eps > s_early_eps;
        if (n == 0 || early) {
            // The phase is complete (every expert full): stop after the last
            // phase; otherwise the duality check, then the next phase.
            if (s_last) {
                if (tid == 0) ctrl->done = 1;
                break;
            }
            if (checks && !early) {
                // D(p) - objective as a sum of per-token slacks over the held
                // tokens (slot order), in double, in a fixed order.
                double acc = 0.0;
                for (int i0 = 0; i0 < T; i0 += per * kSmallRows) {
                    value_t v1[kSmallRows], v2[kSmallRows], s1[kSmallRows];
                    int e1[kSmallRows], tk[kSmallRows];
                    bool ok[kSmallRows];
#pragma unroll
                    for (int u = 0; u < kSmallRows; ++u) {
                        const int i = i0 + gid + u * per;
                        int t = i < T ? key_token(hk[i]) : 0;
                        tk[u] = (t >= 0 && t < T) ? t : 0;
                        ok[u] = i < T;
                    }
                    small_top2<M, G>(c, tk, ok, gl, pr, pmin, v1, e1, v2, s1);
#pragma unroll
                    for (int u = 0; u < kSmallRows; ++u) {
                        const int i = i0 + gid + u * per;
                        if (i < T && gl == 0) {
                            const int e = i / C;
                            acc += (double)v1[u] -
                                   ((double)M::load(c.S, (int64_t)tk[u] * E + e, c.scale) -
                                    (double)pr[e]);
                        }
                    }
                }
                double pm = 0.0;
                for (int e = tid; e < E; e += kSmallThreads) pm = fmax(pm, fabs((double)pr[e]));
#pragma unroll
                for (int off = 32; off > 0; off >>= 1) {
                    acc += __shfl_xor(acc, off);
                    pm = fmax(pm, __shfl_xor(pm, off));
                }
                if (lane == 0) {
                    s_part[wave] = acc;
                    s_pmax[wave] = pm;
                }
                __syncthreads();
                if (tid == 0) {
                    double gap = 0.0, pmax = 0.0;
                    for (int w = 0; w < kSmallWaves; ++w) {
                        gap += s_part[w];
                        pmax = fmax(pmax, s_pmax[w]);
                    }
                    double allowance = 0.0;
                    if (!M::kInteger) {
                        const double smax = fmax(fabs((double)f32_unord(ctrl->smax_ord)),
                                                 fabs((double)f32_unord(ctrl->smin_ord)));
                        allowance = (double)T * ldexp(smax + pmax, -22);
                    }
                    if (gap + allowance <= (double)T * ctrl->eps_final_eff) {
                        ctrl->certified = 1;
                        ctrl->done = 1;
                        s_stop = 1;
                    } else {
                        ctrl->check_gap = gap + allowance;
                    }
                }
                __syncthreads();
                if (s_stop) break;
            }
            if (tid == 0) {
                begin_phase_scalar(ctrl, p, T);
                s_eps = (value_t)ctrl->eps;
                s_last = ctrl->last_phase;
                s_n = T;
            }
            for (int e = tid; e < E; e += kSmallThreads) {
                cnt[e] = 0;
                mk[e] = ~0ull;
                ms[e] = 0;
            }
            for (int i = tid; i < T; i += kSmallThreads) act[i] = i;
            __syncthreads();
            continue;
        }
        if (cap > 0 && n <= cap) break;   // the shortest-path finish takes the rest
        if (ctrl_rounds0 + rounds >= p.max_rounds) {
            if (tid == 0) {
                ctrl->not_converged = 1;
                ctrl->done = 1;
            }
            break;
        }
        // (1) Bids against the prices at the start of the round.
        const value_t eps = s_eps;
        for (int i0 = 0; i0 < n; i0 += per * kSmallRows) {
            value_t v1[kSmallRows], v2[kSmallRows], s1[kSmallRows];
            int e1[kSmallRows], tk[kSmallRows];
            bool ok[kSmallRows];
#pragma unroll
            for (int u = 0; u < kSmallRows; ++u) {
                const int i = i0 + gid + u * per;
                ok[u] = i < n;
                tk[u] = ok[u] ? act[i] : 0;
            }
            small_top2<M, G>(c, tk, ok, gl, pr, pmin, v1, e1, v2, s1);
#pragma unroll
            for (int u = 0; u < kSmallRows; ++u) {
                const int i = i0 + gid + u * per;
                if (i < n && gl == 0) {
                    int ex = e1[u];
                    value_t sc = s1[u];
                    if (ex >= E) {
                        ex = 0;
                        sc = 0;   // with v2 = lowest the bid overflows and is flagged
                    }
                    const value_t bid = (value_t)((sc - v2[u]) + eps);
                    int overflow = 0;
                    const uint64_t key = M::make_key(bid, tk[u], &overflow);
                    if (overflow) ctrl->overflow = 1;
                    bkey[i] = key;
                    bexp[i] = ex;
                    if (atomicAdd(&bcnt[ex], 1) == 0) tch[atomicAdd(&s_ntch, 1)] = ex;
                }
            }
        }
        __syncthreads();
        const int nt = s_ntch < E ? s_ntch : E;
        // (2) Offsets of the touched experts' bids (one wave).
        if (wave == 0) {
            int base = 0;
            for (int j0 = 0; j0 < nt; j0 += 64) {
                const int j = j0 + lane;
                const int cj = j < nt ? bcnt[tch[j]] : 0;
                int incl = cj;
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const int o = __shfl_up(incl, off);
                    if (lane >= off) incl += o;
                }
                if (j < nt) boff[tch[j]] = base + incl - cj;
                base += __shfl(incl, 63);
            }
        }
        if (tid == 0) s_nnext = 0;
        __syncthreads();
        // (3) The bids grouped by expert.
        for (int i = tid; i < n; i += kSmallThreads) {
            const int e = bexp[i];
            const int pos = boff[e] + atomicAdd(&bfill[e], 1);
            if (pos < T) bsort[pos] = bkey[i];
        }
        __syncthreads();
        // (4) Each touched expert streams its bids through its held keys, one
        // wave per expert (touched experts dealt to the waves in turn: a
        // loop whose trip count is the same for every lane of a wave, so
        // the wave stays converged through it). Lane 0 writes the LDS state;
        // the wave's LDS accesses take effect in program order.
        for (int j = wave; j < nt; j += kSmallWaves) {
            const int e = tch[j];
            const int nb = bcnt[e];
            const int b0 = boff[e];
            uint64_t *h = hk + (size_t)e * C;
            int ce = cnt[e];
            uint64_t mke = mk[e];
            int mse = ms[e];
            for (int k = 0; k < nb && b0 + k < T; ++k) {
                const uint64_t b = bsort[b0 + k];
                int out = -1;
                if (ce < C) {
                    if (lane == 0) h[ce] = b;
                    if (b < mke) {
                        mke = b;
                        mse = ce;
                    }
                    ++ce;
                } else if (b > mke) {
                    out = key_token(mke);
                    if (lane == 0) h[mse] = b;
                    asm volatile("" ::: "memory");
                    uint64_t m = ~0ull;
                    int mq = 0;
                    for (int q = lane; q < C; q += 64) {
                        const uint64_t v = h[q];
                        if (v < m) {
                            m = v;
                            mq = q;
                        }
                    }
                    wave_min_key(m, mq);
                    mke = m;
                    mse = mq;
                } else {
                    out = key_token(b);
                }
                if (out >= 0 && lane == 0) {
                    const int at = atomicAdd(&s_nnext, 1);
                    if (at < T && out >= 0 && out < T) nxt[at] = out;
                    else flag_internal(ctrl);
                }
                asm volatile("" ::: "memory");
            }
            if (lane == 0) {
                cnt[e] = ce;
                mk[e] = mke;
                ms[e] = mse;
                if (ce == C) pr[e] = M::key_bid(mke);
                bcnt[e] = 0;
                bfill[e] = 0;
            }
        }
        __syncthreads();
        rounds += 1;
        bids += (unsigned long long)n;
        {
            int *tmp = act;
            act = nxt;
            nxt = tmp;
        }
        if (tid == 0) {
            s_n = s_nnext < T ? s_nnext : T;
            s_ntch = 0;
            if (ctrl->internal_error) s_stop = 1;
        }
        __syncthreads();
    }
    __syncthreads();
    // Hand the state back in the multi-kernel path's layout (holder table 0).
    for (int e = tid; e < E; e += kSmallThreads) {
        c.prices[e] = pr[e];
        c.hcount[e] = cnt[e];
        c.hsel[e] = 0;
        c.bcount[e] = 0;
    }
    for (int i = tid; i < T; i += kSmallThreads) {
        const int e = i / C, q = i - e * C;
        if (q < cnt[e]) c.holders[i] = hk[i];
    }
    for (int i = tid; i < s_n; i += kSmallThreads) c.active[i] = act[i];
    if (tid == 0) {
        ctrl->rounds += rounds;
        ctrl->bids += bids;
        ctrl->cur = 0;
        ctrl->all_active = 0;
        ctrl->active_count[0] = s_n;
        ctrl->active_count[1] = 0;
        ctrl->pad0 = 0;
    }
}

// ------------------------------------------------------------- finalising --

// The finalising kernels write assign and perm from the holder tables. An
// expert's rows of perm are its tokens in ascending order; with at most
// kRankMaxC tokens per expert they are ranked in LDS, expert by expert
// (larger C takes the counting sort below over assign instead).
constexpr int kRankMaxC = 1024;

// out[rank of tok[i] among tok[0..n)] = tok[i] (ascending order for distinct
// tokens). tok has room for n rounded up to 4; entries from n on are padded
// here. rank < n whatever the values, so the writes stay in out[0..n).
__device__ inline void rank_write(int *tok, int n, int32_t *out) {
    const int n4 = (n + 3) & ~3;
    for (int i = n + (int)threadIdx.x; i < n4; i += blockDim.x) tok[i] = 0x7fffffff;
    __syncthreads();
    const int4 *t4 = reinterpret_cast<const int4 *>(tok);
    for (int i = threadIdx.x; i < n; i += blockDim.x) {
        const int t = tok[i];
        int r = 0;
        for (int j = 0; j < n4 / 4; ++j) {
            const int4 q = t4[j];
            r += (q.x < t) + (q.y < t) + (q.z < t) + (q.w < t);
        }
        out[r] = t;
    }
    __syncthreads();
}

// One block per expert: assign[t] = e for every held token (the prologue set
// every entry to -1), the expert's rows of perm when C <= kRankMaxC (its
// tokens in ascending order, then -1 for the rows of an expert that is not
// full), its price into prices_out (when not NULL), and a count of the
// experts that are not full.
template <class M>
__global__ __launch_bounds__(256) void finalise_kernel(Ctx<M> c0, int32_t *assign, int32_t *perm,
                                                       typename M::value_t *prices_out,
                                                       int rank_perm) {
    const Ctx<M> c = c0.at(blockIdx.y);
    assign += (int64_t)blockIdx.y * c.T;
    perm += (int64_t)blockIdx.y * c.T;
    __shared__ __align__(16) int tok[kRankMaxC];
    const int e = blockIdx.x;
    int h = c.hcount[e];
    if (h < 0 || h > c.C) {
        if (threadIdx.x == 0) flag_internal(c.ctrl);
        h = h < 0 ? 0 : c.C;
    }
    const uint64_t *hold = c.holders + (int64_t)(c.hsel[e] & 1) * c.T + (int64_t)e * c.C;
    const bool ranked = rank_perm != 0;
    for (int i = threadIdx.x; i < h; i += blockDim.x) {
        const int t = key_token(hold[i]);
        const bool ok = t >= 0 && t < c.T;
        if (ok) assign[t] = e;
        else flag_internal(c.ctrl);
        if (ranked) tok[i] = ok ? t : 0x7fffffff;
    }
    if (threadIdx.x == 0) {
        if (h != c.C) atomicAdd(&c.ctrl->unconverged_experts, 1);
        if (prices_out != nullptr) prices_out[(int64_t)blockIdx.y * c.E + e] = c.prices[e];
    }
    if (!ranked) return;
    __syncthreads();
    rank_write(tok, h, perm + (int64_t)e * c.C);
    for (int i = h + (int)threadIdx.x; i < c.C; i += blockDim.x) perm[(int64_t)e * c.C + i] = -1;
}

// After the greedy completion (one block per expert): the rows of perm of
// every expert that took tokens in it, ranked again (complete_kernel marks
// them in the overflow-expert list, unused once the rounds have ended).
template <class M>
__global__ __launch_bounds__(256) void rank_filled_kernel(Ctx<M> c0, int32_t *perm) {
    const Ctx<M> c = c0.at(blockIdx.y);
    perm += (int64_t)blockIdx.y * c.T;
    __shared__ __align__(16) int tok[kRankMaxC];
    const int e = blockIdx.x;
    if (!ld_relaxed(&c.ctrl->fell_back) || c.ovf_exp[e] == 0) return;
    int h = c.hcount[e];
    if (h < 0 || h > c.C) {
        if (threadIdx.x == 0) flag_internal(c.ctrl);
        h = h < 0 ? 0 : c.C;
    }
    const uint64_t *hold = c.holders + (int64_t)(c.hsel[e] & 1) * c.T + (int64_t)e * c.C;
    for (int i = threadIdx.x; i < h; i += blockDim.x) {
        const int t = key_token(hold[i]);
        tok[i] = (t >= 0 && t < c.T) ? t : 0x7fffffff;
    }
    __syncthreads();
    rank_write(tok, h, perm + (int64_t)e * c.C);
    for (int i = h + (int)threadIdx.x; i < c.C; i += blockDim.x) perm[(int64_t)e * c.C + i] = -1;
}

int lanes_per_token(int64_t E);

// The duality gap of the result (statistics only): D(p) - objective =
//     sum_t [max_e (S[t,e] - p[e]) - S[t, a_t]] + C sum_e p[e],
// per-token values in the solve's arithmetic, the sum in double. For a
// balanced assignment it bounds the distance to the optimum from above.
template <class M, int G>
__global__ __launch_bounds__(kThreads) void dual_gap_kernel(Ctx<M> c0, const int32_t *assign) {
    using value_t = typename M::value_t;
    const Ctx<M> c = c0.at(blockIdx.y);
    assign += (int64_t)blockIdx.y * c.T;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    value_t *pr = reinterpret_cast<value_t *>(smem_raw);
    __shared__ double part[kThreads / 64];
    for (int e = threadIdx.x; e < c.E; e += kThreads) pr[e] = c.prices[e];
    __syncthreads();
    const int gl = lane_id() & (G - 1);
    const int per_block = kThreads / G;
    const int ngroups = per_block * gridDim.x;
    const int n_round = ((c.T + ngroups - 1) / ngroups) * ngroups;
    double acc = 0.0;
    for (int t = blockIdx.x * per_block + threadIdx.x / G; t < n_round; t += ngroups) {
        const bool valid = t < c.T;
        value_t v1, v2, s1;
        int e1;
        top2_token<M, G>(c, valid ? t : 0, valid, pr, v1, e1, v2, s1);
        if (valid && gl == 0) {
            int a = assign[t];
            a = (a >= 0 && a < c.E) ? a : 0;
            acc += (double)v1 - (double)M::load(c.S, (int64_t)t * c.E + a, c.scale);
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < 64) {
        double sp = 0.0;
        for (int e = threadIdx.x; e < c.E; e += 64) sp += (double)pr[e];
        acc += (double)c.C * sp;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (lane_id() == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        double sum = 0.0;
        for (int w = 0; w < kThreads / 64; ++w) sum += part[w];
        atomicAdd(&c.ctrl->dual_gap, sum);
    }
}

template <class M>
hipError_t launch_dual_gap(const Ctx<M> &c, int B, const int32_t *assign, hipStream_t s) {
    const size_t pr_bytes = (size_t)c.E * sizeof(typename M::value_t);
    int blocks = (int)((c.T + 255) / 256);
    if (blocks > 1024) blocks = 1024;
    const dim3 grid(blocks, B);
    switch (lanes_per_token(c.E)) {
        case 1: hipLaunchKernelGGL((dual_gap_kernel<M, 1>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
        case 2: hipLaunchKernelGGL((dual_gap_kernel<M, 2>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
        case 4: hipLaunchKernelGGL((dual_gap_kernel<M, 4>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
        case 8: hipLaunchKernelGGL((dual_gap_kernel<M, 8>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
        case 16: hipLaunchKernelGGL((dual_gap_kernel<M, 16>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
        case 32: hipLaunchKernelGGL((dual_gap_kernel<M, 32>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
        default: hipLaunchKernelGGL((dual_gap_kernel<M, 64>), grid, dim3(kThreads), pr_bytes, s, c, assign); break;
    }
    return hipGetLastError();
}

constexpr int kCompThreads = 1024;
constexpr int kCompWaves = kCompThreads / 64;
constexpr int kCompStageBytes = 32 * 1024;   // score rows staged per step of the greedy walk
constexpr int kCompMaxRows = 256;
static_assert(kCompMaxRows <= kCompThreads, "a chunk token per thread");

__host__ __device__ inline size_t a16(size_t x) { return (x + 15) & ~size_t(15); }

// LDS of complete_kernel (within the default 64 KiB): prices, the counts
// before the completion, the live counts, the holder-table selectors, the
// staged tokens and their choices, the open experts and the tokens' orders
// of preference over them, then the staged values: R tokens' rows of E, or
// R64 tokens' values at the (at most 64) open experts.
constexpr int kCompOrdRows = 128;
constexpr int kCompOpenStride = 65;   // staged open-expert values per token (odd: no bank conflicts)
struct CompLds {
    size_t pr, hc0, cnt, sel, stok, chs, slot, oe, ord, vst, total;
    int R, R64;
};
__host__ __device__ inline CompLds comp_lds(int E, int vbytes) {
    CompLds L{};
    const size_t budget = 62 * 1024;
    const size_t fixed = a16((size_t)E * vbytes) + 3 * a16((size_t)E * 4) +
                         3 * a16((size_t)kCompMaxRows * 4) + a16(64 * 4) + kCompOrdRows * 64;
    const size_t avail = budget > fixed ? budget - fixed : 0;
    const size_t stage_max = avail < (size_t)kCompStageBytes ? avail : (size_t)kCompStageBytes;
    size_t r = stage_max / ((size_t)E * vbytes);
    L.R = r < 1 ? 1 : (r > (size_t)kCompMaxRows ? kCompMaxRows : (int)r);
    const size_t r64 = stage_max / ((size_t)kCompOpenStride * vbytes);
    L.R64 = r64 < 1 ? 1 : (r64 > (size_t)kCompOrdRows ? kCompOrdRows : (int)r64);
    const int rows = L.R > L.R64 ? L.R : L.R64;
    const size_t sa = (size_t)L.R * E * vbytes, sb = (size_t)L.R64 * kCompOpenStride * vbytes;
    const size_t stage = sa > sb ? sa : sb;
    size_t off = 0;
    L.pr = off;   off += a16((size_t)E * vbytes);
    L.hc0 = off;  off += a16((size_t)E * 4);
    L.cnt = off;  off += a16((size_t)E * 4);
    L.sel = off;  off += a16((size_t)E * 4);
    L.stok = off; off += a16((size_t)rows * 4);
    L.chs = off;  off += a16((size_t)rows * 4);
    L.slot = off; off += a16((size_t)rows * 4);
    L.oe = off;   off += a16(64 * 4);
    L.ord = off;  off += kCompOrdRows * 64;
    L.vst = off;  off += stage;
    L.total = off;
    return L;
}

// With BASE_ASSIGN_GREEDY_FALLBACK, after the finalising kernel, when some
// expert is not full after max_rounds (one block per problem; returns at
// once otherwise): the greedy completion. Every still-unassigned token, in
// ascending token order, takes its best expert by S[t,e] - p[e] (ties to
// the lowest expert) among those with room. The unassigned tokens are first
// compacted into a list (all threads; a block scan orders them). Then, chunk
// by chunk: with at most 64 experts open at the chunk's start (float
// scores), each token's open experts are sorted by preference (all waves in
// parallel) and one wave walks the tokens in order, each taking its first
// entry that is not full. Otherwise the tokens' rows are staged in LDS,
// every wave finds each token's best expert among those with room at the
// chunk's start, and one wave walks the chunk with the live counts: a token
// whose expert filled earlier in the walk takes its best expert again over
// the experts still open. Either way the result is the sequential rule's,
// token by token. Placed tokens join their expert's holder table;
// the experts that took any are marked for rank_filled_kernel, which ranks
// their rows of perm again (one block each).
template <class M>
__global__ __launch_bounds__(kCompThreads) void complete_kernel(Ctx<M> c0, int32_t *assign,
                                                                uint32_t flags) {
    using value_t = typename M::value_t;
    const Ctx<M> c = c0.at(blockIdx.y);
    assign += (int64_t)blockIdx.y * c.T;
    SolveCtrl *ctrl = c.ctrl;
    if ((ld_relaxed(&ctrl->unconverged_experts) & ~(1 << 30)) == 0) return;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int E = c.E, C = c.C, T = c.T;
    const CompLds LY = comp_lds(E, (int)sizeof(value_t));
    const int R = LY.R;
    value_t *pr = reinterpret_cast<value_t *>(smem_raw + LY.pr);
    int *hc0 = reinterpret_cast<int *>(smem_raw + LY.hc0);
    int *cntl = reinterpret_cast<int *>(smem_raw + LY.cnt);
    int *sell = reinterpret_cast<int *>(smem_raw + LY.sel);
    int *stok = reinterpret_cast<int *>(smem_raw + LY.stok);
    int *chs = reinterpret_cast<int *>(smem_raw + LY.chs);
    int *slot = reinterpret_cast<int *>(smem_raw + LY.slot);
    int *oel = reinterpret_cast<int *>(smem_raw + LY.oe);
    uint8_t *ordl = reinterpret_cast<uint8_t *>(smem_raw + LY.ord);
    value_t *vst = reinterpret_cast<value_t *>(smem_raw + LY.vst);
    __shared__ int s_fill, s_base, s_no, s_wsum[kCompWaves];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    for (int e = tid; e < E; e += kCompThreads) {
        pr[e] = c.prices[e];
        int h = c.hcount[e];
        h = h < 0 ? 0 : (h > C ? C : h);
        hc0[e] = h;
        cntl[e] = h;
        sell[e] = c.hsel[e] & 1;
    }
    if (tid == 0) {
        s_fill = ctrl->not_converged && (flags & BASE_ASSIGN_GREEDY_FALLBACK) &&
                 !ctrl->internal_error;
        if (s_fill) {
            ctrl->fell_back = 1;
            ctrl->unconverged_experts &= (1 << 30);
        }
        s_base = 0;
    }
    __syncthreads();
    if (s_fill) {
        // The unassigned tokens, in ascending order, into the (no longer
        // used) first active list. A pass covers kCompThreads * 32 tokens:
        // wave w the 2048 from base + 2048 w, in eight steps of 256 in which
        // lane l holds four consecutive tokens (one 16-byte load when the
        // caller's buffer allows: each load of a wave reads a contiguous
        // KiB). Offsets inside a wave come from ballots of the lanes' counts
        // (0..4, three bits), across waves from their totals.
        int *list = c.active;
        const int one_chunk = R > LY.R64 ? R : LY.R64;   // the rows of stok
        const bool vec = (reinterpret_cast<uintptr_t>(assign) & 15) == 0;
        const uint64_t lt = (1ull << lane) - 1;
        for (int base = 0; base < T; base += kCompThreads * 32) {
            const int wb = base + wave * 2048 + 4 * lane;
            int4 q[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int t0 = wb + k * 256;
                if (vec && t0 + 4 <= T) {
                    q[k] = *reinterpret_cast<const int4 *>(assign + t0);
                } else {
                    q[k].x = t0 < T ? assign[t0] : 0;
                    q[k].y = t0 + 1 < T ? assign[t0 + 1] : 0;
                    q[k].z = t0 + 2 < T ? assign[t0 + 2] : 0;
                    q[k].w = t0 + 3 < T ? assign[t0 + 3] : 0;
                }
            }
            int pre[8];
            int wtot = 0;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int cnt = (q[k].x < 0) + (q[k].y < 0) + (q[k].z < 0) + (q[k].w < 0);
                const uint64_t b0 = __builtin_amdgcn_ballot_w64((cnt & 1) != 0);
                const uint64_t b1 = __builtin_amdgcn_ballot_w64((cnt & 2) != 0);
                const uint64_t b2 = __builtin_amdgcn_ballot_w64((cnt & 4) != 0);
                pre[k] = wtot + __popcll(b0 & lt) + 2 * __popcll(b1 & lt) + 4 * __popcll(b2 & lt);
                wtot += __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2);
            }
            if (lane == 0) s_wsum[wave] = wtot;
            __syncthreads();
            // The waves' totals: one read per lane, summed from registers.
            const int wsv = lane < kCompWaves ? s_wsum[lane] : 0;
            int before = s_base, all = 0;
#pragma unroll
            for (int w = 0; w < kCompWaves; ++w) {
                const int x = __builtin_amdgcn_readlane(wsv, w);
                before += w < wave ? x : 0;
                all += x;
            }
            // All of them in one pass and within the rows of the chunks'
            // token array: straight into it (LDS), not the list.
            int *dst = T <= kCompThreads * 32 && all <= one_chunk ? stok : list;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int4 v = q[k];
                if ((v.x | v.y | v.z | v.w) >= 0) continue;   // none of the four
                const int t0 = wb + k * 256;
                int at = before + pre[k];
                if (v.x < 0) dst[at++] = t0;
                if (v.y < 0) dst[at++] = t0 + 1;
                if (v.z < 0) dst[at++] = t0 + 2;
                if (v.w < 0) dst[at++] = t0 + 3;
            }
            __syncthreads();
            if (tid == 0) {
                int tot = s_base;
                for (int w = 0; w < kCompWaves; ++w) tot += s_wsum[w];
                s_base = tot;
            }
            __syncthreads();
        }
        const int n = s_base;
        const bool in_lds = T <= kCompThreads * 32 && n <= one_chunk;   // the tokens are in stok
        for (int j0 = 0; j0 < n;) {
            if (wave == 0) {
                // The experts open at the chunk's start, ascending (the
                // first 64 of them, and how many there are).
                int no = 0;
                for (int e0 = 0; e0 < E; e0 += 64) {
                    const int e = e0 + lane;
                    const bool open = e < E && cntl[e] < C;
                    const uint64_t bm = __ballot(open);
                    const int at = no + __popcll(bm & ((1ull << lane) - 1));
                    if (open && at < 64) oel[at] = e;
                    no += __popcll(bm);
                }
                if (lane == 0) s_no = no;
            }
            __syncthreads();
            const int no = s_no;
            const bool fast = !M::kInteger && no <= 64;
            const int cap = fast ? LY.R64 : R;
            const int m = n - j0 < cap ? n - j0 : cap;
            // The chunk's tokens to the front of stok (m <= kCompMaxRows <
            // kCompThreads: one each).
            int t = 0;
            if (tid < m) t = in_lds ? stok[j0 + tid] : list[j0 + tid];
            if (in_lds) __syncthreads();
            if (tid < m) stok[tid] = (t >= 0 && t < T) ? t : 0;
            __syncthreads();
            if (fast) {
                // At most 64 experts open (a completion never reopens one):
                // only their values are staged; each token's open experts
                // are ranked by preference (value, then the lower expert):
                // every (token, open expert) pair counts the entries that
                // precede it, and the token's order lists them by rank. The
                // walk then takes each token's first entry that is not full,
                // from a 64-bit mask of the full ones (no reduction per
                // token).
                for (int q = tid; q < m * no; q += kCompThreads) {
                    const int r = q / no;
                    const int i = q - r * no;
                    const int e = oel[i];
                    vst[r * kCompOpenStride + i] =
                        M::load(c.S, (int64_t)stok[r] * E + e, c.scale) - pr[e];
                }
                __syncthreads();
                for (int q = tid; q < m * no; q += kCompThreads) {
                    const int r = q / no;
                    const int i = q - r * no;
                    const value_t *row = vst + r * kCompOpenStride;
                    const value_t v = row[i];
                    int rank = 0;
                    for (int k = 0; k < no; ++k) {
                        const value_t w = row[k];
                        rank += (w > v || (w == v && k < i)) ? 1 : 0;
                    }
                    ordl[r * 64 + rank] = (uint8_t)i;
                }
                __syncthreads();
                if (wave == 0) {
                    // Lane i: the slots left at open expert i (none past the
                    // list, which therefore counts as full); bit i of full:
                    // none left, one ballot of them, off the read of the slot
                    // a token takes. An order's entries past no are stale,
                    // and masked.
                    int rem = lane < no ? C - cntl[oel[lane]] : 0;
                    const uint64_t inl = no >= 64 ? ~0ull : (1ull << no) - 1;   // entries of the order
                    uint64_t full = __builtin_amdgcn_ballot_w64(rem <= 0);
                    for (int b0 = 0; b0 < m; b0 += 64) {
                        const int mb = m - b0 < 64 ? m - b0 : 64;
                        int di = -1, ds = 0;   // lane j: the decision on entry b0 + j (open index, slot)
                        // Two tokens a step, both against the same mask: the
                        // second chooses again only when the first has just
                        // filled the expert it picked.
                        int na = ordl[b0 * 64 + lane];
                        int nb = ordl[(b0 + (mb > 1 ? 1 : 0)) * 64 + lane];
                        for (int j = 0; j < mb; j += 2) {
                            const int orda = na, ordb = nb;   // lane k: the tokens' k-th choices
                            const int j2 = j + 2 < mb ? j + 2 : mb - 1;
                            const int j3 = j + 3 < mb ? j + 3 : mb - 1;
                            na = ordl[(b0 + j2) * 64 + lane];
                            nb = ordl[(b0 + j3) * 64 + lane];
                            const uint64_t ra = __builtin_amdgcn_ballot_w64(((full >> orda) & 1) == 0) & inl;
                            const uint64_t rb = __builtin_amdgcn_ballot_w64(((full >> ordb) & 1) == 0) & inl;
                            if (ra == 0) continue;   // (uniform) no expert has room: nor for the next
                            // oa, ob: the open-list indices the two tokens take
                            const int oa = __builtin_amdgcn_readlane(orda, (int)__builtin_ctzll(ra));
                            const int la = __builtin_amdgcn_readlane(rem, oa);
                            rem -= lane == oa ? 1 : 0;
                            di = lane == j ? oa : di;
                            ds = lane == j ? C - la : ds;
                            if (j + 1 < mb) {
                                int ob = __builtin_amdgcn_readlane(ordb, (int)__builtin_ctzll(rb));
                                if (ob == oa && la == 1) {   // the first filled it: again
                                    full = __builtin_amdgcn_ballot_w64(rem <= 0);
                                    const uint64_t r2 = __builtin_amdgcn_ballot_w64(((full >> ordb) & 1) == 0) & inl;
                                    ob = r2 != 0 ? __builtin_amdgcn_readlane(ordb, (int)__builtin_ctzll(r2)) : -1;
                                }
                                if (ob >= 0) {
                                    const int lb = __builtin_amdgcn_readlane(rem, ob);
                                    rem -= lane == ob ? 1 : 0;
                                    di = lane == j + 1 ? ob : di;
                                    ds = lane == j + 1 ? C - lb : ds;
                                }
                            }
                            full = __builtin_amdgcn_ballot_w64(rem <= 0);
                        }
                        if (lane < mb) {
                            chs[b0 + lane] = di >= 0 ? oel[di] : -1;
                            slot[b0 + lane] = ds;
                        }
                    }
                    if (lane < no) cntl[oel[lane]] = C - rem;
                }
            } else {
#pragma unroll 8
                for (int q = tid; q < m * E; q += kCompThreads) {
                    const int r = q / E;
                    const int e = q - r * E;
                    vst[q] = M::load(c.S, (int64_t)stok[r] * E + e, c.scale) - pr[e];
                }
                __syncthreads();
                // Each staged token's best expert among those open now.
                for (int r = wave; r < m; r += kCompWaves) {
                    value_t bv = M::lowest();
                    int be = 0x7fffffff;
                    for (int e = lane; e < E; e += 64) {
                        const value_t v = vst[r * E + e];
                        if (cntl[e] < C && (v > bv || be == 0x7fffffff)) {
                            bv = v;
                            be = e;
                        }
                    }
                    wave_max_pair(bv, be);
                    if (lane == 0) chs[r] = be;
                }
                __syncthreads();
                // The walk in token order. Lane j of a batch of 64 holds the
                // choice of entry j. With E <= 128 the live counts sit in two
                // registers (lane l: experts l and l + 64) and each decision is
                // a few cross-lane reads; otherwise they are in LDS. Lane 0
                // records each decision (expert and slot, into chs and slot).
                // One wave's LDS accesses take effect in program order, so the
                // walk needs no memory wait: the empty asm statements only keep
                // the compiler from reordering them.
                if (wave == 0 && E <= 128) {
                    int cnt0 = lane < E ? cntl[lane] : C;   // experts past E count as full
                    int cnt1 = lane + 64 < E ? cntl[lane + 64] : C;
                    for (int r0 = 0; r0 < m; r0 += 64) {
                        const int cj = r0 + lane < m ? chs[r0 + lane] : 0;
                        const int mm = m - r0 < 64 ? m - r0 : 64;
                        int de = -1, ds = 0;   // lane j: the decision on entry j
                        // The entry's values for a second choice, read one entry
                        // ahead (a choice that filled up is common once few
                        // slots are left, and the LDS read is then not waited for).
                        value_t nv0 = vst[r0 * E + (lane < E ? lane : 0)];
                        value_t nv1 = vst[r0 * E + (lane + 64 < E ? lane + 64 : 0)];
                        for (int j = 0; j < mm; ++j) {
                            const value_t v0 = nv0, v1 = nv1;
                            if (j + 1 < mm) {
                                nv0 = vst[(r0 + j + 1) * E + (lane < E ? lane : 0)];
                                nv1 = vst[(r0 + j + 1) * E + (lane + 64 < E ? lane + 64 : 0)];
                            }
                            int e = __builtin_amdgcn_readlane(cj, j);
                            int have = e < 64 ? __builtin_amdgcn_readlane(cnt0, e & 63)
                                              : (e < E ? __builtin_amdgcn_readlane(cnt1, e & 63) : C);
                            if (have >= C) {   // (uniform) the choice filled up: again
                                const bool o0 = cnt0 < C, o1 = lane + 64 < E && cnt1 < C;
                                value_t bv = o0 ? v0 : M::lowest();
                                int be = o0 ? lane : 0x7fffffff;
                                const bool t1 = o1 && v1 > bv;
                                bv = t1 ? v1 : bv;
                                be = t1 ? lane + 64 : be;
                                wave_max_pair(bv, be);
                                e = be;
                                have = e < 64 ? __builtin_amdgcn_readlane(cnt0, e & 63)
                                              : (e < E ? __builtin_amdgcn_readlane(cnt1, e & 63) : C);
                            }
                            const bool ok = e < E && have < C;
                            if (ok && lane == (e & 63)) {
                                if (e < 64) cnt0 += 1;
                                else cnt1 += 1;
                            }
                            if (lane == j) {
                                de = ok ? e : -1;
                                ds = have;
                            }
                        }
                        if (lane < mm) {
                            chs[r0 + lane] = de;
                            slot[r0 + lane] = ds;
                        }
                    }
                    if (lane < E) cntl[lane] = cnt0;
                    if (lane + 64 < E) cntl[lane + 64] = cnt1;
                } else if (wave == 0) {
                    for (int r0 = 0; r0 < m; r0 += 64) {
                        const int cj = r0 + lane < m ? chs[r0 + lane] : 0;
                        const int mm = m - r0 < 64 ? m - r0 : 64;
                        for (int j = 0; j < mm; ++j) {
                            int e = __builtin_amdgcn_readlane(cj, j);
                            int have = e < E ? cntl[e] : C;
                            if (have >= C) {   // (uniform) the choice filled up: again
                                value_t bv = M::lowest();
                                int be = 0x7fffffff;
                                for (int e2 = lane; e2 < E; e2 += 64) {
                                    const value_t v = vst[(r0 + j) * E + e2];
                                    if (cntl[e2] < C && (v > bv || be == 0x7fffffff)) {
                                        bv = v;
                                        be = e2;
                                    }
                                }
                                wave_max_pair(bv, be);
                                e = be;
                                have = e < E ? cntl[e] : C;
                            }
                            const bool ok = e < E && have < C;
                            if (lane == 0) {
                                if (ok) cntl[e] = have + 1;
                                chs[r0 + j] = ok ? e : -1;
                                slot[r0 + j] = have;
                            }
                            asm volatile("" ::: "memory");
                        }
                    }
                }
            }
            __syncthreads();
            // The chunk's decisions into assign and the holder tables.
            for (int r = tid; r < m; r += kCompThreads) {
                const int e = chs[r];
                if (e >= 0) {
                    const int t = stok[r];
                    c.holders[(int64_t)sell[e] * T + (int64_t)e * C + slot[r]] =
                        (1ull << kTokBits) | (kTokMask - (uint64_t)t);
                    assign[t] = e;
                }
            }
            __syncthreads();
            j0 += m;
        }
        for (int e = tid; e < E; e += kCompThreads) {
            c.hcount[e] = cntl[e];
            c.ovf_exp[e] = cntl[e] != hc0[e] ? 1 : 0;   // rows for rank_filled_kernel
        }
    }
}

// Per block of kCountTile tokens: how many go to each expert.
__global__ __launch_bounds__(kCountTile) void block_count_kernel(const int32_t *assign, int T,
                                                                 int E, int32_t *blk,
                                                                 int64_t ws_stride) {
    assign += (int64_t)blockIdx.y * T;
    blk = Ctx<FloatMode>::shift(blk, (int64_t)blockIdx.y * ws_stride);
    extern __shared__ int hist[];
    for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
    __syncthreads();
    const int t = blockIdx.x * kCountTile + threadIdx.x;
    if (t < T) {
        const int a = assign[t];
        if (a >= 0 && a < E) atomicAdd(&hist[a], 1);
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) blk[(int64_t)blockIdx.x * E + e] = hist[e];
}

// Exclusive scan over the blocks' counts of one expert (one workgroup per
// expert), offset by the expert's first row e*C.
__global__ __launch_bounds__(256) void block_scan_kernel(int32_t *blk, int nblk, int E, int C,
                                                         int64_t ws_stride) {
    blk = Ctx<FloatMode>::shift(blk, (int64_t)blockIdx.y * ws_stride);
    __shared__ int wsum[4];
    __shared__ int carry;
    const int e = blockIdx.x;
    const int lane = lane_id();
    const int wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) carry = e * C;
    __syncthreads();
    for (int b0 = 0; b0 < nblk; b0 += 256) {
        const int b = b0 + threadIdx.x;
        const int v = b < nblk ? blk[(int64_t)b * E + e] : 0;
        int incl = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int o = __shfl_up(incl, off);
            if (lane >= off) incl += o;
        }
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        int before = carry;
        for (int w = 0; w < wave; ++w) before += wsum[w];
        if (b < nblk) blk[(int64_t)b * E + e] = before + incl - v;
        __syncthreads();
        if (threadIdx.x == 0) carry += wsum[0] + wsum[1] + wsum[2] + wsum[3];
        __syncthreads();
    }
}

// perm[offset(block, a_t) + rank of t among the block's tokens of a_t] = t:
// a stable counting sort by expert.
__global__ __launch_bounds__(kCountTile) void perm_scatter_kernel(const int32_t *assign, int T,
                                                                  int E, const int32_t *blk,
                                                                  int32_t *perm, int64_t ws_stride) {
    assign += (int64_t)blockIdx.y * T;
    perm += (int64_t)blockIdx.y * T;
    blk = Ctx<FloatMode>::shift(blk, (int64_t)blockIdx.y * ws_stride);
    __shared__ int loc[kCountTile];
    const int t = blockIdx.x * kCountTile + threadIdx.x;
    const int a = t < T ? assign[t] : -1;
    loc[threadIdx.x] = a;
    __syncthreads();
    if (a < 0 || a >= E) return;
    int rank = 0;
    for (int j = 0; j < (int)threadIdx.x; ++j) rank += (loc[j] == a);
    const int pos = blk[(int64_t)blockIdx.x * E + a] + rank;
    if (pos < T) perm[pos] = t;
}

__global__ void fill_kernel(int32_t *p, int64_t n, int32_t v) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

// E == 1: every token goes to expert 0 and the sort vector is the identity
// (n = B * T entries, problem by problem).
__global__ void single_expert_kernel(int32_t *assign, int32_t *perm, int64_t n, int64_t T) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        assign[i] = 0;
        perm[i] = (int32_t)(i % T);
    }
}

// ------------------------------------------------------------------ driver --

// Lanes per token: 8 experts per lane, a power of two up to a whole wave.
int lanes_per_token(int64_t E) {
    int g = 1;
    while (g < 64 && 8 * g < E) g <<= 1;
    return g;
}

// ------------------------------------------------------------ timing --
//
// Measurement support: while enabled, every engine launch is bracketed by a
// pair of pre-created events (one process-wide record, not thread-safe).

struct EngineTiming {
    int32_t capacity = 0;
    int32_t used = 0;
    int64_t dropped = 0;
    hipEvent_t *ev = nullptr;   // 2 * capacity events
};
EngineTiming g_timing;

void timing_pair(hipEvent_t *begin, hipEvent_t *end) {
    if (g_timing.capacity == 0) return;
    if (g_timing.used == g_timing.capacity) {
        ++g_timing.dropped;
        return;
    }
    *begin = g_timing.ev[2 * g_timing.used];
    *end = g_timing.ev[2 * g_timing.used + 1];
    ++g_timing.used;
}

// Per-device facts the launches depend on, looked up once per device (and
// per kernel and LDS size): the LDS a block may opt in to, the compute
// units, a kernel's resident blocks per compute unit, and the LDS opt-in
// already granted to a kernel.
constexpr int kMaxDevices = 64;
struct DeviceFacts {
    bool known = false;
    int optin = 0;
    int cus = 0;
};
std::mutex g_facts_mutex;
DeviceFacts g_facts[kMaxDevices];
std::map<std::tuple<int, const void *, int, size_t>, int> g_occupancy;
std::map<std::pair<int, const void *>, size_t> g_lds_granted;

// The current device and its facts (optin falls back to 64 KiB, cus to 0
// when the runtime cannot tell).
int device_facts(DeviceFacts *f) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        (void)hipGetLastError();
        *f = DeviceFacts{true, 64 * 1024, 0};
        return -1;
    }
    std::lock_guard<std::mutex> lock(g_facts_mutex);
    if (!g_facts[dev].known) {
        DeviceFacts d;
        d.known = true;
        if (hipDeviceGetAttribute(&d.optin, hipDeviceAttributeSharedMemPerBlockOptin, dev) !=
                hipSuccess ||
            d.optin <= 0)
            d.optin = 64 * 1024;
        if (hipDeviceGetAttribute(&d.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            d.cus = 0;
        (void)hipGetLastError();
        g_facts[dev] = d;
    }
    *f = g_facts[dev];
    return dev;
}

// Resident blocks per compute unit of kernel fn (0 when unknown).
int occupancy(int dev, const void *fn, int threads, size_t lds) {
    std::lock_guard<std::mutex> lock(g_facts_mutex);
    const auto key = std::make_tuple(dev, fn, threads, lds);
    const auto it = g_occupancy.find(key);
    if (it != g_occupancy.end()) return it->second;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds) != hipSuccess)
        per_cu = 0;
    (void)hipGetLastError();
    if (dev >= 0) g_occupancy[key] = per_cu;
    return per_cu;
}

// Lets kernel fn take `bytes` of dynamic LDS (above the default 64 KiB); the
// attribute is set again only for a larger size than granted before.
hipError_t lds_optin(int dev, const void *fn, size_t bytes) {
    if (bytes <= 64 * 1024) return hipSuccess;
    std::lock_guard<std::mutex> lock(g_facts_mutex);
    const auto key = std::make_pair(dev, fn);
    const auto it = g_lds_granted.find(key);
    if (dev >= 0 && it != g_lds_granted.end() && it->second >= bytes) return hipSuccess;
    const hipError_t err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (err == hipSuccess && dev >= 0) g_lds_granted[key] = bytes;
    return err;
}

// The shortest-path finish for Ep padded experts (one block per problem).
template <class M>
void launch_ssp(const Ctx<M> &c, int B, int ssp_r, size_t ssp_bytes, hipStream_t s) {
    const dim3 g(1, B);
    const int small = ssp_fallbacks_setting();
    switch (ssp_r) {
        case 32: hipLaunchKernelGGL((ssp_kernel<M, 32>), g, dim3(ssp_block<32>()), ssp_bytes, s, c, c.ssp_cap, small); break;
        case 64: hipLaunchKernelGGL((ssp_kernel<M, 64>), g, dim3(ssp_block<64>()), ssp_bytes, s, c, c.ssp_cap, small); break;
        case 128: hipLaunchKernelGGL((ssp_kernel<M, 128>), g, dim3(ssp_block<128>()), ssp_bytes, s, c, c.ssp_cap, small); break;
        default: hipLaunchKernelGGL((ssp_kernel<M, 256>), g, dim3(ssp_block<256>()), ssp_bytes, s, c, c.ssp_cap, small); break;
    }
}

template <class M, int G>
hipError_t run_solve(const Ctx<M> &c0, const AssignParams &p, int B, int32_t *assign,
                     uint32_t *rpart, hipStream_t s) {
    using value_t = typename M::value_t;
    Ctx<M> c = c0;
    DeviceFacts facts;
    const int dev = device_facts(&facts);
    // The engine's LDS: the longest per-expert lists that fit the device's
    // per-block limit (with the opt-in above the default 64 KiB).
    bool engine = c.E <= kEngMaxE && c.C <= kEngMaxC;
    size_t eng_bytes = 0;
    if (engine) {
        const size_t limit = (size_t)facts.optin - 1024;   // room for the kernel's static LDS
        int K = kEngMaxK;
        while (K >= 8 && eng_layout(c.E, (int)sizeof(value_t), K).total > limit) K >>= 1;
        if (K < 8) {
            engine = false;
        } else {
            eng_bytes = eng_layout(c.E, (int)sizeof(value_t), K).total;
            const hipError_t err = lds_optin(
                dev, reinterpret_cast<const void *>(&engine_kernel<M, G>), eng_bytes);
            if (err != hipSuccess) {
                (void)hipGetLastError();
                debug_note("engine LDS opt-in refused", err);
                while (K >= 8 && eng_layout(c.E, (int)sizeof(value_t), K).total > 64 * 1024)
                    K >>= 1;
                engine = K >= 8;
                if (engine) eng_bytes = eng_layout(c.E, (int)sizeof(value_t), K).total;
            }
            c.eng_k = K;
        }
    }
    if (engine) c.engine_cap = kEngCap;
    {
        // Early ends of large-epsilon phases; with the full schedule no
        // check reads any phase above the last, so each of them may end
        // early. Also under a caller's round bound: the rounds saved go to
        // the finer phase, whose partial assignment the greedy completion
        // then starts from (T = 32768, E = 128, clustered scores: at 20
        // rounds the certified gap fell from 53 to 31; 100 rounds converge).
        const int n = early_end_tokens_setting(c.T);
        if (n > 0) c.early_n = (p.flags & BASE_ASSIGN_FULL_SCHEDULE) ? -n : n;
    }
    // The shortest-path finish (float mode, E <= kSspMaxE, with the engine):
    // the most unassigned tokens it takes over, as many as its LDS allows.
    size_t ssp_bytes = 0;
    int ssp_r = 0;
    if constexpr (!M::kInteger) {
        int cap = ssp_cap_setting(c.T, c.E);
        if (engine && c.E <= kSspMaxE && c.T <= 65536 && cap > 0) {
            const size_t limit = (size_t)facts.optin - 2048;   // the kernel's static LDS
            if (cap > kSspMaxCap) cap = kSspMaxCap;
            if (cap < kSspMinCap) cap = kSspMinCap;
            while (cap >= kSspMinCap && ssp_lds_bytes(c.E, cap, c.C) > limit) cap >>= 1;
            if (cap >= kSspMinCap) {
                ssp_r = ssp_pad(c.E);
                ssp_bytes = ssp_lds_bytes(c.E, cap, c.C);
                const void *fn = ssp_r == 32    ? reinterpret_cast<const void *>(&ssp_kernel<M, 32>)
                                 : ssp_r == 64  ? reinterpret_cast<const void *>(&ssp_kernel<M, 64>)
                                 : ssp_r == 128 ? reinterpret_cast<const void *>(&ssp_kernel<M, 128>)
                                                : reinterpret_cast<const void *>(&ssp_kernel<M, 256>);
                const hipError_t err = lds_optin(dev, fn, ssp_bytes);
                if (err == hipSuccess) {
                    c.ssp_cap = cap;
                } else {
                    (void)hipGetLastError();
                    debug_note("shortest-path finish LDS opt-in refused", err);
                    ssp_r = 0;
                }
            }
        }
    }
    // The prologue (score summaries, range partials, assign = -1, a fresh
    // control block and starting prices) and the start of the first phase.
    const int per_block = kThreads / G;
    int sblocks = (int)((c.T + per_block - 1) / per_block);
    if (sblocks > kPrologueBlocks) sblocks = kPrologueBlocks;
    hipLaunchKernelGGL((prologue_kernel<M, G>), dim3(sblocks, B), dim3(kThreads), 0, s, c, p,
                       assign, rpart);
    hipLaunchKernelGGL(start_kernel<M>, dim3(1, B), dim3(256), 0, s, c, p, rpart, sblocks);
    // Small problems: every phase's rounds in one workgroup per problem
    // (small_solve_kernel), the shortest-path finish after each; the last
    // slot's launch runs every phase left to the end.
    // By default a batch of at least kSmallBatch problems (each would get a
    // fraction of the device in the multi-kernel path; 256 worker-shape
    // problems take 3.9 ms this way against 12.3 ms) and very small
    // problems; a single worker-shape problem is faster with the whole
    // device (0.88 ms against 1.20 ms).
    const int small_set = small_path_setting();
    const bool small_fits = c.T <= kSmallT && c.E <= kSmallE;
    const bool small = small_fits && (small_set == 1 ||
                                      (small_set < 0 && (B >= kSmallBatch || c.T <= kSmallSoloT)));
    if (small) {
        const size_t bytes = small_lds(c.T, c.E, (int)sizeof(value_t)).total;
        const void *fn = reinterpret_cast<const void *>(&small_solve_kernel<M, G>);
        const hipError_t err = bytes + 1024 <= (size_t)facts.optin ? lds_optin(dev, fn, bytes)
                                                                     : hipErrorInvalidValue;
        if (err == hipSuccess) {
            int nslots = (p.flags & BASE_ASSIGN_FULL_SCHEDULE) ? 6 : 5;
            if (p.eps_initial > 0.0) {
                double e = p.eps_initial;
                nslots = 1;
                while (e > p.eps_final && nslots < 64) {
                    e /= p.eps_factor;
                    ++nslots;
                }
            }
            for (int slot = 0; slot < nslots; ++slot) {
                const bool last = slot == nslots - 1;
                const int cap = (!last && ssp_r > 0) ? c.ssp_cap : 0;
                // (the dominant kernel of this route, timed like the engine)
                hipEvent_t ev0 = nullptr, ev1 = nullptr;
                timing_pair(&ev0, &ev1);
                if (ev0 != nullptr) (void)hipEventRecord(ev0, s);
                hipLaunchKernelGGL((small_solve_kernel<M, G>), dim3(1, B), dim3(kSmallThreads),
                                   bytes, s, c, p, cap);
                if (ev1 != nullptr) (void)hipEventRecord(ev1, s);
                if constexpr (!M::kInteger) {
                    if (cap > 0) {
                        hipLaunchKernelGGL(ssp_build_kernel<M>, dim3(c.E, B),
                                           dim3(ssp_build_threads(c.C, c.E * B)), 0, s, c);
                        launch_ssp<M>(c, B, ssp_r, ssp_bytes, s);
                    }
                }
            }
            return hipGetLastError();
        }
        (void)hipGetLastError();
        debug_note("single-workgroup solve LDS opt-in refused", err);
    }
    const size_t pr_bytes = (size_t)c.E * sizeof(value_t);
    const size_t tail_smem = pr_bytes + (size_t)c.E * sizeof(int);
    // Phase slots enqueued up front; the last one continues on its own (in
    // one workgroup, slowly) if the epsilon schedule needs more phases than
    // were enqueued. A slot the solve no longer needs still costs its empty
    // launches (a few microseconds each). With the default schedule (first epsilon =
    // range / 8, divisor 32) five slots cover score ranges up to 8 * 32^4
    // (about 8 * 10^6) times eps_final even without a certified early stop,
    // which typically comes one or two phases sooner; the full schedule
    // gets six (up to 8 * 32^5, about 3 * 10^8).
    int slots = (p.flags & BASE_ASSIGN_FULL_SCHEDULE) ? 6 : 5;
    if (p.eps_initial > 0.0) {
        double e = p.eps_initial;
        slots = 1;
        while (e > p.eps_final && slots < 64) {
            e /= p.eps_factor;
            ++slots;
        }
    }
    const int wide_rounds = engine ? 3 : 2;
    const int bid_blocks = (int)((c.T + kBidTile - 1) / kBidTile);   // one tile of the list each
    const size_t bid_bytes = bid_smem(c.E, (int)sizeof(value_t)).total;
    int upd_blocks = c.E < 2048 ? c.E : 2048;
    // Round loop for phases that stay large: one block per compute unit,
    // shared out among the problems of a batch (every block of the grid must
    // be resident at once; a batch larger than the device holds skips it).
    // A single problem takes half the units: its grid barriers cost less
    // (1% faster over eight workloads; batches of 64 and 128 problems were
    // slower with half).
    int coop_blocks = 0;
    {
        const int cus = facts.cus;
        const int per_cu =
            cus > 0 ? occupancy(dev, reinterpret_cast<const void *>(&wide_loop_kernel<M, G>),
                                kThreads, bid_bytes)
                    : 0;
        if (per_cu > 0 && cus > 0) {
            coop_blocks = B == 1 ? cus / 2 : cus / B;
            if (coop_blocks == 0 && B <= cus * per_cu) coop_blocks = 1;
        }
    }
    // Each slot: the phase start (with the decision on the previous slot's
    // duality check), the wide rounds, the round loop, the engine, the
    // one-workgroup tail (with the engine only in the last slot: a phase the
    // engine leaves unfinished goes on in the next slot), and the check.
    const bool checks = !(p.flags & BASE_ASSIGN_FULL_SCHEDULE);
    const int check_parts = phase_check_blocks(c.T, G);
    // From the third slot on, the round loop takes the phase's first rounds
    // as well: those slots often come after the solve has stopped (then
    // every launch returns at once, and fewer launches cost less), and when
    // one runs, its first rounds cost little more in the loop.
    for (int slot = 0; slot < slots; ++slot) {
        if (slot > 0)   // (the start kernel began the first phase)
            hipLaunchKernelGGL(phase_begin_kernel<M>, dim3(1, B), dim3(1024), 0, s, c, p,
                               checks ? check_parts : 0);
        const int wr = (slot >= 2 && coop_blocks > 0) ? 0 : wide_rounds;
        for (int r = 0; r < wr; ++r) {
            hipLaunchKernelGGL((bid_wide_kernel<M, G>), dim3(bid_blocks, B), dim3(kThreads),
                               bid_bytes, s, c);
            hipLaunchKernelGGL(update_wide_kernel<M>, dim3(upd_blocks, B), dim3(kThreads), 0, s, c);
        }
        if (coop_blocks > 0)
            hipLaunchKernelGGL((wide_loop_kernel<M, G>), dim3(coop_blocks, B), dim3(kThreads),
                               bid_bytes, s, c, kWideLoopRounds, p.max_rounds, barrier_polls());
        if (engine) {
            // Summary readers: multiples of 8 blocks per problem, 256 in all
            // when one problem.
            const int pf = B >= 32 ? 8 : 8 * (32 / B);
            hipLaunchKernelGGL(engine_entry_kernel<M>, dim3(c.E + pf, B), dim3(256), 0, s, c, pf);
            hipEvent_t ev0 = nullptr, ev1 = nullptr;
            timing_pair(&ev0, &ev1);
            if (ev0 != nullptr) (void)hipEventRecord(ev0, s);
            hipLaunchKernelGGL((engine_kernel<M, G>), dim3(1, B), dim3(kEngThreads), eng_bytes, s,
                               c, p);
            if (ev1 != nullptr) (void)hipEventRecord(ev1, s);
        }
        if constexpr (!M::kInteger) {
            if (ssp_r > 0) {
                hipLaunchKernelGGL(ssp_build_kernel<M>, dim3(c.E, B),
                                   dim3(ssp_build_threads(c.C, c.E * B)), 0, s, c);
                launch_ssp<M>(c, B, ssp_r, ssp_bytes, s);
            }
        }
        if (!engine || slot == slots - 1)
            hipLaunchKernelGGL((tail_kernel<M, G>), dim3(1, B), dim3(kThreads), tail_smem, s, c,
                               p, slot == slots - 1 ? 1 : 0);
        if (checks && slot < slots - 1) {
            const hipError_t err = launch_phase_check<M, G>(c, B, s);
            if (err != hipSuccess) return err;
        }
    }
    return hipGetLastError();
}

template <class M>
hipError_t solve_mode(const void *S, const AssignParams &p, int B, int32_t *assign, int32_t *perm,
                      void *prices_out, void *workspace, hipStream_t s) {
    using value_t = typename M::value_t;
    char *ws = static_cast<char *>(workspace);
    const Layout L = make_layout(p.T, p.E);
    Ctx<M> c = make_ctx<M>(S, p, ws);
    const int64_t wst = c.ws_stride;
    uint32_t *rpart = reinterpret_cast<uint32_t *>(ws + L.rpart);
    hipError_t err = hipSuccess;
    switch (lanes_per_token(p.E)) {
        case 1: err = run_solve<M, 1>(c, p, B, assign, rpart, s); break;
        case 2: err = run_solve<M, 2>(c, p, B, assign, rpart, s); break;
        case 4: err = run_solve<M, 4>(c, p, B, assign, rpart, s); break;
        case 8: err = run_solve<M, 8>(c, p, B, assign, rpart, s); break;
        case 16: err = run_solve<M, 16>(c, p, B, assign, rpart, s); break;
        case 32: err = run_solve<M, 32>(c, p, B, assign, rpart, s); break;
        default: err = run_solve<M, 64>(c, p, B, assign, rpart, s); break;
    }
    if (err != hipSuccess) {
        debug_note("solver launches", err);
        return err;
    }

    // assign, perm (ranked per expert when C <= kRankMaxC) and the prices;
    // with the fallback flag, the greedy completion and the rows of perm of
    // the experts it filled.
    const int rank_perm = c.C <= kRankMaxC ? 1 : 0;
    hipLaunchKernelGGL(finalise_kernel<M>, dim3(c.E, B), dim3(256), 0, s, c, assign, perm,
                       static_cast<value_t *>(prices_out), rank_perm);
    if (p.flags & BASE_ASSIGN_GREEDY_FALLBACK) {
        hipLaunchKernelGGL(complete_kernel<M>, dim3(1, B), dim3(kCompThreads),
                           comp_lds(c.E, (int)sizeof(value_t)).total, s, c, assign, p.flags);
        if (rank_perm)
            hipLaunchKernelGGL(rank_filled_kernel<M>, dim3(c.E, B), dim3(256), 0, s, c, perm);
    }
    if (!rank_perm) {
        int32_t *blk = reinterpret_cast<int32_t *>(ws + L.blk);
        hipLaunchKernelGGL(block_count_kernel, dim3((unsigned)L.nblk, B), dim3(kCountTile),
                           (size_t)p.E * sizeof(int), s, assign, c.T, c.E, blk, wst);
        hipLaunchKernelGGL(block_scan_kernel, dim3((unsigned)p.E, B), dim3(256), 0, s, blk,
                           (int)L.nblk, c.E, c.C, wst);
        hipLaunchKernelGGL(perm_scatter_kernel, dim3((unsigned)L.nblk, B), dim3(kCountTile), 0, s,
                           assign, c.T, c.E, blk, perm, wst);
    }
    if (p.flags & BASE_ASSIGN_SYNC_STATS) {
        err = launch_dual_gap<M>(c, B, assign, s);
        if (err != hipSuccess) return err;
    }
    return hipGetLastError();
}

}  // namespace

size_t assign_workspace_size(int64_t T, int64_t E) {
    if (T <= 0 || E <= 0 || T % E) return 0;
    return make_layout(T, E).total;
}

hipError_t launch_assign(const void *S, const AssignParams &p, int64_t B, int32_t *assign,
                         int32_t *perm, void *prices_out, void *workspace, hipStream_t stream) {
    if (p.E == 1) {
        // Control blocks and prices are cleared by kernels, not memset nodes,
        // so that a caller may capture the call in a graph.
        const int64_t wst = (int64_t)make_layout(p.T, p.E).total;
        AssignParams q = p;
        q.warm_prices = nullptr;
        hipLaunchKernelGGL(init_kernel, dim3(1, (unsigned)B), dim3(256), 0, stream,
                           static_cast<SolveCtrl *>(workspace), (void *)nullptr, 0, q, wst);
        int blocks = (int)((p.T * B + 255) / 256);
        if (blocks > 2048) blocks = 2048;
        hipLaunchKernelGGL(single_expert_kernel, dim3(blocks), dim3(256), 0, stream, assign, perm,
                           p.T * B, p.T);
        if (prices_out != nullptr) {
            // one price per problem: 0 (fp32 zero and int64 zero share the bit pattern)
            const int64_t words = B * (p.integer ? 2 : 1);
            hipLaunchKernelGGL(fill_kernel, dim3(1), dim3(256), 0, stream,
                               static_cast<int32_t *>(prices_out), words, 0);
        }
        return hipGetLastError();
    }
    if (p.integer)
        return solve_mode<IntMode>(S, p, (int)B, assign, perm, prices_out, workspace, stream);
    return solve_mode<FloatMode>(S, p, (int)B, assign, perm, prices_out, workspace, stream);
}

hipError_t timing_enable(int32_t capacity) {
    for (int32_t i = 0; i < 2 * g_timing.capacity; ++i) (void)hipEventDestroy(g_timing.ev[i]);
    free(g_timing.ev);
    g_timing = EngineTiming{};
    if (capacity <= 0) return hipSuccess;
    g_timing.ev = static_cast<hipEvent_t *>(calloc((size_t)2 * capacity, sizeof(hipEvent_t)));
    if (g_timing.ev == nullptr) return hipErrorOutOfMemory;
    for (int32_t i = 0; i < 2 * capacity; ++i) {
        const hipError_t e = hipEventCreate(&g_timing.ev[i]);
        if (e != hipSuccess) {
            for (int32_t j = 0; j < i; ++j) (void)hipEventDestroy(g_timing.ev[j]);
            free(g_timing.ev);
            g_timing = EngineTiming{};
            return e;
        }
    }
    g_timing.capacity = capacity;
    return hipSuccess;
}

hipError_t timing_read(int64_t *launches, double *total_ms) {
    double sum = 0.0;
    for (int32_t i = 0; i < g_timing.used; ++i) {
        hipError_t e = hipEventSynchronize(g_timing.ev[2 * i + 1]);
        if (e != hipSuccess) return e;
        float ms = 0.0f;
        e = hipEventElapsedTime(&ms, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]);
        if (e != hipSuccess) return e;
        sum += ms;
    }
    *launches = g_timing.used;
    *total_ms = sum;
    g_timing.used = 0;
    g_timing.dropped = 0;
    return hipSuccess;
}

hipError_t read_assign_stats(const void *workspace, int64_t T, int64_t E, int64_t B,
                             SolveCtrl *out, hipStream_t stream) {
    const size_t wst = make_layout(T, E).total;
    hipError_t err = hipMemcpy2DAsync(out, sizeof(SolveCtrl), workspace, wst, sizeof(SolveCtrl),
                                      (size_t)B, hipMemcpyDeviceToHost, stream);
    if (err != hipSuccess) return err;
    return hipStreamSynchronize(stream);
}

hipError_t check_scores_finite(const float *S, int64_t n, int64_t T, int64_t E, void *workspace,
                               int *bad, hipStream_t stream) {
    SolveCtrl *ctrl = static_cast<SolveCtrl *>(workspace);
    uint32_t *rpart =
        reinterpret_cast<uint32_t *>(static_cast<char *>(workspace) + make_layout(T, E).rpart);
    AssignParams p{};
    hipLaunchKernelGGL(init_kernel, dim3(1), dim3(256), 0, stream, ctrl, (void *)nullptr, 0, p,
                       (int64_t)0);
    hipLaunchKernelGGL(range_kernel<FloatMode>, dim3(kRangeBlocks), dim3(256), 0, stream, S, n,
                       rpart, (int64_t)0);
    hipLaunchKernelGGL(range_finish_kernel, dim3(1), dim3(256), 0, stream, ctrl, rpart,
                       kRangeBlocks, (int64_t)0);
    SolveCtrl h{};
    hipError_t err = read_assign_stats(workspace, T, E, 1, &h, stream);
    if (err != hipSuccess) return err;
    *bad = (h.unconverged_experts & (1 << 30)) ? 1 : 0;
    return hipSuccess;
}

}  // namespace base
