// Test-time routing and the gated residual of a BASE layer.
//
// Sec. 3.2.2: at test time every token goes to its highest-scoring expert
// (no balance). Sec. 3.1, Eq. 1: the layer returns
//     y_t = sigmoid(h_t . w_{a_t}) f_{a_t}(h_t) + h_t,
// where the expert output f arrives in routed (expert-contiguous) order:
// row k belongs to token perm[k] (Fig. 2 caption; Sec. 3, the output returns
// to the token's position). The gate score h_t . w_{a_t} is the affinity
// S[t, a_t] already computed for the routing.
//
// Kernels:
//   greedy_route_kernel    E <= 512: the whole routing in one launch (argmax,
//                          counts, grid barrier, offsets, placement), see below
//   otherwise, or when the device cannot hold the blocks at once:
//   greedy_count_kernel    argmax per token (16 lanes per token, 8 experts
//                          per lane per chunk of 128) + per-block expert counts
//   greedy_place_kernel    E <= 512: offsets and placement in one launch
//   greedy_scan_kernel     per-expert exclusive scan over the blocks
//   greedy_offsets_kernel  exclusive scan of the expert totals -> offsets
//   greedy_scatter_kernel  stable counting sort -> perm
//   gate_combine_kernel    y = g * F[k] + H[t] for t = perm[k] (16-byte chunks);
//                          also over B problems of T tokens with a shuffle
//                          index (Sec. 3.2.1, Shuffling), see below
//   gate_rows_kernel       backward per routed row: dS, dF, dH
//   gate_dw_kernel         dW[e] = sum over expert e's rows of dS_t h_t
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <mutex>
#include <random>

#include "base.h"
#include "internal.hpp"

namespace base {
namespace {

constexpr int kGreedyTile = 64;    // tokens per block of the greedy count
constexpr int kGroup = 16;         // lanes per token in the argmax

__device__ inline int lane_of() { return threadIdx.x & 63; }

__device__ inline float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// fp32 -> bf16, round to nearest even (NaN kept quiet).
__device__ inline uint32_t f32_to_bf16_bits(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ inline float gate_of(float s) { return 1.0f / (1.0f + expf(-s)); }

// ---------------------------------------------------------------- greedy --

__global__ __launch_bounds__(256) void greedy_count_kernel(const float *S, int T, int E,
                                                           int32_t *assign, int32_t *blk) {
    extern __shared__ int hist[];
    for (int e = threadIdx.x; e < E; e += blockDim.x) hist[e] = 0;
    __syncthreads();
    const int gl = lane_of() & (kGroup - 1);
    const int per_pass = blockDim.x / kGroup;
    const int t0 = blockIdx.x * kGreedyTile;
    for (int j = threadIdx.x / kGroup; j < kGreedyTile; j += per_pass) {
        const int t = t0 + j;
        const bool valid = t < T;
        float best = -INFINITY;
        int be = 0x7fffffff;
        if (valid) {
            const float *row = S + (int64_t)t * E;
            for (int base = 0; base < E; base += 8 * kGroup) {
                const int e0 = base + 8 * gl;
                if (e0 >= E) break;
                float v[8];
                if (e0 + 8 <= E && (E & 3) == 0) {   // 16-byte aligned rows
                    const float4 x = *reinterpret_cast<const float4 *>(row + e0);
                    const float4 y = *reinterpret_cast<const float4 *>(row + e0 + 4);
                    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
                    v[4] = y.x; v[5] = y.y; v[6] = y.z; v[7] = y.w;
                } else {
#pragma unroll
                    for (int q = 0; q < 8; ++q) v[q] = e0 + q < E ? row[e0 + q] : -INFINITY;
                }
#pragma unroll
                for (int q = 0; q < 8; ++q) {   // ascending scan: ties keep the lower expert
                    const bool better = (e0 + q < E) & (v[q] > best);
                    best = better ? v[q] : best;
                    be = better ? e0 + q : be;
                }
            }
        }
#pragma unroll
        for (int off = kGroup / 2; off > 0; off >>= 1) {
            // (selects, not branches: the lanes of a wave disagree here)
            const float ob = __shfl_xor(best, off);
            const int oe = __shfl_xor(be, off);
            const bool take = (ob > best) | ((ob == best) & (oe < be));
            best = take ? ob : best;
            be = take ? oe : be;
        }
        if (valid && gl == 0) {
            const int a = (be >= 0 && be < E) ? be : 0;   // a row of NaN/-inf goes to expert 0
            assign[t] = a;
            atomicAdd(&hist[a], 1);
        }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < E; e += blockDim.x) blk[(int64_t)blockIdx.x * E + e] = hist[e];
}

// Expert e's block counts -> exclusive running sums (in place); the total goes
// to offsets[e + 1].
__global__ __launch_bounds__(256) void greedy_scan_kernel(int32_t *blk, int nblk, int E,
                                                          int32_t *offsets) {
    __shared__ int wsum[4];
    __shared__ int carry;
    const int e = blockIdx.x;
    const int lane = lane_of();
    const int wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) carry = 0;
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
    if (threadIdx.x == 0) offsets[e + 1] = carry;
}

// offsets[1..E] hold the totals; turn them into the exclusive scan (one block).
__global__ __launch_bounds__(1024) void greedy_offsets_kernel(int32_t *offsets, int E) {
    __shared__ int wsum[16];
    __shared__ int carry;
    const int lane = lane_of();
    const int wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) {
        carry = 0;
        offsets[0] = 0;
    }
    __syncthreads();
    for (int e0 = 0; e0 < E; e0 += 1024) {
        const int e = e0 + threadIdx.x;
        const int v = e < E ? offsets[e + 1] : 0;
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
        __syncthreads();
        if (e < E) offsets[e + 1] = before + incl;
        __syncthreads();
        if (threadIdx.x == 0) {
            int tot = 0;
            for (int w = 0; w < 16; ++w) tot += wsum[w];
            carry += tot;
        }
        __syncthreads();
    }
}

// The placement after greedy_count_kernel, in one launch: every block takes
// kPlaceTiles consecutive count tiles (one token per thread). Each block
// reads the whole tile-count matrix (coalesced rows, many loads in flight)
// into the experts' totals and the counts of the tiles before its own,
// scans the totals into the expert offsets (block 0 writes offsets[0..E]),
// and places every token at
//     offsets[a] + (tokens of a in all earlier tiles)
//                + (rank of t among its own tile's tokens of a),
// the stable counting sort of greedy_scatter_kernel. E <= kPlaceMaxE.
constexpr int kPlaceTiles = 16;
constexpr int kPlaceThreads = kPlaceTiles * kGreedyTile;   // 1024
constexpr int kPlaceMaxE = 512;

__global__ __launch_bounds__(kPlaceThreads) void greedy_place_kernel(const int32_t *assign, int T,
                                                                     int E, const int32_t *blk,
                                                                     int nblk, int32_t *offsets,
                                                                     int32_t *perm) {
    __shared__ int tot[kPlaceMaxE];                  // totals, then exclusive offsets
    __shared__ int own[kPlaceTiles + 1][kPlaceMaxE];  // counts before each of the block's tiles
    __shared__ int part[kPlaceThreads / 64];
    __shared__ int loc[kPlaceThreads];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int tile0 = blockIdx.x * kPlaceTiles;
    for (int i = tid; i < (kPlaceTiles + 1) * kPlaceMaxE; i += kPlaceThreads) (&own[0][0])[i] = 0;
    for (int e = tid; e < E; e += kPlaceThreads) tot[e] = 0;
    __syncthreads();
    // (1) Thread (c, r): column c of the counts, rows r, r + rows, ...;
    // totals and the tiles before the block's first by LDS atomics, the
    // block's own tiles by row. Four columns per 16-byte load when E allows.
    if ((E & 3) == 0) {
        const int q4 = E / 4;
        const int rows = kPlaceThreads / q4;
        const int c = tid % q4, r0 = tid / q4;
        if (r0 < rows) {
            int tb[4] = {0, 0, 0, 0}, ta[4] = {0, 0, 0, 0};
            const int4 *b4 = reinterpret_cast<const int4 *>(blk);
            for (int b0 = r0; b0 < nblk; b0 += 16 * rows) {
                int4 v[16];
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int b = b0 + u * rows;
                    v[u] = b < nblk ? b4[(int64_t)b * q4 + c] : make_int4(0, 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < 16; ++u) {
                    const int b = b0 + u * rows;
                    const int w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        if (b < tile0) tb[k] += w[k];
                        else ta[k] += w[k];
                        if (b >= tile0 && b < tile0 + kPlaceTiles) own[b - tile0 + 1][4 * c + k] = w[k];
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                atomicAdd(&own[0][4 * c + k], tb[k]);
                atomicAdd(&tot[4 * c + k], tb[k] + ta[k]);
            }
        }
    } else {
    const int rows = kPlaceThreads / E;   // >= 2 as E <= kPlaceMaxE
    const int c = tid % E, r0 = tid / E;
    if (r0 < rows) {
        int tb = 0, ta = 0;
        for (int b0 = r0; b0 < nblk; b0 += 8 * rows) {
            int v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int b = b0 + u * rows;
                v[u] = b < nblk ? blk[(int64_t)b * E + c] : 0;
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int b = b0 + u * rows;
                if (b < tile0) tb += v[u];
                else ta += v[u];
                if (b >= tile0 && b < tile0 + kPlaceTiles) own[b - tile0 + 1][c] = v[u];
            }
        }
        atomicAdd(&own[0][c], tb);
        atomicAdd(&tot[c], tb + ta);
    }
    }
    const int t = tile0 * kGreedyTile + tid;
    const int a = t < T ? assign[t] : -1;
    loc[tid] = a;
    __syncthreads();
    // (2) own[q][e]: tokens of e in every tile before the block's tile q
    for (int e = tid; e < E; e += kPlaceThreads) {
        int run = own[0][e];
        for (int q = 1; q <= kPlaceTiles; ++q) {
            const int v = own[q][e];
            own[q][e] = run;
            run += v;
        }
        own[0][e] = 0;
    }
    // exclusive scan of the totals over the experts
    {
        const int v = tid < E ? tot[tid] : 0;
        int incl = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int o = __shfl_up(incl, off);
            if (lane >= off) incl += o;
        }
        if (lane == 63) part[wave] = incl;
        __syncthreads();
        int base = 0;
        for (int w = 0; w < wave; ++w) base += part[w];
        if (tid < E) tot[tid] = base + incl - v;
        if (blockIdx.x == 0 && tid < E) offsets[tid + 1] = base + incl;
        if (blockIdx.x == 0 && tid == 0) offsets[0] = 0;
    }
    __syncthreads();
    if (a < 0 || a >= E) return;
    // (3) the token's place
    const int tl = tid / kGreedyTile;
    int pos = tot[a] + own[tl + 1][a];
    for (int j = tl * kGreedyTile; j < tid; ++j) pos += (loc[j] == a);
    if (pos >= 0 && pos < T) perm[pos] = t;
}

// Greedy routing in one launch (E <= kPlaceMaxE): block b takes tokens
// [b TB, (b + 1) TB), TB a multiple of kRouteTile.
//   (1) argmax, 8 lanes per token (up to four 16-byte loads per lane in
//       flight), the block's expert counts (LDS) to row b of the count
//       matrix, and each token's expert kept in LDS;
//   (2) a grid barrier;
//   (3) every block sums the count matrix into the experts' totals and the
//       counts of the blocks before its own, scans the totals into the
//       offsets (block 0 writes them) and places each token at
//           offsets[a] + (tokens of a in earlier blocks)
//                      + (tokens of a before t in its own block),
//       the same stable counting sort as the multi-launch path.
// The host launches no more blocks than are resident at once, so every
// block reaches the barrier. Its words sit in the workspace header and hold
// anything at entry: block 0 clears the arrival count and the release word
// and then publishes the launch's tag (nonzero); the other blocks arrive
// only after they see the tag, the last arrival stores the tag into the
// release word (on its own line, so the waits do not slow the arrivals),
// and block 0 clears the published tag once every block has arrived, so
// the next launch on the stream starts from a clean one. Waits are bounded: a block
// that gives up (a block never scheduled) leaves its tokens unplaced and
// marks them assign[t] = -1.
constexpr int kRouteThreads = 1024;
constexpr int kRouteLanes = 8;                                  // lanes per token
constexpr int kRouteTile = kRouteThreads / kRouteLanes;         // 128 tokens per pass
constexpr int kRouteMaxTB = 4096;                               // tokens per block (LDS)
// Blocks per launch: more compute units read the scores sooner, more blocks
// make the barrier and every block's read of the count matrix longer; the
// measured optimum at 32768 x 128 and 65536 x 256 scores lies near 128-192.
constexpr int kRouteMaxBlocks = 192;
constexpr size_t kRouteHeader = 1024;                           // barrier words
constexpr uint32_t kRoutePolls = 1u << 24;

__device__ inline bool route_wait(const uint64_t *w, uint64_t want) {
    for (uint32_t polls = 0;; ++polls) {
        if (__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == want) return true;
        if (polls >= kRoutePolls) return false;
        __builtin_amdgcn_s_sleep(2);
    }
}

__global__ __launch_bounds__(kRouteThreads) void greedy_route_kernel(
    const float *S, int T, int E, int TB, int32_t *assign, int32_t *perm, int32_t *offsets,
    uint64_t *bar, int32_t *cnt, uint64_t tag) {
    __shared__ int hist[kPlaceMaxE];   // the block's counts
    __shared__ int pre[kPlaceMaxE];    // counts of the blocks before this one
    __shared__ int tot[kPlaceMaxE];    // totals, then exclusive offsets
    __shared__ int loc[kRouteMaxTB];   // experts of the block's tokens (-1: none)
    __shared__ int part[kRouteThreads / 64];
    __shared__ int ok;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int b = blockIdx.x, G = gridDim.x;
    uint64_t *arrivals = bar;        // own 256-byte lines
    uint64_t *armed = bar + 32;
    uint64_t *release = bar + 64;
    if (b == 0 && tid == 0) {
        __hip_atomic_store(arrivals, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(release, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __hip_atomic_store(armed, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    for (int e = tid; e < E; e += kRouteThreads) { hist[e] = 0; pre[e] = 0; tot[e] = 0; }
    __syncthreads();
    // (1)
    const int g = tid / kRouteLanes, gl = tid % kRouteLanes;
    const int t0 = b * TB;
    for (int i0 = 0; i0 < TB; i0 += kRouteTile) {
        const int i = i0 + g;
        const int t = t0 + i;
        float best = -INFINITY;
        int be = 0x7fffffff;
        if (t < T) {
            const float *row = S + (int64_t)t * E;
            if ((E & 3) == 0) {
                for (int base = 0; base < E; base += 16 * kRouteLanes) {
                    float4 v[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int e = base + 4 * (kRouteLanes * u + gl);
                        v[u] = e < E ? *reinterpret_cast<const float4 *>(row + e)
                                     : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {   // ascending: ties keep the lower expert
                        const int e = base + 4 * (kRouteLanes * u + gl);
                        const float x[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            const bool better = (e + q < E) & (x[q] > best);
                            best = better ? x[q] : best;
                            be = better ? e + q : be;
                        }
                    }
                }
            } else {
                for (int e = gl; e < E; e += kRouteLanes) {
                    const float x = row[e];
                    const bool better = x > best;
                    best = better ? x : best;
                    be = better ? e : be;
                }
            }
        }
#pragma unroll
        for (int off = kRouteLanes / 2; off > 0; off >>= 1) {
            const float ob = __shfl_xor(best, off);
            const int oe = __shfl_xor(be, off);
            const bool take = (ob > best) | ((ob == best) & (oe < be));
            best = take ? ob : best;
            be = take ? oe : be;
        }
        if (gl == 0) {
            int a = -1;
            if (t < T) {
                a = (be >= 0 && be < E) ? be : 0;   // a row of NaN/-inf goes to expert 0
                assign[t] = a;
                atomicAdd(&hist[a], 1);
            }
            loc[i] = a;
        }
    }
    __syncthreads();
    for (int e = tid; e < E; e += kRouteThreads) cnt[(int64_t)b * E + e] = hist[e];
    // (2)
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this thread's stores are done
    __syncthreads();
    if (tid == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        bool fine = b == 0 || route_wait(armed, tag);
        if (fine) {
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            const uint64_t arrived = __hip_atomic_fetch_add(arrivals, 1ull, __ATOMIC_RELAXED,
                                                            __HIP_MEMORY_SCOPE_AGENT) + 1;
            if (arrived == (uint64_t)G) {   // the last arrival releases the others
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                __hip_atomic_store(release, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            } else {
                fine = route_wait(release, tag);
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        if (fine && b == 0)   // every block has arrived, so none still waits for the tag
            __hip_atomic_store(armed, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = fine ? 1 : 0;
    }
    __syncthreads();
    if (!ok) {
        for (int i = tid; i < TB; i += kRouteThreads)
            if (t0 + i < T) assign[t0 + i] = -1;
        return;
    }
    // (3) thread (c, r): column c of the counts, rows r, r + rows, ...
    if ((E & 3) == 0) {
        const int q4 = E / 4;
        const int rows = kRouteThreads / q4;
        const int c = tid % q4, r0 = tid / q4;
        if (r0 < rows) {
            int tb[4] = {0, 0, 0, 0}, ta[4] = {0, 0, 0, 0};
            const int4 *c4 = reinterpret_cast<const int4 *>(cnt);
            for (int k0 = r0; k0 < G; k0 += 8 * rows) {
                int4 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int k = k0 + u * rows;
                    v[u] = k < G ? c4[(int64_t)k * q4 + c] : make_int4(0, 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int k = k0 + u * rows;
                    const int w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        if (k < b) tb[q] += w[q];
                        ta[q] += w[q];
                    }
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                atomicAdd(&pre[4 * c + q], tb[q]);
                atomicAdd(&tot[4 * c + q], ta[q]);
            }
        }
    } else {
        const int rows = kRouteThreads / E;   // >= 2 as E <= kPlaceMaxE
        const int c = tid % E, r0 = tid / E;
        if (r0 < rows) {
            int tb = 0, ta = 0;
            for (int k = r0; k < G; k += rows) {
                const int v = cnt[(int64_t)k * E + c];
                if (k < b) tb += v;
                ta += v;
            }
            atomicAdd(&pre[c], tb);
            atomicAdd(&tot[c], ta);
        }
    }
    __syncthreads();
    {   // exclusive scan of the totals over the experts
        const int v = tid < E ? tot[tid] : 0;
        int incl = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int o = __shfl_up(incl, off);
            if (lane >= off) incl += o;
        }
        if (lane == 63) part[wave] = incl;
        __syncthreads();
        int base = 0;
        for (int w = 0; w < wave; ++w) base += part[w];
        if (tid < E) tot[tid] = base + incl - v + pre[tid];
        if (b == 0 && tid < E) offsets[tid + 1] = base + incl;
        if (b == 0 && tid == 0) offsets[0] = 0;
    }
    __syncthreads();
    // rank within the block: the token's 8 lanes split the earlier tokens
    for (int i0 = 0; i0 < TB; i0 += kRouteTile) {
        const int i = i0 + g;
        const int a = loc[i];
        int r = 0;
        if (a >= 0)
            for (int j = gl; j < i; j += kRouteLanes) r += loc[j] == a;
#pragma unroll
        for (int off = kRouteLanes / 2; off > 0; off >>= 1) r += __shfl_xor(r, off);
        if (gl == 0 && a >= 0) {
            const int pos = tot[a] + r;
            if (pos >= 0 && pos < T) perm[pos] = t0 + i;
        }
    }
}

// perm[offsets[a] + blk[block][a] + rank of t among the block's tokens of a] = t.
__global__ __launch_bounds__(kGreedyTile) void greedy_scatter_kernel(const int32_t *assign, int T,
                                                                     int E, const int32_t *blk,
                                                                     const int32_t *offsets,
                                                                     int32_t *perm) {
    __shared__ int loc[kGreedyTile];
    const int t = blockIdx.x * kGreedyTile + threadIdx.x;
    const int a = t < T ? assign[t] : -1;
    loc[threadIdx.x] = a;
    __syncthreads();
    if (a < 0 || a >= E) return;
    int rank = 0;
    for (int j = 0; j < (int)threadIdx.x; ++j) rank += (loc[j] == a);
    const int pos = offsets[a] + blk[(int64_t)blockIdx.x * E + a] + rank;
    if (pos >= 0 && pos < T) perm[pos] = t;
}

// ---------------------------------------------------------- gated residual --

// One 16-byte chunk of a row: 8 bf16 or 4 fp32 values, widened to fp32.
template <bool BF16>
struct Chunk {
    static constexpr int kN = BF16 ? 8 : 4;
    __device__ static void load(const void *base, int64_t chunk, float (&v)[8]) {
        const uint4 x = reinterpret_cast<const uint4 *>(base)[chunk];
        const uint32_t w[4] = {x.x, x.y, x.z, x.w};
        if (BF16) {
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = bf16_bits_to_f32((w[i >> 1] >> (16 * (i & 1))) & 0xffffu);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) v[i] = __uint_as_float(w[i]);
        }
    }
    __device__ static void store(void *base, int64_t chunk, const float (&v)[8]) {
        uint32_t w[4];
        if (BF16) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                w[i] = f32_to_bf16_bits(v[2 * i]) | (f32_to_bf16_bits(v[2 * i + 1]) << 16);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) w[i] = __float_as_uint(v[i]);
        }
        reinterpret_cast<uint4 *>(base)[chunk] = make_uint4(w[0], w[1], w[2], w[3]);
    }
};

// N = B T routed rows. Row k of problem b = k / T holds worker token
// w = b T + perm[k], whose gate is g = sigmoid(S[w, assign[w]]) (S and
// assign in worker order); its original token is t = shuffle[w] (t = w
// without a shuffle). y[t] = g F[k] + H[t]. Each thread takes 16-byte
// chunks; a row is ncs chunks.
template <bool BF16>
__global__ __launch_bounds__(256) void gate_combine_kernel(const void *F, const void *H,
                                                           const float *S,
                                                           const int32_t *assign,
                                                           const int32_t *perm,
                                                           const int32_t *shuffle, void *Y,
                                                           int N, int T, int E, int ncs) {
    using Ck = Chunk<BF16>;
    const int64_t total = (int64_t)N * ncs;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int k = (int)(i / ncs);
        const int j = (int)(i - (int64_t)k * ncs);
        const int p = perm[k];
        if (p < 0 || p >= T) continue;   // not a permutation: undefined, but in bounds
        const int w = (N == T ? 0 : (k / T) * T) + p;
        const int t = shuffle == nullptr ? w : shuffle[w];
        if (t < 0 || t >= N) continue;
        int a = assign[w];
        a = (a >= 0 && a < E) ? a : 0;
        const float g = gate_of(S[(int64_t)w * E + a]);
        float f[8], h[8], y[8];
        Ck::load(F, (int64_t)k * ncs + j, f);
        Ck::load(H, (int64_t)t * ncs + j, h);
#pragma unroll
        for (int q = 0; q < Ck::kN; ++q) y[q] = fmaf(g, f[q], h[q]);
        Ck::store(Y, (int64_t)t * ncs + j, y);
    }
}

// Backward per routed row k (one block per row, grid-stride): with t =
// perm[k], a = assign[t], g = sigmoid(S[t, a]):
//   dS[t] = g (1 - g) (dY[t] . F[k]);  dF[k] = g dY[t];  dH[t] = dY[t] + dS[t] W[a].
constexpr int kRowRegs = 2;   // 16-byte chunks of a row a thread keeps in registers

template <bool BF16>
__global__ __launch_bounds__(256) void gate_rows_kernel(const void *dY, const void *F,
                                                        const void *W, const float *S,
                                                        const int32_t *assign,
                                                        const int32_t *perm, void *dH, void *dF,
                                                        float *dS, int T, int E, int ncs) {
    using Ck = Chunk<BF16>;
    __shared__ float part[4];
    if (ncs <= kRowRegs * (int)blockDim.x) {
        // The row fits the block's registers: dY, F and W are loaded once,
        // before the reduction, and dF needs no dS, so it is stored first;
        // after the reduction only dH remains. Same arithmetic, same order.
        for (int k = blockIdx.x; k < T; k += gridDim.x) {
            const int t = perm[k];
            const bool ok = t >= 0 && t < T;
            const int tt = ok ? t : 0;
            int a = assign[tt];
            a = (a >= 0 && a < E) ? a : 0;
            const float g = gate_of(S[(int64_t)tt * E + a]);
            float y[kRowRegs][8], f[kRowRegs][8], w[kRowRegs][8];
#pragma unroll
            for (int r = 0; r < kRowRegs; ++r) {
                const int j = threadIdx.x + r * blockDim.x;
                if (j < ncs) {
                    Ck::load(dY, (int64_t)tt * ncs + j, y[r]);
                    Ck::load(F, (int64_t)k * ncs + j, f[r]);
                    Ck::load(W, (int64_t)a * ncs + j, w[r]);
                }
            }
            float dot = 0.0f;
#pragma unroll
            for (int r = 0; r < kRowRegs; ++r) {
                const int j = threadIdx.x + r * blockDim.x;
                if (j < ncs) {
#pragma unroll
                    for (int q = 0; q < Ck::kN; ++q) dot = fmaf(y[r][q], f[r][q], dot);
                    if (ok) {
                        float o[8];
#pragma unroll
                        for (int q = 0; q < Ck::kN; ++q) o[q] = g * y[r][q];
                        Ck::store(dF, (int64_t)k * ncs + j, o);
                    }
                }
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) dot += __shfl_xor(dot, off);
            if (lane_of() == 0) part[threadIdx.x >> 6] = dot;
            __syncthreads();
            dot = 0.0f;
            for (int v = 0; v < (int)(blockDim.x >> 6); ++v) dot += part[v];
            __syncthreads();
            const float ds = g * (1.0f - g) * dot;
            if (!ok) continue;
            if (threadIdx.x == 0) dS[t] = ds;
#pragma unroll
            for (int r = 0; r < kRowRegs; ++r) {
                const int j = threadIdx.x + r * blockDim.x;
                if (j < ncs) {
                    float o[8];
#pragma unroll
                    for (int q = 0; q < Ck::kN; ++q) o[q] = fmaf(ds, w[r][q], y[r][q]);
                    Ck::store(dH, (int64_t)t * ncs + j, o);
                }
            }
        }
        return;
    }
    for (int k = blockIdx.x; k < T; k += gridDim.x) {
        const int t = perm[k];
        const bool ok = t >= 0 && t < T;
        const int tt = ok ? t : 0;
        int a = assign[tt];
        a = (a >= 0 && a < E) ? a : 0;
        const float g = gate_of(S[(int64_t)tt * E + a]);
        float dot = 0.0f;
        for (int j = threadIdx.x; j < ncs; j += blockDim.x) {
            float y[8], f[8];
            Ck::load(dY, (int64_t)tt * ncs + j, y);
            Ck::load(F, (int64_t)k * ncs + j, f);
#pragma unroll
            for (int q = 0; q < Ck::kN; ++q) dot = fmaf(y[q], f[q], dot);
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) dot += __shfl_xor(dot, off);
        if (lane_of() == 0) part[threadIdx.x >> 6] = dot;
        __syncthreads();
        dot = 0.0f;
        for (int w = 0; w < (int)(blockDim.x >> 6); ++w) dot += part[w];
        __syncthreads();
        const float ds = g * (1.0f - g) * dot;
        if (!ok) continue;
        if (threadIdx.x == 0) dS[t] = ds;
        for (int j = threadIdx.x; j < ncs; j += blockDim.x) {
            float y[8], w[8], o[8];
            Ck::load(dY, (int64_t)t * ncs + j, y);
#pragma unroll
            for (int q = 0; q < Ck::kN; ++q) o[q] = g * y[q];
            Ck::store(dF, (int64_t)k * ncs + j, o);
            Ck::load(W, (int64_t)a * ncs + j, w);
#pragma unroll
            for (int q = 0; q < Ck::kN; ++q) o[q] = fmaf(ds, w[q], y[q]);
            Ck::store(dH, (int64_t)t * ncs + j, o);
        }
    }
}

// dW[e][c] = sum over routed rows k in [offsets[e], offsets[e + 1]) of
// dS[t] H[t][c], t = perm[k]: per expert, a weighted sum of its tokens' rows,
// bound by reading each row of H once. Block = (expert, slab of 64 16-byte
// chunks of a row); lane l owns chunk l of the slab. The block's kDwWaves
// waves split the expert's rows (wave w takes k0 + w, k0 + w + kDwWaves, ...
// in ascending order, kDwRows rows in flight), then the wave partials are
// added in wave order: a fixed summation order, so the result is
// deterministic.
constexpr int kDwWaves = 8;
constexpr int kDwRows = 4;

template <bool BF16>
__global__ __launch_bounds__(64 * kDwWaves) void gate_dw_kernel(const void *H, const float *dS,
                                                                const int32_t *perm,
                                                                const int32_t *offsets,
                                                                float *dW, int T, int E,
                                                                int ncs) {
    using Ck = Chunk<BF16>;
    __shared__ float part[kDwWaves][64][Ck::kN];
    const int e = blockIdx.x;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int j = blockIdx.y * 64 + lane;
    int k0 = offsets[e], k1 = offsets[e + 1];
    k0 = k0 < 0 ? 0 : (k0 > T ? T : k0);
    k1 = k1 < k0 ? k0 : (k1 > T ? T : k1);
    float acc[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    if (j < ncs) {
        for (int k = k0 + wave; k < k1; k += kDwWaves * kDwRows) {
            int t[kDwRows];
            float w[kDwRows], h[kDwRows][8];
#pragma unroll
            for (int u = 0; u < kDwRows; ++u) {
                const int kk = k + u * kDwWaves;
                t[u] = kk < k1 ? perm[kk] : -1;
                if (t[u] >= T) t[u] = -1;
            }
#pragma unroll
            for (int u = 0; u < kDwRows; ++u) {
                w[u] = 0.0f;
                if (t[u] >= 0) {
                    w[u] = dS[t[u]];
                    Ck::load(H, (int64_t)t[u] * ncs + j, h[u]);
                }
            }
#pragma unroll
            for (int u = 0; u < kDwRows; ++u)
                if (t[u] >= 0) {
#pragma unroll
                    for (int q = 0; q < Ck::kN; ++q) acc[q] = fmaf(w[u], h[u][q], acc[q]);
                }
        }
    }
#pragma unroll
    for (int q = 0; q < Ck::kN; ++q) part[wave][lane][q] = acc[q];
    __syncthreads();
    if (wave == 0 && j < ncs) {
        float o[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int q = 0; q < Ck::kN; ++q) {
            float v = part[0][lane][q];
            for (int w = 1; w < kDwWaves; ++w) v += part[w][lane][q];
            o[q] = v;
        }
        float4 *dst = reinterpret_cast<float4 *>(dW + ((int64_t)e * ncs + j) * Ck::kN);
        dst[0] = make_float4(o[0], o[1], o[2], o[3]);
        if (BF16) dst[1] = make_float4(o[4], o[5], o[6], o[7]);
    }
}

}  // namespace

size_t greedy_workspace_size(int64_t T, int64_t E) {
    const int64_t nblk = (T + kGreedyTile - 1) / kGreedyTile;
    return kRouteHeader + ((size_t)(nblk * E * 4 + 255) & ~size_t(255));
}

namespace {

// Compute units and resident blocks of greedy_route_kernel per compute unit
// on the current device (0 when the runtime cannot tell), looked up once.
int route_capacity() {
    constexpr int kDevices = 64;
    static std::mutex mu;
    static int known[kDevices] = {}, cap[kDevices] = {};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kDevices) {
        (void)hipGetLastError();
        return 0;
    }
    std::lock_guard<std::mutex> lock(mu);
    if (!known[dev]) {
        int cus = 0, per_cu = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per_cu, reinterpret_cast<const void *>(greedy_route_kernel), kRouteThreads, 0) !=
            hipSuccess)
            per_cu = 0;
        (void)hipGetLastError();
        cap[dev] = cus > 0 && per_cu > 0 ? cus * per_cu : 0;
        known[dev] = 1;
    }
    return cap[dev];
}

// A nonzero tag per launch, from a per-process random start.
uint64_t route_tag() {
    static std::atomic<uint64_t> next{[] {
        std::random_device rd;
        const uint64_t r = ((uint64_t)rd() << 32) ^ rd();
        return r ^ (uint64_t)std::chrono::steady_clock::now().time_since_epoch().count();
    }()};
    const uint64_t t = next.fetch_add(1, std::memory_order_relaxed);
    return t == 0 ? 1 : t;
}

}  // namespace

hipError_t launch_greedy(const float *S, int64_t T, int64_t E, int32_t *assign, int32_t *perm,
                         int32_t *offsets, void *workspace, hipStream_t s) {
    const int nblk = (int)((T + kGreedyTile - 1) / kGreedyTile);
    uint64_t *bar = static_cast<uint64_t *>(workspace);
    int32_t *blk = reinterpret_cast<int32_t *>(static_cast<char *>(workspace) + kRouteHeader);
    if (E <= kPlaceMaxE) {
        // One launch when every block can be resident: as few blocks as keep
        // the tokens per block within the LDS list.
        const int64_t cap = std::min<int64_t>(route_capacity(), kRouteMaxBlocks);
        const int64_t tiles = (T + kRouteTile - 1) / kRouteTile;
        if (cap > 0 && tiles <= cap * (kRouteMaxTB / kRouteTile)) {
            const int64_t per = (tiles + cap - 1) / cap;          // passes per block
            const int64_t TB = per * kRouteTile;
            const int64_t G = (T + TB - 1) / TB;                  // <= cap, <= nblk
            hipLaunchKernelGGL(greedy_route_kernel, dim3((unsigned)G), dim3(kRouteThreads), 0, s,
                               S, (int)T, (int)E, (int)TB, assign, perm, offsets, bar, blk,
                               route_tag());
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL(greedy_count_kernel, dim3(nblk), dim3(256), (size_t)E * sizeof(int), s, S,
                       (int)T, (int)E, assign, blk);
    if (E <= kPlaceMaxE) {
        const int pblk = (nblk + kPlaceTiles - 1) / kPlaceTiles;
        hipLaunchKernelGGL(greedy_place_kernel, dim3(pblk), dim3(kPlaceThreads), 0, s, assign,
                           (int)T, (int)E, blk, nblk, offsets, perm);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(greedy_scan_kernel, dim3((unsigned)E), dim3(256), 0, s, blk, nblk, (int)E,
                       offsets);
    hipLaunchKernelGGL(greedy_offsets_kernel, dim3(1), dim3(1024), 0, s, offsets, (int)E);
    hipLaunchKernelGGL(greedy_scatter_kernel, dim3(nblk), dim3(kGreedyTile), 0, s, assign, (int)T,
                       (int)E, blk, offsets, perm);
    return hipGetLastError();
}

hipError_t launch_gate_combine(const void *F, const void *H, const float *S,
                               const int32_t *assign, const int32_t *perm,
                               const int32_t *shuffle, void *Y, int64_t B, int64_t T, int64_t E,
                               int64_t d, int bf16, hipStream_t s) {
    const int ncs = (int)(d / (bf16 ? 8 : 4));
    const int64_t N = B * T;
    int64_t total = N * ncs;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (bf16)
        hipLaunchKernelGGL(gate_combine_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, s, F,
                           H, S, assign, perm, shuffle, Y, (int)N, (int)T, (int)E, ncs);
    else
        hipLaunchKernelGGL(gate_combine_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, s, F,
                           H, S, assign, perm, shuffle, Y, (int)N, (int)T, (int)E, ncs);
    return hipGetLastError();
}

hipError_t launch_gate_backward(const void *dY, const void *F, const void *H, const void *W,
                                const float *S, const int32_t *assign, const int32_t *perm,
                                const int32_t *offsets, void *dH, void *dF, float *dW, float *dS,
                                int64_t T, int64_t E, int64_t d, int bf16, hipStream_t s) {
    const int ncs = (int)(d / (bf16 ? 8 : 4));
    const int rows = (int)(T < 65536 ? T : 65536);
    const dim3 dwg((unsigned)E, (unsigned)((ncs + 63) / 64));
    if (bf16) {
        hipLaunchKernelGGL(gate_rows_kernel<true>, dim3(rows), dim3(256), 0, s, dY, F, W, S, assign,
                           perm, dH, dF, dS, (int)T, (int)E, ncs);
        hipLaunchKernelGGL(gate_dw_kernel<true>, dwg, dim3(64 * kDwWaves), 0, s, H, dS, perm,
                           offsets, dW, (int)T, (int)E, ncs);
    } else {
        hipLaunchKernelGGL(gate_rows_kernel<false>, dim3(rows), dim3(256), 0, s, dY, F, W, S,
                           assign, perm, dH, dF, dS, (int)T, (int)E, ncs);
        hipLaunchKernelGGL(gate_dw_kernel<false>, dwg, dim3(64 * kDwWaves), 0, s, H, dS, perm,
                           offsets, dW, (int)T, (int)E, ncs);
    }
    return hipGetLastError();
}

}  // namespace base
