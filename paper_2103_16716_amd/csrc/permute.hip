// Routing permute (Fig. 2 caption; Sec. 3): gather token rows into
// expert-contiguous order, out[k] = in[src(k)], or scatter them back,
// out[src(k)] = in[k]. Pure data movement, bound by HBM bandwidth: every
// byte of a row is read once and written once with 16-byte vector accesses.
//
// The rows form B problems of T rows each (B = 1: one problem). Row k of
// problem b = k / T takes its source from that problem's sort vector,
// j = b T + perm[k], and, when a shuffle index is given, src(k) = rows[j]
// (Sec. 3.2.1, Shuffling: worker b's token j came from row rows[j] of the
// unshuffled batch), else src(k) = j. Routing a shuffled batch is then one
// pass over the rows, with no shuffled copy. Entries out of range skip the
// row (memory-safe; the result is then not a permutation).
#include "common.hpp"
#include "internal.hpp"

namespace base {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
// 16-byte chunks in flight per thread. Two (8 KiB blocks) against four
// (16 KiB): 59 -> 53 us for 32768 rows of 4 KiB, 199 -> 184 us for 65536
// rows of 8 KiB, 921 -> 808 us for 256 shuffled problems of 2048 rows (one
// chunk, or 128-thread blocks, about the same as two; eight slower).
constexpr int kPerThread = 2;
constexpr int kChunksPerBlock = kThreads * kPerThread; // 8 KiB per block

// Source row of routed row k (see above), or -1 when an index is out of range.
__device__ inline int64_t routed_source(const int32_t *__restrict__ perm,
                                        const int32_t *__restrict__ shuffle, int k, int T,
                                        int N) {
    const int p = perm[k];
    if (p < 0 || p >= T) return -1;
    const int j = (T == N ? 0 : (k / T) * T) + p;
    if (shuffle == nullptr) return j;
    const int r = shuffle[j];
    return (r >= 0 && r < N) ? r : -1;
}

// A block owns `rows_per_block` consecutive rows k of the permuted index
// space, flattened into (row, chunk) pairs that its threads stride over.
// N = B T rows in all.
__global__ __launch_bounds__(kThreads) void permute_rows_kernel(
    const u32x4 *__restrict__ in, const int32_t *__restrict__ perm,
    const int32_t *__restrict__ shuffle, u32x4 *__restrict__ out, int N, int T,
    int64_t chunks_per_row, int64_t rows_per_block, int inverse) {
    const int64_t k0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t rows = (N - k0) < rows_per_block ? (N - k0) : rows_per_block;
    const int64_t total = rows * chunks_per_row;
    for (int64_t base = 0; base < total; base += kChunksPerBlock) {
        u32x4 v[kPerThread];
        int64_t dst[kPerThread];
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int64_t f = base + threadIdx.x + (int64_t)u * kThreads;
            dst[u] = -1;
            if (f < total) {
                const int64_t r = f / chunks_per_row;
                const int64_t c = f - r * chunks_per_row;
                const int64_t k = k0 + r;
                const int64_t p = routed_source(perm, shuffle, (int)k, T, N);
                if (p >= 0) {
                    const int64_t src = inverse ? k : p;
                    dst[u] = (inverse ? p : k) * chunks_per_row + c;
                    v[u] = __builtin_nontemporal_load(in + src * chunks_per_row + c);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kPerThread; ++u)
            if (dst[u] >= 0) __builtin_nontemporal_store(v[u], out + dst[u]);
    }
}

}  // namespace

hipError_t launch_permute(const void *in, const int32_t *perm, const int32_t *shuffle,
                          void *out, int64_t B, int64_t T, int64_t row_bytes, int inverse,
                          hipStream_t stream) {
    const int64_t chunks = row_bytes / 16;
    const int64_t N = B * T;
    int64_t rows_per_block = kChunksPerBlock / chunks;
    if (rows_per_block < 1) rows_per_block = 1;
    const int64_t blocks = (N + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL(permute_rows_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                       static_cast<const u32x4 *>(in), perm, shuffle, static_cast<u32x4 *>(out),
                       (int)N, (int)T, chunks, rows_per_block, inverse);
    return hipGetLastError();
}

}  // namespace base
