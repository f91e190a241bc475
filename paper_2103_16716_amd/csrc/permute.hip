// Routing permute (Fig. 2 caption; Sec. 3): gather token rows into
// expert-contiguous order, out[k] = in[perm[k]], or scatter them back,
// out[perm[k]] = in[k]. Pure data movement, bound by HBM bandwidth: every
// byte of a row is read once and written once with 16-byte vector accesses.
#include "common.hpp"
#include "internal.hpp"

namespace base {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kPerThread = 4;                          // 16-byte chunks in flight per thread
constexpr int kChunksPerBlock = kThreads * kPerThread; // 16 KiB per block

// A block owns `rows_per_block` consecutive rows k of the permuted index
// space, flattened into (row, chunk) pairs that its threads stride over.
__global__ __launch_bounds__(kThreads) void permute_rows_kernel(
    const u32x4 *__restrict__ in, const int32_t *__restrict__ perm, u32x4 *__restrict__ out,
    int64_t T, int64_t chunks_per_row, int64_t rows_per_block, int inverse) {
    const int64_t k0 = (int64_t)blockIdx.x * rows_per_block;
    const int64_t rows = (T - k0) < rows_per_block ? (T - k0) : rows_per_block;
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
                const int64_t p = perm[k];
                const int64_t src = inverse ? k : p;
                dst[u] = (inverse ? p : k) * chunks_per_row + c;
                v[u] = __builtin_nontemporal_load(in + src * chunks_per_row + c);
            }
        }
#pragma unroll
        for (int u = 0; u < kPerThread; ++u)
            if (dst[u] >= 0) __builtin_nontemporal_store(v[u], out + dst[u]);
    }
}

}  // namespace

hipError_t launch_permute(const void *in, const int32_t *perm, void *out, int64_t T,
                          int64_t row_bytes, int inverse, hipStream_t stream) {
    const int64_t chunks = row_bytes / 16;
    int64_t rows_per_block = kChunksPerBlock / chunks;
    if (rows_per_block < 1) rows_per_block = 1;
    const int64_t blocks = (T + rows_per_block - 1) / rows_per_block;
    hipLaunchKernelGGL(permute_rows_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                       static_cast<const u32x4 *>(in), perm, static_cast<u32x4 *>(out), T, chunks,
                       rows_per_block, inverse);
    return hipGetLastError();
}

}  // namespace base
