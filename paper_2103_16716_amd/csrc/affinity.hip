// Token-expert affinity S = H . W^T (Sec. 3.1, Eq. 2), S[t, e] = h_t . w_e.
//
// bf16 path: a tiled GEMM on the CDNA4 matrix cores (v_mfma_f32_32x32x16_bf16,
// fp32 accumulation). The contraction dimension is the model dimension d,
// contiguous in both H and W. The GEMM is bandwidth-bound at every shape of
// interest (arithmetic intensity about 2E/(2+4E/d) flop per byte, well below
// the MFMA ridge): H is streamed from HBM exactly once, W (at most a few MiB)
// is re-read from L2 by every block, and the kernel is organised around
// keeping enough HBM reads in flight.
//
// With d % 64 == 0 (affinity_bf16_pipe_kernel): a block owns 128 tokens x
// 128 experts (one block per compute unit at T = 32768), eight waves of
// 32 x 64 outputs. Chunks of 64 elements of d of both operands go straight
// from global memory into a ring of kStages LDS stages (16-byte LDS-direct
// loads, no register staging), kStages - 1 chunks ahead of the one being
// multiplied; a 16-byte slot s of LDS row r holds the row's chunk s ^ (r % 8),
// so the matrix-core operand reads (eight rows per 128-byte row group) fall
// on distinct banks. When those tiles would cover fewer than 128 blocks
// (affinity_bf16_small_kernel): 32 x 32 tiles, four waves splitting d and
// summing in a fixed order. Otherwise (affinity_bf16_kernel) 64 x 128
// blocks with register-staged double buffering.
//
// fp32 path: a plain LDS-tiled FMA kernel (fp32 products and sums, no
// reduced-precision matrix instructions).
//
// Every kernel can read H through a row index (`rows`, null for the
// identity): output row i is then h_{rows[i]} . W^T. This is the random
// shuffle of tokens to workers (Sec. 3.2.1, Shuffling) folded into the GEMM's
// loads, so the shuffled copy of H is never written. An index outside
// [0, h_rows) gives a zero row (memory-safe; not a valid shuffle).
#include <mutex>

#include "common.hpp"
#include "internal.hpp"

namespace base {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kBM = 64;             // tokens per block
constexpr int kBN = 128;            // experts per block
constexpr int kBK = 64;             // bf16 elements of d per chunk
constexpr int kLdsRow = kBK + 8;    // padded LDS row (elements): 144 B, shifts 4 banks per row

__device__ inline int64_t source_row(const int32_t *rows, int64_t h_rows, int i) {
    if (rows == nullptr) return i;
    const int64_t r = rows[i];
    return (r >= 0 && r < h_rows) ? r : -1;
}

__global__ __launch_bounds__(256) void affinity_bf16_kernel(const uint16_t *__restrict__ H,
                                                            const int32_t *__restrict__ rows,
                                                            int64_t h_rows,
                                                            const uint16_t *__restrict__ W,
                                                            float *__restrict__ S, int T, int E,
                                                            int d) {
    __shared__ __attribute__((aligned(16))) uint16_t As[kBM * kLdsRow];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[kBN * kLdsRow];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int m0 = blockIdx.x * kBM;
    const int n0 = blockIdx.y * kBN;

    // Source rows of H for this thread's two staging chunks (fixed over k).
    int64_t hrow[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int r = (tid + 256 * i) >> 3;
        hrow[i] = m0 + r < T ? source_row(rows, h_rows, m0 + r) : -1;
    }

    // Global -> register staging: chunk c covers row c/8, elements (c%8)*8 .. +8.
    uint4 ra[2], rb[4];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int c = tid + 256 * i;
            const int k = k0 + (c & 7) * 8;
            ra[i] = make_uint4(0, 0, 0, 0);
            if (hrow[i] >= 0 && k < d)
                ra[i] = *reinterpret_cast<const uint4 *>(H + hrow[i] * d + k);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 256 * i;
            const int r = c >> 3;
            const int k = k0 + (c & 7) * 8;
            rb[i] = make_uint4(0, 0, 0, 0);
            if (n0 + r < E && k < d)
                rb[i] = *reinterpret_cast<const uint4 *>(W + (int64_t)(n0 + r) * d + k);
        }
    };
    auto sstore = [&]() {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int c = tid + 256 * i;
            *reinterpret_cast<uint4 *>(&As[(c >> 3) * kLdsRow + (c & 7) * 8]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = tid + 256 * i;
            *reinterpret_cast<uint4 *>(&Bs[(c >> 3) * kLdsRow + (c & 7) * 8]) = rb[i];
        }
    };

    // Wave layout: 2 x 2 waves, each 32 tokens x 64 experts = two 32x32 MFMA tiles.
    const int wm = wave & 1;
    const int wn = wave >> 1;
    f32x16_t acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[j][i] = 0.0f;

    const int lrow = lane & 31;     // operand row inside a 32-row tile
    const int lk = (lane >> 5) * 8; // this lane's 8 elements of the 16-wide k step

    gload(0);
    for (int k0 = 0; k0 < d; k0 += kBK) {
        __syncthreads();
        sstore();
        __syncthreads();
        if (k0 + kBK < d) gload(k0 + kBK);
#pragma unroll
        for (int ks = 0; ks < kBK; ks += 16) {
            const bf16x8_t a =
                *reinterpret_cast<const bf16x8_t *>(&As[(32 * wm + lrow) * kLdsRow + ks + lk]);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const bf16x8_t b = *reinterpret_cast<const bf16x8_t *>(
                    &Bs[(64 * wn + 32 * j + lrow) * kLdsRow + ks + lk]);
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
            }
        }
    }

    // 32x32 accumulator layout: lane holds column lane%32; register i holds
    // row 8*(i/4) + 4*(lane/32) + i%4.
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int e = n0 + 64 * wn + 32 * j + lrow;
        if (e >= E) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int t = m0 + 32 * wm + 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3);
            if (t < T) S[(int64_t)t * E + e] = acc[j][i];
        }
    }
}

// ---------------------------------------------------- pipelined bf16 GEMM --

constexpr int kPM = 128;                    // tokens per block
constexpr int kPN = 128;                    // experts per block
constexpr int kPK = 64;                     // elements of d per chunk (128 bytes a row)
constexpr int kPThreads = 512;              // 4 (tokens) x 2 (experts) waves
constexpr int kPTile = kPM * kPK * 2;       // bytes of one operand's chunk (16 KiB)
constexpr int kPStage = 2 * kPTile;
constexpr int kStages = 4;
constexpr size_t kPipeLds = (size_t)kStages * kPStage;   // 128 KiB
#define BASE_LDS __attribute__((address_space(3)))

// Waits until at most N vector-memory operations of this wave are in flight
// (the LDS-direct loads count until their data is in LDS).
template <int N>
__device__ inline void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt field");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Workgroup barrier with no memory wait of its own: each wave has already
// waited for the loads the barrier publishes. The empty asm statements keep
// the compiler from moving memory accesses across it.
__device__ inline void bare_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__global__ __launch_bounds__(kPThreads) void affinity_bf16_pipe_kernel(
    const uint16_t *__restrict__ H, const int32_t *__restrict__ rows, int64_t h_rows,
    const uint16_t *__restrict__ W, float *__restrict__ S, int T, int E, int d) {
    extern __shared__ __attribute__((aligned(1024))) unsigned char lds[];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // Blocks go to the eight XCDs in turn (block L to XCD L % 8). The nn
    // expert tiles of a token tile are placed on one XCD one after another
    // (the same L % 8, consecutive L / 8), so that the token tile's rows of H
    // come from memory once and from that XCD's L2 for the other expert
    // tiles. With one expert tile this is the identity.
    const int nn = (E + kPN - 1) / kPN;
    const int L = blockIdx.x;
    const int u = L >> 3;
    const int mt = (u / nn) * 8 + (L & 7);
    if (mt * kPM >= T) return;   // padding of the grid to whole groups of eight
    const int m0 = mt * kPM;
    const int n0 = (u % nn) * kPN;
    // This thread's two 16-byte slots of each operand's chunk: slot q = i *
    // 512 + tid is row q / 8, position q % 8, and holds the row's chunk
    // (q % 8) ^ (row % 8). Rows past T or E, and invalid source rows, read
    // a valid row; their outputs are not stored (or stored as zero).
    const uint16_t *ga[2], *gb[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int q = i * kPThreads + tid;
        const int r = q >> 3;
        const int c = (q & 7) ^ (r & 7);
        int64_t hr = m0 + r < T ? source_row(rows, h_rows, m0 + r) : 0;
        if (hr < 0) hr = 0;
        const int er = n0 + r < E ? n0 + r : E - 1;
        ga[i] = H + hr * d + c * 8;
        gb[i] = W + (int64_t)er * d + c * 8;
    }
    auto issue = [&](int kc) {
        BASE_LDS unsigned char *base = (BASE_LDS unsigned char *)lds + (kc % kStages) * kPStage;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int slot = (i * kPThreads + wave * 64) * 16;   // the wave's 1 KiB
            __builtin_amdgcn_global_load_lds((const void *)(ga[i] + (int64_t)kc * kPK),
                                             (BASE_LDS void *)(base + slot), 16, 0, 0);
            __builtin_amdgcn_global_load_lds((const void *)(gb[i] + (int64_t)kc * kPK),
                                             (BASE_LDS void *)(base + kPTile + slot), 16, 0, 0);
        }
    };
    const int wm = wave & 3;
    const int wn = wave >> 2;
    const int lrow = lane & 31;
    const int lhalf = lane >> 5;
    f32x16_t acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[j][i] = 0.0f;
    const int nk = d / kPK;
#pragma unroll
    for (int st = 0; st < kStages - 1; ++st)
        if (st < nk) issue(st);
    for (int kc = 0; kc < nk; ++kc) {
        // Chunk kc has landed once at most the later chunks' loads (four
        // per chunk) are in flight; after the barrier every wave's part of
        // it is in LDS and every wave is done with the stage refilled next.
        if (kc + kStages - 2 < nk) wait_vmcnt<4 * (kStages - 2)>();
        else wait_vmcnt<0>();
        bare_barrier();
        if (kc + kStages - 1 < nk) issue(kc + kStages - 1);
        const unsigned char *A = lds + (kc % kStages) * kPStage;
        const unsigned char *B = A + kPTile;
        const int ra = 32 * wm + lrow;
#pragma unroll
        for (int ks = 0; ks < kPK / 16; ++ks) {
            const int c = 2 * ks + lhalf;
            const bf16x8_t a =
                *reinterpret_cast<const bf16x8_t *>(A + ra * 128 + ((c ^ (ra & 7)) * 16));
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int rb = 64 * wn + 32 * j + lrow;
                const bf16x8_t b =
                    *reinterpret_cast<const bf16x8_t *>(B + rb * 128 + ((c ^ (rb & 7)) * 16));
                acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[j], 0, 0, 0);
            }
        }
    }
    // 32x32 accumulator layout: lane holds column lane % 32; register i holds
    // row 8 (i / 4) + 4 (lane / 32) + i % 4.
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int e = n0 + 64 * wn + 32 * j + lrow;
        if (e >= E) continue;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int t = m0 + 32 * wm + 8 * (i >> 2) + 4 * lhalf + (i & 3);
            if (t < T) S[(int64_t)t * E + e] = source_row(rows, h_rows, t) >= 0 ? acc[j][i] : 0.0f;
        }
    }
}

// ------------------------------------------------- small bf16 problems --
//
// When the 128 x 128 tiles would occupy few compute units (the per-worker
// shape T = 2048, E = 128 is 16 tiles), a block owns 32 tokens x 32 experts
// and its four waves split d: wave w takes the contiguous quarter of the
// 16-element steps, loading its MFMA operands straight from memory (eight
// steps in flight per lane), and the waves' partial tiles are added in LDS
// in wave order (a fixed order: the result does not depend on scheduling).
constexpr int kST = 32;
constexpr int kSWaves = 4;
constexpr int kSU = 4;   // steps per register set (two sets in flight)

__global__ __launch_bounds__(64 * kSWaves) void affinity_bf16_small_kernel(
    const uint16_t *__restrict__ H, const int32_t *__restrict__ rows, int64_t h_rows,
    const uint16_t *__restrict__ W, float *__restrict__ S, int T, int E, int d) {
    __shared__ float red[kSWaves - 1][16][64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int lrow = lane & 31;
    const int lhalf = lane >> 5;
    const int m0 = blockIdx.x * kST;
    const int n0 = blockIdx.y * kST;
    // A operand: token row m0 + lane % 32; B operand: expert row n0 + lane % 32;
    // lane / 32 picks the upper 8 of each 16-element step.
    int64_t hr = m0 + lrow < T ? source_row(rows, h_rows, m0 + lrow) : 0;
    if (hr < 0) hr = 0;
    const int er = n0 + lrow < E ? n0 + lrow : E - 1;
    const int q = d / 16 / kSWaves;   // steps per wave (d % 64 == 0)
    const uint16_t *pa = H + hr * d + (int64_t)wave * q * 16 + lhalf * 8;
    const uint16_t *pb = W + (int64_t)er * d + (int64_t)wave * q * 16 + lhalf * 8;
    f32x16_t acc;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
    bf16x8_t a0[kSU], b0[kSU], a1[kSU], b1[kSU];
    auto load = [&](bf16x8_t (&a)[kSU], bf16x8_t (&b)[kSU], int s0) {
#pragma unroll
        for (int u = 0; u < kSU; ++u) {
            if (s0 + u < q) {   // (uniform)
                a[u] = *reinterpret_cast<const bf16x8_t *>(pa + (int64_t)(s0 + u) * 16);
                b[u] = *reinterpret_cast<const bf16x8_t *>(pb + (int64_t)(s0 + u) * 16);
            }
        }
    };
    auto mma = [&](bf16x8_t (&a)[kSU], bf16x8_t (&b)[kSU], int s0) {
#pragma unroll
        for (int u = 0; u < kSU; ++u)
            if (s0 + u < q) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[u], b[u], acc, 0, 0, 0);
    };
    load(a0, b0, 0);
    for (int s0 = 0; s0 < q; s0 += 2 * kSU) {
        load(a1, b1, s0 + kSU);
        mma(a0, b0, s0);
        load(a0, b0, s0 + 2 * kSU);
        mma(a1, b1, s0 + kSU);
    }
    if (wave > 0) {
#pragma unroll
        for (int i = 0; i < 16; ++i) red[wave - 1][i][lane] = acc[i];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int w = 0; w < kSWaves - 1; ++w)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[i] += red[w][i][lane];
    // 32x32 accumulator layout: lane holds column lane % 32; register i holds
    // row 8 (i / 4) + 4 (lane / 32) + i % 4.
    const int e = n0 + lrow;
    if (e >= E) return;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int t = m0 + 8 * (i >> 2) + 4 * lhalf + (i & 3);
        if (t < T) S[(int64_t)t * E + e] = source_row(rows, h_rows, t) >= 0 ? acc[i] : 0.0f;
    }
}

// fp32: 64 x 64 output tile per block, 16 x 16 threads, 4 x 4 outputs each.
constexpr int kFT = 64;
constexpr int kFK = 16;

__global__ __launch_bounds__(256) void affinity_f32_kernel(const float *__restrict__ H,
                                                           const int32_t *__restrict__ rows,
                                                           int64_t h_rows,
                                                           const float *__restrict__ W,
                                                           float *__restrict__ S, int T, int E,
                                                           int d) {
    __shared__ float As[kFK][kFT + 4];   // As[k][token]
    __shared__ float Bs[kFK][kFT + 4];   // Bs[k][expert]
    const int tid = threadIdx.x;
    const int tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.x * kFT, n0 = blockIdx.y * kFT;
    // Loader: thread covers row tid/4, elements (tid%4)*4 .. +4 of the chunk.
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    const int64_t hrow = m0 + lr < T ? source_row(rows, h_rows, m0 + lr) : -1;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < d; k0 += kFK) {
        float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
        if (hrow >= 0 && k0 + lk < d)
            a = *reinterpret_cast<const float4 *>(H + hrow * d + k0 + lk);
        if (n0 + lr < E && k0 + lk < d)
            b = *reinterpret_cast<const float4 *>(W + (int64_t)(n0 + lr) * d + k0 + lk);
        __syncthreads();
        As[lk + 0][lr] = a.x; As[lk + 1][lr] = a.y; As[lk + 2][lr] = a.z; As[lk + 3][lr] = a.w;
        Bs[lk + 0][lr] = b.x; Bs[lk + 1][lr] = b.y; Bs[lk + 2][lr] = b.z; Bs[lk + 3][lr] = b.w;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kFK; ++k) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = As[k][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = Bs[k][tx * 4 + j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int t = m0 + ty * 4 + i;
        if (t >= T) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = n0 + tx * 4 + j;
            if (e < E) S[(int64_t)t * E + e] = acc[i][j];
        }
    }
}

}  // namespace

hipError_t launch_affinity_bf16(const uint16_t *H, const int32_t *rows, int64_t h_rows,
                                const uint16_t *W, float *S, int64_t T, int64_t E, int64_t d,
                                hipStream_t stream) {
    if (d % kPK == 0 && ((T + kPM - 1) / kPM) * ((E + kPN - 1) / kPN) < 128) {
        // Fewer 128 x 128 tiles than half the compute units: 32 x 32 tiles.
        dim3 grid((unsigned)((T + kST - 1) / kST), (unsigned)((E + kST - 1) / kST));
        hipLaunchKernelGGL(affinity_bf16_small_kernel, grid, dim3(64 * kSWaves), 0, stream, H,
                           rows, h_rows, W, S, (int)T, (int)E, (int)d);
        return hipGetLastError();
    }
    if (d % kPK == 0) {
        // The LDS ring is above the default 64 KiB: opted in once per device.
        static std::mutex m;
        static bool granted[64] = {};
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return hipErrorInvalidDevice;
        {
            std::lock_guard<std::mutex> lock(m);
            if (!granted[dev]) {
                const hipError_t err = hipFuncSetAttribute(
                    reinterpret_cast<const void *>(&affinity_bf16_pipe_kernel),
                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)kPipeLds);
                if (err != hipSuccess) return err;
                granted[dev] = true;
            }
        }
        const int64_t nm8 = ((T + kPM - 1) / kPM + 7) / 8 * 8;   // token tiles, whole eights
        const int64_t nn = (E + kPN - 1) / kPN;
        hipLaunchKernelGGL(affinity_bf16_pipe_kernel, dim3((unsigned)(nm8 * nn)), dim3(kPThreads),
                           kPipeLds, stream, H, rows, h_rows, W, S, (int)T, (int)E, (int)d);
        return hipGetLastError();
    }
    dim3 grid((unsigned)((T + kBM - 1) / kBM), (unsigned)((E + kBN - 1) / kBN));
    hipLaunchKernelGGL(affinity_bf16_kernel, grid, dim3(256), 0, stream, H, rows, h_rows, W, S,
                       (int)T, (int)E, (int)d);
    return hipGetLastError();
}

hipError_t launch_affinity_f32(const float *H, const int32_t *rows, int64_t h_rows,
                               const float *W, float *S, int64_t T, int64_t E, int64_t d,
                               hipStream_t stream) {
    dim3 grid((unsigned)((T + kFT - 1) / kFT), (unsigned)((E + kFT - 1) / kFT));
    hipLaunchKernelGGL(affinity_f32_kernel, grid, dim3(256), 0, stream, H, rows, h_rows, W, S,
                       (int)T, (int)E, (int)d);
    return hipGetLastError();
}

}  // namespace base
