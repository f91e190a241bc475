// Device-side helpers shared by the HIP kernels of the assignment path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace base {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Bid keys. Every bid is packed into one 64-bit unsigned key so that a plain
// integer comparison orders bids the way the auction needs: higher bid first,
// and among equal bids the lower token index first (the tie rule that makes
// the result independent of scheduling).
//
//   bits 63..24  bid field (40 bits): float mode holds the order-preserving
//                image of the fp32 bid; integer mode holds bid + 2^39
//   bits 23..0   2^24 - 1 - token
//
// Key 0 is below every valid key and marks an empty slot.
// ---------------------------------------------------------------------------
constexpr int kTokBits = 24;
constexpr uint64_t kTokMask = (1ull << kTokBits) - 1;
constexpr int64_t kIntBias = 1ll << 39;
constexpr int64_t kIntFieldMax = (1ll << 40) - 1;

__host__ __device__ inline uint32_t f32_ord(float x) {
    uint32_t u = __float_as_uint(x);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__host__ __device__ inline float f32_unord(uint32_t o) {
    uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}

__device__ inline int32_t key_token(uint64_t key) {
    return (int32_t)(kTokMask - (key & kTokMask));
}
__device__ inline uint64_t key_field(uint64_t key) { return key >> kTokBits; }

// Float mode: values, prices and bids are fp32.
struct FloatMode {
    using score_t = float;
    using value_t = float;
    static constexpr bool kInteger = false;
    __device__ static inline value_t load(const score_t *S, int64_t i, int64_t /*scale*/) {
        return S[i];
    }
    __device__ static inline value_t lowest() { return -INFINITY; }
    // Returns the key and flags (in *overflow) a bid that cannot be encoded.
    __device__ static inline uint64_t make_key(value_t bid, int32_t tok, int *overflow) {
        if (!(bid < INFINITY)) *overflow = 1;
        return ((uint64_t)f32_ord(bid) << kTokBits) | (kTokMask - (uint64_t)tok);
    }
    __device__ static inline value_t key_bid(uint64_t key) {
        return f32_unord((uint32_t)key_field(key));
    }
};

// Integer mode: int16 scores scaled by K (a power of two), int64 arithmetic.
struct IntMode {
    using score_t = int16_t;
    using value_t = int64_t;
    static constexpr bool kInteger = true;
    __device__ static inline value_t load(const score_t *S, int64_t i, int64_t scale) {
        return (int64_t)S[i] * scale;
    }
    __device__ static inline value_t lowest() { return INT64_MIN / 4; }
    __device__ static inline uint64_t make_key(value_t bid, int32_t tok, int *overflow) {
        int64_t f = bid + kIntBias;
        if (f < 1 || f > kIntFieldMax) {
            *overflow = 1;
            f = f < 1 ? 1 : kIntFieldMax;
        }
        return ((uint64_t)f << kTokBits) | (kTokMask - (uint64_t)tok);
    }
    __device__ static inline value_t key_bid(uint64_t key) {
        return (int64_t)key_field(key) - kIntBias;
    }
};

}  // namespace base
