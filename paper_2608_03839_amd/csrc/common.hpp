// Shared device helpers for the gfx950 kernels of the retrieval path.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace oil {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short short2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// bf16 bit pattern -> float (a bf16 is the upper half of a binary32).
__device__ __forceinline__ float bf16_bits_to_float(uint32_t b) { return __uint_as_float(b << 16); }

// Round a double to bf16, nearest-even, straight from the binary64 fields
// (one rounding: no detour through binary32).
__device__ __forceinline__ uint16_t double_to_bf16_rne(double x)
{
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    const uint32_t sign = (uint32_t)(u >> 63) << 15;
    const int e = (int)((u >> 52) & 0x7FF);
    const uint64_t frac = u & ((1ull << 52) - 1);
    if (e == 0x7FF)
        return frac ? (uint16_t)0x7FC0 : (uint16_t)(sign | 0x7F80);
    if (e == 0)  // zero or binary64 subnormal: far below the smallest bf16
        return (uint16_t)sign;
    const int E = e - 1023 + 127;  // biased binary32/bf16 exponent
    uint64_t sig = frac | (1ull << 52);  // 53-bit significand
    int shift;                           // bits dropped to keep the bf16 significand
    uint32_t base;
    if (E >= 1) {
        shift = 45;                      // keep 8 significant bits
        base = (uint32_t)E << 7;
        sig &= (1ull << 52) - 1;         // normal: implicit bit lives in the exponent
    } else {
        shift = 45 + (1 - E);            // bf16 subnormal: spacing 2^-133
        base = 0;
        if (shift > 60)
            return (uint16_t)sign;
    }
    const uint64_t keep = sig >> shift;
    const uint64_t rem = sig & ((1ull << shift) - 1);
    const uint64_t half = 1ull << (shift - 1);
    uint32_t mag = base + (uint32_t)keep;  // carries into the exponent when keep overflows
    if (rem > half || (rem == half && (keep & 1)))
        mag += 1;
    if (mag >= 0x7F80)
        mag = 0x7F80;                    // overflow to infinity
    return (uint16_t)(sign | mag);
}

// MurmurHash3's 32-bit finaliser (public domain): the hash of the LDS tables
// that map tokens to requests (lexical source, recycled pool).
__device__ __forceinline__ uint32_t mix32(uint32_t h)
{
    h ^= h >> 16;
    h *= 0x85EBCA6Bu;
    h ^= h >> 13;
    h *= 0xC2B2AE35u;
    h ^= h >> 16;
    return h;
}

// Order-preserving 32-bit code of a float score: a larger code is a larger
// score.  0 is reserved: the bit pattern 0xFFFFFFFF (a NaN) marks "no
// position" (outside the pool, or excluded) and maps to it.
__device__ __forceinline__ uint32_t score_code(float s)
{
    const uint32_t b = __float_as_uint(s) == 0x80000000u ? 0u : __float_as_uint(s);  // -0 ranks as +0
    return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ float code_score(uint32_t c)
{
    const uint32_t b = (c & 0x80000000u) ? (c & 0x7FFFFFFFu) : ~c;
    return __uint_as_float(b);
}

constexpr uint32_t kNoScoreBits = 0xFFFFFFFFu;

// Total order key of a (score, position) pair: score descending, then
// position ascending, as one unsigned 64-bit integer (larger = better).
// Key 0 means "no position".
__device__ __forceinline__ uint64_t rank_key(float s, uint32_t pos)
{
    const uint32_t c = score_code(s);
    if (c == 0)
        return 0ull;
    return ((uint64_t)c << 32) | (uint64_t)(0xFFFFFFFFu - pos);
}

__device__ __forceinline__ uint32_t key_pos(uint64_t key) { return 0xFFFFFFFFu - (uint32_t)key; }

}  // namespace oil
