// Device helpers shared by the UFP4 kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ufp4 {

constexpr int kBlock = 16;  // quantization block = RHT block (Table 1)

// ------------------------------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11). One round maps (c0, c1, c2, c3) with key (k0, k1) to
// (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0)); the key advances by the Weyl
// constants between rounds. The key schedule only depends on the seed, so it stays in scalar registers.
// ------------------------------------------------------------------------------------------------
struct Philox4 {
    uint32_t x, y, z, w;
};

// a ^ b ^ k in one gfx950 three-input bitwise instruction (truth table 0x96); k is wave-uniform (a key word).
// The compiler emits two XORs for this pattern, and XORs dual-issue no better than the one instruction.
__device__ __forceinline__ uint32_t xor3_key(uint32_t a, uint32_t b, uint32_t k) {
    uint32_t r;
    asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
    return r;
}

__device__ __forceinline__ Philox4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3, uint32_t k0,
                                                 uint32_t k1) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        // round 0 keeps plain XORs so that constant counter words fold
        const uint32_t n0 = r == 0 ? (uint32_t)(p1 >> 32) ^ c1 ^ k0 : xor3_key((uint32_t)(p1 >> 32), c1, k0);
        const uint32_t n2 = r == 0 ? (uint32_t)(p0 >> 32) ^ c3 ^ k1 : xor3_key((uint32_t)(p0 >> 32), c3, k1);
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
        k0 += 0x9E3779B9u;
        k1 += 0xBB67AE85u;
    }
    return {c0, c1, c2, c3};
}

// ------------------------------------------------------------------------------------------------
// bf16 <-> fp32
// ------------------------------------------------------------------------------------------------
__device__ __forceinline__ float bf16_lo(uint32_t pair) { return __uint_as_float(pair << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t pair) { return __uint_as_float(pair & 0xFFFF0000u); }

// fp32 -> bf16 bits, round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

}  // namespace ufp4
