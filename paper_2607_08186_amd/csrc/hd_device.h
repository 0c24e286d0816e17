// hd_device.h -- gfx950 device helpers: buffer addressing, MFMA, bf16 packing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "hd_internal.h"

namespace hd {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Byte offset that lies beyond every buffer range we build (ranges stay below 2^31):
// buffer loads at such an offset return zeros and buffer stores are dropped.
constexpr uint32_t kOob = 0x80000000u;

typedef __amdgpu_buffer_rsrc_t rsrc_t;

// Raw (unswizzled, stride 0) buffer resource covering `bytes` bytes from `base`.
__device__ inline rsrc_t make_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ inline u32x4 ld16(rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ inline uint32_t ld4(rsrc_t r, uint32_t off)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ inline void st16(rsrc_t r, uint32_t off, u32x4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((__vector_size__(16))) unsigned int, v), r, off, 0, 0);
}
__device__ inline void st8(rsrc_t r, uint32_t off, u32x2 v)
{
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((__vector_size__(8))) unsigned int, v), r, off, 0, 0);
}
// Non-temporal store (cache policy "nt"): data written once and read back much later
// by another kernel, marked so that it does not push reused lines out of L2.
__device__ inline void st16_nt(rsrc_t r, uint32_t off, u32x4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(__attribute__((__vector_size__(16))) unsigned int, v), r, off, 0, 2);
}
__device__ inline void st4(rsrc_t r, uint32_t off, uint32_t v)
{
    __builtin_amdgcn_raw_buffer_store_b32(v, r, off, 0, 0);
}

// D(32x32 fp32) += A(32x16 bf16) * B(16x32 bf16).  Lane l supplies row/column l % 32 of
// A/B and 8 consecutive k-slots chosen by l / 32 (A and B use the same slot->k map).
// Result register r of lane l holds row 8*(r/4) + 4*(l/32) + r%4, column l % 32.
__device__ inline f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Two floats -> packed bf16x2 (round to nearest even), low half = a.
__device__ inline uint32_t pack_bf16(float a, float b)
{
    f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Max / sum of v over lanes l and l ^ 32 (the two halves of the wave), in registers:
// v_permlane32_swap exchanges the upper half of one copy with the lower half of the
// other, so the two results hold v of both halves for every lane (no LDS round trip,
// which a cross-half shuffle otherwise takes).
__device__ inline float max_xor32(float v)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float sum_xor32(float v)
{
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup id -> (problem, row tile).  Tiles with the longest causal extent go first.
// Consecutive workgroup ids are spread round-robin over the 8 XCDs, so when the
// problem count allows it each XCD gets a contiguous band of problems (the query heads
// of one key/value head) and its L2 serves their shared K/V.
__device__ inline void decode_tile(int bid, int nprob, int ntiles, int &prob, int &tile)
{
    if ((nprob & 7) == 0) {
        const int per = nprob >> 3, r = bid >> 3;
        tile = ntiles - 1 - r / per;
        prob = (bid & 7) * per + r % per;
    } else {
        tile = ntiles - 1 - bid / nprob;
        prob = bid % nprob;
    }
}

// Same for key tiles in the dK/dV pass: heavy (early) key tiles first.
__device__ inline void decode_key_tile(int bid, int nprob, int ntiles, int &prob, int &tile)
{
    decode_tile(bid, nprob, ntiles, prob, tile);
    tile = ntiles - 1 - tile;
}

}  // namespace hd
