// sfa_tiles.h -- staging of 64-row bf16 tiles from HBM into LDS for the MFMA kernels.
//
// A tile is 64 consecutive rows (row stride given in bytes, so intra-stream rows at
// stride n are gathered directly) of D bf16 values.  Each active thread loads a quad of
// 4 consecutive rows x 8 consecutive dims (four 16-byte loads; 16 lanes cover one
// 256-byte row, so loads coalesce) and can write it to LDS in two layouts:
//   row-major   [64][D + 8]      -- 16-byte padded rows; read as MFMA operands whose
//                                   k-slots run along D;
//   transposed  [D][64]          -- one LDS row per dim, rows of the tile contiguous in
//                                   swap23 order, 16-byte chunks XOR-swizzled per dim;
//                                   read as MFMA operands whose k-slots run along rows.
#pragma once

#include "hd_device.h"

namespace hd {

constexpr int kTileRows = 64;

__device__ inline int tr_swizzle(int d) { return ((d >> 1) ^ (d >> 3)) & 7; }

// element offset of (dim d, 16-byte chunk c of rows) in a transposed tile
__device__ inline int tr_offset(int d, int c) { return d * kTileRows + ((c ^ tr_swizzle(d)) << 3); }

template <int D>
struct QuadStager {
    static constexpr int CH = D / 8;                     // 16-byte chunks per row
    static constexpr int ACTIVE = (kTileRows / 4) * CH;  // threads with a quad
    static constexpr int RM_STRIDE = D + 8;              // row-major LDS row (elements)
    u32x4 reg[4];

    __device__ inline void load(rsrc_t r, uint32_t base, uint32_t stride, int row0, int len,
                                int tid)
    {
        if (tid < ACTIVE) {
            const int ch = tid % CH, quad = tid / CH;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = row0 + quad * 4 + i;
                const uint32_t off = row < len ? base + (uint32_t)row * stride + ch * 16 : kOob;
                reg[i] = ld16(r, off);
            }
        }
    }

    __device__ inline void store_rm(bf16 *lds, int tid) const
    {
        if (tid < ACTIVE) {
            const int ch = tid % CH, quad = tid / CH;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *reinterpret_cast<u32x4 *>(&lds[(quad * 4 + i) * RM_STRIDE + ch * 8]) = reg[i];
        }
    }

    __device__ inline void store_tr(bf16 *lds, int tid) const
    {
        if (tid < ACTIVE) {
            const int ch = tid % CH, quad = tid / CH;
            const int pos = swap23(quad * 4);  // rows quad*4 .. +3 land on pos .. pos+3
            const int c16 = pos >> 3, within = pos & 7;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int d = ch * 8 + e, w = e >> 1;
                uint32_t lo, hi;
                if ((e & 1) == 0) {
                    lo = (reg[0][w] & 0xffffu) | (reg[1][w] << 16);
                    hi = (reg[2][w] & 0xffffu) | (reg[3][w] << 16);
                } else {
                    lo = (reg[0][w] >> 16) | (reg[1][w] & 0xffff0000u);
                    hi = (reg[2][w] >> 16) | (reg[3][w] & 0xffff0000u);
                }
                *reinterpret_cast<u32x2 *>(&lds[tr_offset(d, c16) + within]) = u32x2{lo, hi};
            }
        }
    }
};

// MFMA operand (8 bf16) from a row-major tile: row `row`, dims kk*16 + half*8 .. +7
template <int D>
__device__ inline bf16x8 rm_operand(const bf16 *lds, int row, int kk, int half)
{
    return *reinterpret_cast<const bf16x8 *>(&lds[row * (D + 8) + kk * 16 + half * 8]);
}

// MFMA operand (8 bf16) from a transposed tile: dim d, rows of 16-row group kk as the
// lane half `half` of an MFMA result block holds them (swap23 order)
__device__ inline bf16x8 tr_operand(const bf16 *lds, int d, int kk, int half)
{
    return *reinterpret_cast<const bf16x8 *>(&lds[tr_offset(d, kk * 2 + half)]);
}

}  // namespace hd
