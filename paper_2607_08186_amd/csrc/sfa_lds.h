// sfa_lds.h -- 64-row bf16 tiles staged HBM -> LDS by direct-to-LDS buffer loads, and
// the MFMA operand reads from them.
//
// Tile layout: 64 rows (consecutive rows of one causal problem; the row stride in HBM
// is free, so intra-stream rows at stride n are gathered directly) x D bf16, row-major,
// D*2 bytes per row with no padding.  Inside a row the 16-byte chunks are permuted:
// logical chunk c of row r sits at physical chunk c ^ swz(r).  LDS has 64 banks of 4
// bytes; a 16-byte read serves 16 lanes per cycle, an 8-byte read 32 lanes.  swz is
// chosen per head dim so that both read patterns are bank-conflict free:
//   * row reads (16 lanes = 16 consecutive rows, same logical chunk, 16 bytes each);
//   * transposed reads (ds_read_b64_tr_b16: 32 lanes cover 4 aligned rows x 4 aligned
//     logical chunks, 8 bytes each), which need the 4 rows to select 4 different
//     groups of 4 physical chunks.
//   D = 128 (16 chunks, one row spans all banks): swz(r) = (r & 3) << 2 | (r >> 2) & 3
//   D = 64  (8 chunks, rows alternate bank halves): swz(r) = (r >> 1 & 1) << 2 | (r >> 2) & 3
//   D = 32  (4 chunks, 4 rows per bank line):      swz(r) = (r >> 2) & 3
// A direct-to-LDS load writes 64 lanes x 16 bytes to consecutive LDS slots; each lane
// picks the HBM chunk that belongs in its slot, which realises the permutation.
#pragma once

#include "hd_device.h"

namespace hd {

constexpr int kRows = 64;  // rows per staged tile

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// Direct-to-LDS buffer loads (lane l writes LDS bytes lds + 16 l, resp. 4 l).  They are
// issued from inline assembly on purpose: the compiler tracks the builtin form as a
// pending LDS write and then waits for every such load before any LDS read, which
// would expose the full HBM latency of the prefetch in every tile step.  Completion
// is instead awaited explicitly (wait_vmcnt_le) before the barrier that publishes a
// tile.  M0 carries the LDS base; no compiler-generated code in these kernels keeps a
// value in M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ inline void dma_lds16(rsrc_t rs, const char *lds, uint32_t voff)
{
    const uint32_t m0 = (uint32_t)(uintptr_t)(lds_void *)lds;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :: "s"(m0), "v"(voff), "s"(rs) : "memory", "m0");
}
// Same with the non-temporal cache policy, for data read exactly once.
__device__ inline void dma_lds16_nt(rsrc_t rs, const char *lds, uint32_t voff)
{
    const uint32_t m0 = (uint32_t)(uintptr_t)(lds_void *)lds;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen nt lds"
                 :: "s"(m0), "v"(voff), "s"(rs) : "memory", "m0");
}
__device__ inline void dma_lds4(rsrc_t rs, const char *lds, uint32_t voff)
{
    const uint32_t m0 = (uint32_t)(uintptr_t)(lds_void *)lds;
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :: "s"(m0), "v"(voff), "s"(rs) : "memory", "m0");
}
#pragma clang diagnostic pop

// Workgroup barrier for LDS tiles: this wave's LDS reads have completed
// (lgkmcnt 0), without __syncthreads' wait for every outstanding global load, so
// prefetches stay in flight across it.  Tile data written by direct-to-LDS loads
// must have been waited for (wait_vmcnt_le) by every issuing wave beforehand.
// The scheduling barriers keep the compiler from moving any instruction across it.
__device__ inline void lds_barrier()
{
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Force values to be computed at this point of the program (an empty asm that reads
// them); used to keep work inside the phase it belongs to.
template <typename T>
__device__ inline void pin(const T &v)
{
    asm volatile("" ::"v"(v));
}
template <typename T, typename... Ts>
__device__ inline void pin(const T &v, const Ts &...rest)
{
    pin(v);
    pin(rest...);
}

template <int D, int R = kRows>
struct Tile {
    static_assert(R % 16 == 0, "the swizzle repeats every 16 rows");
    static constexpr int CH = D / 8;           // 16-byte chunks per row
    static constexpr int BYTES = R * D * 2;    // one tile of R rows
    static constexpr int INSTR = R * CH / 64;  // direct-to-LDS instructions per tile

    // physical chunk = logical chunk ^ swz(row)
    __device__ static inline int swz(int r)
    {
        if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
        else if constexpr (D == 64) return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
        else return (r >> 2) & 3;
    }

    // byte offset of element (row, col) inside the tile
    __device__ static inline int offset(int row, int col)
    {
        const int c = (col >> 3) ^ swz(row);
        return row * (D * 2) + c * 16 + (col & 7) * 2;
    }

    // Issue this wave's share of the direct-to-LDS loads of rows row0 .. row0+63 of a
    // problem whose row r lives at byte base + r*stride of buffer `rs`; rows >= len
    // load zeros.  Waves wave, wave+nwaves, ... take the tile's INSTR instructions.
    __device__ static inline void load(char *lds_tile, rsrc_t rs, uint32_t base,
                                       uint32_t stride, int row0, int len, int wave,
                                       int nwaves, int lane)
    {
#pragma unroll
        for (int t = wave; t < INSTR; t += nwaves) {
            const int slot = t * 64 + lane;
            const int row = slot / CH;
            const int c = (slot % CH) ^ swz(row);
            const int grow = row0 + row;
            const uint32_t off = grow < len ? base + (uint32_t)grow * stride + c * 16 : kOob;
            dma_lds16(rs, lds_tile + t * 1024, off);
        }
    }

    // Per-lane parts of the addresses, computed once per kernel so that the tile base,
    // whole 16-row groups and the row-within-tile offsets below are immediates.
    //
    // DMA: with NW waves loading, this wave's share of a tile is slots t*64 + lane for
    // t = wave, wave+NW, ...; slot -> (row, logical chunk).  voff[i] is the HBM byte
    // offset of that chunk relative to the tile's first row (row stride `stride`).
    template <int NW>
    struct Dma {
        static constexpr int MAXL = (INSTR + NW - 1) / NW;  // loads per wave, at most
        uint32_t voff[MAXL];
        int n;  // loads this wave issues per tile
    };
    template <int NW>
    __device__ static inline Dma<NW> dma_plan(uint32_t base, uint32_t stride, int wave, int lane)
    {
        Dma<NW> p;
        p.n = 0;
#pragma unroll
        for (int i = 0; i < Dma<NW>::MAXL; ++i) {
            const int t = wave + i * NW;
            const int slot = t * 64 + lane;
            const int row = slot / CH;
            const int c = (slot % CH) ^ swz(row);
            p.voff[i] = base + (uint32_t)row * stride + c * 16;
            if (t < INSTR) p.n = i + 1;
        }
        return p;
    }
    // Load rows row0 .. row0+63 (row0 * stride + p.voff < 2^31).  Rows past the end of
    // the problem must lie past the end of the buffer range, which returns zeros.
    template <int NW>
    __device__ static inline void load(char *lds_tile, rsrc_t rs, const Dma<NW> &p, uint32_t row0_off,
                                       int wave)
    {
#pragma unroll
        for (int i = 0; i < Dma<NW>::MAXL; ++i) {
            const int t = wave + i * NW;
            if (t < INSTR) dma_lds16(rs, lds_tile + t * 1024, p.voff[i] + row0_off);
        }
    }

    // Row reads: byte offsets of row (lane % 32) at k-step kk, lane half `half`; rows
    // r + 16 m add 16 m rows (swz depends on r % 16 only).
    __device__ static inline void row_offsets(int l32, int half, uint32_t (&off)[D / 16])
    {
#pragma unroll
        for (int kk = 0; kk < D / 16; ++kk)
            off[kk] = l32 * (D * 2) + (((kk * 2 + half) ^ swz(l32 & 15)) * 16);
    }
    __device__ static inline bf16x8 row_at(const char *lds_tile, uint32_t off, int row_group16)
    {
        return *reinterpret_cast<const bf16x8 *>(lds_tile + off + row_group16 * 16 * (D * 2));
    }

    // Transposed reads (see tr_operand): offsets for 32-dim block db and the two
    // 8-row halves of a 16-row group; 16-row group kk adds kk*16 rows.
    __device__ static inline void tr_offsets(int lane, uint32_t (&off)[D / 32][2])
    {
        const int s = lane & 15, g = lane >> 4, half = g >> 1;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
            for (int p = 0; p < 2; ++p)
                off[db][p] = offset(4 * half + (s >> 2) + 8 * p, db * 32 + 16 * (g & 1) + 4 * (s & 3));
    }
    __device__ static inline bf16x8 tr_at(const char *lds_tile, const uint32_t (&off)[2], int kk)
    {
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_v4i16 *)(lds_tile + off[0] + kk * 16 * (D * 2)));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_v4i16 *)(lds_tile + off[1] + kk * 16 * (D * 2)));
        const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
        return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], b[0], b[1]});
    }

    // MFMA operand whose k-slots run along D: row `row`, dims kk*16 + half*8 .. +7
    __device__ static inline bf16x8 row_operand(const char *lds_tile, int row, int kk, int half)
    {
        const int c = (kk * 2 + half) ^ swz(row);
        return *reinterpret_cast<const bf16x8 *>(lds_tile + row * (D * 2) + c * 16);
    }

    // MFMA operand whose k-slots run along the tile rows, for output row (dim)
    // d = d0 + (lane % 32): the rows of 16-row group kk that lane half `half` of an MFMA
    // result block holds, i.e. rows kk*16 + 4*half + {0..3} and kk*16 + 8 + 4*half +
    // {0..3}.  Two transposed 8-byte reads: in each 16-lane group, lane i returns element
    // i%4 of the 4-element pieces addressed by lanes i/4, i/4+4, i/4+8, i/4+12.
    __device__ static inline bf16x8 tr_operand(const char *lds_tile, int d0, int kk, int lane)
    {
        const int s = lane & 15, g = lane >> 4, half = g >> 1;
        const int col = d0 + 16 * (g & 1) + 4 * (s & 3);
        const int row = kk * 16 + 4 * half + (s >> 2);
        const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_v4i16 *)(lds_tile + offset(row, col)));
        const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_v4i16 *)(lds_tile + offset(row + 8, col)));
        const u32x2 a = __builtin_bit_cast(u32x2, lo), b = __builtin_bit_cast(u32x2, hi);
        return __builtin_bit_cast(bf16x8, u32x4{a[0], a[1], b[0], b[1]});
    }
};

// Scheduling hint for the basic block it ends: P LDS reads up front, then N
// repetitions of (M MFMAs, R LDS reads, V other vector ALU instructions), so that each
// MFMA's operands were requested about P reads earlier.
template <int P, int N, int M, int R, int V>
__device__ inline void sched_pattern()
{
    __builtin_amdgcn_sched_group_barrier(0x100, P, 0);  // LDS read
#pragma unroll
    for (int i = 0; i < N; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, M, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, R, 0);  // LDS read
        if constexpr (V > 0) __builtin_amdgcn_sched_group_barrier(0x002, V, 0);  // VALU
    }
}

// Wait until every direct-to-LDS load this wave issued has landed.
__device__ inline void wait_lds_loads() { __builtin_amdgcn_s_waitcnt(0); }

// Wait until at most n (0..15) of this wave's vector-memory loads are still in flight
// (s_waitcnt vmcnt(n); the expcnt and lgkmcnt fields are left at "no wait").
__device__ inline void wait_vmcnt_le(int n)
{
    switch (n) {
#define HD_VMCNT(k) \
    case k: __builtin_amdgcn_s_waitcnt(0x0F70 | k); break;
        HD_VMCNT(1) HD_VMCNT(2) HD_VMCNT(3) HD_VMCNT(4) HD_VMCNT(5) HD_VMCNT(6) HD_VMCNT(7)
        HD_VMCNT(8) HD_VMCNT(9) HD_VMCNT(10) HD_VMCNT(11) HD_VMCNT(12) HD_VMCNT(13)
        HD_VMCNT(14) HD_VMCNT(15)
#undef HD_VMCNT
    default: __builtin_amdgcn_s_waitcnt(0x0F70); break;
    }
}

// Direct-to-LDS instructions a wave issues per tile when nwaves share INSTR of them.
__device__ inline int loads_per_wave(int instr, int wave, int nwaves)
{
    return wave < instr ? (instr - wave + nwaves - 1) / nwaves : 0;
}

}  // namespace hd
