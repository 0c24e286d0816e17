// sfa_fwd_bf16.hip -- Stream-Factorized Attention forward, bf16 in/out, fp32 softmax.
//
// Computes, per causal problem (see SfaGeom), O = softmax(scale Q K^T + mask) V and the
// natural-log row log-sum-exp: the forward of the intra-stream layer (eq. (mask_intra))
// and of the full cross-stream layer (causal mask of Fig. "masks"(a)).
//
// Tiling (gfx950, wave64):
//   workgroup = 8 waves = 256 query rows of one problem (two waves per SIMD); wave w
//   owns rows 32w..32w+31 and each lane keeps one query row (column l%32 of the MFMA
//   results).  The transposed score tile S^T = K Q^T puts a row's scores in one lane,
//   so the row max / row sum need one cross-half exchange, and P^T feeds the second
//   MFMA (O^T += V^T P^T) straight from registers.
//   Key/value tiles of 64 rows are loaded HBM -> LDS by direct-to-LDS buffer loads
//   into a double buffer (one barrier per tile); K is read row-wise, V through
//   transposed LDS reads, both from the same swizzled row-major layout.
//   Only tiles at or below a wave's diagonal are computed; the causal mask is applied
//   on diagonal tiles alone.  The running max is refreshed only when it grows by more
//   than 2^8 (log2 units), so the O rescale is rare; results are exact either way
//   because the normaliser uses the same reference.
#include <type_traits>

#include "sfa_lds.h"

namespace hd {

namespace {

constexpr int kWaves = 8;
constexpr int kBM = kWaves * 32;           // query rows per workgroup
constexpr int kStages = 2;                 // K/V tiles in flight (LDS double buffer)
constexpr float kRescaleThreshold = 8.0f;  // log2 units

template <int D>
__global__ __launch_bounds__(kWaves * 64, 1) void sfa_fwd_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    bf16 *__restrict__ o, float *__restrict__ lse, SfaGeom g)
{
    constexpr int KS = D / 16;  // MFMA k-steps over the head dim
    constexpr int DB = D / 32;  // 32-wide head-dim blocks of O
    using T = Tile<D>;
    __shared__ __attribute__((aligned(1024))) char smem[kStages][2 * T::BYTES];  // [stage][K | V]

    const int ntiles = (g.len + kBM - 1) / kBM;
    const int nprob = g.B * g.Hq * g.streams;
    int prob, tile;
    decode_tile(blockIdx.x, nprob, ntiles, prob, tile);
    const int s = prob % g.streams;
    const int hq = (prob / g.streams) % g.Hq;
    const int b = prob / (g.streams * g.Hq);
    const int hk = hq / g.G;

    // per-batch slices; all in-slice byte offsets fit in 31 bits
    const size_t qslice = (size_t)g.N * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const rsrc_t rq = make_rsrc(q + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rv = make_rsrc(v + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t ro = make_rsrc(o + b * qslice, (uint32_t)(qslice * 2));
    const uint32_t qstride = (uint32_t)g.rowmul * g.Hq * D * 2;
    const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase0 = (uint32_t)(s * g.Hkv + hk) * D * 2;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
    const int l32 = lane & 31, hi = lane >> 5;
    const int q0 = tile * kBM;
    const int row = q0 + wave * 32 + l32;

    const int kend = min(g.len, q0 + kBM);
    const int nkt = (kend + kRows - 1) / kRows;
    auto issue = [&](int j) __attribute__((always_inline)) {
        char *st = smem[j & 1];
        T::load(st, rk, kbase0, kstride, j * kRows, g.len, wave, kWaves, lane);
        T::load(st + T::BYTES, rv, kbase0, kstride, j * kRows, g.len, wave, kWaves, lane);
    };
    // loads this wave issues per tile, and a wait for "tile j has landed" given how
    // many later tiles were issued after it
    const int per_tile = 2 * loads_per_wave(T::INSTR, wave, kWaves);
    auto wait_tile = [&](int later) __attribute__((always_inline)) { wait_vmcnt_le(per_tile * later); };
    for (int j = 0; j < kStages - 1 && j < nkt; ++j) issue(j);

    // this lane's query row as the B operand of S^T = K Q^T
    bf16x8 qr[KS];
    {
        const uint32_t off = row < g.len ? qbase + (uint32_t)row * qstride : kOob;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
            qr[kk] = __builtin_bit_cast(bf16x8, ld16(rq, off + (kk * 16 + hi * 8) * 2));
    }

    f32x16 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
    float m2 = -INFINITY;  // reference max in log2 units
    float lsum = 0.f;      // this lane half's share of the row sum

    const float c2 = g.scale_log2;
    const int wrow_min = q0 + wave * 32, wrow_max = wrow_min + 31;

    wait_tile(min(kStages - 2, nkt - 1));
    __syncthreads();

    // one key tile; the stage index is a compile-time constant so LDS addresses are a
    // per-lane base plus an immediate offset
    auto step = [&](int j, auto stage) __attribute__((always_inline)) {
        constexpr int kSt = decltype(stage)::value;
        if (j + kStages - 1 < nkt) issue(j + kStages - 1);
        const int kbase = j * kRows;
        if (kbase <= wrow_max) {  // wave-uniform: tile holds keys visible to this wave
            const char *kt = smem[kSt];
            const char *vt = kt + T::BYTES;
            // MFMA bursts run at raised wave priority, the softmax at normal priority, so
            // the two waves sharing a SIMD tend to alternate matrix and vector work
            __builtin_amdgcn_s_setprio(1);
            f32x16 sacc[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                sacc[mb] = f32x16{};
#pragma unroll
                for (int kk = 0; kk < KS; ++kk)
                    sacc[mb] = mfma32(T::row_operand(kt, mb * 32 + l32, kk, hi), qr[kk], sacc[mb]);
            }
            __builtin_amdgcn_s_setprio(0);
            if (kbase + kRows - 1 > wrow_min) {  // diagonal tile: causal mask
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = kbase + mb * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
                        if (key > row) sacc[mb][r] = -INFINITY;
                    }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[mb][r]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float mcand = fmaxf(m2, mx * c2);
            if (__any(mcand > m2 + kRescaleThreshold)) {
                const float alpha = mcand == -INFINITY ? 1.f : fast_exp2(m2 - mcand);
                m2 = mcand;
                lsum *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
            }
            bf16x8 pb[4];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float p0 = fast_exp2(__builtin_fmaf(sacc[mb][h * 8 + 2 * e], c2, -m2));
                        const float p1 = fast_exp2(__builtin_fmaf(sacc[mb][h * 8 + 2 * e + 1], c2, -m2));
                        lsum += p0 + p1;
                        w[e] = pack_bf16(p0, p1);
                    }
                    pb[mb * 2 + h] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
                }
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    oacc[db] = mfma32(T::tr_operand(vt, db * 32, kk, lane), pb[kk], oacc[db]);
            __builtin_amdgcn_s_setprio(0);
        }
        // tile j+1 must have landed; tiles j+2 .. j+kStages-1 may still be in flight
        wait_tile(max(0, min(kStages - 2, nkt - 2 - j)));
        __syncthreads();
    };
    static_assert(kStages == 2, "the tile loop below alternates two stages");
    for (int j = 0; j < nkt; j += 2) {
        step(j, std::integral_constant<int, 0>{});
        if (j + 1 < nkt) step(j + 1, std::integral_constant<int, 1>{});
    }

    const float l = lsum + __shfl_xor(lsum, 32);
    if (row < g.len) {
        const float inv = 1.f / l;
        const uint32_t obase = qbase + (uint32_t)row * qstride;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const int d0 = db * 32 + 8 * rq + 4 * hi;
                const u32x2 w = {pack_bf16(oacc[db][4 * rq] * inv, oacc[db][4 * rq + 1] * inv),
                                 pack_bf16(oacc[db][4 * rq + 2] * inv, oacc[db][4 * rq + 3] * inv)};
                st8(ro, obase + d0 * 2, w);
            }
        if (hi == 0) {
            const size_t li = ((size_t)b * g.Hq + hq) * g.N + (size_t)row * g.rowmul + s;
            lse[li] = (m2 + log2f(l)) * 0.6931471805599453f;
        }
    }
}

}  // namespace

hipError_t launch_fwd_bf16(const void *q, const void *k, const void *v, void *o, float *lse,
                           const SfaGeom &g, hipStream_t s)
{
    const int ntiles = (g.len + kBM - 1) / kBM;
    const int nprob = g.B * g.Hq * g.streams;
    const dim3 grid(ntiles * nprob), block(kWaves * 64);
    const bf16 *qq = static_cast<const bf16 *>(q), *kk = static_cast<const bf16 *>(k),
               *vv = static_cast<const bf16 *>(v);
    bf16 *oo = static_cast<bf16 *>(o);
    switch (g.D) {
    case 32:
        timing_before("sfa_fwd_bf16_d32", s);
        sfa_fwd_bf16_kernel<32><<<grid, block, 0, s>>>(qq, kk, vv, oo, lse, g);
        break;
    case 64:
        timing_before("sfa_fwd_bf16_d64", s);
        sfa_fwd_bf16_kernel<64><<<grid, block, 0, s>>>(qq, kk, vv, oo, lse, g);
        break;
    default:
        timing_before("sfa_fwd_bf16_d128", s);
        sfa_fwd_bf16_kernel<128><<<grid, block, 0, s>>>(qq, kk, vv, oo, lse, g);
        break;
    }
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace hd
