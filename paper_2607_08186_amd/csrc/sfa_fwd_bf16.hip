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
constexpr int kSlots = 4;                  // K and V ring slots (64-key tiles)
constexpr float kRescaleThreshold = 8.0f;  // log2 units

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <int D>
__global__ __launch_bounds__(kWaves * 64, 1) void sfa_fwd_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    bf16 *__restrict__ o, float *__restrict__ lse, SfaGeom g)
{
    constexpr int KS = D / 16;  // MFMA k-steps over the head dim
    constexpr int DB = D / 32;  // 32-wide head-dim blocks of O
    using T = Tile<D>;
    // separate K and V rings: every slot is an immediate offset (< 64 KB) from one
    // per-lane address
    __shared__ __attribute__((aligned(1024))) char ks[kSlots][T::BYTES];
    __shared__ __attribute__((aligned(1024))) char vs[kSlots][T::BYTES];

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
    const int wrow_min = q0 + wave * 32, wrow_max = wrow_min + 31;

    const int kend = min(g.len, q0 + kBM);
    const int nkt = (kend + kRows - 1) / kRows;
    const int jlast = min(nkt - 1, wrow_max / kRows);  // last tile with keys this wave sees

    // this lane's query row as the B operand of S^T = K Q^T
    bf16x8 qr[KS];
    {
        const uint32_t off = row < g.len ? qbase + (uint32_t)row * qstride : kOob;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
            qr[kk] = __builtin_bit_cast(bf16x8, ld16(rq, off + (kk * 16 + hi * 8) * 2));
    }

    // per-lane address parts (K and V share the row layout)
    const typename T::Dma dma = T::dma_plan(kbase0, kstride, wave, kWaves, lane);
    uint32_t kro[KS], vto[DB][2];
    T::row_offsets(l32, hi, kro);
    T::tr_offsets(lane, vto);
    auto issue_k = [&](int j) __attribute__((always_inline)) {
        if (j < nkt) T::load(ks[j % kSlots], rk, dma, (uint32_t)(j * kRows) * kstride, wave, kWaves);
    };
    auto issue_v = [&](int j) __attribute__((always_inline)) {
        if (j < nkt) T::load(vs[j % kSlots], rv, dma, (uint32_t)(j * kRows) * kstride, wave, kWaves);
    };

    f32x16 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
    float m2 = -INFINITY;         // reference max in log2 units
    float lsum0 = 0.f, lsum1 = 0.f;  // this lane half's share of the row sum (two chains)
    const float c2 = g.scale_log2;
    const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3f803f80u);

    auto is_diag = [&](int j) __attribute__((always_inline)) { return j * kRows + kRows - 1 > wrow_min; };
    // S^T of one 64-key tile (two 32-key blocks).  On the tile that holds this wave's
    // diagonal the accumulators start at -inf for keys past the lane's row, so masked
    // scores come out as -inf (exp2 -> 0) and nothing downstream needs a mask; other
    // tiles start from the MFMA's literal zero.
    auto scores = [&](f32x16 (&sc)[2], const char *kt, int j) __attribute__((always_inline)) {
        const bf16x8 a0 = T::row_at(kt, kro[0], 0), a1 = T::row_at(kt, kro[0], 2);
        if (is_diag(j)) {
            // key = j*64 + mb*32 + 8*(r/4) + 4*hi + r%4, compared against a per-lane
            // limit so the per-element constants stay immediates
            const int lim = row - 4 * hi - j * kRows;
            f32x16 bias[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    bias[mb][r] = mb * 32 + 8 * (r >> 2) + (r & 3) > lim ? -INFINITY : 0.f;
            sc[0] = mfma32(a0, qr[0], bias[0]);
            sc[1] = mfma32(a1, qr[0], bias[1]);
        } else {
            sc[0] = mfma32(a0, qr[0], f32x16{});
            sc[1] = mfma32(a1, qr[0], f32x16{});
        }
#pragma unroll
        for (int kk = 1; kk < KS; ++kk)
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
                sc[mb] = mfma32(T::row_at(kt, kro[kk], mb * 2), qr[kk], sc[mb]);
    };
    auto rowmax = [&](const f32x16 (&sc)[2]) __attribute__((always_inline)) {
        float mx = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[mb][r]);
        return fmaxf(mx, __shfl_xor(mx, 32));
    };

    // K of tiles 0..2 and V of tiles 0..1 resident before the loop (and the query row)
    issue_k(0);
    issue_k(1);
    issue_v(0);
    issue_v(1);
    issue_k(2);
    wait_vmcnt_le(0);
    lds_barrier();

    f32x16 sa[2], sb[2];
    scores(sa, ks[0], 0);
    float mx = rowmax(sa);
    lds_barrier();  // every wave is done with K of tile 0 before its slot is refilled

    // One tile j (ring slot kSl): the softmax of tile j runs on the vector unit while
    // the scores of tile j+1 run on the matrix unit, then O^T += V^T P^T with the row
    // max of tile j+1 in between.  Scores of a tile past this wave's diagonal (or past
    // the last tile) are computed from whatever the ring slot holds and discarded.
    auto tile_step = [&](int j, auto slot, f32x16 (&sc)[2], f32x16 (&sn)[2]) __attribute__((always_inline)) {
        constexpr int kSl = decltype(slot)::value;
        constexpr int kNx = (kSl + 1) % kSlots;
        if (j > jlast) return;  // wave-uniform
        const float mcand = fmaxf(m2, mx * c2);
        if (__any(mcand > m2 + kRescaleThreshold)) {
            const float alpha = mcand == -INFINITY ? 1.f : fast_exp2(m2 - mcand);
            m2 = mcand;
            lsum0 *= alpha;
            lsum1 *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
        }
        scores(sn, ks[kNx], j + 1);
        bf16x8 pb[4];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = fast_exp2(__builtin_fmaf(sc[mb][h * 8 + 2 * e], c2, -m2));
                    const float p1 = fast_exp2(__builtin_fmaf(sc[mb][h * 8 + 2 * e + 1], c2, -m2));
                    w[e] = pack_bf16(p0, p1);
                    // the row sum adds the bf16 weights that the P V product uses
                    if (mb == 0)
                        lsum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, lsum0, false);
                    else
                        lsum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, lsum1, false);
                }
                pb[mb * 2 + h] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
            }
        // K reads three MFMAs ahead, a slice of the softmax after each MFMA
        sched_pattern<3, 2 * KS - 2, 1, 1, 6>();
        asm volatile("; P V" ::: "memory");
        const char *vt = vs[kSl];
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                oacc[db] = mfma32(T::tr_at(vt, vto[db], kk), pb[kk], oacc[db]);
        mx = rowmax(sn);
        // transposed V reads three MFMAs ahead, the row max in between
        sched_pattern<6, 4 * DB, 1, 2, 3>();
    };
    // Two tiles per barrier.  At entry K of tiles j+1, j+2 and V of tiles j, j+1 are
    // resident; K of j+3, j+4 and V of j+2, j+3 go to the slots freed by the previous
    // pair and must have landed at the closing barrier.
    auto pair_step = [&](int j, auto slot) __attribute__((always_inline)) {
        constexpr int kSl = decltype(slot)::value;
        issue_k(j + 3);
        issue_k(j + 4);
        issue_v(j + 2);
        issue_v(j + 3);
        tile_step(j, std::integral_constant<int, kSl>{}, sa, sb);
        tile_step(j + 1, std::integral_constant<int, kSl + 1>{}, sb, sa);
        wait_vmcnt_le(0);
        lds_barrier();
    };
    static_assert(kSlots == 4, "the loop below cycles through four ring slots");
    for (int j = 0; j < nkt; j += 4) {
        pair_step(j, std::integral_constant<int, 0>{});
        if (j + 2 < nkt) pair_step(j + 2, std::integral_constant<int, 2>{});
    }

    const float l = lsum0 + lsum1 + __shfl_xor(lsum0 + lsum1, 32);
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
