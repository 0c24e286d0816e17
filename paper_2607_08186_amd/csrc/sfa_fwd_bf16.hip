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
constexpr int kLoaders = 4;                // group B (waves 4-7) issues the tile loads
constexpr float kRescaleThreshold = 8.0f;  // log2 units

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// FINAL: final-stream layer (query row i at key coordinate i*n + n - 1, strided wave
// rows); otherwise query row i is key coordinate i and waves take consecutive rows.
template <int D, bool FINAL>
__global__ __launch_bounds__(kWaves * 64, 1) void sfa_fwd_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    bf16 *__restrict__ o, float *__restrict__ lse, SfaGeom g)
{
    constexpr int KS = D / 16;  // MFMA k-steps over the head dim
    constexpr int DB = D / 32;  // 32-wide head-dim blocks of O
    using T = Tile<D>;
    // two-slot K and V rings (tile t in slot t % 2); every slot is an immediate offset
    // from one per-lane address
    __shared__ __attribute__((aligned(1024))) char ks[2][T::BYTES];
    __shared__ __attribute__((aligned(1024))) char vs[2][T::BYTES];

    const int ntiles = (g.qlen + kBM - 1) / kBM;
    const int nprob = g.B * g.Hq * g.streams;
    int prob, tile;
    decode_tile(blockIdx.x, nprob, ntiles, prob, tile);
    const int s = prob % g.streams;
    const int hq = (prob / g.streams) % g.Hq;
    const int b = prob / (g.streams * g.Hq);
    const int hk = hq / g.G;

    // per-batch slices; all in-slice byte offsets fit in 31 bits
    const size_t qslice = (size_t)g.qN * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const rsrc_t rq = make_rsrc(q + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rv = make_rsrc(v + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t ro = make_rsrc(o + b * qslice, (uint32_t)(qslice * 2));
    const uint32_t qstride = (uint32_t)g.qrowmul * g.Hq * D * 2;
    const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase0 = (uint32_t)(s * g.Hkv + hk) * D * 2;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
    const int group = wave >> 2;  // 0: A, 1: B (one wave of each per SIMD)
    const int l32 = lane & 31, hi = lane >> 5;
    const int q0 = tile * kBM;
    // This wave's 32 query rows: 32 consecutive rows, or, in final-stream layers (whose
    // queries advance n key positions per row), rows wave, wave + 8, ... of the block,
    // so that all eight waves reach (about) the same last key tile.
    auto P = [&](int i) __attribute__((always_inline)) { return FINAL ? qpos(g, i) : i; };
    const int row = FINAL ? q0 + wave + 8 * l32 : q0 + wave * 32 + l32;
    const int wrow_min = FINAL ? q0 + wave : q0 + wave * 32;
    const int wrow_max = FINAL ? wrow_min + 8 * 31 : wrow_min + 31;

    // keys of the block: up to the key coordinate of its last query row
    const int kend = min(g.len, P(min(q0 + kBM, g.qlen) - 1) + 1);
    const int nkt = (kend + kRows - 1) / kRows;
    // Tiles are numbered from jf, the first one holding a key that a row of this
    // workgroup sees (0 unless the layer is local); t below is relative to jf.
    const int jf = max(0, P(q0) - g.window + 1) / kRows;
    const int ntl = nkt - jf;
    // last tile with keys this wave sees
    const int jlast = min(nkt - 1, P(wrow_max) / kRows) - jf;

    // this lane's query row as the B operand of S^T = K Q^T
    bf16x8 qr[KS];
    {
        const uint32_t off = row < g.qlen ? qbase + (uint32_t)row * qstride : kOob;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
            qr[kk] = __builtin_bit_cast(bf16x8, ld16(rq, off + (kk * 16 + hi * 8) * 2));
    }

    // per-lane address parts (K and V share the row layout)
    const bool loader = wave >= kWaves - kLoaders;  // the waves of group B
    const int lw = loader ? wave - (kWaves - kLoaders) : 0;
    const auto dma = T::template dma_plan<kLoaders>(kbase0, kstride, lw, lane);
    uint32_t kro[KS], vto[DB][2];
    T::row_offsets(l32, hi, kro);
    T::tr_offsets(lane, vto);
    // loader waves queue their shares of K of tile t+2 and V of tile t+1 in their
    // vector phase of tile t (or, once past their last tile, before the barrier that
    // ends it) and wait for them at the end of their next phase
    auto issue = [&](int t) __attribute__((always_inline)) {
        if (loader) {
            if (t + 2 < ntl)
                T::load(ks[t & 1], rk, dma, (uint32_t)((jf + t + 2) * kRows) * kstride, lw);
            if (t + 1 < ntl)
                T::load(vs[(t + 1) & 1], rv, dma, (uint32_t)((jf + t + 1) * kRows) * kstride, lw);
        }
    };

    f32x16 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
    f32x16 sc[2];               // scores of the tile whose softmax comes next
    bf16x8 pb[4];               // bf16 weights of the tile whose P V product comes next
    float m2 = -INFINITY;       // reference max in log2 units
    float lsum0 = 0.f, lsum1 = 0.f;  // this lane half's share of the row sum (two chains)
    const float c2 = g.scale_log2;
    const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3f803f80u);

    // the tile holds keys past this wave's first row (diagonal) or, in a local layer,
    // keys at least a window before its last row
    auto needs_mask = [&](int t) __attribute__((always_inline)) {
        const int kb = (jf + t) * kRows;
        return kb + kRows - 1 > P(wrow_min) || kb <= P(wrow_max) - g.window;
    };

    // Matrix phase of tile t: the scores of tile t+1 (DO_S) and O^T += V^T P^T of
    // tile t (DO_PV).  On the tile that holds this wave's diagonal the score
    // accumulators start at -inf for keys past the lane's row, so masked scores come
    // out as -inf (exp2 -> 0) and the softmax needs no mask; other tiles start from the
    // MFMA's literal zero.  KSL/VSL: ring slots of K of tile t+1 and V of tile t.
    auto mfma_phase = [&](int t, auto do_s_, auto do_pv_, auto ksl, auto vsl) __attribute__((always_inline)) {
        constexpr bool DO_S = decltype(do_s_)::value, DO_PV = decltype(do_pv_)::value;
        const char *kt = ks[decltype(ksl)::value];
        const char *vt = vs[decltype(vsl)::value];
        if constexpr (DO_S) {
            const bf16x8 a0 = T::row_at(kt, kro[0], 0), a1 = T::row_at(kt, kro[0], 2);
            if (needs_mask(t + 1)) {
                // key = kb + c with c = mb*32 + 8*(r/4) + r%4 + 4*hi; masked if key > row
                // or row - key >= window, compared against a per-lane limit so the
                // per-element constants stay immediates
                const int lim = P(row) - 4 * hi - (jf + t + 1) * kRows;
                const int lo = lim - g.window;
                f32x16 bias[2];
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int c = mb * 32 + 8 * (r >> 2) + (r & 3);
                        bias[mb][r] = c > lim || c <= lo ? -INFINITY : 0.f;
                    }
                sc[0] = mfma32(a0, qr[0], bias[0]);
                sc[1] = mfma32(a1, qr[0], bias[1]);
            } else {
                sc[0] = mfma32(a0, qr[0], f32x16{});
                sc[1] = mfma32(a1, qr[0], f32x16{});
            }
        }
        // the S and P V chains interleaved
        constexpr int NS = DO_S ? 2 * KS - 2 : 0, NP = DO_PV ? 4 * DB : 0;
#pragma unroll
        for (int i = 0; i < (NS > NP ? NS : NP); ++i) {
            if (i < NP) {
                const int db = i / 4, kk = i % 4;
                oacc[db] = mfma32(T::tr_at(vt, vto[db], kk), pb[kk], oacc[db]);
            }
            if (i < NS) {
                const int kk2 = 1 + i / 2, mb = i % 2;
                sc[mb] = mfma32(T::row_at(kt, kro[kk2], mb * 2), qr[kk2], sc[mb]);
            }
        }
        // operand reads about six ahead of their MFMAs
        sched_pattern<6, NS + NP, 1, 2, 0>();
        if constexpr (DO_S) pin(sc[0], sc[1]);
    };
    // Vector phase of tile t: row max, rare rescale, P = exp2(S c2 - m2) as bf16 and
    // the row sum of those bf16 weights.
    auto vector_phase = [&]() __attribute__((always_inline)) {
        float mx = -INFINITY;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[mb][r]);
        mx = max_xor32(mx);
        const float mcand = fmaxf(m2, mx * c2);
        if (__any(mcand > m2 + kRescaleThreshold)) {
            const float alpha = mcand == -INFINITY ? 1.f : fast_exp2(m2 - mcand);
            m2 = mcand;
            lsum0 *= alpha;
            lsum1 *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
        }
        // a row that has seen only masked keys so far (local layers) keeps m2 = -inf;
        // its weights are then exp2(-inf) = 0, not NaN
        const float m2e = m2 == -INFINITY ? 0.f : m2;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float p0 = fast_exp2(__builtin_fmaf(sc[mb][h * 8 + 2 * e], c2, -m2e));
                    const float p1 = fast_exp2(__builtin_fmaf(sc[mb][h * 8 + 2 * e + 1], c2, -m2e));
                    w[e] = pack_bf16(p0, p1);
                    // the row sum adds the bf16 weights that the P V product uses
                    if (mb == 0)
                        lsum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, lsum0, false);
                    else
                        lsum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones, lsum1, false);
                }
                pb[mb * 2 + h] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
            }
        pin(pb[0], pb[1], pb[2], pb[3]);
    };

    // Prologue: K of tiles 0, 1 and V of tile 0 resident (and the query row).
    if (loader) {
        T::load(ks[0], rk, dma, (uint32_t)(jf * kRows) * kstride, lw);
        if (ntl > 1) T::load(ks[1], rk, dma, (uint32_t)((jf + 1) * kRows) * kstride, lw);
        T::load(vs[0], rv, dma, (uint32_t)(jf * kRows) * kstride, lw);
    }
    wait_vmcnt_le(0);
    lds_barrier();

    // Ping-pong.  Each wave runs: matrix phase of tile -1 (scores of tile 0), then for
    // t = 0 .. jlast the vector phase of tile t and the matrix phase of tile t, one
    // phase per workgroup barrier.  Group B starts one phase after group A, so on every
    // SIMD one wave feeds the matrix unit while the other uses the vector unit.  Waves
    // that finish early pass the remaining barriers idle; every wave passes
    // 2*ntl + 2 of them.  Loads (the four waves of group B, each a quarter of a tile,
    // also those whose rows end before the block's last key tile): K of t+2 goes to
    // the slot of K of t, V of t+1 to the slot of V of t-1, both last read in the
    // matrix phases of tile t-1 (phases 2t, 2t+1); they are queued in phase 2t+2 and
    // published by the barrier of phase 2t+3, before group A's matrix phase of tile
    // t+1 (phase 2t+4).  A group B wave passes barrier 2t+2 right after queueing the
    // loads of tile t and barrier 2t+3 right after waiting for them.
    using F = std::false_type;
    using Tr = std::true_type;
    using Z = std::integral_constant<int, 0>;
    using O = std::integral_constant<int, 1>;
    int nb = 0;  // barriers passed
    auto bar = [&]() __attribute__((always_inline)) { lds_barrier(); ++nb; };
    if (group == 1) bar();
    mfma_phase(-1, Tr{}, F{}, Z{}, Z{});
    bar();
    int t = 0;
    for (; t + 1 < jlast; t += 2) {
        vector_phase();
        issue(t);
        bar();
        mfma_phase(t, Tr{}, Tr{}, O{}, Z{});
        if (loader) wait_vmcnt_le(0);
        bar();
        vector_phase();
        issue(t + 1);
        bar();
        mfma_phase(t + 1, Tr{}, Tr{}, Z{}, O{});
        if (loader) wait_vmcnt_le(0);
        bar();
    }
    if (t < jlast) {  // t even
        vector_phase();
        issue(t);
        bar();
        mfma_phase(t, Tr{}, Tr{}, O{}, Z{});
        if (loader) wait_vmcnt_le(0);
        bar();
        ++t;
    }
    // t == jlast: last softmax and P V product
    vector_phase();
    issue(t);
    bar();
    if (t & 1)
        mfma_phase(t, F{}, Tr{}, Z{}, O{});
    else
        mfma_phase(t, F{}, Tr{}, Z{}, Z{});
    if (loader) wait_vmcnt_le(0);
    bar();
    while (nb < 2 * ntl + 2) {  // idle: past this wave's last tile
        if (loader) {
            if ((nb & 1) == 0)
                issue((nb - 2) >> 1);  // barrier 2t+2 ends the vector phase of tile t
            else
                wait_vmcnt_le(0);      // barrier 2t+3 ends its matrix phase
        }
        bar();
    }

    const float l = sum_xor32(lsum0 + lsum1);
    if (row < g.qlen) {
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
            const size_t li = ((size_t)b * g.Hq + hq) * g.qN + (size_t)row * g.qrowmul + s;
            lse[li] = (m2 + log2f(l)) * 0.6931471805599453f;
        }
    }
}

}  // namespace

hipError_t launch_fwd_bf16(const void *q, const void *k, const void *v, void *o, float *lse,
                           const SfaGeom &g, hipStream_t s)
{
    const int ntiles = (g.qlen + kBM - 1) / kBM;
    const int nprob = g.B * g.Hq * g.streams;
    const dim3 grid(ntiles * nprob), block(kWaves * 64);
    const bf16 *qq = static_cast<const bf16 *>(q), *kk = static_cast<const bf16 *>(k),
               *vv = static_cast<const bf16 *>(v);
    bf16 *oo = static_cast<bf16 *>(o);
    auto launch = [&](auto dk, const char *name) {
        constexpr int DD = decltype(dk)::value;
        timing_before(name, s);
        if (g.strided_waves)
            sfa_fwd_bf16_kernel<DD, true><<<grid, block, 0, s>>>(qq, kk, vv, oo, lse, g);
        else
            sfa_fwd_bf16_kernel<DD, false><<<grid, block, 0, s>>>(qq, kk, vv, oo, lse, g);
    };
    const bool f = g.strided_waves;
    switch (g.D) {
    case 32: launch(std::integral_constant<int, 32>{}, f ? "sfa_fwd_final_bf16_d32" : "sfa_fwd_bf16_d32"); break;
    case 64: launch(std::integral_constant<int, 64>{}, f ? "sfa_fwd_final_bf16_d64" : "sfa_fwd_bf16_d64"); break;
    default: launch(std::integral_constant<int, 128>{}, f ? "sfa_fwd_final_bf16_d128" : "sfa_fwd_bf16_d128"); break;
    }
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace hd
