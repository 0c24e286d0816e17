// sfa_bwd_bf16.hip -- Stream-Factorized Attention backward, bf16 in/out, fp32 math.
//
// Gradients of O = softmax(scale Q K^T + mask) V with the probabilities recomputed
// from the forward's log-sum-exp; the workspace holds, per query row, -lse/scale and
// -Delta:
//   P = exp2(scale*log2(e) (q.k - lse/scale)),  dP = dO V^T,  dS = P (dP - Delta),
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K,   Delta = rowsum(dO * O).
// Three deterministic kernels (no atomics):
//   stats: -Delta and -lse/scale of every query row.
//   dK/dV: a workgroup owns 128 keys of one (b, kv-head[, stream]) problem (K and V
//          resident in LDS), 32 per pair of waves, and sweeps the query tiles that see
//          them for every query head of the group, so the grouped-query sum happens in
//          registers; the two waves of a pair split each query tile and add their
//          partials once at the end.  Scores are formed as
//          S = Q K^T (one key per lane), which makes P and dS the B operands of
//          dV^T += dO^T P and dK^T += Q^T dS; Q and dO tiles are staged row-major and
//          read transposed for those two products.  The bf16 dS it forms is also
//          stored, as 64 x 128 tiles in the workspace.
//   dQ:    dQ = scale dS K from the stored tiles: a workgroup owns 256 query rows (32
//          per wave, one row per lane) and streams the dS tiles and key rows at or
//          below the diagonal through an LDS ring (32 keys x 2 stages, several
//          workgroups per CU, unless that would make the whole grid resident at
//          once; then 64 keys x 3 stages), dQ^T += K^T dS^T with
//          both operands read transposed from LDS.  No S or dP is recomputed, so this
//          pass is bound by the dS reads from HBM.
// All tiles move HBM -> LDS through direct-to-LDS buffer loads.
#include <atomic>
#include <type_traits>

#include "sfa_lds.h"

namespace hd {

namespace {

constexpr int kKeysPerWg = 128;  // dK/dV: 4 key groups of 32, each shared by 2 waves
constexpr int kDkdvWaves = 8;
constexpr int kDqWaves = 8;
constexpr int kRowsPerWg = kDqWaves * 32;  // dQ: 8 waves (two per SIMD) x 32 rows
static_assert(kRowsPerWg == kBandUnit * kDsRows, "a query band unit is one dQ workgroup's rows");

// Row statistics for the dK/dV pass: -Delta = -rowsum(dO * O) (fp32 sum of the bf16
// products) and -lse/scale, both fp32 [B][Hq][N].  A workgroup takes 64 consecutive
// rows p of one (b, hq): D/8 lanes per row read 16 bytes each of O and dO (every
// thread issues all of its loads first; streaming loads, 12% faster than cached ones),
// and the 64 results go out through LDS as two contiguous 256-byte runs.
constexpr int kStatRows = 64;

template <int D>
__global__ __launch_bounds__(256) void bwd_stats_bf16_kernel(const bf16 *__restrict__ o,
                                                             const bf16 *__restrict__ dO,
                                                             const float *__restrict__ lse,
                                                             float *__restrict__ nstat_d,
                                                             float *__restrict__ nstat_l, SfaGeom g)
{
    constexpr int LPR = D / 8;             // lanes per row
    constexpr int RPP = 256 / LPR;         // rows per pass
    constexpr int PASSES = kStatRows / RPP;
    __shared__ float sh[kStatRows];
    const int nblk = (g.qN + kStatRows - 1) / kStatRows;
    const int bh = blockIdx.x / nblk;  // b * Hq + hq
    const int b = bh / g.Hq, hq = bh % g.Hq;
    const int p0 = (blockIdx.x % nblk) * kStatRows;
    const int part = threadIdx.x % LPR, r = threadIdx.x / LPR;
    u32x4 ow[PASSES], dw[PASSES];
#pragma unroll
    for (int i = 0; i < PASSES; ++i) {
        const int p = p0 + i * RPP + r;
        ow[i] = dw[i] = u32x4{0u, 0u, 0u, 0u};
        if (p < g.qN) {
            const int64_t off = (((int64_t)b * g.qN + p) * g.Hq + hq) * D + part * 8;
            ow[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(o + off));
            dw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(dO + off));
        }
    }
#pragma unroll
    for (int i = 0; i < PASSES; ++i) {
        float acc = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            acc = __builtin_fmaf(bf16_lo(dw[i][w]), bf16_lo(ow[i][w]), acc);
            acc = __builtin_fmaf(bf16_hi(dw[i][w]), bf16_hi(ow[i][w]), acc);
        }
#pragma unroll
        for (int m = LPR / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m);
        if (part == 0) sh[i * RPP + r] = acc;
    }
    __syncthreads();
    const int t = threadIdx.x;
    if (t < kStatRows && p0 + t < g.qN) {
        const size_t li = (size_t)bh * g.qN + p0 + t;
        nstat_d[li] = -sh[t];
        nstat_l[li] = -lse[li] / g.scale;
    }
}

template <int D>
__global__ __launch_bounds__(kDkdvWaves * 64, 1) void sfa_dkdv_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    const bf16 *__restrict__ dO, const float *__restrict__ delta, const float *__restrict__ lse2,
    bf16 *__restrict__ dk, bf16 *__restrict__ dv, bf16 *__restrict__ ds, int64_t ds_tiles, SfaGeom g,
    QBand bd, int nsplit, float *__restrict__ split, SplitOrder order)
{
    constexpr int DB = D / 32, KS = D / 16;
    using T = Tile<D>;
    constexpr int STAGE = 2 * T::BYTES + 2 * kRows * 4;       // Q | dO | lse2 | delta
    constexpr int KV = 2 * (kKeysPerWg / kRows) * T::BYTES;  // K tiles | V tiles
    constexpr int LDS = 2 * STAGE + KV;
    static_assert(2 * (kDkdvWaves / 2) * DB * 16 * 64 * 4 <= LDS, "partials must fit in LDS");
    __shared__ __attribute__((aligned(1024))) char smem[LDS];
    char *const kvt = smem + 2 * STAGE;

    const int nkt = (g.len + kKeysPerWg - 1) / kKeysPerWg;
    const int nprob = g.B * g.Hkv * g.streams;
    // work item: a key tile's whole sweep, or with split sweeps (nsplit > 0) one half of
    // the sweep of one of the first nsplit key tiles, the items taken longest first
    int prob, ktile, half;
    if (nsplit > 0) {
        int rank;
        decode_key_tile(blockIdx.x, nprob, nkt + nsplit, prob, rank);
        const int code = order.item[rank];
        ktile = code >> 2;
        half = (code & 3) - 1;  // -1: the whole sweep, 0: its later half, 1: its earlier half
    } else {
        decode_key_tile(blockIdx.x, nprob, nkt, prob, ktile);
        half = -1;
    }
    const int s = prob % g.streams;
    const int hk = (prob / g.streams) % g.Hkv;
    const int b = prob / (g.streams * g.Hkv);

    const size_t qslice = (size_t)g.qN * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const size_t lslice = (size_t)g.Hq * g.qN;
    const rsrc_t rq = make_rsrc(q + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rdo = make_rsrc(dO + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rv = make_rsrc(v + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rdk = make_rsrc(dk + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rdv = make_rsrc(dv + b * kslice, (uint32_t)(kslice * 2));
    const uint32_t qstride = (uint32_t)g.qrowmul * g.Hq * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase = (uint32_t)(s * g.Hkv + hk) * D * 2;

    // waves w and w + 4 own the same 32 keys; w takes query rows 0..31 of every
    // 64-row tile and w + 4 rows 32..63; their dK/dV partials are summed at the end
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
    const int l32 = lane & 31, hi = lane >> 5;
    const int kw = wave & 3, qb = wave >> 2;
    const int k0 = ktile * kKeysPerWg;
    const int kw0 = k0 + kw * 32;
    const int key = kw0 + l32;

    // Sweep: the query tiles from the last one down to the one holding the first key,
    // and for each tile every query head of the group in turn.  Workgroups of one
    // problem that run together (decode_key_tile keeps a problem's key tiles on one
    // XCD) then read the same Q/dO tiles at about the same time, and the group's heads
    // follow each other, so most of those reads hit in L2.
    // first query tile with a row that sees the first key (P(i) >= k0)
    const int qt_first_all = max(0, (k0 - g.qpoff + g.qpmul - 1) / g.qpmul) / kRows;
    const int band = ds_band(g);
    // last query tile that sees a key of this workgroup: the end of the sequence, or for
    // local layers the window's end past the last key (P(i) <= k0 + 126 + window)
    const int qt_end_all = (int)min((int64_t)(g.qlen + kRows - 1) / kRows,
                                    ((int64_t)k0 + kKeysPerWg - 2 + g.window - g.qpoff) / g.qpmul / kRows + 1);
    // this query band's part of the sweep; dK/dV go out as bf16 from the band holding
    // the last query tile of the sweep and as fp32 partials from earlier bands, and a
    // band after the one holding the first query tile adds to the partials.  Keys that
    // no query sees are written (as zeros) by the first band.
    int qt_first = max(qt_first_all, bd.qt_lo), qt_end = min(qt_end_all, bd.qt_hi);
    const bool unseen = qt_first_all >= qt_end_all;
    if (unseen ? bd.qt_lo != 0 : qt_first >= qt_end) return;  // uniform: nothing to do here
    const bool first_band = unseen || qt_first_all >= bd.qt_lo;
    const bool last_band = unseen || qt_end_all <= bd.qt_hi;
    if (half >= 0) {  // one half of a split sweep (one pass only): the later tiles, or the earlier
        const int mid = qt_first + (qt_end - qt_first) / 2;
        if (half == 0)
            qt_first = mid;
        else
            qt_end = mid;
    }
    const int nqt = max(0, qt_end - qt_first);
    const int iters = g.G * nqt;

    // this workgroup's 128 keys and values, resident in LDS for the whole sweep
#pragma unroll
    for (int t = 0; t < kKeysPerWg / kRows; ++t) {
        T::load(kvt + t * T::BYTES, rk, kbase, kstride, k0 + t * kRows, g.len, wave, kDkdvWaves, lane);
        T::load(kvt + (kKeysPerWg / kRows + t) * T::BYTES, rv, kbase, kstride, k0 + t * kRows,
                g.len, wave, kDkdvWaves, lane);
    }
    // dS tiles of query head hq[, stream s]: this wave writes the 32 x 32 block of its
    // keys and query half of tile (query tile qt, this key tile); the tile's byte
    // offset inside the problem is its index times kDsTileBytes
    auto ds_problem = [&](int gi) __attribute__((always_inline)) {
        const int64_t prob_q = ((int64_t)b * g.Hq + hk * g.G + gi) * g.streams + s;
        return ds + prob_q * ds_tiles * (kDsTileBytes / 2);
    };
    const uint32_t dsoff = (uint32_t)(qb * kDsKeys + kw * 32 + l32) * 64 + hi * 32;
    const char *ktl = kvt + (kw >> 1) * T::BYTES;                              // tile of my keys
    const char *vtl = kvt + (kKeysPerWg / kRows + (kw >> 1)) * T::BYTES;
    const int krow = (kw & 1) * 32 + l32;                                      // my key's row there

    // Loads of a query tile: per-lane offsets computed once (rows are relative to the
    // tile's first row); rows past the end of the problem lie past the end of the
    // batch's buffer range and load zeros.  The row statistics take a buffer range of
    // one query head, so their rows past the end load zeros as well.
    const auto qplan = T::template dma_plan<kDkdvWaves>(0, qstride, wave, lane);
    const uint32_t stat_lane = (uint32_t)(lane * g.qrowmul + s) * 4;
    auto issue = [&](int gi, int qt, int st) __attribute__((always_inline)) {
        const int hq = hk * g.G + gi;
        const int row0 = qt * kRows;
        const uint32_t row0_off = (uint32_t)(s * g.Hq + hq) * D * 2 + (uint32_t)row0 * qstride;
        char *base = smem + st * STAGE;
        T::load(base, rq, qplan, row0_off, wave);
        T::load(base + T::BYTES, rdo, qplan, row0_off, wave);
        if (wave < 2) {  // per-row lse2 (wave 0) and delta (wave 1), 4 bytes per lane
            const float *sbase = (wave == 0 ? lse2 : delta) + b * lslice + (size_t)hq * g.qN;
            dma_lds4(make_rsrc(sbase, (uint32_t)g.qN * 4), base + 2 * T::BYTES + wave * kRows * 4,
                     stat_lane + (uint32_t)row0 * g.qrowmul * 4);
        }
    };
    if (iters > 0) issue(0, qt_end - 1, 0);

    f32x16 adk[DB], adv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) adk[db] = adv[db] = f32x16{};

    const float c2 = g.scale_log2;
    wait_lds_loads();
    lds_barrier();

    // P = exp2(c2 (S - lse/scale)) and dS = P (dP - Delta) of my 32 keys x 32 queries,
    // packed as bf16 B operands (two 16-query groups)
    auto softmax = [&](const f32x16 &sacc, const f32x16 &pacc, int qlo, uint32_t (&pw)[8],
                       uint32_t (&dw)[8], auto mask) __attribute__((always_inline)) {
        constexpr bool kMask = decltype(mask)::value;
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
            float p[4], ds[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int r = rq * 4 + e;
                float x = sacc[r];
                if constexpr (kMask) {  // causal and, for local layers, windowed
                    const int qd = qpos(g, qlo + 8 * rq + 4 * hi + e) - key;  // query - key
                    if (qd < 0 || qd >= g.window) x = -INFINITY;  // exp2 -> 0
                }
                p[e] = fast_exp2(x * c2);
                ds[e] = p[e] * pacc[r];
            }
            pw[rq * 2] = pack_bf16(p[0], p[1]);
            pw[rq * 2 + 1] = pack_bf16(p[2], p[3]);
            dw[rq * 2] = pack_bf16(ds[0], ds[1]);
            dw[rq * 2 + 1] = pack_bf16(ds[2], ds[3]);
        }
    };
    // Sweep position (query head gi, query tile qt) of the current step; the next step
    // takes the next head of the group, or after the last one the first head of the
    // tile below.
    int cur_gi = 0, cur_qt = qt_end - 1;
    const bf16 *ds_head = ds_problem(0);
    auto step = [&](int it, auto stage) __attribute__((always_inline)) {
        constexpr int st = decltype(stage)::value;
        const bool wrap = cur_gi + 1 == g.G;
        const int nxt_gi = wrap ? 0 : cur_gi + 1;
        const int nxt_qt = wrap ? cur_qt - 1 : cur_qt;
        if (it + 1 < iters) issue(nxt_gi, nxt_qt, st ^ 1);
        const int qlo = cur_qt * kRows + qb * 32;
        const rsrc_t rds = make_rsrc(
            ds_head + (ds_tile_index(band, ds_kt_lo(g, cur_qt), cur_qt, ktile) - bd.ds_base) *
                          (kDsTileBytes / 2),
            kDsTileBytes);
        uint32_t dsw[8];
        // wave-uniform: some of my 32 queries see some of my keys
        if (qpos(g, qlo + 31) >= kw0 && qpos(g, qlo) - kw0 < 31 + g.window) {
            const char *qt = smem + st * STAGE;
            const char *dot = qt + T::BYTES;
            const float *sl = reinterpret_cast<const float *>(qt + 2 * T::BYTES) + qb * 32;
            const float *sdl = sl + kRows;
            // S and dP accumulators start at -lse/scale and -Delta of their query rows
            // (register r of a lane: row 8*(r/4) + 4*hi + r%4 of my 32 queries)
            f32x16 sacc, pacc;
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const f32x4 l4 = *reinterpret_cast<const f32x4 *>(&sl[8 * rq + 4 * hi]);
                const f32x4 d4 = *reinterpret_cast<const f32x4 *>(&sdl[8 * rq + 4 * hi]);
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    sacc[4 * rq + e] = l4[e];
                    pacc[4 * rq + e] = d4[e];
                }
            }
            // operands of k-step kk + 2 read while the MFMAs of k-step kk run (two
            // k-steps in flight); scheduling barriers keep the reads where they are
            bf16x8 oq[2], ok[2], od[2], ov[2];
            auto rd = [&](int kk, int sl) __attribute__((always_inline)) {
                oq[sl] = T::row_operand(qt, qb * 32 + l32, kk, hi);
                ok[sl] = T::row_operand(ktl, krow, kk, hi);
                od[sl] = T::row_operand(dot, qb * 32 + l32, kk, hi);
                ov[sl] = T::row_operand(vtl, krow, kk, hi);
            };
            rd(0, 0);
            rd(1, 1);
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
                sacc = mfma32(oq[kk & 1], ok[kk & 1], sacc);
                pacc = mfma32(od[kk & 1], ov[kk & 1], pacc);
                if (kk + 2 < KS) rd(kk + 2, kk & 1);
                __builtin_amdgcn_sched_barrier(0);
            }
            uint32_t pw[8], dw[8];
            // dV += dO^T P and dK += Q^T dS in 4*DB MFMAs; operand i belongs to 16-query
            // group h, dim block db and dV (i even) or dK (i odd).  Each operand is read
            // three MFMAs ahead, the first three while the softmax runs.
            constexpr int NOP = 4 * DB, AHEAD = 3;
            bf16x8 ot[AHEAD + 1];
            auto rdt = [&](int i) __attribute__((always_inline)) {
                ot[i % (AHEAD + 1)] = T::tr_operand((i & 1) ? qt : dot, ((i >> 1) % DB) * 32,
                                                    qb * 2 + i / (2 * DB), lane);
            };
#pragma unroll
            for (int i = 0; i < AHEAD; ++i) rdt(i);
            __builtin_amdgcn_sched_barrier(0);
            if (qpos(g, qlo) < kw0 + 31 || qpos(g, qlo + 31) - kw0 >= g.window)  // diagonal or window edge
                softmax(sacc, pacc, qlo, pw, dw, std::true_type{});
            else
                softmax(sacc, pacc, qlo, pw, dw, std::false_type{});
            bf16x8 pb[2], dsb[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                pb[h] = __builtin_bit_cast(
                    bf16x8, u32x4{pw[h * 4], pw[h * 4 + 1], pw[h * 4 + 2], pw[h * 4 + 3]});
                dsb[h] = __builtin_bit_cast(
                    bf16x8, u32x4{dw[h * 4], dw[h * 4 + 1], dw[h * 4 + 2], dw[h * 4 + 3]});
            }
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < NOP; ++i) {
                const int h = i / (2 * DB), db = (i >> 1) % DB;
                if (i & 1)
                    adk[db] = mfma32(ot[i % (AHEAD + 1)], dsb[h], adk[db]);
                else
                    adv[db] = mfma32(ot[i % (AHEAD + 1)], pb[h], adv[db]);
                if (i + AHEAD < NOP) rdt(i + AHEAD);
                __builtin_amdgcn_sched_barrier(0);
            }
            // dw[0..7] hold queries 8 rq + 4 hi .. +3 of my key (rq = 0..3) in the order of
            // the tile layout: 32 contiguous bytes per lane
#pragma unroll
            for (int i = 0; i < 8; ++i) dsw[i] = dw[i];
        } else {
            // no visible pair in this block: its part of the tile is zero
#pragma unroll
            for (int i = 0; i < 8; ++i) dsw[i] = 0u;
        }
        st16_nt(rds, dsoff, u32x4{dsw[0], dsw[1], dsw[2], dsw[3]});
        st16_nt(rds, dsoff + 16, u32x4{dsw[4], dsw[5], dsw[6], dsw[7]});
        // the next tile's loads were issued before this step's two dS stores; vector
        // memory operations complete in order, so once at most those stores are
        // outstanding the tile has landed
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("" ::: "memory");
        wait_vmcnt_le(2);
        lds_barrier();
        cur_gi = nxt_gi;
        cur_qt = nxt_qt;
        ds_head = ds_problem(nxt_gi);
    };
    for (int it = 0; it < iters; it += 2) {
        step(it, std::integral_constant<int, 0>{});
        if (it + 1 < iters) step(it + 1, std::integral_constant<int, 1>{});
    }

    // sum the two query halves: waves 4..7 park their partials in LDS (one 16-byte
    // slot per lane and register quad), waves 0..3 add them and write dK/dV
    f32x4 *park = reinterpret_cast<f32x4 *>(smem) + kw * (2 * DB * 4 * 64);
    if (qb == 1) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                park[((0 * DB + db) * 4 + r4) * 64 + lane] =
                    f32x4{adk[db][4 * r4], adk[db][4 * r4 + 1], adk[db][4 * r4 + 2], adk[db][4 * r4 + 3]};
                park[((1 * DB + db) * 4 + r4) * 64 + lane] =
                    f32x4{adv[db][4 * r4], adv[db][4 * r4 + 1], adv[db][4 * r4 + 2], adv[db][4 * r4 + 3]};
            }
    }
    __syncthreads();
    if (half >= 0 && qb == 0 && key < g.len) {
        // one half of a split sweep: fp32 sums [half][dK, dV][problem][key][D]
        const size_t slice = (size_t)nsplit * kKeysPerWg * D;
        float *pk = split + ((size_t)(half * 2) * nprob + prob) * slice + (size_t)key * D;
        float *pv = split + ((size_t)(half * 2 + 1) * nprob + prob) * slice + (size_t)key * D;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const f32x4 a = park[((0 * DB + db) * 4 + rq) * 64 + lane];
                const f32x4 c = park[((1 * DB + db) * 4 + rq) * 64 + lane];
                const int d0 = db * 32 + 8 * rq + 4 * hi;
                *reinterpret_cast<f32x4 *>(pk + d0) = f32x4{adk[db][4 * rq] + a[0], adk[db][4 * rq + 1] + a[1],
                                                            adk[db][4 * rq + 2] + a[2], adk[db][4 * rq + 3] + a[3]};
                *reinterpret_cast<f32x4 *>(pv + d0) = f32x4{adv[db][4 * rq] + c[0], adv[db][4 * rq + 1] + c[1],
                                                            adv[db][4 * rq + 2] + c[2], adv[db][4 * rq + 3] + c[3]};
            }
        return;
    }
    if (qb == 0 && key < g.len) {
        const uint32_t off = kbase + (uint32_t)key * kstride;
        // fp32 partials of this problem's keys (query bands only): [key][D]
        const size_t pslice = (size_t)g.len * D;
        const rsrc_t rpk = make_rsrc(bd.part_k + prob * pslice, (uint32_t)(pslice * 4));
        const rsrc_t rpv = make_rsrc(bd.part_v + prob * pslice, (uint32_t)(pslice * 4));
        const uint32_t poff = (uint32_t)key * D * 4;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const f32x4 pk = park[((0 * DB + db) * 4 + rq) * 64 + lane];
                const f32x4 pv = park[((1 * DB + db) * 4 + rq) * 64 + lane];
                const int d0 = db * 32 + 8 * rq + 4 * hi;
                f32x4 sk = {adk[db][4 * rq] + pk[0], adk[db][4 * rq + 1] + pk[1],
                            adk[db][4 * rq + 2] + pk[2], adk[db][4 * rq + 3] + pk[3]};
                f32x4 sv = {adv[db][4 * rq] + pv[0], adv[db][4 * rq + 1] + pv[1],
                            adv[db][4 * rq + 2] + pv[2], adv[db][4 * rq + 3] + pv[3]};
                if (!first_band) {
                    sk += __builtin_bit_cast(f32x4, ld16(rpk, poff + d0 * 4));
                    sv += __builtin_bit_cast(f32x4, ld16(rpv, poff + d0 * 4));
                }
                if (last_band) {
                    const float sc = g.scale;
                    st8(rdk, off + d0 * 2, u32x2{pack_bf16(sk[0] * sc, sk[1] * sc), pack_bf16(sk[2] * sc, sk[3] * sc)});
                    st8(rdv, off + d0 * 2, u32x2{pack_bf16(sv[0], sv[1]), pack_bf16(sv[2], sv[3])});
                } else {
                    st16(rpk, poff + d0 * 4, __builtin_bit_cast(u32x4, sk));
                    st16(rpv, poff + d0 * 4, __builtin_bit_cast(u32x4, sv));
                }
            }
    }
}

// dK, dV of the split key tiles: the two halves' fp32 sums added in a fixed order
// (half 0, then half 1), scaled (dK) and rounded to bf16; four dims per thread.
template <int D>
__global__ __launch_bounds__(256) void dkdv_split_combine_kernel(const float *__restrict__ split,
                                                                 int nsplit, bf16 *__restrict__ dk,
                                                                 bf16 *__restrict__ dv, SfaGeom g)
{
    const int nprob = g.B * g.Hkv * g.streams;
    const int keys = nsplit * kKeysPerWg;
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= (int64_t)nprob * keys * (D / 4)) return;
    const int d0 = (int)(idx % (D / 4)) * 4;
    const int key = (int)(idx / (D / 4) % keys);
    const int prob = (int)(idx / (D / 4) / keys);
    if (key >= g.len) return;
    const int s = prob % g.streams;
    const int hk = (prob / g.streams) % g.Hkv;
    const int b = prob / (g.streams * g.Hkv);
    const size_t slice = (size_t)keys * D, at = (size_t)key * D + d0;
    const f32x4 k0 = *reinterpret_cast<const f32x4 *>(split + (size_t)prob * slice + at);
    const f32x4 v0 = *reinterpret_cast<const f32x4 *>(split + ((size_t)nprob + prob) * slice + at);
    const f32x4 k1 = *reinterpret_cast<const f32x4 *>(split + ((size_t)2 * nprob + prob) * slice + at);
    const f32x4 v1 = *reinterpret_cast<const f32x4 *>(split + ((size_t)3 * nprob + prob) * slice + at);
    const f32x4 ks = (k0 + k1) * g.scale, vs = v0 + v1;
    const size_t off = ((size_t)b * g.N + (size_t)key * g.rowmul + s) * g.Hkv * D + (size_t)hk * D + d0;
    *reinterpret_cast<u32x2 *>(dk + off) = u32x2{pack_bf16(ks[0], ks[1]), pack_bf16(ks[2], ks[3])};
    *reinterpret_cast<u32x2 *>(dv + off) = u32x2{pack_bf16(vs[0], vs[1]), pack_bf16(vs[2], vs[3])};
}

// KK keys per ring step, S ring stages.  <32, 2> takes 48 KB of LDS at D=128, so two
// workgroups share a CU and each one's loads overlap the other's MFMAs; <64, 3> takes
// 144 KB, one workgroup per CU, and wins when the whole grid would otherwise be resident
// at once (the dispatcher then cannot pair long causal row blocks with short ones).
template <int D, int KK, int S>
__global__ __launch_bounds__(kDqWaves * 64, 1) void sfa_dq_bf16_kernel(
    const bf16 *__restrict__ k, const bf16 *__restrict__ ds, bf16 *__restrict__ dq, SfaGeom g,
    int64_t ds_tiles, QBand bd)
{
    constexpr int DB = D / 32;
    static_assert(kDsKeys % KK == 0 && KK % 16 == 0 && S >= 2, "ring shape");
    using T = Tile<D, KK>;
    // a wave's dS slab of one step: KK keys x 32 queries, 64 bytes per key
    constexpr int kSlab = KK * 64;
    constexpr int kStage = T::BYTES + kDqWaves * kSlab;  // K rows | dS slabs
    static_assert(S * kStage <= 160 * 1024, "the ring must fit in LDS");
    __shared__ __attribute__((aligned(1024))) char smem[S][kStage];

    // the 256-row blocks of this query band (its first tile is a multiple of four)
    const int rb_lo = bd.qt_lo / kBandUnit;
    const int ntiles = (min(bd.qt_hi * kDsRows, g.qlen) + kRowsPerWg - 1) / kRowsPerWg - rb_lo;
    const int nprob = g.B * g.Hq * g.streams;
    int prob, tile;
    decode_tile(blockIdx.x, nprob, ntiles, prob, tile);
    tile += rb_lo;
    const int s = prob % g.streams;
    const int hq = (prob / g.streams) % g.Hq;
    const int b = prob / (g.streams * g.Hq);
    const int hk = hq / g.G;

    const size_t qslice = (size_t)g.qN * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const rsrc_t rdq = make_rsrc(dq + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const uint32_t qstride = (uint32_t)g.qrowmul * g.Hq * D * 2;
    const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase = (uint32_t)(s * g.Hkv + hk) * D * 2;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
    const int l32 = lane & 31, hi = lane >> 5;
    const int q0 = tile * kRowsPerWg;
    // MFMA column l32 holds the query at position l32 of the dS tile layout
    const int row = q0 + wave * 32 + ds_query_at(l32);
    const int wrow_min = q0 + wave * 32, wrow_max = wrow_min + 31;
    // my rows are half (wave & 1) of dS query tile qt
    const int qt = wrow_min / kDsRows;
    const int band = ds_band(g);
    const int kt_lo = ds_kt_lo(g, qt);
    const bf16 *ds_prob = ds + (int64_t)prob * ds_tiles * (kDsTileBytes / 2);

    // keys of the block: up to the key coordinate of its last query row
    const int kend = min(g.len, qpos(g, min(q0 + kRowsPerWg, g.qlen) - 1) + 1);
    const int nkt = (kend + KK - 1) / KK;
    // first key step any row of the workgroup sees (0 unless the layer is local)
    const int jf = max(0, qpos(g, q0) - g.window + 1) / KK;
    // wave-uniform: key step j holds a key that a row of this wave sees (then the dS
    // tile that holds it exists)
    auto active = [&](int j) __attribute__((always_inline)) {
        const int kb0 = j * KK;
        return wrow_min < g.qlen && kb0 <= qpos(g, wrow_max) &&
               qpos(g, wrow_min) - (kb0 + KK - 1) < g.window;
    };
    constexpr int kSteps = kDsKeys / KK;  // key steps per dS tile
    const int kloads = loads_per_wave(T::INSTR, wave, kDqWaves);
    // this wave's loads of step j (in-order completion makes counts enough to wait on)
    auto nloads = [&](int j) __attribute__((always_inline)) {
        return j < nkt ? kloads + (active(j) ? kSlab / 1024 : 0) : 0;
    };
    static_assert((S - 2) * (T::INSTR / kDqWaves + 1 + kSlab / 1024) <= 15,
                  "outstanding loads must fit the vmcnt wait");
    // K rows of a step: per-lane offsets computed once; rows past the end of the
    // problem lie past the end of the batch's buffer range and load zeros
    const auto kplan = T::template dma_plan<kDqWaves>(kbase, kstride, wave, lane);
    auto issue = [&](int j) __attribute__((always_inline)) {
        if (j >= nkt) return;
        char *st = smem[(j - jf) % S];
        T::load(st, rk, kplan, (uint32_t)(j * KK) * kstride, wave);
        if (active(j)) {
            const int64_t t = ds_tile_index(band, kt_lo, qt, j / kSteps) - bd.ds_base;
            const rsrc_t rt = make_rsrc(ds_prob + t * (kDsTileBytes / 2), kDsTileBytes);
            char *slab = st + T::BYTES + wave * kSlab;
            const uint32_t off =
                (uint32_t)((wave & 1) * kDsKeys + (j % kSteps) * KK) * 64 + lane * 16;
#pragma unroll
            for (int oc = 0; oc < kSlab / 1024; ++oc)
                dma_lds16_nt(rt, slab + oc * 1024, off + oc * 1024);
        }
    };

    // B operand dS^T (k-slots along keys, one query per lane): lane i of 16-lane group
    // gr reads the 8-byte pieces of key rows 4*(gr>>1) + (i>>2) (+8) and queries
    // 16*(gr&1) + 4*(i&3) .. +3, which the transposed read turns into query
    // 16*(gr&1) + i with 4 keys, in the key order of T::tr_operand's A operand.  The
    // 32 lanes of a half read 4 rows x 8 pieces: 32 distinct 8-byte bank slots.
    const int sl = lane & 15, gr = lane >> 4;
    const uint32_t dso = (uint32_t)((4 * (gr >> 1) + (sl >> 2)) * 64 + (16 * (gr & 1) + 4 * (sl & 3)) * 2);
    uint32_t kto[DB][2];
    T::tr_offsets(lane, kto);

    f32x16 adq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) adq[db] = f32x16{};

    // steps jf .. jf+S-2 in flight; step j's stage is free again once every wave has
    // passed the barrier that ends step j - 1
#pragma unroll
    for (int i = 0; i < S - 1; ++i) issue(jf + i);
    {
        int pend = 0;
#pragma unroll
        for (int i = 1; i < S - 1; ++i) pend += nloads(jf + i);
        wait_vmcnt_le(pend);
    }
    lds_barrier();
    for (int j = jf; j < nkt; ++j) {
        issue(j + S - 1);
        if (active(j)) {
            const char *kt = smem[(j - jf) % S];
            const char *slab = kt + T::BYTES + wave * kSlab;
#pragma unroll
            for (int kk = 0; kk < KK / 16; ++kk) {
                const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4i16 *)(slab + dso + kk * 1024));
                const v4i16 hi8 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (lds_v4i16 *)(slab + dso + kk * 1024 + 512));
                const u32x2 x = __builtin_bit_cast(u32x2, lo), y = __builtin_bit_cast(u32x2, hi8);
                const bf16x8 bop = __builtin_bit_cast(bf16x8, u32x4{x[0], x[1], y[0], y[1]});
#pragma unroll
                for (int db = 0; db < DB; ++db) adq[db] = mfma32(T::tr_at(kt, kto[db], kk), bop, adq[db]);
            }
        }
        // step j + 1 has landed once at most the loads of steps j + 2 .. j + S - 1 are
        // outstanding
        {
            int pend = 0;
#pragma unroll
            for (int i = 2; i < S; ++i) pend += nloads(j + i);
            wait_vmcnt_le(pend);
        }
        lds_barrier();
    }

    if (row < g.qlen) {
        const uint32_t off = qbase + (uint32_t)row * qstride;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const int d0 = db * 32 + 8 * rq + 4 * hi;
                const u32x2 w = {pack_bf16(adq[db][4 * rq] * g.scale, adq[db][4 * rq + 1] * g.scale),
                                 pack_bf16(adq[db][4 * rq + 2] * g.scale, adq[db][4 * rq + 3] * g.scale)};
                st8(rdq, off + d0 * 2, w);
            }
    }
}

template <int D>
hipError_t bwd_bf16_d(const bf16 *q, const bf16 *k, const bf16 *v, const bf16 *o,
                      const float *lse, const bf16 *dO, float *delta, float *lse2, char *wsb,
                      const BwdWorkspace &w, size_t ws_bytes, bf16 *dq, bf16 *dk, bf16 *dv,
                      const SfaGeom &g, hipStream_t s, const char *st_name, const char *dq_name,
                      const char *dkdv_name)
{
    timing_before(st_name, s);
    bwd_stats_bf16_kernel<D><<<(unsigned)((g.qN + kStatRows - 1) / kStatRows * g.B * g.Hq), 256, 0, s>>>(
        o, dO, lse, delta, lse2, g);
    hipError_t e = hipGetLastError();
    timing_after(s);
    if (e != hipSuccess) return e;

    // the co-resident dQ ring, unless the whole grid would then be resident at once
    static std::atomic<int> co_resident{0};  // its workgroups per CU (a property of the code)
    int dev = 0, cus = 0, per_cu = co_resident.load(std::memory_order_relaxed);
    if (per_cu == 0) {
        if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
                 &per_cu, reinterpret_cast<const void *>(&sfa_dq_bf16_kernel<D, 32, 2>),
                 kDqWaves * 64, 0)) != hipSuccess)
            return e;
        co_resident.store(per_cu, std::memory_order_relaxed);
    }
    if ((e = hipGetDevice(&dev)) != hipSuccess ||
        (e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
        return e;

    const int nkt = (g.len + kKeysPerWg - 1) / kKeysPerWg;
    const int nqt = (g.qlen + kDsRows - 1) / kDsRows;
    const int band = ds_band(g);
    const int64_t nprob_q = (int64_t)g.B * g.Hq * g.streams;
    // one pass when every dS tile fits, else query bands as large as the workspace allows
    const bool one_pass = ws_bytes >= w.total;
    if (!one_pass && ws_bytes < w.min_total) return hipErrorInvalidValue;  // checked by the caller
    bf16 *ds = reinterpret_cast<bf16 *>(wsb + (one_pass ? w.ds : w.ds_banded));
    const int64_t ds_room = one_pass ? w.ds_tiles : (int64_t)((ws_bytes - w.ds_banded) / kDsTileBytes / nprob_q);
    auto tiles = [&](int qa, int qb) { return ds_tile_base(band, qb) - ds_tile_base(band, qa); };
    for (int qa = 0; qa < nqt;) {
        int qb = one_pass ? nqt : min(nqt, qa + kBandUnit);
        while (qb < nqt && tiles(qa, min(nqt, qb + kBandUnit)) <= ds_room) qb = min(nqt, qb + kBandUnit);
        QBand bd;
        bd.qt_lo = qa;
        bd.qt_hi = qb;
        bd.ds_base = ds_tile_base(band, qa);
        bd.part_k = one_pass ? nullptr : reinterpret_cast<float *>(wsb + w.part_k);
        bd.part_v = one_pass ? nullptr : reinterpret_cast<float *>(wsb + w.part_v);
        const int64_t band_tiles = tiles(qa, qb);
        // one pass only: the longest sweeps of a small grid are split in halves
        const int nsplit = one_pass ? w.nsplit : 0;
        float *split = reinterpret_cast<float *>(wsb + w.split);
        SplitOrder order;
        if (nsplit > 0) order = dkdv_split_order(g, nsplit);
        timing_before(dkdv_name, s);
        sfa_dkdv_bf16_kernel<D><<<(nkt + nsplit) * g.B * g.Hkv * g.streams, kDkdvWaves * 64, 0, s>>>(
            q, k, v, dO, delta, lse2, dk, dv, ds, band_tiles, g, bd, nsplit, split, order);
        e = hipGetLastError();
        timing_after(s);
        if (e != hipSuccess) return e;
        if (nsplit > 0) {
            const int64_t n4 = (int64_t)g.B * g.Hkv * g.streams * nsplit * kKeysPerWg * (D / 4);
            timing_before(D == 32 ? "sfa_dkdv_split_combine_d32"
                                  : D == 64 ? "sfa_dkdv_split_combine_d64" : "sfa_dkdv_split_combine_d128",
                          s);
            dkdv_split_combine_kernel<D><<<(unsigned)((n4 + 255) / 256), 256, 0, s>>>(split, nsplit, dk, dv, g);
            e = hipGetLastError();
            timing_after(s);
            if (e != hipSuccess) return e;
        }
        const int nrb = (min(qb * kDsRows, g.qlen) + kRowsPerWg - 1) / kRowsPerWg - qa / kBandUnit;
        const int64_t wgs = nrb * nprob_q;
        timing_before(dq_name, s);
        if (wgs > (int64_t)per_cu * cus)
            sfa_dq_bf16_kernel<D, 32, 2><<<(unsigned)wgs, kDqWaves * 64, 0, s>>>(k, ds, dq, g, band_tiles, bd);
        else
            sfa_dq_bf16_kernel<D, 64, 3><<<(unsigned)wgs, kDqWaves * 64, 0, s>>>(k, ds, dq, g, band_tiles, bd);
        e = hipGetLastError();
        timing_after(s);
        if (e != hipSuccess) return e;
        qa = qb;
    }
    return hipSuccess;
}

}  // namespace

hipError_t launch_bwd_bf16(const void *q, const void *k, const void *v, const void *o,
                           const float *lse, const void *dO, void *dq, void *dk, void *dv,
                           const SfaGeom &g, void *ws, size_t ws_bytes, hipStream_t s)
{
    const BwdWorkspace w = bwd_workspace(g, 2);
    char *wsb = static_cast<char *>(ws);
    float *delta = reinterpret_cast<float *>(wsb + w.delta);
    float *lse2 = reinterpret_cast<float *>(wsb + w.lse2);
    const bf16 *qq = static_cast<const bf16 *>(q), *kk = static_cast<const bf16 *>(k),
               *vv = static_cast<const bf16 *>(v), *dd = static_cast<const bf16 *>(dO),
               *oo = static_cast<const bf16 *>(o);
    bf16 *gq = static_cast<bf16 *>(dq), *gk = static_cast<bf16 *>(dk), *gv = static_cast<bf16 *>(dv);
    const bool f = g.qpmul != 1;  // final-stream layer: tagged in the timing names
    if (g.D == 32)
        return bwd_bf16_d<32>(qq, kk, vv, oo, lse, dd, delta, lse2, wsb, w, ws_bytes, gq, gk, gv, g,
                              s, f ? "sfa_bwd_final_stats_d32" : "sfa_bwd_stats_d32",
                              f ? "sfa_dq_final_bf16_d32" : "sfa_dq_bf16_d32",
                              f ? "sfa_dkdv_final_bf16_d32" : "sfa_dkdv_bf16_d32");
    if (g.D == 64)
        return bwd_bf16_d<64>(qq, kk, vv, oo, lse, dd, delta, lse2, wsb, w, ws_bytes, gq, gk, gv, g,
                              s, f ? "sfa_bwd_final_stats_d64" : "sfa_bwd_stats_d64",
                              f ? "sfa_dq_final_bf16_d64" : "sfa_dq_bf16_d64",
                              f ? "sfa_dkdv_final_bf16_d64" : "sfa_dkdv_bf16_d64");
    return bwd_bf16_d<128>(qq, kk, vv, oo, lse, dd, delta, lse2, wsb, w, ws_bytes, gq, gk, gv, g, s,
                           f ? "sfa_bwd_final_stats_d128" : "sfa_bwd_stats_d128",
                           f ? "sfa_dq_final_bf16_d128" : "sfa_dq_bf16_d128",
                           f ? "sfa_dkdv_final_bf16_d128" : "sfa_dkdv_bf16_d128");
}

}  // namespace hd
