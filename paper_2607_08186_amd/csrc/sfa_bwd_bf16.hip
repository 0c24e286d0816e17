// sfa_bwd_bf16.hip -- Stream-Factorized Attention backward, bf16 in/out, fp32 math.
//
// Gradients of O = softmax(scale Q K^T + mask) V with the probabilities recomputed
// from the forward's log-sum-exp; the workspace holds, per query row, -lse/scale and
// -Delta:
//   P = exp2(scale*log2(e) (q.k - lse/scale)),  dP = dO V^T,  dS = P (dP - Delta),
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K,   Delta = rowsum(dO * O).
// Two deterministic kernels (no atomics):
//   dK/dV: a workgroup owns 128 keys of one (b, kv-head[, stream]) problem (K and V
//          resident in LDS), 32 per pair of waves, and sweeps the query tiles that see
//          them for every query head of the group, so the grouped-query sum happens in
//          registers; the two waves of a pair split each query tile and add their
//          partials once at the end.  Scores are formed as
//          S = Q K^T (one key per lane), which makes P and dS the B operands of
//          dV^T += dO^T P and dK^T += Q^T dS; Q and dO tiles are staged row-major and
//          read transposed for those two products.
//   dQ:    a workgroup owns 256 query rows (32 per wave, one row per lane as in the
//          forward) and sweeps the key tiles at or below the diagonal:
//          S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T, with K^T read from the
//          transposed copy in the workspace.
// All tiles move HBM -> LDS through direct-to-LDS buffer loads into double buffers.
#include <type_traits>

#include "sfa_lds.h"

namespace hd {

namespace {

constexpr int kKeysPerWg = 128;  // dK/dV: 4 key groups of 32, each shared by 2 waves
constexpr int kDkdvWaves = 8;
constexpr int kDqWaves = 8;
constexpr int kRowsPerWg = kDqWaves * 32;  // dQ: 8 waves (two per SIMD) x 32 rows

// Transposed copy of k for the dQ pass: for each key/value problem (b, hk, s) and each
// 64-row tile, rows i of k (expanded position i*rowmul + s) become columns of
// kt[prob][d][len_pad], position i stored at column swap23(i) of its 16-group; columns
// past len are zero.
template <int D>
__global__ __launch_bounds__(256) void transpose_k_kernel(const bf16 *__restrict__ k,
                                                          bf16 *__restrict__ kt, SfaGeom g,
                                                          int len_pad)
{
    constexpr int CH = D / 8;
    constexpr int STR = D + 2;  // padded LDS row (elements)
    __shared__ uint16_t sm[kRows * STR];
    const int H = g.Hkv;
    const int ntiles = len_pad / kRows;
    const int tile = blockIdx.x % ntiles, prob = blockIdx.x / ntiles;
    const int s = prob % g.streams, h = (prob / g.streams) % H, b = prob / (g.streams * H);
    const size_t slice = (size_t)g.N * H * D;
    const rsrc_t rx = make_rsrc(k + b * slice, (uint32_t)(slice * 2));
    const uint32_t stride = (uint32_t)g.rowmul * H * D * 2;
    const uint32_t base = (uint32_t)(s * H + h) * D * 2;
    const int tid = threadIdx.x;
    for (int idx = tid; idx < kRows * CH; idx += 256) {
        const int r = idx / CH, ch = idx % CH, row = tile * kRows + r;
        const u32x4 v = ld16(rx, row < g.len ? base + (uint32_t)row * stride + ch * 16 : kOob);
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            sm[r * STR + ch * 8 + 2 * w] = (uint16_t)(v[w] & 0xffffu);
            sm[r * STR + ch * 8 + 2 * w + 1] = (uint16_t)(v[w] >> 16);
        }
    }
    __syncthreads();
    bf16 *out = kt + ((size_t)prob * D) * len_pad + (size_t)tile * kRows;
    for (int idx = tid; idx < D * (kRows / 8); idx += 256) {
        const int d = idx / (kRows / 8), c = idx % (kRows / 8);
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const uint32_t lo = sm[swap23(c * 8 + 2 * e) * STR + d];
            const uint32_t hi = sm[swap23(c * 8 + 2 * e + 1) * STR + d];
            w[e] = lo | (hi << 16);
        }
        *reinterpret_cast<u32x4 *>(out + (size_t)d * len_pad + c * 8) = u32x4{w[0], w[1], w[2], w[3]};
    }
}

template <int D>
__global__ __launch_bounds__(kDkdvWaves * 64, 1) void sfa_dkdv_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    const bf16 *__restrict__ dO, const float *__restrict__ delta, const float *__restrict__ lse2,
    bf16 *__restrict__ dk, bf16 *__restrict__ dv, SfaGeom g)
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
    int prob, ktile;
    decode_key_tile(blockIdx.x, nprob, nkt, prob, ktile);
    const int s = prob % g.streams;
    const int hk = (prob / g.streams) % g.Hkv;
    const int b = prob / (g.streams * g.Hkv);

    const size_t qslice = (size_t)g.N * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const size_t lslice = (size_t)g.Hq * g.N;
    const rsrc_t rq = make_rsrc(q + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rdo = make_rsrc(dO + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rv = make_rsrc(v + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rdk = make_rsrc(dk + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rdv = make_rsrc(dv + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rl2 = make_rsrc(lse2 + b * lslice, (uint32_t)(lslice * 4));
    const rsrc_t rdl = make_rsrc(delta + b * lslice, (uint32_t)(lslice * 4));
    const uint32_t qstride = (uint32_t)g.rowmul * g.Hq * D * 2;
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

    // Sweep: for each query head of the group, the query tiles from the last one down
    // to the one holding the first key.  Workgroups of one problem that run together
    // (decode_key_tile keeps a problem's key tiles on one XCD) then read the same Q/dO
    // tiles at about the same time, so most of those reads hit in L2.
    const int qt_first = k0 / kRows;
    // last query tile that sees a key of this workgroup: the end of the sequence, or for
    // local layers the window's end past the last key
    const int qt_end = (int)min((int64_t)(g.len + kRows - 1) / kRows,
                                ((int64_t)k0 + kKeysPerWg - 2 + g.window) / kRows + 1);
    const int nqt = qt_end - qt_first;
    const int iters = g.G * nqt;

    // this workgroup's 128 keys and values, resident in LDS for the whole sweep
#pragma unroll
    for (int t = 0; t < kKeysPerWg / kRows; ++t) {
        T::load(kvt + t * T::BYTES, rk, kbase, kstride, k0 + t * kRows, g.len, wave, kDkdvWaves, lane);
        T::load(kvt + (kKeysPerWg / kRows + t) * T::BYTES, rv, kbase, kstride, k0 + t * kRows,
                g.len, wave, kDkdvWaves, lane);
    }
    const char *ktl = kvt + (kw >> 1) * T::BYTES;                              // tile of my keys
    const char *vtl = kvt + (kKeysPerWg / kRows + (kw >> 1)) * T::BYTES;
    const int krow = (kw & 1) * 32 + l32;                                      // my key's row there

    auto issue = [&](int it, int st) __attribute__((always_inline)) {
        const int gi = it / nqt, qt = qt_end - 1 - it % nqt;
        const int hq = hk * g.G + gi;
        const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
        const int row0 = qt * kRows;
        char *base = smem + st * STAGE;
        T::load(base, rq, qbase, qstride, row0, g.len, wave, kDkdvWaves, lane);
        T::load(base + T::BYTES, rdo, qbase, qstride, row0, g.len, wave, kDkdvWaves, lane);
        if (wave < 2) {  // per-row lse2 (wave 0) and delta (wave 1), 4 bytes per lane
            const int row = row0 + lane;
            const uint32_t off =
                row < g.len ? (uint32_t)(((size_t)hq * g.N + (size_t)row * g.rowmul + s) * 4) : kOob;
            dma_lds4(wave == 0 ? rl2 : rdl, base + 2 * T::BYTES + wave * kRows * 4, off);
        }
    };
    if (iters > 0) issue(0, 0);

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
                    const int qd = qlo + 8 * rq + 4 * hi + e - key;  // query - key
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
    auto step = [&](int it, auto stage) __attribute__((always_inline)) {
        constexpr int st = decltype(stage)::value;
        if (it + 1 < iters) issue(it + 1, st ^ 1);
        const int qlo = (qt_end - 1 - it % nqt) * kRows + qb * 32;
        // wave-uniform: some of my 32 queries see some of my keys
        if (qlo + 31 >= kw0 && qlo - kw0 < 31 + g.window) {
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
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
                sacc = mfma32(T::row_operand(qt, qb * 32 + l32, kk, hi),
                              T::row_operand(ktl, krow, kk, hi), sacc);
                pacc = mfma32(T::row_operand(dot, qb * 32 + l32, kk, hi),
                              T::row_operand(vtl, krow, kk, hi), pacc);
            }
            uint32_t pw[8], dw[8];
            if (qlo < kw0 + 31 || qlo + 31 - kw0 >= g.window)  // diagonal or window edge
                softmax(sacc, pacc, qlo, pw, dw, std::true_type{});
            else
                softmax(sacc, pacc, qlo, pw, dw, std::false_type{});
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const bf16x8 pb = __builtin_bit_cast(
                    bf16x8, u32x4{pw[h * 4], pw[h * 4 + 1], pw[h * 4 + 2], pw[h * 4 + 3]});
                const bf16x8 dsb = __builtin_bit_cast(
                    bf16x8, u32x4{dw[h * 4], dw[h * 4 + 1], dw[h * 4 + 2], dw[h * 4 + 3]});
                const int kk = qb * 2 + h;  // 16-row group of the 64-row tile
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    adv[db] = mfma32(T::tr_operand(dot, db * 32, kk, lane), pb, adv[db]);
                    adk[db] = mfma32(T::tr_operand(qt, db * 32, kk, lane), dsb, adk[db]);
                }
            }
        }
        wait_lds_loads();
        lds_barrier();
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
    if (qb == 0 && key < g.len) {
        const uint32_t off = kbase + (uint32_t)key * kstride;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const f32x4 pk = park[((0 * DB + db) * 4 + rq) * 64 + lane];
                const f32x4 pv = park[((1 * DB + db) * 4 + rq) * 64 + lane];
                const int d0 = db * 32 + 8 * rq + 4 * hi;
                const float sc = g.scale;
                const u32x2 wk = {pack_bf16((adk[db][4 * rq] + pk[0]) * sc, (adk[db][4 * rq + 1] + pk[1]) * sc),
                                  pack_bf16((adk[db][4 * rq + 2] + pk[2]) * sc, (adk[db][4 * rq + 3] + pk[3]) * sc)};
                const u32x2 wv = {pack_bf16(adv[db][4 * rq] + pv[0], adv[db][4 * rq + 1] + pv[1]),
                                  pack_bf16(adv[db][4 * rq + 2] + pv[2], adv[db][4 * rq + 3] + pv[3])};
                st8(rdk, off + d0 * 2, wk);
                st8(rdv, off + d0 * 2, wv);
            }
    }
}

template <int D>
__global__ __launch_bounds__(kDqWaves * 64, 1) void sfa_dq_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    const bf16 *__restrict__ o, const float *__restrict__ lse, const bf16 *__restrict__ dO,
    float *__restrict__ nstat_d, float *__restrict__ nstat_l, const bf16 *__restrict__ kt,
    bf16 *__restrict__ dq, SfaGeom g, int len_pad)
{
    constexpr int KS = D / 16, DB = D / 32;
    using T = Tile<D>;
    using TT = TileT<D>;
    // [stage][K rows | V rows | K transposed]
    __shared__ __attribute__((aligned(1024))) char smem[2][2 * T::BYTES + TT::BYTES];

    const int ntiles = (g.len + kRowsPerWg - 1) / kRowsPerWg;
    const int nprob = g.B * g.Hq * g.streams;
    int prob, tile;
    decode_tile(blockIdx.x, nprob, ntiles, prob, tile);
    const int s = prob % g.streams;
    const int hq = (prob / g.streams) % g.Hq;
    const int b = prob / (g.streams * g.Hq);
    const int hk = hq / g.G;

    const size_t qslice = (size_t)g.N * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const rsrc_t rq = make_rsrc(q + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rdo = make_rsrc(dO + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rdq = make_rsrc(dq + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rv = make_rsrc(v + b * kslice, (uint32_t)(kslice * 2));
    const size_t ktslice = (size_t)D * len_pad;  // one key/value problem, transposed
    const rsrc_t rkt = make_rsrc(kt + ((size_t)(b * g.Hkv + hk) * g.streams + s) * ktslice,
                                 (uint32_t)(ktslice * 2));
    const uint32_t qstride = (uint32_t)g.rowmul * g.Hq * D * 2;
    const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase = (uint32_t)(s * g.Hkv + hk) * D * 2;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
    const int l32 = lane & 31, hi = lane >> 5;
    const int q0 = tile * kRowsPerWg;
    const int row = q0 + wave * 32 + l32;

    const int kend = min(g.len, q0 + kRowsPerWg);
    const int nkt = (kend + kRows - 1) / kRows;
    // first key tile any row of the workgroup sees (0 unless the layer is local); the
    // LDS stage of tile j is (j - jf) % 2
    const int jf = max(0, q0 - g.window + 1) / kRows;
    auto issue = [&](int j) __attribute__((always_inline)) {
        char *st = smem[(j - jf) & 1];
        T::load(st, rk, kbase, kstride, j * kRows, g.len, wave, kDqWaves, lane);
        T::load(st + T::BYTES, rv, kbase, kstride, j * kRows, g.len, wave, kDqWaves, lane);
        TT::load(st + 2 * T::BYTES, rkt, 0, (uint32_t)len_pad * 2, j * kRows, wave, kDqWaves, lane);
    };
    issue(jf);

    // This lane's query row (dims kk*16 + hi*8 .. +7 of every k-step) of Q and dO, and
    // the row statistics: lse in log2 units and Delta = rowsum(dO * O), from the
    // forward's O and lse.  Every query row belongs to exactly one workgroup, which
    // also stores -Delta and -lse/scale for the dK/dV pass.
    bf16x8 qr[KS], dor[KS];
    float lrow = 0.f, drow = 0.f;
    {
        const rsrc_t ro = make_rsrc(o + b * qslice, (uint32_t)(qslice * 2));
        const uint32_t off = row < g.len ? qbase + (uint32_t)row * qstride : kOob;
        float dpart = 0.f;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            qr[kk] = __builtin_bit_cast(bf16x8, ld16(rq, off + (kk * 16 + hi * 8) * 2));
            const u32x4 dw = ld16(rdo, off + (kk * 16 + hi * 8) * 2);
            const u32x4 ow = ld16(ro, off + (kk * 16 + hi * 8) * 2);
            dor[kk] = __builtin_bit_cast(bf16x8, dw);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                dpart = __builtin_fmaf(bf16_lo(dw[w]), bf16_lo(ow[w]), dpart);
                dpart = __builtin_fmaf(bf16_hi(dw[w]), bf16_hi(ow[w]), dpart);
            }
        }
        drow = dpart + __shfl_xor(dpart, 32);
        if (row < g.len) {
            const size_t li = ((size_t)b * g.Hq + hq) * g.N + (size_t)row * g.rowmul + s;
            const float l = lse[li];
            lrow = l * 1.4426950408889634f;
            if (hi == 0) {
                nstat_d[li] = -drow;
                nstat_l[li] = -l / g.scale;
            }
        }
    }

    f32x16 adq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) adq[db] = f32x16{};

    const float c2 = g.scale_log2;
    const int wrow_min = q0 + wave * 32, wrow_max = wrow_min + 31;
    wait_lds_loads();
    lds_barrier();

    // dS^T of one 32-key half as two B operands; MASK selects the diagonal variant
    auto softmax = [&](const f32x16 &sacc, const f32x16 &pacc, int k0, bf16x8 (&dsb)[2], auto mask) {
        constexpr bool kMask = decltype(mask)::value;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            uint32_t w[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float ds2[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    const int r = h * 8 + 2 * e + u;
                    float p = fast_exp2(__builtin_fmaf(sacc[r], c2, -lrow));
                    if constexpr (kMask) {  // causal and, for local layers, windowed
                        const int key = k0 + 8 * (r >> 2) + 4 * hi + (r & 3);
                        if (key > row || row - key >= g.window) p = 0.f;
                    }
                    ds2[u] = p * (pacc[r] - drow);
                }
                w[e] = pack_bf16(ds2[0], ds2[1]);
            }
            dsb[h] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
        }
    };
    // One 64-key tile as two 32-key halves (S^T and dP^T, softmax, dQ^T each), which
    // keeps registers free for operand prefetch.
    auto tile_body = [&](const char *ktl, const char *vt, const char *ktt, int kb0, bool diag) __attribute__((always_inline)) {
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            f32x16 sacc = f32x16{}, pacc = f32x16{};
#pragma unroll
            for (int kk = 0; kk < KS; ++kk) {
                sacc = mfma32(T::row_operand(ktl, mb * 32 + l32, kk, hi), qr[kk], sacc);
                pacc = mfma32(T::row_operand(vt, mb * 32 + l32, kk, hi), dor[kk], pacc);
            }
            bf16x8 dsb[2];
            if (diag)
                softmax(sacc, pacc, kb0 + mb * 32, dsb, std::true_type{});
            else
                softmax(sacc, pacc, kb0 + mb * 32, dsb, std::false_type{});
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    adq[db] = mfma32(TT::operand(ktt, db * 32 + l32, mb * 2 + h, hi), dsb[h], adq[db]);
        }
    };
    auto step = [&](int j, auto stage) __attribute__((always_inline)) {
        constexpr int kSt = decltype(stage)::value;
        if (j + 1 < nkt) issue(j + 1);
        const int kb0 = j * kRows;
        // wave-uniform: the tile holds a key that some row of this wave sees
        if (kb0 <= wrow_max && wrow_min - (kb0 + kRows - 1) < g.window) {
            const char *ktl = smem[kSt];
            const char *vt = ktl + T::BYTES;
            const char *ktt = ktl + 2 * T::BYTES;
            // mask on the diagonal tile and on tiles reaching a window before a row
            tile_body(ktl, vt, ktt, kb0, kb0 + kRows - 1 > wrow_min || wrow_max - kb0 >= g.window);
        }
        wait_lds_loads();
        lds_barrier();
    };
    for (int j = jf; j < nkt; j += 2) {
        step(j, std::integral_constant<int, 0>{});
        if (j + 1 < nkt) step(j + 1, std::integral_constant<int, 1>{});
    }

    if (row < g.len) {
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
                      const float *lse, const bf16 *dO, float *delta, float *lse2, bf16 *kt,
                      int len_pad, bf16 *dq, bf16 *dk, bf16 *dv, const SfaGeom &g, hipStream_t s,
                      const char *tr_name, const char *dq_name, const char *dkdv_name)
{
    timing_before(tr_name, s);
    transpose_k_kernel<D><<<g.B * g.Hkv * g.streams * (len_pad / kRows), 256, 0, s>>>(k, kt, g,
                                                                                     len_pad);
    hipError_t e = hipGetLastError();
    timing_after(s);
    if (e != hipSuccess) return e;
    const int nqt = (g.len + kRowsPerWg - 1) / kRowsPerWg;
    timing_before(dq_name, s);
    sfa_dq_bf16_kernel<D><<<nqt * g.B * g.Hq * g.streams, kDqWaves * 64, 0, s>>>(
        q, k, v, o, lse, dO, delta, lse2, kt, dq, g, len_pad);
    e = hipGetLastError();
    timing_after(s);
    if (e != hipSuccess) return e;
    const int nkt = (g.len + kKeysPerWg - 1) / kKeysPerWg;
    timing_before(dkdv_name, s);
    sfa_dkdv_bf16_kernel<D><<<nkt * g.B * g.Hkv * g.streams, kDkdvWaves * 64, 0, s>>>(q, k, v, dO, delta,
                                                                           lse2, dk, dv, g);
    e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace

hipError_t launch_bwd_bf16(const void *q, const void *k, const void *v, const void *o,
                           const float *lse, const void *dO, void *dq, void *dk, void *dv,
                           const SfaGeom &g, void *ws, hipStream_t s)
{
    const BwdWorkspace w = bwd_workspace(g, 2);
    char *wsb = static_cast<char *>(ws);
    float *delta = reinterpret_cast<float *>(wsb + w.delta);
    float *lse2 = reinterpret_cast<float *>(wsb + w.lse2);
    bf16 *kt = reinterpret_cast<bf16 *>(wsb + w.kt);
    const bf16 *qq = static_cast<const bf16 *>(q), *kk = static_cast<const bf16 *>(k),
               *vv = static_cast<const bf16 *>(v), *dd = static_cast<const bf16 *>(dO),
               *oo = static_cast<const bf16 *>(o);
    bf16 *gq = static_cast<bf16 *>(dq), *gk = static_cast<bf16 *>(dk), *gv = static_cast<bf16 *>(dv);
    if (g.D == 32)
        return bwd_bf16_d<32>(qq, kk, vv, oo, lse, dd, delta, lse2, kt, w.len_pad, gq, gk, gv, g, s,
                              "sfa_bwd_transpose_d32", "sfa_dq_bf16_d32", "sfa_dkdv_bf16_d32");
    if (g.D == 64)
        return bwd_bf16_d<64>(qq, kk, vv, oo, lse, dd, delta, lse2, kt, w.len_pad, gq, gk, gv, g, s,
                              "sfa_bwd_transpose_d64", "sfa_dq_bf16_d64", "sfa_dkdv_bf16_d64");
    return bwd_bf16_d<128>(qq, kk, vv, oo, lse, dd, delta, lse2, kt, w.len_pad, gq, gk, gv, g, s,
                           "sfa_bwd_transpose_d128", "sfa_dq_bf16_d128", "sfa_dkdv_bf16_d128");
}

}  // namespace hd
