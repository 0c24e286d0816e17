// sfa_bwd_bf16.hip -- Stream-Factorized Attention backward, bf16 in/out, fp32 math.
//
// Gradients of O = softmax(scale Q K^T + mask) V with the probabilities recomputed
// from the forward's log-sum-exp (kept in log2 units in the workspace):
//   P = exp2(scale*log2(e) q.k - lse2),  dP = dO V^T,  dS = P (dP - Delta),
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K,   Delta = rowsum(dO * O).
// Two deterministic kernels (no atomics):
//   dK/dV: a workgroup owns 128 keys of one (b, kv-head[, stream]) problem, 32 per wave,
//          and sweeps the query tiles that see them for every query head of the group,
//          so the grouped-query sum happens in registers.  Scores are formed as
//          S = Q K^T (one key per lane), which makes P and dS the B operands of
//          dV^T += dO^T P and dK^T += Q^T dS; Q and dO are staged in LDS both
//          row-major and transposed.
//   dQ:    a workgroup owns 128 query rows (32 per wave, one row per lane as in the
//          forward) and sweeps the key tiles at or below the diagonal:
//          S^T = K Q^T, dP^T = V dO^T, dQ^T += K^T dS^T.
#include "sfa_tiles.h"

namespace hd {

namespace {

constexpr int kKeysPerWg = 128;
constexpr int kRowsPerWg = 128;

template <int D>
struct DkdvLds {
    static constexpr int RM = kTileRows * (D + 8);  // elements
    static constexpr int TR = D * kTileRows;
    static constexpr int Q_RM = 0, DO_RM = RM, Q_TR = 2 * RM, DO_TR = 2 * RM + TR;
    static constexpr int ELEMS = 2 * RM + 2 * TR;
    static constexpr int BYTES = ELEMS * 2 + 2 * kTileRows * 4;  // + lse2, delta
};

template <int D>
__global__ __launch_bounds__(256, 1) void sfa_dkdv_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    const bf16 *__restrict__ dO, const float *__restrict__ delta, const float *__restrict__ lse2,
    bf16 *__restrict__ dk, bf16 *__restrict__ dv, SfaGeom g)
{
    constexpr int KS = D / 16, DB = D / 32;
    using LY = DkdvLds<D>;
    __shared__ __attribute__((aligned(16))) char smem[2][LY::BYTES];

    const int nkt = (g.len + kKeysPerWg - 1) / kKeysPerWg;
    const int nprob = g.B * g.Hkv * g.streams;
    int prob, ktile;
    decode_key_tile(blockIdx.x, nprob, nkt, prob, ktile);
    const int s = prob % g.streams;
    const int hk = (prob / g.streams) % g.Hkv;
    const int b = prob / (g.streams * g.Hkv);

    const size_t qslice = (size_t)g.N * g.Hq * D, kslice = (size_t)g.N * g.Hkv * D;
    const rsrc_t rq = make_rsrc(q + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rdo = make_rsrc(dO + b * qslice, (uint32_t)(qslice * 2));
    const rsrc_t rk = make_rsrc(k + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rv = make_rsrc(v + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rdk = make_rsrc(dk + b * kslice, (uint32_t)(kslice * 2));
    const rsrc_t rdv = make_rsrc(dv + b * kslice, (uint32_t)(kslice * 2));
    const uint32_t qstride = (uint32_t)g.rowmul * g.Hq * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase = (uint32_t)(s * g.Hkv + hk) * D * 2;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;
    const int k0 = ktile * kKeysPerWg;
    const int kw0 = k0 + wave * 32;
    const int key = kw0 + l32;

    // this lane's key and value rows as B operands
    bf16x8 kr[KS], vr[KS];
    {
        const uint32_t off = key < g.len ? kbase + (uint32_t)key * kstride : kOob;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            kr[kk] = __builtin_bit_cast(bf16x8, ld16(rk, off + (kk * 16 + hi * 8) * 2));
            vr[kk] = __builtin_bit_cast(bf16x8, ld16(rv, off + (kk * 16 + hi * 8) * 2));
        }
    }

    f32x16 adk[DB], adv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) adk[db] = adv[db] = f32x16{};

    const int qt_first = k0 / kTileRows;
    const int qt_end = (g.len + kTileRows - 1) / kTileRows;
    const int nqt = qt_end - qt_first;
    const int iters = g.G * nqt;

    QuadStager<D> stq, stdo;
    float lrow = 0.f;

    auto prefetch = [&](int it) {
        const int gi = it / nqt, qt = qt_first + it % nqt;
        const int hq = hk * g.G + gi;
        const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
        const int row0 = qt * kTileRows;
        stq.load(rq, qbase, qstride, row0, g.len, tid);
        stdo.load(rdo, qbase, qstride, row0, g.len, tid);
        if (tid < 2 * kTileRows) {
            const int row = row0 + (tid & (kTileRows - 1));
            const size_t li = ((size_t)b * g.Hq + hq) * g.N + (size_t)row * g.rowmul + s;
            const float *src = tid < kTileRows ? lse2 : delta;
            lrow = row < g.len ? src[li] : 0.f;
        }
    };
    auto commit = [&](int buf) {
        bf16 *base = reinterpret_cast<bf16 *>(smem[buf]);
        stq.store_rm(base + LY::Q_RM, tid);
        stq.store_tr(base + LY::Q_TR, tid);
        stdo.store_rm(base + LY::DO_RM, tid);
        stdo.store_tr(base + LY::DO_TR, tid);
        if (tid < 2 * kTileRows) reinterpret_cast<float *>(base + LY::ELEMS)[tid] = lrow;
    };

    const float c2 = g.scale_log2;
    if (iters > 0) {
        prefetch(0);
        commit(0);
    }
    __syncthreads();

    for (int it = 0; it < iters; ++it) {
        const int buf = it & 1;
        if (it + 1 < iters) prefetch(it + 1);
        const int qrow0 = (qt_first + it % nqt) * kTileRows;
        if (qrow0 + kTileRows - 1 >= kw0) {  // wave-uniform: some query sees some key
            const bf16 *base = reinterpret_cast<const bf16 *>(smem[buf]);
            const float *sl = reinterpret_cast<const float *>(base + LY::ELEMS);
            const float *sdl = sl + kTileRows;
            f32x16 sacc[2], pacc[2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                sacc[qb] = f32x16{};
                pacc[qb] = f32x16{};
#pragma unroll
                for (int kk = 0; kk < KS; ++kk) {
                    sacc[qb] = mfma32(rm_operand<D>(base + LY::Q_RM, qb * 32 + l32, kk, hi), kr[kk],
                                      sacc[qb]);
                    pacc[qb] = mfma32(rm_operand<D>(base + LY::DO_RM, qb * 32 + l32, kk, hi),
                                      vr[kk], pacc[qb]);
                }
            }
            const bool need_mask = qrow0 < kw0 + 31;
            bf16x8 pb[4], dsb[4];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                uint32_t pw[8], dw[8];
#pragma unroll
                for (int rq = 0; rq < 4; ++rq) {
                    const f32x4 l4 = *reinterpret_cast<const f32x4 *>(&sl[qb * 32 + 8 * rq + 4 * hi]);
                    const f32x4 d4 = *reinterpret_cast<const f32x4 *>(&sdl[qb * 32 + 8 * rq + 4 * hi]);
                    float p[4], ds[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int r = rq * 4 + e;
                        p[e] = fast_exp2(__builtin_fmaf(sacc[qb][r], c2, -l4[e]));
                        if (need_mask) {
                            const int query = qrow0 + qb * 32 + 8 * rq + 4 * hi + e;
                            if (query < key) p[e] = 0.f;
                        }
                        ds[e] = p[e] * (pacc[qb][r] - d4[e]);
                    }
                    pw[rq * 2] = pack_bf16(p[0], p[1]);
                    pw[rq * 2 + 1] = pack_bf16(p[2], p[3]);
                    dw[rq * 2] = pack_bf16(ds[0], ds[1]);
                    dw[rq * 2 + 1] = pack_bf16(ds[2], ds[3]);
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    pb[qb * 2 + h] = __builtin_bit_cast(
                        bf16x8, u32x4{pw[h * 4], pw[h * 4 + 1], pw[h * 4 + 2], pw[h * 4 + 3]});
                    dsb[qb * 2 + h] = __builtin_bit_cast(
                        bf16x8, u32x4{dw[h * 4], dw[h * 4 + 1], dw[h * 4 + 2], dw[h * 4 + 3]});
                }
            }
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int d = db * 32 + l32;
#pragma unroll
                for (int kk = 0; kk < 4; ++kk) {
                    adv[db] = mfma32(tr_operand(base + LY::DO_TR, d, kk, hi), pb[kk], adv[db]);
                    adk[db] = mfma32(tr_operand(base + LY::Q_TR, d, kk, hi), dsb[kk], adk[db]);
                }
            }
        }
        if (it + 1 < iters) commit(buf ^ 1);
        __syncthreads();
    }

    if (key < g.len) {
        const uint32_t off = kbase + (uint32_t)key * kstride;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int rq = 0; rq < 4; ++rq) {
                const int d0 = db * 32 + 8 * rq + 4 * hi;
                const u32x2 wk = {pack_bf16(adk[db][4 * rq] * g.scale, adk[db][4 * rq + 1] * g.scale),
                                  pack_bf16(adk[db][4 * rq + 2] * g.scale, adk[db][4 * rq + 3] * g.scale)};
                const u32x2 wv = {pack_bf16(adv[db][4 * rq], adv[db][4 * rq + 1]),
                                  pack_bf16(adv[db][4 * rq + 2], adv[db][4 * rq + 3])};
                st8(rdk, off + d0 * 2, wk);
                st8(rdv, off + d0 * 2, wv);
            }
    }
}

template <int D>
struct DqLds {
    static constexpr int RM = kTileRows * (D + 8);
    static constexpr int TR = D * kTileRows;
    static constexpr int K_RM = 0, V_RM = RM, K_TR = 2 * RM;
    static constexpr int BYTES = (2 * RM + TR) * 2;
};

template <int D>
__global__ __launch_bounds__(256, 1) void sfa_dq_bf16_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    const bf16 *__restrict__ dO, const float *__restrict__ delta, const float *__restrict__ lse2,
    bf16 *__restrict__ dq, SfaGeom g)
{
    constexpr int KS = D / 16, DB = D / 32;
    using LY = DqLds<D>;
    __shared__ __attribute__((aligned(16))) char smem[2][LY::BYTES];

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
    const uint32_t qstride = (uint32_t)g.rowmul * g.Hq * D * 2;
    const uint32_t qbase = (uint32_t)(s * g.Hq + hq) * D * 2;
    const uint32_t kstride = (uint32_t)g.rowmul * g.Hkv * D * 2;
    const uint32_t kbase = (uint32_t)(s * g.Hkv + hk) * D * 2;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;
    const int q0 = tile * kRowsPerWg;
    const int row = q0 + wave * 32 + l32;

    bf16x8 qr[KS], dor[KS];
    float lrow = 0.f, drow = 0.f;
    {
        const uint32_t off = row < g.len ? qbase + (uint32_t)row * qstride : kOob;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk) {
            qr[kk] = __builtin_bit_cast(bf16x8, ld16(rq, off + (kk * 16 + hi * 8) * 2));
            dor[kk] = __builtin_bit_cast(bf16x8, ld16(rdo, off + (kk * 16 + hi * 8) * 2));
        }
        if (row < g.len) {
            const size_t li = ((size_t)b * g.Hq + hq) * g.N + (size_t)row * g.rowmul + s;
            lrow = lse2[li];
            drow = delta[li];
        }
    }

    f32x16 adq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) adq[db] = f32x16{};

    const int kend = min(g.len, q0 + kRowsPerWg);
    const int nkt = (kend + kTileRows - 1) / kTileRows;
    QuadStager<D> stk, stv;
    auto prefetch = [&](int j) {
        stk.load(rk, kbase, kstride, j * kTileRows, g.len, tid);
        stv.load(rv, kbase, kstride, j * kTileRows, g.len, tid);
    };
    auto commit = [&](int buf) {
        bf16 *base = reinterpret_cast<bf16 *>(smem[buf]);
        stk.store_rm(base + LY::K_RM, tid);
        stk.store_tr(base + LY::K_TR, tid);
        stv.store_rm(base + LY::V_RM, tid);
    };

    const float c2 = g.scale_log2;
    const int wrow_min = q0 + wave * 32, wrow_max = wrow_min + 31;
    prefetch(0);
    commit(0);
    __syncthreads();

    for (int j = 0; j < nkt; ++j) {
        const int buf = j & 1;
        if (j + 1 < nkt) prefetch(j + 1);
        const int kb0 = j * kTileRows;
        if (kb0 <= wrow_max) {
            const bf16 *base = reinterpret_cast<const bf16 *>(smem[buf]);
            f32x16 sacc[2], pacc[2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb) {
                sacc[mb] = f32x16{};
                pacc[mb] = f32x16{};
#pragma unroll
                for (int kk = 0; kk < KS; ++kk) {
                    sacc[mb] = mfma32(rm_operand<D>(base + LY::K_RM, mb * 32 + l32, kk, hi), qr[kk],
                                      sacc[mb]);
                    pacc[mb] = mfma32(rm_operand<D>(base + LY::V_RM, mb * 32 + l32, kk, hi), dor[kk],
                                      pacc[mb]);
                }
            }
            const bool need_mask = kb0 + kTileRows - 1 > wrow_min;
            bf16x8 dsb[4];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    uint32_t w[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        float ds2[2];
#pragma unroll
                        for (int u = 0; u < 2; ++u) {
                            const int r = h * 8 + 2 * e + u;
                            float p = fast_exp2(__builtin_fmaf(sacc[mb][r], c2, -lrow));
                            if (need_mask) {
                                const int kidx = kb0 + mb * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
                                if (kidx > row) p = 0.f;
                            }
                            ds2[u] = p * (pacc[mb][r] - drow);
                        }
                        w[e] = pack_bf16(ds2[0], ds2[1]);
                    }
                    dsb[mb * 2 + h] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
                }
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int d = db * 32 + l32;
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
                    adq[db] = mfma32(tr_operand(base + LY::K_TR, d, kk, hi), dsb[kk], adq[db]);
            }
        }
        if (j + 1 < nkt) commit(buf ^ 1);
        __syncthreads();
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
hipError_t bwd_bf16_d(const bf16 *q, const bf16 *k, const bf16 *v, const bf16 *dO,
                      const float *delta, const float *lse2, bf16 *dq, bf16 *dk, bf16 *dv,
                      const SfaGeom &g, hipStream_t s, const char *dq_name, const char *dkdv_name)
{
    const int nqt = (g.len + kRowsPerWg - 1) / kRowsPerWg;
    timing_before(dq_name, s);
    sfa_dq_bf16_kernel<D><<<nqt * g.B * g.Hq * g.streams, 256, 0, s>>>(q, k, v, dO, delta, lse2,
                                                                        dq, g);
    hipError_t e = hipGetLastError();
    timing_after(s);
    if (e != hipSuccess) return e;
    const int nkt = (g.len + kKeysPerWg - 1) / kKeysPerWg;
    timing_before(dkdv_name, s);
    sfa_dkdv_bf16_kernel<D><<<nkt * g.B * g.Hkv * g.streams, 256, 0, s>>>(q, k, v, dO, delta,
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
    const size_t half = bwd_workspace_bytes(g) / 2;
    float *delta = static_cast<float *>(ws);
    float *lse2 = reinterpret_cast<float *>(static_cast<char *>(ws) + half);
    hipError_t e = launch_bwd_preprocess(o, dO, lse, delta, lse2, g, 2, s);
    if (e != hipSuccess) return e;
    const bf16 *qq = static_cast<const bf16 *>(q), *kk = static_cast<const bf16 *>(k),
               *vv = static_cast<const bf16 *>(v), *dd = static_cast<const bf16 *>(dO);
    bf16 *gq = static_cast<bf16 *>(dq), *gk = static_cast<bf16 *>(dk), *gv = static_cast<bf16 *>(dv);
    if (g.D == 32)
        return bwd_bf16_d<32>(qq, kk, vv, dd, delta, lse2, gq, gk, gv, g, s, "sfa_dq_bf16_d32",
                              "sfa_dkdv_bf16_d32");
    if (g.D == 64)
        return bwd_bf16_d<64>(qq, kk, vv, dd, delta, lse2, gq, gk, gv, g, s, "sfa_dq_bf16_d64",
                              "sfa_dkdv_bf16_d64");
    return bwd_bf16_d<128>(qq, kk, vv, dd, delta, lse2, gq, gk, gv, g, s, "sfa_dq_bf16_d128",
                           "sfa_dkdv_bf16_d128");
}

}  // namespace hd
