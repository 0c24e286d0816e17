// sfa_f32.hip -- fp32 Stream-Factorized Attention forward/backward (with its backward
// preprocess, which forms Delta and the base-2 lse of every query row; the bf16 path
// forms its row statistics in a kernel of its own before the dK/dV pass).
//
// The fp32 kernels serve small, accuracy-first workloads: one lane owns one query row
// (forward, dQ) or one key row (dK/dV), tiles of the other operand are staged in LDS
// and read as broadcasts.  Arithmetic is plain fp32 FMA with an fp32 online softmax.
// Same problem decomposition as the bf16 path (see SfaGeom).
#include "hd_device.h"

namespace hd {

namespace {

constexpr int kRows = 64;  // rows per workgroup (one wave)
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kLog2e = 1.4426950408889634f;

template <int D>
__global__ __launch_bounds__(64) void sfa_fwd_f32_kernel(const float *__restrict__ q,
                                                         const float *__restrict__ k,
                                                         const float *__restrict__ v,
                                                         float *__restrict__ o,
                                                         float *__restrict__ lse, SfaGeom g)
{
    __shared__ float sk[kRows][D];
    __shared__ float sv[kRows][D];
    const int ntiles = (g.len + kRows - 1) / kRows;
    const int nprob = g.B * g.Hq * g.streams;
    int prob, tile;
    decode_tile(blockIdx.x, nprob, ntiles, prob, tile);
    const int s = prob % g.streams, hq = (prob / g.streams) % g.Hq;
    const int b = prob / (g.streams * g.Hq), hk = hq / g.G;
    const int tid = threadIdx.x, row = tile * kRows + tid;
    const size_t qs = (size_t)g.rowmul * g.Hq * D, ks = (size_t)g.rowmul * g.Hkv * D;
    const float *qb = q + (size_t)b * g.N * g.Hq * D + (size_t)(s * g.Hq + hq) * D;
    const float *kb = k + (size_t)b * g.N * g.Hkv * D + (size_t)(s * g.Hkv + hk) * D;
    const float *vb = v + (size_t)b * g.N * g.Hkv * D + (size_t)(s * g.Hkv + hk) * D;

    float qv[D], acc[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
        qv[d] = row < g.len ? qb[row * qs + d] : 0.f;
        acc[d] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    const int kend = min(g.len, tile * kRows + kRows);
    // first key any row of the tile sees (local layers: window)
    const int kbeg = max(0, tile * kRows - g.window + 1) / kRows * kRows;
    for (int j0 = kbeg; j0 < kend; j0 += kRows) {
        __syncthreads();
        const int key = j0 + tid;
#pragma unroll
        for (int d = 0; d < D; ++d) {
            sk[tid][d] = key < g.len ? kb[key * ks + d] : 0.f;
            sv[tid][d] = key < g.len ? vb[key * ks + d] : 0.f;
        }
        __syncthreads();
        if (row >= g.len) continue;
        const int jn = min(kRows, row - j0 + 1);  // causal: keys j0 .. row
        for (int jj = max(0, row - g.window + 1 - j0); jj < jn; ++jj) {
            float dot = 0.f;
#pragma unroll
            for (int d = 0; d < D; ++d) dot = __builtin_fmaf(qv[d], sk[jj][d], dot);
            const float x = dot * g.scale_log2;
            if (x > m) {
                const float alpha = exp2f(m - x);
                l *= alpha;
#pragma unroll
                for (int d = 0; d < D; ++d) acc[d] *= alpha;
                m = x;
            }
            const float p = exp2f(x - m);
            l += p;
#pragma unroll
            for (int d = 0; d < D; ++d) acc[d] = __builtin_fmaf(p, sv[jj][d], acc[d]);
        }
    }
    if (row < g.len) {
        float *ob = o + (size_t)b * g.N * g.Hq * D + (size_t)(s * g.Hq + hq) * D + row * qs;
        const float inv = 1.f / l;
#pragma unroll
        for (int d = 0; d < D; ++d) ob[d] = acc[d] * inv;
        lse[((size_t)b * g.Hq + hq) * g.N + (size_t)row * g.rowmul + s] = (m + log2f(l)) * kLn2;
    }
}

// Per (b, hq, p) query row: delta = sum_d dO * O and lse2 = lse * log2(e).  One group
// of lanes per row, 16 bytes per lane, reduced with xor shuffles.
template <int D>
__global__ __launch_bounds__(256) void bwd_preprocess_kernel(const float *__restrict__ o,
                                                             const float *__restrict__ dO,
                                                             const float *__restrict__ lse,
                                                             float *__restrict__ delta,
                                                             float *__restrict__ lse2, SfaGeom g)
{
    constexpr int LPR = D / 4;      // lanes per row, 4 floats each
    constexpr int RPB = 256 / LPR;  // rows per workgroup
    const size_t rows = (size_t)g.B * g.N * g.Hq;
    const size_t r = (size_t)blockIdx.x * RPB + threadIdx.x / LPR;
    const int part = threadIdx.x % LPR;
    float acc = 0.f;
    if (r < rows) {
        const u32x4 a = *reinterpret_cast<const u32x4 *>(o + r * D + part * 4);
        const u32x4 c = *reinterpret_cast<const u32x4 *>(dO + r * D + part * 4);
#pragma unroll
        for (int w = 0; w < 4; ++w) acc = __builtin_fmaf(__uint_as_float(a[w]), __uint_as_float(c[w]), acc);
    }
#pragma unroll
    for (int off = LPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (r < rows && part == 0) {
        const int hq = (int)(r % g.Hq);
        const size_t bp = r / g.Hq;  // b * N + p
        const size_t b = bp / g.N, p = bp % g.N;
        const size_t li = (b * g.Hq + hq) * g.N + p;
        delta[li] = acc;
        lse2[li] = lse[li] * kLog2e;
    }
}

template <int D>
__global__ __launch_bounds__(64) void sfa_dq_f32_kernel(const float *__restrict__ q,
                                                        const float *__restrict__ k,
                                                        const float *__restrict__ v,
                                                        const float *__restrict__ dO,
                                                        const float *__restrict__ delta,
                                                        const float *__restrict__ lse2,
                                                        float *__restrict__ dq, SfaGeom g)
{
    __shared__ float sk[kRows][D];
    __shared__ float sv[kRows][D];
    const int ntiles = (g.len + kRows - 1) / kRows;
    const int nprob = g.B * g.Hq * g.streams;
    int prob, tile;
    decode_tile(blockIdx.x, nprob, ntiles, prob, tile);
    const int s = prob % g.streams, hq = (prob / g.streams) % g.Hq;
    const int b = prob / (g.streams * g.Hq), hk = hq / g.G;
    const int tid = threadIdx.x, row = tile * kRows + tid;
    const size_t qs = (size_t)g.rowmul * g.Hq * D, ks = (size_t)g.rowmul * g.Hkv * D;
    const size_t qoff = (size_t)b * g.N * g.Hq * D + (size_t)(s * g.Hq + hq) * D;
    const float *kb = k + (size_t)b * g.N * g.Hkv * D + (size_t)(s * g.Hkv + hk) * D;
    const float *vb = v + (size_t)b * g.N * g.Hkv * D + (size_t)(s * g.Hkv + hk) * D;
    const size_t li = ((size_t)b * g.Hq + hq) * g.N + (size_t)row * g.rowmul + s;

    float qv[D], dov[D], acc[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
        qv[d] = row < g.len ? q[qoff + row * qs + d] : 0.f;
        dov[d] = row < g.len ? dO[qoff + row * qs + d] : 0.f;
        acc[d] = 0.f;
    }
    const float l2 = row < g.len ? lse2[li] : 0.f;
    const float dl = row < g.len ? delta[li] : 0.f;
    const int kend = min(g.len, tile * kRows + kRows);
    const int kbeg = max(0, tile * kRows - g.window + 1) / kRows * kRows;
    for (int j0 = kbeg; j0 < kend; j0 += kRows) {
        __syncthreads();
        const int key = j0 + tid;
#pragma unroll
        for (int d = 0; d < D; ++d) {
            sk[tid][d] = key < g.len ? kb[key * ks + d] : 0.f;
            sv[tid][d] = key < g.len ? vb[key * ks + d] : 0.f;
        }
        __syncthreads();
        if (row >= g.len) continue;
        const int jn = min(kRows, row - j0 + 1);
        for (int jj = max(0, row - g.window + 1 - j0); jj < jn; ++jj) {
            float dot = 0.f, dp = 0.f;
#pragma unroll
            for (int d = 0; d < D; ++d) {
                dot = __builtin_fmaf(qv[d], sk[jj][d], dot);
                dp = __builtin_fmaf(dov[d], sv[jj][d], dp);
            }
            const float p = exp2f(dot * g.scale_log2 - l2);
            const float ds = p * (dp - dl);
#pragma unroll
            for (int d = 0; d < D; ++d) acc[d] = __builtin_fmaf(ds, sk[jj][d], acc[d]);
        }
    }
    if (row < g.len) {
#pragma unroll
        for (int d = 0; d < D; ++d) dq[qoff + row * qs + d] = acc[d] * g.scale;
    }
}

// One lane per key row of problem (b, hk, s); loops over the group's query heads and
// the query rows that see the key.
template <int D>
__global__ __launch_bounds__(64) void sfa_dkdv_f32_kernel(const float *__restrict__ q,
                                                          const float *__restrict__ k,
                                                          const float *__restrict__ v,
                                                          const float *__restrict__ dO,
                                                          const float *__restrict__ delta,
                                                          const float *__restrict__ lse2,
                                                          float *__restrict__ dk,
                                                          float *__restrict__ dv, SfaGeom g)
{
    __shared__ float sq[kRows][D];
    __shared__ float sd[kRows][D];
    __shared__ float sl[kRows], sdl[kRows];
    const int ntiles = (g.len + kRows - 1) / kRows;
    const int nprob = g.B * g.Hkv * g.streams;
    int prob, tile;
    decode_key_tile(blockIdx.x, nprob, ntiles, prob, tile);
    const int s = prob % g.streams, hk = (prob / g.streams) % g.Hkv;
    const int b = prob / (g.streams * g.Hkv);
    const int tid = threadIdx.x, key = tile * kRows + tid;
    const size_t qs = (size_t)g.rowmul * g.Hq * D, ks = (size_t)g.rowmul * g.Hkv * D;
    const size_t koff = (size_t)b * g.N * g.Hkv * D + (size_t)(s * g.Hkv + hk) * D;

    float kv[D], vv[D], ak[D], av[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
        kv[d] = key < g.len ? k[koff + key * ks + d] : 0.f;
        vv[d] = key < g.len ? v[koff + key * ks + d] : 0.f;
        ak[d] = 0.f;
        av[d] = 0.f;
    }
    for (int gi = 0; gi < g.G; ++gi) {
        const int hq = hk * g.G + gi;
        const size_t qoff = (size_t)b * g.N * g.Hq * D + (size_t)(s * g.Hq + hq) * D;
        const size_t lbase = ((size_t)b * g.Hq + hq) * g.N + s;
        // queries that see a key of this tile (local layers: up to the window's end)
        const int qend = (int)min((int64_t)g.len, (int64_t)tile * kRows + kRows - 1 + g.window);
        for (int i0 = tile * kRows; i0 < qend; i0 += kRows) {
            __syncthreads();
            const int qrow = i0 + tid;
#pragma unroll
            for (int d = 0; d < D; ++d) {
                sq[tid][d] = qrow < g.len ? q[qoff + qrow * qs + d] : 0.f;
                sd[tid][d] = qrow < g.len ? dO[qoff + qrow * qs + d] : 0.f;
            }
            sl[tid] = qrow < g.len ? lse2[lbase + (size_t)qrow * g.rowmul] : 0.f;
            sdl[tid] = qrow < g.len ? delta[lbase + (size_t)qrow * g.rowmul] : 0.f;
            __syncthreads();
            if (key >= g.len) continue;
            const int in = min(kRows, g.len - i0);
            // causal and windowed: key <= query < key + window
            const int iend = (int)min((int64_t)in, (int64_t)key + g.window - i0);
            for (int ii = max(0, key - i0); ii < iend; ++ii) {
                float dot = 0.f, dp = 0.f;
#pragma unroll
                for (int d = 0; d < D; ++d) {
                    dot = __builtin_fmaf(sq[ii][d], kv[d], dot);
                    dp = __builtin_fmaf(sd[ii][d], vv[d], dp);
                }
                const float p = exp2f(dot * g.scale_log2 - sl[ii]);
                const float ds = p * (dp - sdl[ii]);
#pragma unroll
                for (int d = 0; d < D; ++d) {
                    av[d] = __builtin_fmaf(p, sd[ii][d], av[d]);
                    ak[d] = __builtin_fmaf(ds, sq[ii][d], ak[d]);
                }
            }
        }
    }
    if (key < g.len) {
#pragma unroll
        for (int d = 0; d < D; ++d) {
            dk[koff + key * ks + d] = ak[d] * g.scale;
            dv[koff + key * ks + d] = av[d];
        }
    }
}

template <int D>
hipError_t fwd_f32_d(const float *q, const float *k, const float *v, float *o, float *lse,
                     const SfaGeom &g, hipStream_t s)
{
    const int ntiles = (g.len + kRows - 1) / kRows;
    timing_before("sfa_fwd_f32", s);
    sfa_fwd_f32_kernel<D><<<ntiles * g.B * g.Hq * g.streams, kRows, 0, s>>>(q, k, v, o, lse, g);
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

template <int D>
hipError_t bwd_f32_d(const float *q, const float *k, const float *v, const float *dO,
                     float *dq, float *dk, float *dv, const SfaGeom &g, float *delta,
                     float *lse2, hipStream_t s)
{
    const int ntiles = (g.len + kRows - 1) / kRows;
    timing_before("sfa_dq_f32", s);
    sfa_dq_f32_kernel<D><<<ntiles * g.B * g.Hq * g.streams, kRows, 0, s>>>(q, k, v, dO, delta,
                                                                            lse2, dq, g);
    hipError_t e = hipGetLastError();
    timing_after(s);
    if (e != hipSuccess) return e;
    timing_before("sfa_dkdv_f32", s);
    sfa_dkdv_f32_kernel<D><<<ntiles * g.B * g.Hkv * g.streams, kRows, 0, s>>>(
        q, k, v, dO, delta, lse2, dk, dv, g);
    e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace

hipError_t launch_bwd_preprocess_f32(const float *o, const float *dO, const float *lse,
                                     float *delta, float *lse2, const SfaGeom &g, hipStream_t s)
{
    const size_t rows = (size_t)g.B * g.N * g.Hq;
    const int lpr = g.D * 4 / 16;
    const int rpb = 256 / lpr;
    const dim3 grid((unsigned)((rows + rpb - 1) / rpb));
    timing_before("sfa_bwd_preprocess_f32", s);
    if (g.D == 32)
        bwd_preprocess_kernel<32><<<grid, 256, 0, s>>>(o, dO, lse, delta, lse2, g);
    else if (g.D == 64)
        bwd_preprocess_kernel<64><<<grid, 256, 0, s>>>(o, dO, lse, delta, lse2, g);
    else
        bwd_preprocess_kernel<128><<<grid, 256, 0, s>>>(o, dO, lse, delta, lse2, g);
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

hipError_t launch_fwd_f32(const float *q, const float *k, const float *v, float *o, float *lse,
                          const SfaGeom &g, hipStream_t s)
{
    if (g.D == 32) return fwd_f32_d<32>(q, k, v, o, lse, g, s);
    if (g.D == 64) return fwd_f32_d<64>(q, k, v, o, lse, g, s);
    return fwd_f32_d<128>(q, k, v, o, lse, g, s);
}

hipError_t launch_bwd_f32(const float *q, const float *k, const float *v, const float *o,
                          const float *lse, const float *dO, float *dq, float *dk, float *dv,
                          const SfaGeom &g, void *ws, hipStream_t s)
{
    const BwdWorkspace w = bwd_workspace(g, 4);
    float *delta = reinterpret_cast<float *>(static_cast<char *>(ws) + w.delta);
    float *lse2 = reinterpret_cast<float *>(static_cast<char *>(ws) + w.lse2);
    hipError_t e = launch_bwd_preprocess_f32(o, dO, lse, delta, lse2, g, s);
    if (e != hipSuccess) return e;
    if (g.D == 32) return bwd_f32_d<32>(q, k, v, dO, dq, dk, dv, g, delta, lse2, s);
    if (g.D == 64) return bwd_f32_d<64>(q, k, v, dO, dq, dk, dv, g, delta, lse2, s);
    return bwd_f32_d<128>(q, k, v, dO, dq, dk, dv, g, delta, lse2, s);
}

}  // namespace hd
