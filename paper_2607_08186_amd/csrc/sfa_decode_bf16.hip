// sfa_decode_bf16.hip -- parallel-stream decode for Stream-Factorized Attention.
//
// At a decode step the n streams of each sequence's new token are run together: query
// row s of sequence b sits at expanded position ctx[b]*n + s and attends, under the
// layer's mask, to the sequence's cached rows (the new token's own n keys and values
// are already appended at rows ctx[b]*n .. ctx[b]*n + n - 1).  An intra-stream layer
// reads only its stream's rows (1/n of the cache), a full cross-stream layer the whole
// prefix, a local one the last `window` positions.
//
// HBM-bound: every cached key/value row is read once for all the query rows that use it
// (the heads of its group, and for cross-stream layers all n streams: up to 32 query
// slots per problem).  Split over the cache:
//   partial: a workgroup takes 256 cached rows of one problem (b, kv-head[, head chunk]
//            [, stream]), one 64-row tile per wave, K to registers and V to LDS (all
//            loads issued up front; two workgroups per CU, so one's loads overlap the
//            other's arithmetic), S^T = K Q^T and O^T += V^T P^T on the matrix cores,
//            the four waves merged through LDS into one (max, sum, unnormalised O) per
//            query slot in the workspace;
//   combine: per query row, the chunks' partials reduced to o and lse.
#include <mutex>

#include "decode_internal.h"
#include "sfa_lds.h"

namespace hd {

namespace {

constexpr int kDecWaves = 4;
constexpr int kDecChunk = kDecWaves * kRows;  // cached rows per workgroup
constexpr int kSlots = 32;                    // query slots per problem (MFMA columns)

// problem index -> (b, kv head, head chunk, stream) and the problem's query slots:
// cross-stream layers: slot = s * gchunk + head-in-chunk (all streams of the token);
// intra-stream layers: one problem per stream, slot = head-in-chunk.
struct DecProblem {
    int b, hk, gc, s;
};

__device__ inline DecProblem dec_problem(const DecGeom &g, int p)
{
    DecProblem r;
    r.s = 0;
    if (g.mode == 0) {
        r.s = p % g.n;
        p /= g.n;
    }
    r.gc = p % g.ngc;
    p /= g.ngc;
    r.hk = p % g.Hkv;
    r.b = p / g.Hkv;
    return r;
}

template <int D>
__global__ __launch_bounds__(kDecWaves * 64, 2) void sfa_decode_partial_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ kc, const bf16 *__restrict__ vc,
    const int32_t *__restrict__ ctx_tokens, float *__restrict__ part, DecGeom g)
{
    constexpr int KS = D / 16, DB = D / 32;
    using T = Tile<D>;
    // LDS: the V tile of each wave (read transposed), reused at the end as the scratch of
    // the merge of the four waves ([wave][slot][D] of O, then [wave][slot] max and sum)
    constexpr int MERGE = kDecWaves * kSlots * D * 4 + 2 * kDecWaves * kSlots * 4;
    static_assert(MERGE >= kDecWaves * T::BYTES, "V tiles must fit in the merge scratch");
    __shared__ __attribute__((aligned(1024))) char smem[MERGE];

    const int chunk = blockIdx.x;
    const DecProblem pr = dec_problem(g, blockIdx.y);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l32 = lane & 31, hi = lane >> 5;

    const int ctx = ctx_tokens[pr.b];
    // cached rows of the problem: cross-stream rows 0 .. (ctx+1)n - 1; intra-stream rows
    // j*n + s for j <= ctx (problem row j)
    const int kvlen = g.mode == 0 ? ctx + 1 : (ctx + 1) * g.n;
    const int pos0 = ctx * g.n;  // expanded position of the new token's stream 0
    const int kb = chunk * kDecChunk + wave * kRows;  // first problem row of my tile

    const size_t cslice = (size_t)g.n * g.Lcap * g.Hkv * D;  // one sequence's cache
    const rsrc_t rk = make_rsrc(kc + pr.b * cslice, (uint32_t)(cslice * 2));
    const rsrc_t rv = make_rsrc(vc + pr.b * cslice, (uint32_t)(cslice * 2));
    const uint32_t kstride = (uint32_t)(g.mode == 0 ? g.n : 1) * g.Hkv * D * 2;
    const uint32_t kbase = (uint32_t)((g.mode == 0 ? pr.s : 0) * g.Hkv + pr.hk) * D * 2;

    // first row any query row sees: 0, or for local layers the window start of stream 0
    const int klo = g.mode == 2 ? max(0, pos0 - g.window + 1) : 0;
    // a chunk without a visible row is skipped whole; the combine reads only the chunks
    // from klo / kDecChunk to the last row
    const int c0 = chunk * kDecChunk;
    if (c0 >= kvlen || c0 + kDecChunk - 1 < klo) return;
    // wave-uniform: my tile holds a visible row (else it is neither loaded nor used)
    const bool any = kb < kvlen && kb + kRows - 1 >= klo;
    // K rows go straight to registers as the A operand of S^T = K Q^T (lane: row l32 of
    // block mb, dims kk*16 + hi*8 ..); V moves to LDS by direct loads for the transposed
    // reads of the P V product.  Rows past kvlen read zeros.
    char *vtile = smem + wave * T::BYTES;
    bf16x8 ka[2][KS];
    if (any) {
        T::load(vtile, rv, kbase, kstride, kb, kvlen, 0, 1, lane);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int row = kb + mb * 32 + l32;
            const uint32_t off = row < kvlen ? kbase + (uint32_t)row * kstride : kOob;
#pragma unroll
            for (int kk = 0; kk < KS; ++kk)
                ka[mb][kk] = __builtin_bit_cast(bf16x8, ld16(rk, off + (kk * 16 + hi * 8) * 2));
        }
    }

    // my query slot (column l32 of the MFMA results): its head and stream
    const int nslot = g.nslot;
    const int slot = l32;
    const int sl_s = g.mode == 0 ? pr.s : slot / g.gchunk;
    const int hq = pr.hk * g.G + pr.gc * g.gchunk + (g.mode == 0 ? slot : slot % g.gchunk);
    const int qp = pos0 + sl_s;  // key coordinate of my query (cross-stream layers)
    bf16x8 qr[KS];
    {
        const size_t qslice = (size_t)g.B * g.n * g.Hq * D;
        const rsrc_t rq = make_rsrc(q, (uint32_t)(qslice * 2));
        const uint32_t off =
            slot < nslot ? (uint32_t)((((size_t)pr.b * g.n + sl_s) * g.Hq + hq) * D * 2) : kOob;
#pragma unroll
        for (int kk = 0; kk < KS; ++kk)
            qr[kk] = __builtin_bit_cast(bf16x8, ld16(rq, off + (kk * 16 + hi * 8) * 2));
    }
    wait_lds_loads();
    __syncthreads();

    // S^T = K Q^T for my 64 rows (two blocks of 32), then the mask: a row is visible if
    // it exists and, for cross-stream layers, lies at or before my query and within
    // the window.  A tile without a visible row contributes an empty partial.
    float mx = -INFINITY, lsum = 0.f;
    f32x16 oacc[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
    if (any) {
        f32x16 sc[2];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            sc[mb] = f32x16{};
#pragma unroll
            for (int kk = 0; kk < KS; ++kk)
                sc[mb] = mfma32(ka[mb][kk], qr[kk], sc[mb]);
        }
        const float c2 = g.scale_log2;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int j = kb + mb * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
                bool vis = j < kvlen && slot < nslot;
                if (g.mode != 0) vis = vis && j <= qp && qp - j < g.window;
                sc[mb][r] = vis ? sc[mb][r] * c2 : -INFINITY;
                mx = fmaxf(mx, sc[mb][r]);
            }
        mx = max_xor32(mx);
        const float me = mx == -INFINITY ? 0.f : mx;  // no visible row: weights exp2(-inf) = 0
        bf16x8 pb[4];
        const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3f803f80u);
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                uint32_t w[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    w[e] = pack_bf16(fast_exp2(sc[mb][h * 8 + 2 * e] - me),
                                     fast_exp2(sc[mb][h * 8 + 2 * e + 1] - me));
                    // the sum adds the bf16 weights that the P V product uses
                    lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[e]), ones,
                                                           lsum, false);
                }
                pb[mb * 2 + h] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
            }
        lsum = sum_xor32(lsum);
        // O^T (dims x slots) = V^T P^T over my 64 rows
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
                oacc[db] = mfma32(T::tr_operand(vtile, db * 32, kk, lane), pb[kk], oacc[db]);
    }

    // merge the four waves: scratch [wave][slot][D] of O, then [wave][slot] max and sum
    __syncthreads();
    float *so = reinterpret_cast<float *>(smem);
    float *sm = so + kDecWaves * kSlots * D;
    float *sl = sm + kDecWaves * kSlots;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int d = db * 32 + 8 * (r >> 2) + 4 * hi + (r & 3);
            so[(wave * kSlots + slot) * D + d] = oacc[db][r];
        }
    if (hi == 0) {
        sm[wave * kSlots + slot] = mx;
        sl[wave * kSlots + slot] = lsum;
    }
    __syncthreads();
    // partials [problem][chunk][slot][D + 2]: O, then max and sum, for the problem's
    // nslot slots only
    float *dst = part + ((size_t)blockIdx.y * g.nchunk + chunk) * nslot * (D + 2);
    for (int e = tid; e < nslot * D; e += kDecWaves * 64) {  // the problem's slots only
        const int sl_i = e / D, d = e % D;
        float m = -INFINITY;
#pragma unroll
        for (int w = 0; w < kDecWaves; ++w) m = fmaxf(m, sm[w * kSlots + sl_i]);
        float o = 0.f, l = 0.f;
        if (m != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kDecWaves; ++w) {
                const float a = fast_exp2(sm[w * kSlots + sl_i] - m);
                o += a * so[(w * kSlots + sl_i) * D + d];
                l += a * sl[w * kSlots + sl_i];
            }
        }
        dst[sl_i * (D + 2) + d] = o;
        if (d == 0) {
            dst[sl_i * (D + 2) + D] = m;
            dst[sl_i * (D + 2) + D + 1] = l;
        }
    }
}

// one workgroup of D threads per query row (b, s, hq): reduce the chunks' partials
template <int D>
__global__ __launch_bounds__(D) void sfa_decode_combine_kernel(const float *__restrict__ part,
                                                               const int32_t *__restrict__ ctx_tokens,
                                                               bf16 *__restrict__ o,
                                                               float *__restrict__ lse, DecGeom g)
{
    const int hq = blockIdx.x % g.Hq;
    const int s = (blockIdx.x / g.Hq) % g.n;
    const int b = blockIdx.x / (g.Hq * g.n);
    const int hk = hq / g.G, gc = (hq % g.G) / g.gchunk, gl = (hq % g.G) % g.gchunk;
    int prob = (b * g.Hkv + hk) * g.ngc + gc;
    int slot;
    if (g.mode == 0) {
        prob = prob * g.n + s;
        slot = gl;
    } else {
        slot = s * g.gchunk + gl;
    }
    // the chunks the partial kernel wrote: those with a row in [klo, kvlen)
    const int ctx = ctx_tokens[b];
    const int kvlen = g.mode == 0 ? ctx + 1 : (ctx + 1) * g.n;
    const int klo = g.mode == 2 ? max(0, ctx * g.n - g.window + 1) : 0;
    const int nc = min(g.nchunk, (kvlen + kDecChunk - 1) / kDecChunk);
    const int cl = klo / kDecChunk;
    const float *src = part + (size_t)prob * g.nchunk * g.nslot * (D + 2) + slot * (D + 2);
    const size_t cstep = (size_t)g.nslot * (D + 2);
    // Every chunk in [cl, nc) has a visible row for some query of the problem, but
    // possibly none for this one (max -inf, sum 0); the query's own key is in one of
    // them, so the largest maximum m is finite.  Two passes, m first and then each
    // chunk's share scaled by exp2(mc - m): no load waits for the previous chunk's
    // arithmetic, as it would with a running maximum.
    float m = -INFINITY;
#pragma unroll 8
    for (int c = cl; c < nc; ++c) m = fmaxf(m, src[c * cstep + D]);
    float acc = 0.f, l = 0.f;
#pragma unroll 8
    for (int c = cl; c < nc; ++c) {
        const float mc = src[c * cstep + D], lc = src[c * cstep + D + 1];
        const float oc = src[c * cstep + threadIdx.x];
        const float w = fast_exp2(mc - m);  // exp2(-inf) = 0
        // a chunk without a visible row is skipped (select, no branch)
        acc = mc == -INFINITY ? acc : __builtin_fmaf(oc, w, acc);
        l = mc == -INFINITY ? l : __builtin_fmaf(lc, w, l);
    }
    const size_t row = ((size_t)b * g.n + s) * g.Hq + hq;
    o[row * D + threadIdx.x] = (bf16)(acc / l);
    if (threadIdx.x == 0) lse[((size_t)b * g.Hq + hq) * g.n + s] = (m + log2f(l)) * 0.6931471805599453f;
}

}  // namespace

DecGeom make_dec_geom(int B, int Lcap, int n, int Hq, int Hkv, int D, int mode, int window,
                      float scale, int max_ctx)
{
    DecGeom g;
    g.B = B; g.Lcap = Lcap; g.n = n; g.Hq = Hq; g.Hkv = Hkv; g.D = D; g.G = Hq / Hkv;
    g.mode = mode;
    g.window = mode == 2 ? window : kNoWindow;
    g.scale_log2 = scale * 1.4426950408889634f;
    // query heads per problem: the largest divisor of G whose slots fit the 32 columns
    const int per_head = mode == 0 ? 1 : n;
    g.gchunk = 1;
    for (int c = g.G; c >= 1; --c)
        if (g.G % c == 0 && c * per_head <= kSlots) {
            g.gchunk = c;
            break;
        }
    g.ngc = g.G / g.gchunk;
    const int64_t rows = mode == 0 ? (int64_t)max_ctx + 1 : ((int64_t)max_ctx + 1) * n;
    g.nchunk = (int)((rows + kDecChunk - 1) / kDecChunk);
    g.problems = B * Hkv * g.ngc * (mode == 0 ? n : 1);
    g.nslot = g.gchunk * per_head;
    return g;
}

size_t decode_workspace_bytes(const DecGeom &g)
{
    return (size_t)g.problems * g.nchunk * g.nslot * (g.D + 2) * sizeof(float);
}

// The scratch array of the allocation-free decode entry point.  In host code its name
// stands for a host-side shadow, not for device memory: kernels get the address that
// hipGetSymbolAddress reports for the current device.
static __device__ __align__(256) char scratch[kDecodeScratchBytes];

hipError_t decode_scratch(void **ptr)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(mu);
    if (addr[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_decode_bf16(const void *q, const void *kc, const void *vc, const int32_t *ctx,
                              void *o, float *lse, const DecGeom &g, void *ws, hipStream_t s)
{
    const bf16 *qq = static_cast<const bf16 *>(q), *kk = static_cast<const bf16 *>(kc),
               *vv = static_cast<const bf16 *>(vc);
    float *part = static_cast<float *>(ws);
    bf16 *oo = static_cast<bf16 *>(o);
    const dim3 grid(g.nchunk, g.problems);
    const int rows = g.B * g.n * g.Hq;
    auto run = [&](auto dk, const char *pname, const char *cname) {
        constexpr int DD = decltype(dk)::value;
        timing_before(pname, s);
        sfa_decode_partial_kernel<DD><<<grid, kDecWaves * 64, 0, s>>>(qq, kk, vv, ctx, part, g);
        hipError_t e = hipGetLastError();
        timing_after(s);
        if (e != hipSuccess) return e;
        timing_before(cname, s);
        sfa_decode_combine_kernel<DD><<<rows, DD, 0, s>>>(part, ctx, oo, lse, g);
        e = hipGetLastError();
        timing_after(s);
        return e;
    };
    if (g.D == 32)
        return run(std::integral_constant<int, 32>{}, "sfa_decode_bf16_d32", "sfa_decode_combine_d32");
    if (g.D == 64)
        return run(std::integral_constant<int, 64>{}, "sfa_decode_bf16_d64", "sfa_decode_combine_d64");
    return run(std::integral_constant<int, 128>{}, "sfa_decode_bf16_d128", "sfa_decode_combine_d128");
}

}  // namespace hd
