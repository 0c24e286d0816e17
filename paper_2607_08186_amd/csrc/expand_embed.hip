// expand_embed.hip -- the two ends of the stream layout: the multi-stream token
// expansion, eq. (expansion):
//   out[b][t*n + s][:] = tables[s][ids[b][t]][:]
// and, at the top, the final-stream gather that feeds the loss (further below).
// A pure gather: one workgroup per token copies its n table rows into the n adjacent
// expanded rows (HBM-bound; every byte is read and written once).  The token's n rows
// are one contiguous run of the output, so the workgroup treats them as a flat array
// of 16-byte words (4- or 2-byte words for other row sizes) and each thread issues
// all of its loads before any store, which keeps enough reads in flight per CU.  Loads
// and stores carry the streaming (non-temporal) hint: the stores measured 5% faster
// than cached ones (the output is not read again by this kernel), and the loads 15-20%
// faster on tables that no earlier launch left in the caches, as at the start of a
// training step (when a previous expansion of the same ids left the rows in the
// Infinity Cache, cached loads are about 10% faster).  An id
// outside [0, V) yields zero rows and bumps *bad once.
#include "hd_device.h"

namespace hd {

namespace {

// Unsigned division by a divisor fixed for the launch as a multiply-high, an add and a
// shift (Granlund and Montgomery, "Division by invariant integers using
// multiplication", 1994): with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1
// (which fits 32 bits), x / d = (umulhi(x, m) + x) >> l for every x < 2^31, where the
// add cannot overflow.  Index arithmetic of the copy kernels below uses it in place of
// a division per element (a 64-bit division is dozens of instructions per word).
struct FastDiv {
    uint32_t d, m, l;
};

FastDiv make_fastdiv(uint32_t d)
{
    uint32_t l = 0;
    while (l < 32 && ((uint64_t)1 << l) < d) ++l;
    const uint64_t m = ((uint64_t)1 << 32) * (((uint64_t)1 << l) - d) / d + 1;
    return FastDiv{d, (uint32_t)m, l};
}

__device__ inline uint32_t fdiv(uint32_t x, FastDiv f) { return (__umulhi(x, f.m) + x) >> f.l; }

// words of one token held in flight per thread
constexpr int kExpandUnroll = 8;

template <typename W>
__global__ __launch_bounds__(256) void expand_embed_kernel(const int32_t *__restrict__ ids,
                                                           const W *__restrict__ tables,
                                                           W *__restrict__ out, int n, int64_t V,
                                                           int row_words, FastDiv frw,
                                                           int32_t *__restrict__ bad)
{
    const int64_t bt = blockIdx.x;  // b * L + t
    const int32_t id = ids[bt];
    const bool ok = id >= 0 && (int64_t)id < V;
    if (!ok && bad != nullptr && threadIdx.x == 0) atomicAdd(bad, 1);
    const int total = n * row_words;  // the token's words (the host bounds it below 2^31)
    W *dst = out + bt * (int64_t)total;
    const W *row0 = tables + (ok ? (int64_t)id : 0) * row_words;
    const int64_t table_words = V * (int64_t)row_words;
    for (int base = 0; base < total; base += 256 * kExpandUnroll) {
        W buf[kExpandUnroll];
        if (ok && base + 256 * kExpandUnroll <= total) {
            // a whole chunk (every chunk at the usual row sizes): no per-lane branches,
            // so that the stores wait only for their own loads (behind a branch the
            // compiler waits for every earlier memory operation, stores included)
#pragma unroll
            for (int i = 0; i < kExpandUnroll; ++i) {
                const int w = base + i * 256 + (int)threadIdx.x;
                const int s = (int)fdiv((uint32_t)w, frw);  // stream of word w
                buf[i] = __builtin_nontemporal_load(row0 + s * table_words + (w - s * row_words));
            }
#pragma unroll
            for (int i = 0; i < kExpandUnroll; ++i)
                __builtin_nontemporal_store(buf[i], dst + base + i * 256 + (int)threadIdx.x);
            continue;
        }
#pragma unroll
        for (int i = 0; i < kExpandUnroll; ++i) {
            const int w = base + i * 256 + (int)threadIdx.x;
            buf[i] = W{};
            if (ok && w < total) {
                const int s = (int)fdiv((uint32_t)w, frw);  // stream of word w
                buf[i] = __builtin_nontemporal_load(row0 + s * table_words + (w - s * row_words));
            }
        }
#pragma unroll
        for (int i = 0; i < kExpandUnroll; ++i) {
            const int w = base + i * 256 + (int)threadIdx.x;
            if (w < total) __builtin_nontemporal_store(buf[i], dst + w);
        }
    }
}

}  // namespace

hipError_t launch_expand_embed(const int32_t *ids, const void *tables, void *out, int B, int L,
                               int n, int64_t V, int Dm, int esize, int32_t *bad, hipStream_t s)
{
    const int64_t row_bytes = (int64_t)Dm * esize;
    const dim3 grid((unsigned)((int64_t)B * L));
    timing_before("expand_embed", s);
    if (row_bytes % 16 == 0)
        expand_embed_kernel<u32x4><<<grid, 256, 0, s>>>(
            ids, static_cast<const u32x4 *>(tables), static_cast<u32x4 *>(out), n, V,
            (int)(row_bytes / 16), make_fastdiv((uint32_t)(row_bytes / 16)), bad);
    else if (row_bytes % 4 == 0)
        expand_embed_kernel<uint32_t><<<grid, 256, 0, s>>>(
            ids, static_cast<const uint32_t *>(tables), static_cast<uint32_t *>(out), n, V,
            (int)(row_bytes / 4), make_fastdiv((uint32_t)(row_bytes / 4)), bad);
    else
        expand_embed_kernel<uint16_t><<<grid, 256, 0, s>>>(
            ids, static_cast<const uint16_t *>(tables), static_cast<uint16_t *>(out), n, V,
            (int)(row_bytes / 2), make_fastdiv((uint32_t)(row_bytes / 2)), bad);
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace hd

// Final-stream gather, eq. (hd_loss): the loss reads token i's hidden state at its final
// stream, expanded position i*n + n - 1.  Both directions are flat copies over W-sized
// words of the output (every thread one word), so reads and writes are coalesced and
// every byte moves once.
namespace hd {

namespace {

template <typename W>
__global__ __launch_bounds__(256) void final_gather_kernel(const W *__restrict__ h,
                                                           W *__restrict__ out, int n,
                                                           FastDiv frw, uint32_t words)
{
    const uint32_t w = blockIdx.x * 256u + threadIdx.x;  // words < 2^31 (checked by the caller)
    if (w >= words) return;
    const uint32_t row = fdiv(w, frw);  // b * L + i
    const uint32_t c = w - row * frw.d;
    out[w] = h[((int64_t)row * n + n - 1) * frw.d + c];
}

// adjoint: dh row p = b*n*L + i*n + s holds dout row b*L + i when s = n - 1, else zero
template <typename W>
__global__ __launch_bounds__(256) void final_gather_bwd_kernel(const W *__restrict__ dout,
                                                               W *__restrict__ dh, FastDiv fn,
                                                               FastDiv frw, uint32_t words)
{
    const uint32_t w = blockIdx.x * 256u + threadIdx.x;
    if (w >= words) return;
    const uint32_t p = fdiv(w, frw);
    const uint32_t c = w - p * frw.d;
    const uint32_t tok = fdiv(p, fn);
    dh[w] = p - tok * fn.d == fn.d - 1 ? dout[(int64_t)tok * frw.d + c] : W{};
}

}  // namespace

hipError_t launch_final_gather(const void *h, void *out, int B, int L, int n, int Dm, int esize,
                               bool backward, hipStream_t s)
{
    const int64_t row_bytes = (int64_t)Dm * esize;
    const int64_t rows = (int64_t)B * L * (backward ? n : 1);  // output rows
    auto go = [&](auto word) {
        using W = decltype(word);
        // the caller bounds the output below 2^31 words
        const int64_t rw = row_bytes / (int64_t)sizeof(W), words = rows * rw;
        const dim3 grid((unsigned)((words + 255) / 256));
        if (backward)
            final_gather_bwd_kernel<W><<<grid, 256, 0, s>>>(
                static_cast<const W *>(h), static_cast<W *>(out), make_fastdiv((uint32_t)n),
                make_fastdiv((uint32_t)rw), (uint32_t)words);
        else
            final_gather_kernel<W><<<grid, 256, 0, s>>>(static_cast<const W *>(h),
                                                        static_cast<W *>(out), n,
                                                        make_fastdiv((uint32_t)rw), (uint32_t)words);
    };
    timing_before(backward ? "final_gather_bwd" : "final_gather", s);
    if (row_bytes % 16 == 0) go(u32x4{});
    else if (row_bytes % 4 == 0) go(uint32_t{});
    else go(uint16_t{});
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace hd
