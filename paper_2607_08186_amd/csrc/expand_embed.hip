// expand_embed.hip -- the two ends of the stream layout: the multi-stream token
// expansion, eq. (expansion):
//   out[b][t*n + s][:] = tables[s][ids[b][t]][:]
// and, at the top, the final-stream gather that feeds the loss (further below).
// A pure gather: one workgroup per token copies its n table rows into the n adjacent
// expanded rows (HBM-bound; every byte is read and written once).  The token's n rows
// are one contiguous run of the output, so the workgroup treats them as a flat array
// of 16-byte words (4- or 2-byte words for other row sizes) and each thread issues
// all of its loads before any store, which keeps enough reads in flight per CU; the
// stores carry the streaming (non-temporal) hint, measured 5% faster than cached
// ones (the output is not read again by this kernel).  An id
// outside [0, V) yields zero rows and bumps *bad once.
#include "hd_device.h"

namespace hd {

namespace {

// words of one token held in flight per thread
constexpr int kExpandUnroll = 8;

template <typename W>
__global__ __launch_bounds__(256) void expand_embed_kernel(const int32_t *__restrict__ ids,
                                                           const W *__restrict__ tables,
                                                           W *__restrict__ out, int n, int64_t V,
                                                           int row_words,
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
#pragma unroll
        for (int i = 0; i < kExpandUnroll; ++i) {
            const int w = base + i * 256 + (int)threadIdx.x;
            buf[i] = W{};
            if (ok && w < total) {
                const int s = w / row_words;  // stream of word w
                buf[i] = row0[s * table_words + (w - s * row_words)];
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
        expand_embed_kernel<u32x4><<<grid, 256, 0, s>>>(ids, static_cast<const u32x4 *>(tables),
                                                        static_cast<u32x4 *>(out), n, V,
                                                        (int)(row_bytes / 16), bad);
    else if (row_bytes % 4 == 0)
        expand_embed_kernel<uint32_t><<<grid, 256, 0, s>>>(
            ids, static_cast<const uint32_t *>(tables), static_cast<uint32_t *>(out), n, V,
            (int)(row_bytes / 4), bad);
    else
        expand_embed_kernel<uint16_t><<<grid, 256, 0, s>>>(
            ids, static_cast<const uint16_t *>(tables), static_cast<uint16_t *>(out), n, V,
            (int)(row_bytes / 2), bad);
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
                                                           int64_t row_words, int64_t words)
{
    const int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (w >= words) return;
    const int64_t row = w / row_words;  // b * L + i
    const int64_t c = w - row * row_words;
    out[w] = h[(row * n + n - 1) * row_words + c];
}

// adjoint: dh row p = b*n*L + i*n + s holds dout row b*L + i when s = n - 1, else zero
template <typename W>
__global__ __launch_bounds__(256) void final_gather_bwd_kernel(const W *__restrict__ dout,
                                                               W *__restrict__ dh, int n,
                                                               int64_t row_words, int64_t words)
{
    const int64_t w = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (w >= words) return;
    const int64_t p = w / row_words;
    const int64_t c = w - p * row_words;
    dh[w] = p % n == n - 1 ? dout[(p / n) * row_words + c] : W{};
}

}  // namespace

hipError_t launch_final_gather(const void *h, void *out, int B, int L, int n, int Dm, int esize,
                               bool backward, hipStream_t s)
{
    const int64_t row_bytes = (int64_t)Dm * esize;
    const int64_t rows = (int64_t)B * L * (backward ? n : 1);  // output rows
    auto go = [&](auto word) {
        using W = decltype(word);
        const int64_t rw = row_bytes / (int64_t)sizeof(W), words = rows * rw;
        const dim3 grid((unsigned)((words + 255) / 256));
        if (backward)
            final_gather_bwd_kernel<W><<<grid, 256, 0, s>>>(static_cast<const W *>(h),
                                                            static_cast<W *>(out), n, rw, words);
        else
            final_gather_kernel<W><<<grid, 256, 0, s>>>(static_cast<const W *>(h),
                                                        static_cast<W *>(out), n, rw, words);
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
