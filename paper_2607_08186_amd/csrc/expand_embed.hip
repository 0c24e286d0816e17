// expand_embed.hip -- multi-stream token expansion, eq. (expansion):
//   out[b][t*n + s][:] = tables[s][ids[b][t]][:]
// A pure gather: one workgroup per token copies its n table rows into the n adjacent
// expanded rows with 16-byte vector loads and stores (HBM-bound; every byte is read
// and written once).  An id outside [0, V) yields zero rows and bumps *bad once.
#include "hd_device.h"

namespace hd {

namespace {

template <typename W>
__global__ __launch_bounds__(256) void expand_embed_kernel(const int32_t *__restrict__ ids,
                                                           const W *__restrict__ tables,
                                                           W *__restrict__ out, int L, int n,
                                                           int64_t V, int row_words,
                                                           int32_t *__restrict__ bad)
{
    const int64_t bt = blockIdx.x;  // b * L + t
    const int32_t id = ids[bt];
    const bool ok = id >= 0 && (int64_t)id < V;
    if (!ok && bad != nullptr && threadIdx.x == 0) atomicAdd(bad, 1);
    const int64_t b = bt / L, t = bt % L;
    for (int s = 0; s < n; ++s) {
        W *dst = out + ((b * L + t) * n + s) * (int64_t)row_words;
        const W *src = tables + ((int64_t)s * V + (ok ? id : 0)) * (int64_t)row_words;
        for (int w = threadIdx.x; w < row_words; w += blockDim.x) dst[w] = ok ? src[w] : W{};
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
                                                        static_cast<u32x4 *>(out), L, n, V,
                                                        (int)(row_bytes / 16), bad);
    else if (row_bytes % 4 == 0)
        expand_embed_kernel<uint32_t><<<grid, 256, 0, s>>>(
            ids, static_cast<const uint32_t *>(tables), static_cast<uint32_t *>(out), L, n, V,
            (int)(row_bytes / 4), bad);
    else
        expand_embed_kernel<uint16_t><<<grid, 256, 0, s>>>(
            ids, static_cast<const uint16_t *>(tables), static_cast<uint16_t *>(out), L, n, V,
            (int)(row_bytes / 2), bad);
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace hd
