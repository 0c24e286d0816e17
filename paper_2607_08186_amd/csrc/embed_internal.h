// embed_internal.h -- host-side declarations of the expansion-gradient and cyclic-
// replication launchers inside libhd.so (kernels in embed_bwd.hip).
#pragma once

#include "hd_internal.h"

namespace hd {

// Gradient of the expansion with respect to the tables (see embed_bwd.hip).  Workspace
// byte offsets for M = B*L tokens, each part 256-byte aligned: two (key, token) buffer
// pairs of the radix sort, digit histograms, scan block sums, a few scalars, segment
// indices and segment starts (M + 1 entries).
struct EmbedBwdWorkspace {
    size_t keys_a, vals_a, keys_b, vals_b, hist, sums, scalars, segidx, seg_start, total;
};
constexpr int kEmbedBwdMaxTokens = 2048 * 2048;  // B*L limit of the single-level scans
constexpr int kSmallSortMax = 16384;              // B*L up to which one counting pass sorts
EmbedBwdWorkspace embed_bwd_workspace(int M);
hipError_t launch_embed_bwd(const int32_t *ids, const void *dout, int B, int L, int n, int64_t V,
                            int Dm, int esize, int32_t *uniq, float *drows, int32_t *num_uniq,
                            void *ws, hipStream_t s);
hipError_t launch_embed_grad_scatter_add(const int32_t *uniq, const float *drows,
                                         const int32_t *num_uniq, int rows_cap, int n, int64_t V,
                                         int Dm, float *dtables, hipStream_t s);
hipError_t launch_cyclic_replicate(const void *src, void *dst, int n, int m, int64_t V, int Dm,
                                   int esize, hipStream_t s);

}  // namespace hd
