// hd_internal.h -- host-side geometry and kernel launchers shared inside libhd.so.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hd {

// One SFA call reduced to independent causal problems over a strided row sequence.
//   MIX  : one problem per (b, hq); rows p = 0 .. N-1            (len = N, rowmul = 1)
//   INTRA: one problem per (b, hq, s); rows p = t*n + s, t < L   (len = L, rowmul = n)
// Row i of a problem is expanded position p = i*rowmul + s, so the intra mask of
// eq. (mask_intra) becomes the ordinary causal mask i' <= i inside the problem and
// the kernels never touch rows of other streams.
struct SfaGeom {
    int B, L, n, Hq, Hkv, D, G;  // G = Hq / Hkv
    int N;                       // n * L
    int mode;                    // 0 intra, 1 mix (full cross-stream), 2 local cross-stream
    int len;                     // rows per problem
    int rowmul;                  // n (intra) or 1 (mix, local)
    int streams;                 // n (intra) or 1 (mix, local): problems per head
    int window;                  // local: row p sees keys p-window+1 .. p; else a huge value
    float scale;                 // softmax scale
    float scale_log2;            // scale * log2(e)
};

constexpr int kNoWindow = 1 << 30;

// Problem geometry of one call.  Local cross-stream layers decompose like the full
// cross-stream layer (one problem per (b, hq) over all N rows) with a window.
inline SfaGeom make_geom(int B, int L, int n, int Hq, int Hkv, int D, int mode, float scale,
                         int window = 0)
{
    SfaGeom g;
    g.B = B; g.L = L; g.n = n; g.Hq = Hq; g.Hkv = Hkv; g.D = D; g.G = Hq / Hkv;
    g.N = n * L;
    g.mode = mode;
    g.len = mode == 0 ? L : n * L;
    g.rowmul = mode == 0 ? n : 1;
    g.streams = mode == 0 ? n : 1;
    g.window = mode == 2 ? window : kNoWindow;
    g.scale = scale;
    g.scale_log2 = scale * 1.4426950408889634f;
    return g;
}

// Launch wrappers record per-kernel timing events when timing is enabled.
void timing_before(const char *name, hipStream_t s);
void timing_after(hipStream_t s);

hipError_t launch_expand_embed(const int32_t *ids, const void *tables, void *out, int B, int L,
                               int n, int64_t V, int Dm, int esize, int32_t *bad,
                               hipStream_t s);

hipError_t launch_fwd_bf16(const void *q, const void *k, const void *v, void *o, float *lse,
                           const SfaGeom &g, hipStream_t s);
hipError_t launch_bwd_bf16(const void *q, const void *k, const void *v, const void *o,
                           const float *lse, const void *dO, void *dq, void *dk, void *dv,
                           const SfaGeom &g, void *ws, hipStream_t s);

hipError_t launch_fwd_f32(const float *q, const float *k, const float *v, float *o, float *lse,
                          const SfaGeom &g, hipStream_t s);
hipError_t launch_bwd_f32(const float *q, const float *k, const float *v, const float *o,
                          const float *lse, const float *dO, float *dq, float *dk, float *dv,
                          const SfaGeom &g, void *ws, hipStream_t s);

// fp32 path: per query row, fp32 [B][Hq][N], delta = rowsum(dO * O) and
// lse2 = lse * log2(e).
hipError_t launch_bwd_preprocess_f32(const float *o, const float *dO, const float *lse,
                                     float *delta, float *lse2, const SfaGeom &g, hipStream_t s);

// Backward workspace, each part 256-byte aligned:
//   per-row statistics, fp32 [B][Hq][N] each: for fp32 those of
//   launch_bwd_preprocess_f32, for bf16 -Delta and -lse/scale (written by the dQ pass);
//   bf16 path only: a transposed copy of k per key/value problem, [problem][D][len_pad]
//   with len_pad = len rounded up to 64 and the positions inside every 16-group in
//   swap23 order (zeros past len).
struct BwdWorkspace {
    size_t delta, lse2, kt, total;
    int len_pad;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline BwdWorkspace bwd_workspace(const SfaGeom &g, int esize)
{
    BwdWorkspace w;
    const size_t rows = (size_t)g.B * g.Hq * g.N;
    w.len_pad = (g.len + 63) / 64 * 64;
    w.delta = 0;
    w.lse2 = align256(rows * 4);
    w.kt = w.lse2 + align256(rows * 4);
    w.total = w.kt;
    if (esize == 2)
        w.total += align256((size_t)g.B * g.Hkv * g.streams * g.D * w.len_pad * 2);
    return w;
}

inline size_t bwd_workspace_bytes(const SfaGeom &g, int esize) { return bwd_workspace(g, esize).total; }

}  // namespace hd
