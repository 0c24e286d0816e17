// decode_internal.h -- host-side geometry and launcher of the parallel-stream decode
// kernels inside libhd.so (sfa_decode_bf16.hip).
#pragma once

#include "hd_internal.h"

namespace hd {

struct DecGeom {
    int B, Lcap, n, Hq, Hkv, D, G;
    int mode;          // 0 intra, 1 full cross-stream, 2 local cross-stream
    int window;        // local layers: positions p - window < p' <= p; else a huge value
    float scale_log2;  // scale * log2(e)
    int gchunk;        // query heads per problem (their query slots fit 32 MFMA columns)
    int ngc;           // head chunks per key/value head, G / gchunk
    int nchunk;        // 256-row chunks of the cache per problem (for the longest context)
    int problems;      // B * Hkv * ngc (* n for intra-stream layers)
    int nslot;         // query slots per problem: gchunk (intra-stream) or n * gchunk
};

DecGeom make_dec_geom(int B, int Lcap, int n, int Hq, int Hkv, int D, int mode, int window,
                      float scale, int max_ctx);
size_t decode_workspace_bytes(const DecGeom &g);
hipError_t launch_decode_bf16(const void *q, const void *kc, const void *vc, const int32_t *ctx,
                              void *o, float *lse, const DecGeom &g, void *ws, hipStream_t s);

// Library-owned scratch for the decode partials of callers that cannot allocate: a
// device array of kDecodeScratchBytes per GPU, held until the process ends and shared
// by every such call on that GPU.  decode_scratch returns its address on the current
// device (looked up once per device).
constexpr size_t kDecodeScratchBytes = (size_t)128 << 20;
hipError_t decode_scratch(void **ptr);

}  // namespace hd
