// hd_api.cpp -- the C ABI of libhd.so: argument validation, dispatch, diagnostics.
//
// Every entry point validates all arguments on the host before enqueuing anything;
// the kernels then run on the caller's stream.  No allocation, no synchronisation.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/hd.h"
#include "decode_internal.h"
#include "embed_internal.h"
#include "hd_internal.h"

namespace {

thread_local char g_err[512] = "";

hd_status_t fail(hd_status_t st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

hd_status_t hip_status(hipError_t e, const char *what)
{
    if (e == hipSuccess) return HD_OK;
    return fail(HD_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

constexpr int64_t kSliceLimit = (int64_t)1 << 31;  // bytes per batch slice

// Shared shape checks of the SFA entry points.
hd_status_t check_sfa(int B, int L, int n, int Hq, int Hkv, int D, int mode, float scale,
                      int dtype)
{
    if (B <= 0 || L <= 0 || n <= 0 || Hq <= 0 || Hkv <= 0 || D <= 0)
        return fail(HD_ERR_INVALID_ARG, "sizes must be positive (B=%d L=%d n=%d Hq=%d Hkv=%d D=%d)",
                    B, L, n, Hq, Hkv, D);
    if (Hq % Hkv != 0)
        return fail(HD_ERR_INVALID_ARG, "Hq=%d is not a multiple of Hkv=%d", Hq, Hkv);
    if (mode != HD_SFA_INTRA && mode != HD_SFA_MIX && mode != HD_SFA_LOCAL)
        return fail(HD_ERR_INVALID_ARG, "unknown mode %d", mode);
    if (!std::isfinite(scale) || !(scale > 0.f))
        return fail(HD_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", (double)scale);
    if (dtype != HD_DTYPE_BF16 && dtype != HD_DTYPE_F32)
        return fail(HD_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (D != 32 && D != 64 && D != 128)
        return fail(HD_ERR_UNSUPPORTED, "head dim D=%d not supported (32, 64 or 128)", D);
    const int64_t N = (int64_t)n * L;
    const int64_t esize = dtype == HD_DTYPE_BF16 ? 2 : 4;
    if (N > (1 << 30))
        return fail(HD_ERR_INVALID_ARG, "expanded length n*L=%lld too large", (long long)N);
    if (N * Hq * D * esize >= kSliceLimit || (int64_t)Hq * N * 4 >= kSliceLimit)
        return fail(HD_ERR_INVALID_ARG,
                    "per-batch tensor slice of %lld bytes exceeds the 2^31-byte limit",
                    (long long)(N * Hq * D * esize));
    const int64_t len = mode == HD_SFA_INTRA ? L : N;
    const int64_t problems = (int64_t)B * Hq * (mode == HD_SFA_INTRA ? n : 1);
    if (problems * ((len + 63) / 64) >= ((int64_t)1 << 31))
        return fail(HD_ERR_INVALID_ARG, "grid too large");
    return HD_OK;
}

// ------------------------------------------------------------------ timing

struct TimingRecord {
    std::string name;
    hipEvent_t start, stop;
};

std::mutex g_tmu;
bool g_timing = false;
std::string g_tfilter;  // time only kernels whose name starts with this (empty: all)
std::vector<hipEvent_t> g_pool;
std::vector<TimingRecord> g_records;
thread_local int g_open = -1;

hipEvent_t take_event()
{
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

namespace hd {

void timing_before(const char *name, hipStream_t s)
{
    std::lock_guard<std::mutex> lk(g_tmu);
    g_open = -1;
    if (!g_timing || strncmp(name, g_tfilter.c_str(), g_tfilter.size()) != 0) return;
    TimingRecord r{name, take_event(), take_event()};
    if (!r.start || !r.stop) return;
    (void)hipEventRecord(r.start, s);
    g_records.push_back(r);
    g_open = (int)g_records.size() - 1;
}

void timing_after(hipStream_t s)
{
    std::lock_guard<std::mutex> lk(g_tmu);
    if (g_open < 0) return;
    (void)hipEventRecord(g_records[g_open].stop, s);
    g_open = -1;
}

}  // namespace hd

extern "C" {

const char *hd_status_str(hd_status_t s)
{
    switch (s) {
    case HD_OK: return "HD_OK";
    case HD_ERR_INVALID_ARG: return "HD_ERR_INVALID_ARG";
    case HD_ERR_UNSUPPORTED: return "HD_ERR_UNSUPPORTED";
    case HD_ERR_HIP: return "HD_ERR_HIP";
    }
    return "HD_ERR_UNKNOWN";
}

const char *hd_last_error(void) { return g_err; }

hd_status_t hd_expand_embed(const int32_t *ids, const void *tables, void *out, int B, int L,
                            int n, int64_t V, int Dm, hd_dtype_t dtype, int32_t *bad_id_count,
                            hd_stream_t stream)
{
    g_err[0] = 0;
    if (!ids || !tables || !out) return fail(HD_ERR_INVALID_ARG, "null ids, tables or out");
    if (B <= 0 || L <= 0 || n <= 0 || Dm <= 0 || V <= 0)
        return fail(HD_ERR_INVALID_ARG, "sizes must be positive (B=%d L=%d n=%d V=%lld Dm=%d)", B,
                    L, n, (long long)V, Dm);
    if (V > INT32_MAX) return fail(HD_ERR_INVALID_ARG, "V=%lld exceeds int32 ids", (long long)V);
    if (dtype != HD_DTYPE_BF16 && dtype != HD_DTYPE_F32)
        return fail(HD_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    if (!aligned16(tables) || !aligned16(out) || (reinterpret_cast<uintptr_t>(ids) & 3))
        return fail(HD_ERR_INVALID_ARG, "tables/out must be 16-byte aligned, ids 4-byte aligned");
    if (bad_id_count && (reinterpret_cast<uintptr_t>(bad_id_count) & 3))
        return fail(HD_ERR_INVALID_ARG, "bad_id_count must be 4-byte aligned");
    if ((int64_t)B * L >= ((int64_t)1 << 31))
        return fail(HD_ERR_INVALID_ARG, "B*L too large");
    const int esize = dtype == HD_DTYPE_BF16 ? 2 : 4;
    if ((int64_t)n * Dm * esize >= ((int64_t)1 << 31))
        return fail(HD_ERR_INVALID_ARG, "one token's n rows exceed 2^31-1 bytes (n=%d Dm=%d)", n, Dm);
    return hip_status(hd::launch_expand_embed(ids, tables, out, B, L, n, V, Dm, esize,
                                              bad_id_count, (hipStream_t)stream),
                      "hd_expand_embed launch");
}

size_t hd_expand_embed_bwd_workspace_bytes(int B, int L)
{
    if (B <= 0 || L <= 0 || (int64_t)B * L > hd::kEmbedBwdMaxTokens) return 0;
    return hd::embed_bwd_workspace(B * L).total;
}

hd_status_t hd_expand_embed_bwd(const int32_t *ids, const void *dout, int B, int L, int n,
                                int64_t V, int Dm, hd_dtype_t dtype, int32_t *uniq_ids,
                                float *drows, int32_t *num_uniq, void *workspace,
                                size_t workspace_bytes, hd_stream_t stream)
{
    g_err[0] = 0;
    if (!ids || !dout || !uniq_ids || !drows || !num_uniq)
        return fail(HD_ERR_INVALID_ARG, "null ids, dout, uniq_ids, drows or num_uniq");
    if (B <= 0 || L <= 0 || n <= 0 || Dm <= 0 || V <= 0)
        return fail(HD_ERR_INVALID_ARG, "sizes must be positive (B=%d L=%d n=%d V=%lld Dm=%d)", B,
                    L, n, (long long)V, Dm);
    if (V > INT32_MAX) return fail(HD_ERR_INVALID_ARG, "V=%lld exceeds int32 ids", (long long)V);
    if (dtype != HD_DTYPE_BF16 && dtype != HD_DTYPE_F32)
        return fail(HD_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    if ((int64_t)B * L > hd::kEmbedBwdMaxTokens)
        return fail(HD_ERR_INVALID_ARG, "B*L=%lld exceeds %d tokens", (long long)B * L,
                    hd::kEmbedBwdMaxTokens);
    if (!aligned16(dout) || !aligned16(drows) || (reinterpret_cast<uintptr_t>(ids) & 3) ||
        (reinterpret_cast<uintptr_t>(uniq_ids) & 3) || (reinterpret_cast<uintptr_t>(num_uniq) & 3))
        return fail(HD_ERR_INVALID_ARG,
                    "dout/drows must be 16-byte aligned, ids/uniq_ids/num_uniq 4-byte aligned");
    const size_t need = hd::embed_bwd_workspace(B * L).total;
    if (!workspace) return fail(HD_ERR_INVALID_ARG, "null workspace (%zu bytes needed)", need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(HD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
        return fail(HD_ERR_INVALID_ARG, "workspace of %zu bytes is short of %zu", workspace_bytes,
                    need);
    const int esize = dtype == HD_DTYPE_BF16 ? 2 : 4;
    return hip_status(hd::launch_embed_bwd(ids, dout, B, L, n, V, Dm, esize, uniq_ids, drows,
                                           num_uniq, workspace, (hipStream_t)stream),
                      "hd_expand_embed_bwd launch");
}

hd_status_t hd_embed_grad_scatter_add(const int32_t *uniq_ids, const float *drows,
                                      const int32_t *num_uniq, int max_rows, int n, int64_t V,
                                      int Dm, float *dtables, hd_stream_t stream)
{
    g_err[0] = 0;
    if (!uniq_ids || !drows || !num_uniq || !dtables)
        return fail(HD_ERR_INVALID_ARG, "null uniq_ids, drows, num_uniq or dtables");
    if (max_rows <= 0 || n <= 0 || Dm <= 0 || V <= 0 || V > INT32_MAX)
        return fail(HD_ERR_INVALID_ARG, "bad sizes (max_rows=%d n=%d V=%lld Dm=%d)", max_rows, n,
                    (long long)V, Dm);
    if ((reinterpret_cast<uintptr_t>(drows) & 3) || (reinterpret_cast<uintptr_t>(dtables) & 3) ||
        (reinterpret_cast<uintptr_t>(uniq_ids) & 3) || (reinterpret_cast<uintptr_t>(num_uniq) & 3))
        return fail(HD_ERR_INVALID_ARG, "pointers must be 4-byte aligned");
    return hip_status(hd::launch_embed_grad_scatter_add(uniq_ids, drows, num_uniq, max_rows, n, V,
                                                        Dm, dtables, (hipStream_t)stream),
                      "hd_embed_grad_scatter_add launch");
}

hd_status_t hd_cyclic_replicate(const void *src, void *dst, int n, int m, int64_t V, int Dm,
                                hd_dtype_t dtype, hd_stream_t stream)
{
    g_err[0] = 0;
    if (!src || !dst) return fail(HD_ERR_INVALID_ARG, "null src or dst");
    if (n <= 0 || m < n || m % n != 0 || m > 65535)
        return fail(HD_ERR_INVALID_ARG, "m=%d must be a multiple of n=%d (at most 65535)", m, n);
    if (V <= 0 || Dm <= 0) return fail(HD_ERR_INVALID_ARG, "V and Dm must be positive");
    if (dtype != HD_DTYPE_BF16 && dtype != HD_DTYPE_F32)
        return fail(HD_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    if (!aligned16(src) || !aligned16(dst))
        return fail(HD_ERR_INVALID_ARG, "src/dst must be 16-byte aligned");
    const int esize = dtype == HD_DTYPE_BF16 ? 2 : 4;
    const uintptr_t a = reinterpret_cast<uintptr_t>(src), b = reinterpret_cast<uintptr_t>(dst);
    const uintptr_t table = (uintptr_t)V * Dm * esize;
    if (src != dst && a < b + (uintptr_t)m * table && b < a + (uintptr_t)n * table)
        return fail(HD_ERR_INVALID_ARG, "src and dst overlap without being the same buffer");
    return hip_status(hd::launch_cyclic_replicate(src, dst, n, m, V, Dm, esize, (hipStream_t)stream),
                      "hd_cyclic_replicate launch");
}

namespace {

hd_status_t final_gather(const void *src, void *dst, int B, int L, int n, int Dm,
                         hd_dtype_t dtype, bool backward, hd_stream_t stream, const char *what)
{
    g_err[0] = 0;
    if (!src || !dst) return fail(HD_ERR_INVALID_ARG, "%s: null pointer", what);
    if (B <= 0 || L <= 0 || n <= 0 || Dm <= 0)
        return fail(HD_ERR_INVALID_ARG, "%s: sizes must be positive (B=%d L=%d n=%d Dm=%d)", what,
                    B, L, n, Dm);
    if (dtype != HD_DTYPE_BF16 && dtype != HD_DTYPE_F32)
        return fail(HD_ERR_INVALID_ARG, "%s: unknown dtype %d", what, (int)dtype);
    if (!aligned16(src) || !aligned16(dst))
        return fail(HD_ERR_INVALID_ARG, "%s: pointers must be 16-byte aligned", what);
    const int esize = dtype == HD_DTYPE_BF16 ? 2 : 4;
    const int64_t row = (int64_t)Dm * esize;
    const int64_t word = row % 16 == 0 ? 16 : row % 4 == 0 ? 4 : 2;
    const int64_t big = (int64_t)B * n * L * row, small = (int64_t)B * L * row;  // h, out bytes
    if ((int64_t)B * n * L > INT32_MAX || (backward ? big : small) / word >= ((int64_t)1 << 31))
        return fail(HD_ERR_INVALID_ARG, "%s: too large (B=%d L=%d n=%d Dm=%d)", what, B, L, n, Dm);
    const uintptr_t a = reinterpret_cast<uintptr_t>(src), b = reinterpret_cast<uintptr_t>(dst);
    const uintptr_t alen = (uintptr_t)(backward ? small : big), blen = (uintptr_t)(backward ? big : small);
    if (a < b + blen && b < a + alen) return fail(HD_ERR_INVALID_ARG, "%s: buffers overlap", what);
    return hip_status(hd::launch_final_gather(src, dst, B, L, n, Dm, esize, backward,
                                              (hipStream_t)stream),
                      what);
}

}  // namespace

hd_status_t hd_final_stream_gather(const void *h, void *out, int B, int L, int n, int Dm,
                                   hd_dtype_t dtype, hd_stream_t stream)
{
    return final_gather(h, out, B, L, n, Dm, dtype, false, stream, "hd_final_stream_gather");
}

hd_status_t hd_final_stream_gather_bwd(const void *dout, void *dh, int B, int L, int n, int Dm,
                                       hd_dtype_t dtype, hd_stream_t stream)
{
    return final_gather(dout, dh, B, L, n, Dm, dtype, true, stream, "hd_final_stream_gather_bwd");
}

namespace {

// Final-stream layers (queries at the final stream of each token only): bf16 kernels,
// and at most 63 streams (the forward's eight waves then all reach the last key tile
// of their 256-row block).
hd_status_t check_final(int n, hd_dtype_t dtype)
{
    if (dtype != HD_DTYPE_BF16)
        return fail(HD_ERR_UNSUPPORTED, "final-stream layers are implemented for bf16 only");
    if (n > 63) return fail(HD_ERR_UNSUPPORTED, "final-stream layers support n <= 63 (got %d)", n);
    return HD_OK;
}

hd::SfaGeom geom(int B, int L, int n, int Hq, int Hkv, int D, int mode, float scale, int window,
                 bool final_q)
{
    return final_q ? hd::make_geom_final(B, L, n, Hq, Hkv, D, mode, scale, window)
                   : hd::make_geom(B, L, n, Hq, Hkv, D, mode, scale, window);
}

hd_status_t sfa_fwd(const void *q, const void *k, const void *v, void *o, float *lse, int B, int L,
                    int n, int Hq, int Hkv, int D, int mode, int window, float scale,
                    hd_dtype_t dtype, hd_stream_t stream, bool final_q = false)
{
    if (!q || !k || !v || !o || !lse) return fail(HD_ERR_INVALID_ARG, "null tensor pointer");
    hd_status_t st = check_sfa(B, L, n, Hq, Hkv, D, mode, scale, dtype);
    if (st != HD_OK) return st;
    if (final_q && (st = check_final(n, dtype)) != HD_OK) return st;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse))
        return fail(HD_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
    const hd::SfaGeom g = geom(B, L, n, Hq, Hkv, D, mode, scale, window, final_q);
    hipError_t e;
    if (dtype == HD_DTYPE_BF16)
        e = hd::launch_fwd_bf16(q, k, v, o, lse, g, (hipStream_t)stream);
    else
        e = hd::launch_fwd_f32(static_cast<const float *>(q), static_cast<const float *>(k),
                               static_cast<const float *>(v), static_cast<float *>(o), lse, g,
                               (hipStream_t)stream);
    return hip_status(e, "sfa forward launch");
}

}  // namespace

hd_status_t hd_sfa_fwd(const void *q, const void *k, const void *v, void *o, float *lse, int B,
                       int L, int n, int Hq, int Hkv, int D, hd_sfa_mode_t mode, float scale,
                       hd_dtype_t dtype, hd_stream_t stream)
{
    g_err[0] = 0;
    if (mode == HD_SFA_LOCAL)
        return fail(HD_ERR_INVALID_ARG, "local layers take a window: use hd_sfa_fwd_local");
    return sfa_fwd(q, k, v, o, lse, B, L, n, Hq, Hkv, D, mode, 0, scale, dtype, stream);
}

hd_status_t hd_sfa_fwd_local(const void *q, const void *k, const void *v, void *o, float *lse,
                             int B, int L, int n, int Hq, int Hkv, int D, int window, float scale,
                             hd_dtype_t dtype, hd_stream_t stream)
{
    g_err[0] = 0;
    if (window < 1) return fail(HD_ERR_INVALID_ARG, "window must be >= 1 (got %d)", window);
    return sfa_fwd(q, k, v, o, lse, B, L, n, Hq, Hkv, D, HD_SFA_LOCAL, window, scale, dtype,
                   stream);
}

}  // extern "C"

namespace {

// Workspace of a backward call: the one-pass size, or (smallest) the least it accepts;
// 0 for arguments the call would reject.  The check leaves hd_last_error untouched.
size_t bwd_ws_size(int B, int L, int n, int Hq, int Hkv, int D, int mode, int window,
                   bool final_q, hd_dtype_t dtype, bool smallest)
{
    char saved[sizeof g_err];
    memcpy(saved, g_err, sizeof g_err);
    hd_status_t st = check_sfa(B, L, n, Hq, Hkv, D, mode, 1.0f, dtype);
    if (st == HD_OK && final_q) st = check_final(n, dtype);
    memcpy(g_err, saved, sizeof g_err);
    if (st != HD_OK) return 0;
    const hd::SfaGeom g = geom(B, L, n, Hq, Hkv, D, mode, 1.0f, window, final_q);
    const int esize = dtype == HD_DTYPE_BF16 ? 2 : 4;
    return smallest ? hd::bwd_workspace_min_bytes(g, esize) : hd::bwd_workspace_bytes(g, esize);
}

}  // namespace

extern "C" {

// without a window a local layer gets the size of the full causal layer, which bounds
// that of every window
size_t hd_sfa_bwd_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                  hd_sfa_mode_t mode, hd_dtype_t dtype)
{
    return bwd_ws_size(B, L, n, Hq, Hkv, D, mode, hd::kNoWindow, false, dtype, false);
}

size_t hd_sfa_bwd_min_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                      hd_sfa_mode_t mode, hd_dtype_t dtype)
{
    return bwd_ws_size(B, L, n, Hq, Hkv, D, mode, hd::kNoWindow, false, dtype, true);
}

size_t hd_sfa_bwd_local_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D, int window,
                                        hd_dtype_t dtype)
{
    if (window < 1) return 0;
    return bwd_ws_size(B, L, n, Hq, Hkv, D, HD_SFA_LOCAL, window, false, dtype, false);
}

size_t hd_sfa_bwd_local_min_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                            int window, hd_dtype_t dtype)
{
    if (window < 1) return 0;
    return bwd_ws_size(B, L, n, Hq, Hkv, D, HD_SFA_LOCAL, window, false, dtype, true);
}

namespace {

hd_status_t sfa_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
                    const void *dO, void *dq, void *dk, void *dv, int B, int L, int n, int Hq,
                    int Hkv, int D, int mode, int window, float scale, hd_dtype_t dtype,
                    void *workspace, size_t workspace_bytes, hd_stream_t stream,
                    bool final_q = false)
{
    if (!q || !k || !v || !o || !lse || !dO || !dq || !dk || !dv)
        return fail(HD_ERR_INVALID_ARG, "null tensor pointer");
    hd_status_t st = check_sfa(B, L, n, Hq, Hkv, D, mode, scale, dtype);
    if (st != HD_OK) return st;
    if (final_q && (st = check_final(n, dtype)) != HD_OK) return st;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse) ||
        !aligned16(dO) || !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
        return fail(HD_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
    const hd::SfaGeom g = geom(B, L, n, Hq, Hkv, D, mode, scale, window, final_q);
    // the bf16 path runs in query bands when the workspace is below the one-pass size
    const size_t need = hd::bwd_workspace_min_bytes(g, dtype == HD_DTYPE_BF16 ? 2 : 4);
    if (!workspace) return fail(HD_ERR_INVALID_ARG, "null workspace (%zu bytes needed)", need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(HD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
        return fail(HD_ERR_INVALID_ARG, "workspace of %zu bytes is short of %zu", workspace_bytes,
                    need);
    hipError_t e;
    if (dtype == HD_DTYPE_BF16)
        e = hd::launch_bwd_bf16(q, k, v, o, lse, dO, dq, dk, dv, g, workspace, workspace_bytes,
                                (hipStream_t)stream);
    else
        e = hd::launch_bwd_f32(static_cast<const float *>(q), static_cast<const float *>(k),
                               static_cast<const float *>(v), static_cast<const float *>(o), lse,
                               static_cast<const float *>(dO), static_cast<float *>(dq),
                               static_cast<float *>(dk), static_cast<float *>(dv), g, workspace,
                               (hipStream_t)stream);
    return hip_status(e, "sfa backward launch");
}

}  // namespace

hd_status_t hd_sfa_bwd(const void *q, const void *k, const void *v, const void *o,
                       const float *lse, const void *dO, void *dq, void *dk, void *dv, int B,
                       int L, int n, int Hq, int Hkv, int D, hd_sfa_mode_t mode, float scale,
                       hd_dtype_t dtype, void *workspace, size_t workspace_bytes,
                       hd_stream_t stream)
{
    g_err[0] = 0;
    if (mode == HD_SFA_LOCAL)
        return fail(HD_ERR_INVALID_ARG, "local layers take a window: use hd_sfa_bwd_local");
    return sfa_bwd(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, mode, 0, scale, dtype,
                   workspace, workspace_bytes, stream);
}

hd_status_t hd_sfa_bwd_local(const void *q, const void *k, const void *v, const void *o,
                             const float *lse, const void *dO, void *dq, void *dk, void *dv,
                             int B, int L, int n, int Hq, int Hkv, int D, int window, float scale,
                             hd_dtype_t dtype, void *workspace, size_t workspace_bytes,
                             hd_stream_t stream)
{
    g_err[0] = 0;
    if (window < 1) return fail(HD_ERR_INVALID_ARG, "window must be >= 1 (got %d)", window);
    return sfa_bwd(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D, HD_SFA_LOCAL, window,
                   scale, dtype, workspace, workspace_bytes, stream);
}

hd_status_t hd_sfa_fwd_final(const void *q, const void *k, const void *v, void *o, float *lse,
                             int B, int L, int n, int Hq, int Hkv, int D, int window, float scale,
                             hd_dtype_t dtype, hd_stream_t stream)
{
    g_err[0] = 0;
    if (window < 0) return fail(HD_ERR_INVALID_ARG, "window must be >= 0 (got %d)", window);
    return sfa_fwd(q, k, v, o, lse, B, L, n, Hq, Hkv, D, window ? HD_SFA_LOCAL : HD_SFA_MIX,
                   window, scale, dtype, stream, true);
}

size_t hd_sfa_bwd_final_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D, int window,
                                        hd_dtype_t dtype)
{
    if (window < 0) return 0;
    return bwd_ws_size(B, L, n, Hq, Hkv, D, window ? HD_SFA_LOCAL : HD_SFA_MIX, window, true,
                       dtype, false);
}

size_t hd_sfa_bwd_final_min_workspace_bytes(int B, int L, int n, int Hq, int Hkv, int D,
                                            int window, hd_dtype_t dtype)
{
    if (window < 0) return 0;
    return bwd_ws_size(B, L, n, Hq, Hkv, D, window ? HD_SFA_LOCAL : HD_SFA_MIX, window, true,
                       dtype, true);
}

hd_status_t hd_sfa_bwd_final(const void *q, const void *k, const void *v, const void *o,
                             const float *lse, const void *dO, void *dq, void *dk, void *dv,
                             int B, int L, int n, int Hq, int Hkv, int D, int window, float scale,
                             hd_dtype_t dtype, void *workspace, size_t workspace_bytes,
                             hd_stream_t stream)
{
    g_err[0] = 0;
    if (window < 0) return fail(HD_ERR_INVALID_ARG, "window must be >= 0 (got %d)", window);
    return sfa_bwd(q, k, v, o, lse, dO, dq, dk, dv, B, L, n, Hq, Hkv, D,
                   window ? HD_SFA_LOCAL : HD_SFA_MIX, window, scale, dtype, workspace,
                   workspace_bytes, stream, true);
}

namespace {

hd_status_t check_decode(int B, int Lcap, int n, int Hq, int Hkv, int D, int mode, int window,
                         int max_ctx, hd_dtype_t dtype)
{
    if (B <= 0 || Lcap <= 0 || n <= 0 || Hq <= 0 || Hkv <= 0 || D <= 0)
        return fail(HD_ERR_INVALID_ARG, "sizes must be positive (B=%d Lcap=%d n=%d Hq=%d Hkv=%d D=%d)",
                    B, Lcap, n, Hq, Hkv, D);
    if (Hq % Hkv != 0) return fail(HD_ERR_INVALID_ARG, "Hq=%d is not a multiple of Hkv=%d", Hq, Hkv);
    if (mode != HD_SFA_INTRA && mode != HD_SFA_MIX && mode != HD_SFA_LOCAL)
        return fail(HD_ERR_INVALID_ARG, "unknown mode %d", mode);
    if (mode == HD_SFA_LOCAL && window < 1)
        return fail(HD_ERR_INVALID_ARG, "local layers need window >= 1 (got %d)", window);
    if (max_ctx < 0 || max_ctx >= Lcap)
        return fail(HD_ERR_INVALID_ARG, "max_ctx_tokens=%d must lie in [0, Lcap-1=%d]", max_ctx,
                    Lcap - 1);
    if (dtype != HD_DTYPE_BF16 && dtype != HD_DTYPE_F32)
        return fail(HD_ERR_INVALID_ARG, "unknown dtype %d", (int)dtype);
    if (dtype != HD_DTYPE_BF16) return fail(HD_ERR_UNSUPPORTED, "decode is implemented for bf16 only");
    if (D != 32 && D != 64 && D != 128)
        return fail(HD_ERR_UNSUPPORTED, "head dim D=%d not supported (32, 64 or 128)", D);
    if ((int64_t)n * Lcap * Hkv * D * 2 >= kSliceLimit || (int64_t)B * n * Hq * D * 2 >= kSliceLimit)
        return fail(HD_ERR_INVALID_ARG, "a sequence's cache or the query tensor exceeds 2^31 bytes");
    const hd::DecGeom g = hd::make_dec_geom(B, Lcap, n, Hq, Hkv, D, mode, window, 1.f, max_ctx);
    if (g.problems > 65535) return fail(HD_ERR_INVALID_ARG, "too many decode problems (%d)", g.problems);
    return HD_OK;
}

}  // namespace

size_t hd_sfa_decode_workspace_bytes(int B, int Lcap, int n, int Hq, int Hkv, int D,
                                     hd_sfa_mode_t mode, int window, int max_ctx_tokens)
{
    char saved[sizeof g_err];
    memcpy(saved, g_err, sizeof g_err);
    hd_status_t st = check_decode(B, Lcap, n, Hq, Hkv, D, mode, window, max_ctx_tokens,
                                  HD_DTYPE_BF16);
    memcpy(g_err, saved, sizeof g_err);
    if (st != HD_OK) return 0;
    return hd::decode_workspace_bytes(
        hd::make_dec_geom(B, Lcap, n, Hq, Hkv, D, mode, window, 1.f, max_ctx_tokens));
}

hd_status_t hd_sfa_decode(const void *q, const void *k_cache, const void *v_cache,
                          const int32_t *ctx_tokens, int max_ctx_tokens, void *o, float *lse,
                          int B, int Lcap, int n, int Hq, int Hkv, int D, hd_sfa_mode_t mode,
                          int window, float scale, hd_dtype_t dtype, void *workspace,
                          size_t workspace_bytes, hd_stream_t stream)
{
    g_err[0] = 0;
    if (!q || !k_cache || !v_cache || !ctx_tokens || !o || !lse)
        return fail(HD_ERR_INVALID_ARG, "null pointer");
    hd_status_t st = check_decode(B, Lcap, n, Hq, Hkv, D, mode, window, max_ctx_tokens, dtype);
    if (st != HD_OK) return st;
    if (!std::isfinite(scale) || !(scale > 0.f))
        return fail(HD_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", (double)scale);
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o) ||
        !aligned16(lse) || (reinterpret_cast<uintptr_t>(ctx_tokens) & 3))
        return fail(HD_ERR_INVALID_ARG, "tensors must be 16-byte aligned, ctx_tokens 4-byte aligned");
    const hd::DecGeom g = hd::make_dec_geom(B, Lcap, n, Hq, Hkv, D, mode, window, scale,
                                            max_ctx_tokens);
    const size_t need = hd::decode_workspace_bytes(g);
    if (!workspace) return fail(HD_ERR_INVALID_ARG, "null workspace (%zu bytes needed)", need);
    if (reinterpret_cast<uintptr_t>(workspace) & 255)
        return fail(HD_ERR_INVALID_ARG, "workspace must be 256-byte aligned");
    if (workspace_bytes < need)
        return fail(HD_ERR_INVALID_ARG, "workspace of %zu bytes is short of %zu", workspace_bytes,
                    need);
    return hip_status(hd::launch_decode_bf16(q, k_cache, v_cache, ctx_tokens, o, lse, g, workspace,
                                             (hipStream_t)stream),
                      "hd_sfa_decode launch");
}

hd_status_t hd_sfa_decode_noalloc(const void *q, const void *k_cache, const void *v_cache,
                                  const int32_t *ctx_tokens, int max_ctx_tokens, void *o,
                                  float *lse, int B, int Lcap, int n, int Hq, int Hkv, int D,
                                  hd_sfa_mode_t mode, int window, float scale, hd_dtype_t dtype,
                                  hd_stream_t stream)
{
    g_err[0] = 0;
    if (!q || !k_cache || !v_cache || !ctx_tokens || !o || !lse)
        return fail(HD_ERR_INVALID_ARG, "null pointer");
    hd_status_t st = check_decode(B, Lcap, n, Hq, Hkv, D, mode, window, max_ctx_tokens, dtype);
    if (st != HD_OK) return st;
    if (!std::isfinite(scale) || !(scale > 0.f))
        return fail(HD_ERR_INVALID_ARG, "scale must be finite and > 0 (got %g)", (double)scale);
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o) ||
        !aligned16(lse) || (reinterpret_cast<uintptr_t>(ctx_tokens) & 3))
        return fail(HD_ERR_INVALID_ARG, "tensors must be 16-byte aligned, ctx_tokens 4-byte aligned");
    const hd::DecGeom g = hd::make_dec_geom(B, Lcap, n, Hq, Hkv, D, mode, window, scale,
                                            max_ctx_tokens);
    const size_t need = hd::decode_workspace_bytes(g);
    if (need > hd::kDecodeScratchBytes)
        return fail(HD_ERR_INVALID_ARG,
                    "these sizes need %zu bytes of decode scratch, more than the %zu bytes the "
                    "library holds per GPU; call hd_sfa_decode with a workspace instead",
                    need, hd::kDecodeScratchBytes);
    void *scratch = nullptr;
    hd_status_t sst = hip_status(hd::decode_scratch(&scratch), "hd_sfa_decode_noalloc scratch");
    if (sst != HD_OK) return sst;
    return hip_status(hd::launch_decode_bf16(q, k_cache, v_cache, ctx_tokens, o, lse, g, scratch,
                                             (hipStream_t)stream),
                      "hd_sfa_decode_noalloc launch");
}

size_t hd_sfa_decode_noalloc_max_bytes(void) { return hd::kDecodeScratchBytes; }

hd_status_t hd_timing_enable(int enable)
{
    std::lock_guard<std::mutex> lk(g_tmu);
    g_timing = enable != 0;
    return HD_OK;
}

hd_status_t hd_timing_filter(const char *prefix)
{
    std::lock_guard<std::mutex> lk(g_tmu);
    g_tfilter = prefix ? prefix : "";
    return HD_OK;
}

int hd_timing_collect(hd_kernel_time_t *out, int max)
{
    std::vector<TimingRecord> recs;
    {
        std::lock_guard<std::mutex> lk(g_tmu);
        recs.swap(g_records);
    }
    std::map<std::string, std::pair<int, double>> acc;
    std::vector<std::string> order;
    bool ok = true;
    for (auto &r : recs) {
        float ms = 0.f;
        if (hipEventSynchronize(r.stop) != hipSuccess ||
            hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
            ok = false;
            continue;
        }
        auto it = acc.find(r.name);
        if (it == acc.end()) {
            order.push_back(r.name);
            acc[r.name] = {1, (double)ms};
        } else {
            it->second.first += 1;
            it->second.second += ms;
        }
    }
    {
        std::lock_guard<std::mutex> lk(g_tmu);
        for (auto &r : recs) {
            g_pool.push_back(r.start);
            g_pool.push_back(r.stop);
        }
    }
    if (!ok) {
        fail(HD_ERR_HIP, "hd_timing_collect: event query failed");
        return -1;
    }
    int nout = 0;
    for (auto &name : order) {
        if (nout >= max || !out) break;
        hd_kernel_time_t &t = out[nout++];
        memset(&t, 0, sizeof t);
        strncpy(t.name, name.c_str(), sizeof t.name - 1);
        t.launches = acc[name].first;
        t.total_ms = acc[name].second;
    }
    return nout;
}

}  // extern "C"
