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
    int len;                     // key rows per problem
    int rowmul;                  // n (intra) or 1 (mix, local)
    int streams;                 // n (intra) or 1 (mix, local): problems per head
    int window;                  // local: row p sees keys p-window+1 .. p; else a huge value
    float scale;                 // softmax scale
    float scale_log2;            // scale * log2(e)
    // Query side.  Query row i of a problem sits at key coordinate P(i) = i*qpmul + qpoff
    // for the mask (key j visible iff j <= P(i) and P(i) - j < window).  Every layer
    // but the final-stream one has one query row per key row: P(i) = i.
    int qlen;                    // query rows per problem
    int qN;                      // rows of q, o, dO, dq per batch ([B][qN][Hq][D]); lse [B][Hq][qN]
    int qrowmul;                 // row stride of q, o, dO, dq in units of Hq*D
    int qpmul, qpoff;
    bool strided_waves;          // forward: wave w of a 256-row block takes rows w, w+8, ...
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
    g.qlen = g.len;
    g.qN = g.N;
    g.qrowmul = g.rowmul;
    g.qpmul = 1;
    g.qpoff = 0;
    g.strided_waves = false;
    return g;
}

// Final-stream layer (full cross-stream mode 1 or local mode 2): queries only at the
// final stream of each token, q [B][L][Hq][D] with row t at expanded position
// t*n + n - 1, keys and values over all N expanded rows.
inline SfaGeom make_geom_final(int B, int L, int n, int Hq, int Hkv, int D, int mode, float scale,
                               int window = 0)
{
    SfaGeom g = make_geom(B, L, n, Hq, Hkv, D, mode, scale, window);
    g.qlen = L;
    g.qN = L;
    g.qrowmul = 1;
    g.qpmul = n;
    g.qpoff = n - 1;
    g.strided_waves = true;
    return g;
}

// key coordinate of query row i
__host__ __device__ inline int qpos(const SfaGeom &g, int i) { return i * g.qpmul + g.qpoff; }

// Launch wrappers record per-kernel timing events when timing is enabled.
void timing_before(const char *name, hipStream_t s);
void timing_after(hipStream_t s);

hipError_t launch_expand_embed(const int32_t *ids, const void *tables, void *out, int B, int L,
                               int n, int64_t V, int Dm, int esize, int32_t *bad,
                               hipStream_t s);
// final-stream gather (backward: its adjoint, dh written in full)
hipError_t launch_final_gather(const void *h, void *out, int B, int L, int n, int Dm, int esize,
                               bool backward, hipStream_t s);

hipError_t launch_fwd_bf16(const void *q, const void *k, const void *v, void *o, float *lse,
                           const SfaGeom &g, hipStream_t s);
// ws_bytes >= bwd_workspace_min_bytes(g, 2); below bwd_workspace_bytes(g, 2) the
// query rows are processed in bands (see QBand)
hipError_t launch_bwd_bf16(const void *q, const void *k, const void *v, const void *o,
                           const float *lse, const void *dO, void *dq, void *dk, void *dv,
                           const SfaGeom &g, void *ws, size_t ws_bytes, hipStream_t s);

hipError_t launch_fwd_f32(const float *q, const float *k, const float *v, float *o, float *lse,
                          const SfaGeom &g, hipStream_t s);
hipError_t launch_bwd_f32(const float *q, const float *k, const float *v, const float *o,
                          const float *lse, const float *dO, float *dq, float *dk, float *dv,
                          const SfaGeom &g, void *ws, hipStream_t s);

// fp32 path: per query row, fp32 [B][Hq][N], delta = rowsum(dO * O) and
// lse2 = lse * log2(e).
hipError_t launch_bwd_preprocess_f32(const float *o, const float *dO, const float *lse,
                                     float *delta, float *lse2, const SfaGeom &g, hipStream_t s);

// dS tiles of the bf16 backward.  The dK/dV pass stores dS = P (dP - Delta), rounded
// to bf16 (the precision its own dK MFMA uses), and the dQ pass reads it back, so dQ
// costs one product instead of a recomputation of S and dP.  A tile covers 64 query
// rows x 128 keys of one causal problem (query tile qt, key tile kt); its 16 KB are
// laid out [query half (2)][key (128)][32 queries], i.e. for query row r (0..63) and
// key c (0..127) of the tile the element sits at ((r >> 5) * 128 + c) * 32 +
// ds_query_pos(r & 31).  Within a key's 32 queries the order is the one in which an
// MFMA result holds them (lane half h, register r: query 8 (r / 4) + 4 h + r % 4), so
// the dK/dV pass stores each lane's 16 values as they are.
// Only tiles holding a visible pair are stored, per problem in query-tile order:
//   causal (no window, or window >= len): query tile qt holds key tiles 0 .. qt/2,
//     so its first tile is m(m+1) (qt = 2m) or (m+1)^2 (qt = 2m+1);
//   local (window < len): key tiles kt_lo(qt) .. qt/2, at most `band` of them, each
//     query tile owning `band` slots.
// position of query q (0..31) inside a key's 32 dS values, and its inverse
__host__ __device__ inline int ds_query_pos(int q) { return ((q >> 2) & 1) * 16 + (q >> 3) * 4 + (q & 3); }
__host__ __device__ inline int ds_query_at(int pos) { return ((pos & 15) >> 2) * 8 + (pos >> 4) * 4 + (pos & 3); }

constexpr int kDsRows = 64;                      // query rows per dS tile
constexpr int kDsKeys = 128;                     // keys per dS tile
constexpr int kDsTileBytes = kDsRows * kDsKeys * 2;

// index of tile (qt, kt) inside its problem; kt_lo = ds_kt_lo(g, qt)
__host__ __device__ inline int64_t ds_tile_index(int band, int kt_lo, int qt, int kt)
{
    if (band == 0) {
        const int64_t m = qt >> 1;
        return ((qt & 1) ? (m + 1) * (m + 1) : m * (m + 1)) + kt;
    }
    return (int64_t)qt * band + (kt - kt_lo);
}

// Slots per query tile, or 0 for triangular packing.  Layers with one query per key
// (P(i) = i) pack triangularly without a window (or one >= len) and whenever a band
// would not be smaller, so the triangular size bounds every window.  Final-stream
// layers always use bands: query tile qt sees at most window + 63*qpmul consecutive
// keys (all key tiles without a window).
__host__ __device__ inline int ds_band(const SfaGeom &g)
{
    const int nkt = (g.len + kDsKeys - 1) / kDsKeys;
    const int nqt = (g.qlen + kDsRows - 1) / kDsRows;
    if (g.qpmul != 1) {
        const int64_t span = (int64_t)(g.window < g.len ? g.window : g.len) + 63 * g.qpmul;
        const int64_t band = (span - 1 + kDsKeys - 1) / kDsKeys + 1;
        return (int)(band < nkt ? band : nkt);
    }
    if (g.window >= g.len) return 0;
    int band = (g.window - 1 + kDsKeys - 1) / kDsKeys + 1;
    band = band < nkt ? band : nkt;
    return (int64_t)nqt * band < ds_tile_index(0, 0, nqt, 0) ? band : 0;
}

// first key tile that query tile qt sees (used by the band index only)
__host__ __device__ inline int ds_kt_lo(const SfaGeom &g, int qt)
{
    if (g.window >= g.len) return 0;
    const int first = qpos(g, qt * kDsRows) - g.window + 1;
    return first > 0 ? first / kDsKeys : 0;
}

// index of the first dS tile of query tile qt inside its problem; qt = the query tile
// count gives the problem's tile count
__host__ __device__ inline int64_t ds_tile_base(int band, int qt)
{
    return band == 0 ? ds_tile_index(0, 0, qt, 0) : (int64_t)qt * band;
}

// Query tiles [first, end) of 64 rows with a row that sees some key of the 128-key
// tile kt (the sweep of the dK/dV workgroup that owns those keys).
__host__ __device__ inline void dkdv_sweep(const SfaGeom &g, int kt, int &first, int &end)
{
    const int k0 = kt * kDsKeys;
    const int f = (k0 - g.qpoff + g.qpmul - 1) / g.qpmul;
    first = (f > 0 ? f : 0) / kDsRows;
    const int64_t e = ((int64_t)k0 + kDsKeys - 2 + g.window - g.qpoff) / g.qpmul / kDsRows + 1;
    const int64_t nqt = (g.qlen + kDsRows - 1) / kDsRows;
    end = (int)(e < nqt ? e : nqt);
}

// Small dK/dV grids (fewer than kSplitGrid workgroups, i.e. under two per CU on
// MI355X) split the longest key-tile sweeps over two workgroups each, which run at the
// same time and leave fp32 partials for a combine pass; without it the step lasts as
// long as the sweep of the first key tile, which sees every query.  Returns the number
// of leading key tiles split this way: those whose sweep is longer than half the
// longest one (0 when the grid is large or has fewer than four key tiles).
constexpr int kSplitGrid = 512;

// Work items of a dK/dV launch with split sweeps, longest first (a key problem's items
// are dispatched in this order, so that the workgroups that finish early take the
// shorter items).  Item i is key tile item[i] >> 2 with code item[i] & 3: 0 the whole
// sweep, 1 its later half, 2 its earlier half.  A launch has at most kSplitGrid key
// tiles, so 2 * kSplitGrid items.
struct SplitOrder {
    uint16_t item[2 * kSplitGrid];
};

inline int dkdv_splits(const SfaGeom &g)
{
    const int nkt = (g.len + kDsKeys - 1) / kDsKeys;
    if (nkt < 4 || (int64_t)nkt * g.B * g.Hkv * g.streams >= kSplitGrid) return 0;
    int maxlen = 0;
    for (int kt = 0; kt < nkt; ++kt) {
        int f, e;
        dkdv_sweep(g, kt, f, e);
        maxlen = e - f > maxlen ? e - f : maxlen;
    }
    int ns = 0;
    for (; ns < nkt; ++ns) {
        int f, e;
        dkdv_sweep(g, ns, f, e);
        if (2 * (e - f) <= maxlen || e - f < 2) break;
    }
    return ns;
}

// The items of a launch with nsplit split key tiles, longest first (ties: lower key
// tile, later half first).
inline SplitOrder dkdv_split_order(const SfaGeom &g, int nsplit)
{
    const int nkt = (g.len + kDsKeys - 1) / kDsKeys;
    struct It {
        int len, code;
    };
    It its[2 * kSplitGrid];
    int n = 0;
    for (int kt = 0; kt < nkt; ++kt) {
        int f, e;
        dkdv_sweep(g, kt, f, e);
        const int len = e > f ? e - f : 0;
        if (kt < nsplit) {
            its[n++] = {len - len / 2, kt << 2 | 1};  // later half: [f + len/2, e)
            its[n++] = {len / 2, kt << 2 | 2};        // earlier half
        } else {
            its[n++] = {len, kt << 2};
        }
    }
    // insertion sort (at most 2 * kSplitGrid items, once per launch)
    for (int i = 1; i < n; ++i) {
        const It x = its[i];
        int j = i - 1;
        while (j >= 0 && (its[j].len < x.len || (its[j].len == x.len && its[j].code > x.code))) {
            its[j + 1] = its[j];
            --j;
        }
        its[j + 1] = x;
    }
    SplitOrder o;
    for (int i = 0; i < n; ++i) o.item[i] = (uint16_t)its[i].code;
    return o;
}

// dS tiles per causal problem
inline int64_t ds_tiles_per_problem(const SfaGeom &g)
{
    return ds_tile_base(ds_band(g), (g.qlen + kDsRows - 1) / kDsRows);
}

// Query bands of the bf16 backward.  With a workspace that holds every dS tile the
// backward runs in one pass.  With less, the query rows are processed in bands of
// whole 256-row units (four dS query tiles, one dQ workgroup's rows), in ascending
// order: the dK/dV pass of a band sweeps only the band's query tiles and stores their
// dS tiles, the dQ pass of the band reads them back.  dK and dV of a key tile are
// carried from band to band in fp32: the band holding the first query tile that sees
// the key tile writes the partials, later ones add to them, and the band holding the
// last such query tile writes the bf16 result.
constexpr int kBandUnit = 4;  // 64-row query tiles per band unit

struct QBand {
    int qt_lo, qt_hi;         // 64-row query tiles [qt_lo, qt_hi) of this band
    int64_t ds_base;          // index of the band's first dS tile in a problem's full numbering
    float *part_k, *part_v;   // fp32 dK / dV partials [B][Hkv][streams][len][D]; null: one band
};

// Backward workspace, each part 256-byte aligned:
//   per-row statistics, fp32 [B][Hq][qN] each: for fp32 those of
//   launch_bwd_preprocess_f32, for bf16 -Delta and -lse/scale;
//   bf16 path only, one pass: the dS tiles of every problem (b, hq[, s]),
//     problem-major (ds, total);
//   bf16 path only, one pass with split sweeps (dkdv_splits > 0): after the dS tiles,
//     the fp32 partials of the two halves of every split sweep (split), laid out
//     [half][dK, dV][key problem][split keys][D];
//   bf16 path only, in query bands: the fp32 dK and dV partials, then the dS tiles of
//     one band (part_k, part_v, ds_banded); the smallest workspace holds the dS tiles of
//     the largest band unit (min_total).  Bands do not split sweeps.
struct BwdWorkspace {
    size_t delta, lse2, ds, total;
    int64_t ds_tiles;  // dS tiles per problem (one pass)
    size_t part_k, part_v, ds_banded, min_total;
    size_t split;      // offset of the split-sweep partials (one pass)
    int nsplit;        // key tiles with a split sweep (one pass)
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline BwdWorkspace bwd_workspace(const SfaGeom &g, int esize)
{
    BwdWorkspace w;
    const size_t rows = (size_t)g.B * g.Hq * g.qN;
    w.delta = 0;
    w.lse2 = align256(rows * 4);
    w.ds = w.lse2 + align256(rows * 4);
    w.total = w.ds;
    w.ds_tiles = 0;
    w.part_k = w.part_v = w.ds_banded = w.ds;
    w.min_total = w.total;
    w.split = w.total;
    w.nsplit = 0;
    if (esize != 2) return w;
    const size_t probs = (size_t)g.B * g.Hq * g.streams;
    w.ds_tiles = ds_tiles_per_problem(g);
    w.total += probs * (size_t)w.ds_tiles * kDsTileBytes;
    w.split = align256(w.total);
    w.nsplit = dkdv_splits(g);
    w.total = w.split + (size_t)4 * g.B * g.Hkv * g.streams * w.nsplit * kDsKeys * g.D * 4;
    w.min_total = w.total;
    // banded layout; it needs each problem's fp32 partials to stay below 2^31 bytes
    const size_t part = (size_t)g.B * g.Hkv * g.streams * g.len * g.D * 4;
    w.part_v = w.part_k + align256(part);
    w.ds_banded = w.part_v + align256(part);
    if ((int64_t)g.len * g.D * 4 >= ((int64_t)1 << 31)) return w;
    const int band = ds_band(g);
    const int nqt = (g.qlen + kDsRows - 1) / kDsRows;
    int64_t unit = 0;  // dS tiles per problem of the largest band unit
    for (int qa = 0; qa < nqt; qa += kBandUnit) {
        const int qb = qa + kBandUnit < nqt ? qa + kBandUnit : nqt;
        const int64_t t = ds_tile_base(band, qb) - ds_tile_base(band, qa);
        unit = t > unit ? t : unit;
    }
    const size_t banded_min = w.ds_banded + probs * (size_t)unit * kDsTileBytes;
    if (banded_min < w.total) w.min_total = banded_min;
    return w;
}

inline size_t bwd_workspace_bytes(const SfaGeom &g, int esize) { return bwd_workspace(g, esize).total; }
inline size_t bwd_workspace_min_bytes(const SfaGeom &g, int esize)
{
    return bwd_workspace(g, esize).min_total;
}

}  // namespace hd
