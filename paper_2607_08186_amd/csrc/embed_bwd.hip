// embed_bwd.hip -- gradient of the multi-stream token expansion with respect to the
// n tables, and cyclic replication of the tables.
//
// The expansion of eq. (expansion) is a gather, out[b][t*n + s] = tables[s][ids[b][t]],
// so its gradient is a scatter-add: table s at token id x receives the sum of the
// upstream rows t*n + s of every token t with id x.  Done deterministically, without
// atomics on the data:
//   1. a stable sort of the (id, token position) pairs by id; ids outside [0, V) get
//      the key V and sort to the end.  Up to kSmallSortMax tokens the sorted position
//      of a token is counted directly (the number of tokens whose (key, position) is
//      smaller; one launch spread over M / 16 workgroups).  Larger batches take an LSD radix
//      sort with 8-bit digits (per-block digit histograms, one device-wide exclusive
//      scan, then a scatter in which every block ranks its chunk stably with eight
//      1-bit splits in LDS);
//   2. segment heads of the sorted ids give the distinct ids in ascending order and
//      each id's run of token positions (ascending, as the sort is stable);
//   3. one gather-reduce per (distinct id, stream): the upstream rows of the run are
//      summed in fp32 in ascending token order (HBM-bound: every upstream row is read
//      once, every gradient row written once).
// The gradient comes out sparse, as (distinct ids, rows), so nothing scales with V;
// hd_embed_grad_scatter_add adds such rows into a dense fp32 table gradient.
//
// Cyclic replication, eq. (cyclic_init): when the expansion factor grows from n to m
// (a multiple of n), table s of the new set is table s mod n of the old one.
#include <algorithm>

#include "embed_internal.h"
#include "hd_device.h"

namespace hd {

namespace {

constexpr int kThreads = 256;
constexpr int kItems = 8;
constexpr int kChunk = kThreads * kItems;  // keys per block in the scan and sort kernels
constexpr int kWaves = kThreads / 64;

// Exclusive scan of one int per thread across a workgroup of W waves; *total gets the
// sum.  `sh` is LDS scratch of W + 1 ints.
template <int W = kWaves>
__device__ inline int block_exclusive_scan(int x, int *total, int *sh)
{
    constexpr int kWaves = W;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int v = x;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(v, o);
        if (lane >= o) v += y;
    }
    if (lane == 63) sh[wave] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        int acc = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const int t = sh[w];
            sh[w] = acc;
            acc += t;
        }
        sh[kWaves] = acc;
    }
    __syncthreads();
    const int r = sh[wave] + v - x;
    *total = sh[kWaves];
    __syncthreads();  // sh may be reused right away
    return r;
}

// ---------------------------------------------------------------- device-wide scan
// Exclusive scan of x[0..n) (n <= kChunk * kChunk) in three launches: per-block sums,
// a one-block scan of the sums (the grand total goes to *total), per-block apply.

__global__ __launch_bounds__(kThreads) void scan_reduce_kernel(const int *__restrict__ x, int n,
                                                               int *__restrict__ sums)
{
    __shared__ int sh[kWaves + 1];
    const int64_t base = (int64_t)blockIdx.x * kChunk + threadIdx.x * kItems;
    int acc = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j)
        if (base + j < n) acc += x[base + j];
    int total;
    block_exclusive_scan(acc, &total, sh);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kThreads) void scan_top_kernel(int *__restrict__ sums, int nb,
                                                            int *__restrict__ total)
{
    __shared__ int sh[kWaves + 1];
    const int base = threadIdx.x * kItems;
    int v[kItems], acc = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        v[j] = base + j < nb ? sums[base + j] : 0;
        acc += v[j];
    }
    int tot;
    int run = block_exclusive_scan(acc, &tot, sh);
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        if (base + j < nb) sums[base + j] = run;
        run += v[j];
    }
    if (threadIdx.x == 0 && total != nullptr) *total = tot;
}

__global__ __launch_bounds__(kThreads) void scan_apply_kernel(int *__restrict__ x, int n,
                                                              const int *__restrict__ sums)
{
    __shared__ int sh[kWaves + 1];
    const int64_t base = (int64_t)blockIdx.x * kChunk + threadIdx.x * kItems;
    int v[kItems], acc = 0;
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        v[j] = base + j < n ? x[base + j] : 0;
        acc += v[j];
    }
    int tot;
    int run = block_exclusive_scan(acc, &tot, sh) + sums[blockIdx.x];
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        if (base + j < n) x[base + j] = run;
        run += v[j];
    }
}

hipError_t scan_exclusive(int *x, int n, int *sums, int *total, hipStream_t s)
{
    const int nb = (n + kChunk - 1) / kChunk;
    scan_reduce_kernel<<<nb, kThreads, 0, s>>>(x, n, sums);
    scan_top_kernel<<<1, kThreads, 0, s>>>(sums, nb, total);
    scan_apply_kernel<<<nb, kThreads, 0, s>>>(x, n, sums);
    return hipGetLastError();
}

// ---------------------------------------------------------------- radix sort

// sort key of token i: its id, or V for an id outside [0, V)
__device__ inline uint32_t id_key(const int32_t *ids, int64_t i, int64_t V)
{
    const int32_t id = ids[i];
    return id >= 0 && (int64_t)id < V ? (uint32_t)id : (uint32_t)V;
}

// digit histogram of each block's chunk, stored digit-major: hist[d * nblk + block]
__global__ __launch_bounds__(kThreads) void radix_hist_kernel(const uint32_t *__restrict__ keys,
                                                              const int32_t *__restrict__ ids,
                                                              int M, int64_t V, int shift,
                                                              int *__restrict__ hist)
{
    __shared__ int h[256];
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = (int64_t)blockIdx.x * kChunk + threadIdx.x * kItems;
#pragma unroll
    for (int j = 0; j < kItems; ++j)
        if (base + j < M) {
            const uint32_t key = ids != nullptr ? id_key(ids, base + j, V) : keys[base + j];
            atomicAdd(&h[(key >> shift) & 255], 1);
        }
    __syncthreads();
    hist[threadIdx.x * gridDim.x + blockIdx.x] = h[threadIdx.x];
}

// Stable scatter of one 8-bit digit pass.  offs = exclusive scan of the histograms
// (digit-major), so offs[d * nblk + block] is where this block's first key of digit d
// goes.  Keys and values come from (ids, token index) on the first pass.
__global__ __launch_bounds__(kThreads) void radix_scatter_kernel(
    const uint32_t *__restrict__ keys, const int32_t *__restrict__ vals,
    const int32_t *__restrict__ ids, int M, int64_t V, int shift, const int *__restrict__ offs,
    uint32_t *__restrict__ keys_out, int32_t *__restrict__ vals_out)
{
    __shared__ uint32_t sk[kChunk];
    __shared__ int32_t sv[kChunk];
    __shared__ int h[256];
    __shared__ int sh[kWaves + 1];
    const int64_t base = (int64_t)blockIdx.x * kChunk;
    const int valid = (int)min((int64_t)kChunk, (int64_t)M - base);
    uint32_t k[kItems];
    int32_t v[kItems];
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int c = threadIdx.x * kItems + j;
        if (c < valid) {
            k[j] = ids != nullptr ? id_key(ids, base + c, V) : keys[base + c];
            v[j] = ids != nullptr ? (int32_t)(base + c) : vals[base + c];
        } else {
            k[j] = 0xffffffffu;  // padding: digit 255, after every real key of the chunk
            v[j] = 0;
        }
    }
    // local stable sort of the chunk by the digit: one stable 1-bit split per bit
    for (int bit = 0; bit < 8; ++bit) {
        int zeros = 0;
#pragma unroll
        for (int j = 0; j < kItems; ++j) zeros += ((k[j] >> (shift + bit)) & 1) ? 0 : 1;
        int ztot;
        const int zb = block_exclusive_scan(zeros, &ztot, sh);  // zeros in earlier threads
        int zc = 0;
#pragma unroll
        for (int j = 0; j < kItems; ++j) {
            const int c = threadIdx.x * kItems + j;
            const bool one = (k[j] >> (shift + bit)) & 1;
            const int zbefore = zb + zc;  // zeros before element c
            const int dst = one ? ztot + (c - zbefore) : zbefore;
            zc += one ? 0 : 1;
            sk[dst] = k[j];
            sv[dst] = v[j];
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kItems; ++j) {
            k[j] = sk[threadIdx.x * kItems + j];
            v[j] = sv[threadIdx.x * kItems + j];
        }
        __syncthreads();
    }
    // start of each digit's run inside the sorted chunk (real keys only)
    h[threadIdx.x] = 0;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kItems; ++j)
        if ((int)threadIdx.x * kItems + j < valid) atomicAdd(&h[(k[j] >> shift) & 255], 1);
    __syncthreads();
    int tot;
    const int start = block_exclusive_scan(h[threadIdx.x], &tot, sh);
    h[threadIdx.x] = start;
    __syncthreads();
    // the chunk's real keys are its first `valid` sorted entries
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int c = threadIdx.x * kItems + j;
        if (c < valid) {
            const int d = (k[j] >> shift) & 255;
            const int64_t dst = (int64_t)offs[d * gridDim.x + blockIdx.x] + (c - h[d]);
            keys_out[dst] = k[j];
            vals_out[dst] = v[j];
        }
    }
}

// ---------------------------------------------------------------- small batches

constexpr int kRankWaves = 16;   // the segment pass: one workgroup of 16 waves
constexpr int kRankTokens = 16;  // tokens a rank workgroup places
constexpr int kRankChunks = 16;  // key chunks per token, one thread each

// Stable sort by counting: token i goes to position #{j : key_j < key_i, or key_j ==
// key_i and j < i}, which is the position the stable radix sort gives it.  A
// workgroup of 256 threads places 16 tokens: thread (c, i) counts over every 16th key
// from c (all M keys staged in LDS) for token i, and the 16 counts of a token are
// added in LDS, so the M x M comparisons spread over M / 16 workgroups (every CU at
// the 36-layer step's 4096 tokens).  PACKED (V < 2^18, so that every key, V included,
// fits 18 bits; vocabularies under 262144): LDS holds key << 14 | j, all distinct, and
// the order above is a single unsigned comparison of those words.
constexpr int kRankIndexBits = 14;  // token indices below kSmallSortMax = 2^14
static_assert((1 << kRankIndexBits) == kSmallSortMax, "packed keys carry the token index");

template <bool PACKED>
__global__ __launch_bounds__(kRankTokens * kRankChunks) void rank_sort_kernel(
    const int32_t *__restrict__ ids, int M, int64_t V, uint32_t *__restrict__ keys_out,
    int32_t *__restrict__ vals_out)
{
    __shared__ uint32_t sk[kSmallSortMax];
    __shared__ int cnt[kRankChunks][kRankTokens];
    // all of a thread's ids in flight at once (64 at kSmallSortMax tokens): buffer loads
    // past the M ids return 0 instead of being branched around, so that no load waits
    // for the one before it
    constexpr int kFill = kSmallSortMax / (kRankTokens * kRankChunks);
    const rsrc_t rid = make_rsrc(ids, (uint32_t)M * 4);
    int32_t fid[kFill];
#pragma unroll
    for (int f = 0; f < kFill; ++f)
        fid[f] = (int32_t)ld4(rid, (uint32_t)(f * kRankTokens * kRankChunks + threadIdx.x) * 4);
#pragma unroll
    for (int f = 0; f < kFill; ++f) {
        const int j = f * kRankTokens * kRankChunks + threadIdx.x;
        if (j < M) {
            const uint32_t key = fid[f] >= 0 && (int64_t)fid[f] < V ? (uint32_t)fid[f] : (uint32_t)V;
            sk[j] = PACKED ? key << kRankIndexBits | (uint32_t)j : key;
        }
    }
    __syncthreads();
    const int t = threadIdx.x % kRankTokens, c = threadIdx.x / kRankTokens;
    const int i = blockIdx.x * kRankTokens + t;
    const uint32_t ki = i < M ? sk[i] : 0xffffffffu;
    // chunk c: keys c, c + 16, ... (the 16 threads of a chunk read the same word, the
    // four chunks of a wave four consecutive words)
    int n = 0;
#pragma unroll 8
    for (int j = c; j < M; j += kRankChunks) {
        const uint32_t kj = sk[j];
        if constexpr (PACKED)
            n += kj < ki ? 1 : 0;
        else
            n += (kj < ki || (kj == ki && j < i)) ? 1 : 0;
    }
    cnt[c][t] = n;
    __syncthreads();
    if (c == 0 && i < M) {
        int r = 0;
#pragma unroll
        for (int cc = 0; cc < kRankChunks; ++cc) r += cnt[cc][t];
        keys_out[r] = PACKED ? ki >> kRankIndexBits : ki;
        vals_out[r] = i;
    }
}

// Segments of a sorted key array of M <= kSmallSortMax entries in one workgroup: the
// head of every run of equal keys gets its run's index (a block scan of the head
// flags), its start and, for in-range keys, its id; the run of key V (if any) is the
// last one and is not counted as a distinct id.  Each thread takes kPer consecutive
// keys and the one before them with branch-free buffer loads (zeros past the end).
__global__ __launch_bounds__(kRankWaves * 64) void small_segments_kernel(
    const uint32_t *__restrict__ keys, int M, int64_t V, int *__restrict__ seg_start,
    int32_t *__restrict__ uniq, int32_t *__restrict__ num_uniq)
{
    constexpr int kPer = kSmallSortMax / (kRankWaves * 64);
    static_assert(kPer % 4 == 0, "whole 16-byte loads");
    __shared__ int sh[kRankWaves + 1];
    const rsrc_t rk = make_rsrc(keys, (uint32_t)M * 4);
    const int i0 = threadIdx.x * kPer;
    uint32_t k[kPer];
#pragma unroll
    for (int e = 0; e < kPer; e += 4) {
        const u32x4 w = ld16(rk, (uint32_t)(i0 + e) * 4);
        k[e] = w[0];
        k[e + 1] = w[1];
        k[e + 2] = w[2];
        k[e + 3] = w[3];
    }
    const uint32_t before = i0 > 0 ? ld4(rk, (uint32_t)(i0 - 1) * 4) : 0u;
    uint32_t head = 0;  // bit e: key i0 + e starts a run
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int i = i0 + e;
        const uint32_t prev = e == 0 ? before : k[e - 1];
        if (i < M && (i == 0 || k[e] != prev)) head |= 1u << e;
    }
    int S;
    int u = block_exclusive_scan<kRankWaves>(__builtin_popcount(head), &S, sh);
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        if ((head >> e) & 1u) {
            seg_start[u] = i0 + e;
            if (k[e] < (uint64_t)V) uniq[u] = (int32_t)k[e];
            ++u;
        }
        // the thread holding the last key closes the last run
        if (i0 + e == M - 1) {
            seg_start[S] = M;
            *num_uniq = S - (k[e] == (uint64_t)V ? 1 : 0);
        }
    }
}

// ---------------------------------------------------------------- segments

__global__ __launch_bounds__(kThreads) void seg_flags_kernel(const uint32_t *__restrict__ keys,
                                                             int M, int *__restrict__ flags)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < M) flags[i] = (i == 0 || keys[i] != keys[i - 1]) ? 1 : 0;
}

// segidx = exclusive scan of the head flags: a head's value is its segment's index
__global__ __launch_bounds__(kThreads) void seg_write_kernel(const uint32_t *__restrict__ keys,
                                                             const int *__restrict__ segidx,
                                                             int M, int64_t V,
                                                             int *__restrict__ seg_start,
                                                             int32_t *__restrict__ uniq)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= M || !(i == 0 || keys[i] != keys[i - 1])) return;
    const int u = segidx[i];
    seg_start[u] = (int)i;
    if (keys[i] < (uint64_t)V) uniq[u] = (int32_t)keys[i];
}

// closes the last segment and counts the distinct in-range ids (the run of key V, if
// any, is the last segment and is left out)
__global__ void seg_finish_kernel(const uint32_t *__restrict__ keys, int M, int64_t V,
                                  const int *__restrict__ nseg, int *__restrict__ seg_start,
                                  int32_t *__restrict__ num_uniq)
{
    const int S = *nseg;
    seg_start[S] = M;
    *num_uniq = S - (keys[M - 1] == (uint64_t)V ? 1 : 0);
}

// ---------------------------------------------------------------- gather-reduce

template <typename E>
__device__ inline float elem(const E *p, int64_t i);
template <>
__device__ inline float elem<bf16>(const bf16 *p, int64_t i)
{
    return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t *>(p)[i] << 16);
}
template <>
__device__ inline float elem<float>(const float *p, int64_t i)
{
    return p[i];
}

// drows[s][u][:] = sum over the run of distinct id u of dout[pos*n + s][:] (fp32, in
// ascending token order).  Work items (u, s) are strided over the grid; the item
// count is read from the device.  VEC consecutive elements per thread and chunk, and
// kReduceChunks chunks of a row per pass, whose loads are all issued before the adds.
constexpr int kReduceChunks = 2;

// The upstream rows are read once: streaming (non-temporal) loads, 14% faster than
// cached ones on rows that are not in the caches.
template <typename E, int VEC>
__device__ inline void load_add(const E *src, float (&acc)[VEC])
{
    if constexpr (VEC == 8 && sizeof(E) == 2) {
        const u32x4 w4 = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(src));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc[2 * e] += bf16_lo(w4[e]);
            acc[2 * e + 1] += bf16_hi(w4[e]);
        }
    } else if constexpr (VEC == 8) {
        const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(src));
        const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(src + 4));
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            acc[e] += a[e];
            acc[4 + e] += b[e];
        }
    } else {
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += elem<E>(src, e);
    }
}

template <typename E, int VEC>
__global__ __launch_bounds__(kThreads) void embed_grad_reduce_kernel(
    const E *__restrict__ dout, const int32_t *__restrict__ pos, const int *__restrict__ seg_start,
    const int32_t *__restrict__ num_uniq, int n, int Dm, int rows_cap, float *__restrict__ drows)
{
    constexpr int kStride = kThreads * VEC;  // elements between a thread's chunks
    const int64_t items = (int64_t)*num_uniq * n;
    for (int64_t w = blockIdx.x; w < items; w += gridDim.x) {
        const int u = (int)(w / n), s = (int)(w % n);
        const int i0 = seg_start[u], i1 = seg_start[u + 1];
        float *dst = drows + ((int64_t)s * rows_cap + u) * Dm;
        for (int d0 = threadIdx.x * VEC; d0 < Dm; d0 += kStride * kReduceChunks) {
            float acc[kReduceChunks][VEC];
#pragma unroll
            for (int c = 0; c < kReduceChunks; ++c)
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc[c][e] = 0.f;
            for (int i = i0; i < i1; ++i) {
                const E *src = dout + ((int64_t)pos[i] * n + s) * Dm + d0;
#pragma unroll
                for (int c = 0; c < kReduceChunks; ++c)
                    if (d0 + c * kStride < Dm) load_add<E, VEC>(src + c * kStride, acc[c]);
            }
#pragma unroll
            for (int c = 0; c < kReduceChunks; ++c) {
                if (d0 + c * kStride >= Dm) continue;
                float *o = dst + d0 + c * kStride;
                if constexpr (VEC == 8) {
                    *reinterpret_cast<f32x4 *>(o) = f32x4{acc[c][0], acc[c][1], acc[c][2], acc[c][3]};
                    *reinterpret_cast<f32x4 *>(o + 4) = f32x4{acc[c][4], acc[c][5], acc[c][6], acc[c][7]};
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) o[e] = acc[c][e];
                }
            }
        }
    }
}

// dtables[s][uniq[u]][:] += drows[s][u][:] for u < *num_uniq (distinct ids: one writer
// per destination row, no atomics)
__global__ __launch_bounds__(kThreads) void embed_grad_scatter_add_kernel(
    const int32_t *__restrict__ uniq, const float *__restrict__ drows,
    const int32_t *__restrict__ num_uniq, int rows_cap, int n, int64_t V, int Dm,
    float *__restrict__ dtables)
{
    const int64_t items = (int64_t)*num_uniq * n;
    for (int64_t w = blockIdx.x; w < items; w += gridDim.x) {
        const int u = (int)(w / n), s = (int)(w % n);
        const int32_t x = uniq[u];
        if (x < 0 || (int64_t)x >= V) continue;
        const float *src = drows + ((int64_t)s * rows_cap + u) * Dm;
        float *dst = dtables + ((int64_t)s * V + x) * Dm;
        for (int d = threadIdx.x; d < Dm; d += kThreads) dst[d] += src[d];
    }
}

// ---------------------------------------------------------------- cyclic replication

// dst table s (s0 <= s < m) = src table s mod n; `words` W-sized words per table
template <typename W>
__global__ __launch_bounds__(kThreads) void cyclic_replicate_kernel(const W *__restrict__ src,
                                                                    W *__restrict__ dst, int n,
                                                                    int s0, int64_t words)
{
    const int s = s0 + blockIdx.y;
    const W *a = src + (int64_t)(s % n) * words;
    W *b = dst + (int64_t)s * words;
    for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < words;
         e += (int64_t)gridDim.x * kThreads)
        b[e] = a[e];
}

}  // namespace

EmbedBwdWorkspace embed_bwd_workspace(int M)
{
    EmbedBwdWorkspace w;
    const size_t m4 = align256((size_t)M * 4);
    const int nblk = (M + kChunk - 1) / kChunk;
    w.keys_a = 0;
    w.vals_a = w.keys_a + m4;
    w.keys_b = w.vals_a + m4;
    w.vals_b = w.keys_b + m4;
    w.hist = w.vals_b + m4;
    w.sums = w.hist + align256((size_t)256 * nblk * 4);
    w.scalars = w.sums + align256((size_t)kChunk * 4);
    w.segidx = w.scalars + 256;
    w.seg_start = w.segidx + m4;
    w.total = w.seg_start + align256(((size_t)M + 1) * 4);
    return w;
}

hipError_t launch_embed_bwd(const int32_t *ids, const void *dout, int B, int L, int n, int64_t V,
                            int Dm, int esize, int32_t *uniq, float *drows, int32_t *num_uniq,
                            void *ws, hipStream_t s)
{
    const int M = B * L;
    const EmbedBwdWorkspace w = embed_bwd_workspace(M);
    char *base = static_cast<char *>(ws);
    uint32_t *ka = reinterpret_cast<uint32_t *>(base + w.keys_a);
    int32_t *va = reinterpret_cast<int32_t *>(base + w.vals_a);
    uint32_t *kb = reinterpret_cast<uint32_t *>(base + w.keys_b);
    int32_t *vb = reinterpret_cast<int32_t *>(base + w.vals_b);
    int *hist = reinterpret_cast<int *>(base + w.hist);
    int *sums = reinterpret_cast<int *>(base + w.sums);
    int *nseg = reinterpret_cast<int *>(base + w.scalars);
    int *segidx = reinterpret_cast<int *>(base + w.segidx);
    int *seg_start = reinterpret_cast<int *>(base + w.seg_start);

    const int nblk = (M + kChunk - 1) / kChunk;
    int bits = 0;
    while (bits < 32 && ((uint64_t)V >> bits) != 0) ++bits;  // the largest key is V
    const int passes = bits == 0 ? 1 : (bits + 7) / 8;

    timing_before("embed_bwd_sort", s);
    hipError_t e = hipSuccess;
    const uint32_t *kin = nullptr;
    const int32_t *vin = nullptr;
    if (M <= kSmallSortMax) {
        const unsigned nb = (M + kRankTokens - 1) / kRankTokens;
        if (V < ((int64_t)1 << (32 - kRankIndexBits)))
            rank_sort_kernel<true><<<nb, kRankTokens * kRankChunks, 0, s>>>(ids, M, V, ka, va);
        else
            rank_sort_kernel<false><<<nb, kRankTokens * kRankChunks, 0, s>>>(ids, M, V, ka, va);
        small_segments_kernel<<<1, kRankWaves * 64, 0, s>>>(ka, M, V, seg_start, uniq, num_uniq);
        kin = ka;
        vin = va;
        e = hipGetLastError();
    }
    for (int p = 0; M > kSmallSortMax && p < passes && e == hipSuccess; ++p) {
        uint32_t *kout = (p & 1) ? kb : ka;
        int32_t *vout = (p & 1) ? vb : va;
        const int32_t *from_ids = p == 0 ? ids : nullptr;
        radix_hist_kernel<<<nblk, kThreads, 0, s>>>(kin, from_ids, M, V, 8 * p, hist);
        e = scan_exclusive(hist, 256 * nblk, sums, nullptr, s);
        radix_scatter_kernel<<<nblk, kThreads, 0, s>>>(kin, vin, from_ids, M, V, 8 * p, hist,
                                                       kout, vout);
        kin = kout;
        vin = vout;
        if (e == hipSuccess) e = hipGetLastError();
    }
    timing_after(s);
    if (e != hipSuccess) return e;

    if (M > kSmallSortMax) {
        timing_before("embed_bwd_segments", s);
        const int nb1 = (M + kThreads - 1) / kThreads;
        seg_flags_kernel<<<nb1, kThreads, 0, s>>>(kin, M, segidx);
        e = scan_exclusive(segidx, M, sums, nseg, s);
        seg_write_kernel<<<nb1, kThreads, 0, s>>>(kin, segidx, M, V, seg_start, uniq);
        seg_finish_kernel<<<1, 1, 0, s>>>(kin, M, V, nseg, seg_start, num_uniq);
        if (e == hipSuccess) e = hipGetLastError();
        timing_after(s);
        if (e != hipSuccess) return e;
    }

    // enough workgroups to keep every CU streaming; items beyond *num_uniq * n are
    // strided over them
    const int64_t max_items = (int64_t)M * n;
    const int grid = (int)(max_items < 8192 ? max_items : 8192);
    timing_before("embed_bwd_reduce", s);
    const bool vec = Dm % 8 == 0;
    if (esize == 2) {
        const bf16 *d = static_cast<const bf16 *>(dout);
        if (vec)
            embed_grad_reduce_kernel<bf16, 8><<<grid, kThreads, 0, s>>>(d, vin, seg_start, num_uniq,
                                                                        n, Dm, M, drows);
        else
            embed_grad_reduce_kernel<bf16, 1><<<grid, kThreads, 0, s>>>(d, vin, seg_start, num_uniq,
                                                                        n, Dm, M, drows);
    } else {
        const float *d = static_cast<const float *>(dout);
        if (vec)
            embed_grad_reduce_kernel<float, 8><<<grid, kThreads, 0, s>>>(d, vin, seg_start,
                                                                         num_uniq, n, Dm, M, drows);
        else
            embed_grad_reduce_kernel<float, 1><<<grid, kThreads, 0, s>>>(d, vin, seg_start,
                                                                         num_uniq, n, Dm, M, drows);
    }
    e = hipGetLastError();
    timing_after(s);
    return e;
}

hipError_t launch_embed_grad_scatter_add(const int32_t *uniq, const float *drows,
                                         const int32_t *num_uniq, int rows_cap, int n, int64_t V,
                                         int Dm, float *dtables, hipStream_t s)
{
    const int64_t max_items = (int64_t)rows_cap * n;
    const int grid = (int)(max_items < 8192 ? max_items : 8192);
    timing_before("embed_grad_scatter_add", s);
    embed_grad_scatter_add_kernel<<<grid, kThreads, 0, s>>>(uniq, drows, num_uniq, rows_cap, n, V,
                                                            Dm, dtables);
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

hipError_t launch_cyclic_replicate(const void *src, void *dst, int n, int m, int64_t V, int Dm,
                                   int esize, hipStream_t s)
{
    const int s0 = src == dst ? n : 0;  // in place: the first n tables are already there
    if (s0 >= m) return hipSuccess;
    const int64_t bytes = V * (int64_t)Dm * esize;
    const dim3 block(kThreads);
    timing_before("cyclic_replicate", s);
    if (bytes % 16 == 0) {
        const int64_t words = bytes / 16;
        const dim3 grid((unsigned)std::min<int64_t>((words + kThreads - 1) / kThreads, 4096),
                        (unsigned)(m - s0));
        cyclic_replicate_kernel<u32x4><<<grid, block, 0, s>>>(
            static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst), n, s0, words);
    } else {
        const int64_t words = bytes / 2;
        const dim3 grid((unsigned)std::min<int64_t>((words + kThreads - 1) / kThreads, 4096),
                        (unsigned)(m - s0));
        cyclic_replicate_kernel<uint16_t><<<grid, block, 0, s>>>(
            static_cast<const uint16_t *>(src), static_cast<uint16_t *>(dst), n, s0, words);
    }
    hipError_t e = hipGetLastError();
    timing_after(s);
    return e;
}

}  // namespace hd
