// Codebook learning (Alg. 3, App. D) for gfx950: block-normalised gradient histogram,
// exact interval DP over the non-empty bins, and installation of a codebook into the
// tables the step kernels read (fp32 entries, midpoints, guide table).
//
// Floating-point choices: the histogram bin and the whole DP are evaluated in float64
// with contraction disabled, in the operation order of the definitions, so that the
// bins, DP costs, split points and codebook entries are reproducible bit for bit.
#include "gefen_internal.h"

#include <math.h>

namespace gefen {
namespace {

constexpr int kMaxBins = 16 * kMaxK;   // 4096

// ---------------------------------------------------------------------------------
// Histogram: x = g / max|g_block| (blocks with max 0 are skipped),
// bin = min(NB - 1, floor((x + 1) * NB / 2)). Each workgroup accumulates its tiles into
// an LDS histogram with integer atomics, then adds the non-zero bins to the global
// uint64 histogram. Integer atomics make the result independent of scheduling.
// ---------------------------------------------------------------------------------
__device__ __forceinline__ float grad_at(const Seg& sg, int64_t i)
{
    if (sg.gdtype == DT_F32) return static_cast<const float*>(sg.grad)[i];
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(sg.grad)[i]) << 16);
}

__device__ __forceinline__ int bin_of(float g, float a, double half_nb, int nbins)
{
    return hist_bin(g, a, half_nb, nbins);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Four gradient elements at vector index v (16-byte fp32 or 8-byte bf16 load).
__device__ __forceinline__ void grad4_at(const Seg& sg, int64_t v, float g[4])
{
    if (sg.gdtype == DT_F32) {
        const f32x4 x = reinterpret_cast<const f32x4*>(sg.grad)[v];
        g[0] = x.x; g[1] = x.y; g[2] = x.z; g[3] = x.w;
    } else {
        const u32x2 x = reinterpret_cast<const u32x2*>(sg.grad)[v];
        g[0] = __uint_as_float(x.x << 16); g[1] = __uint_as_float(x.x & 0xffff0000u);
        g[2] = __uint_as_float(x.y << 16); g[3] = __uint_as_float(x.y & 0xffff0000u);
    }
}

// Range [start, start + len) split into an aligned vector body [vb, ve) (vector units)
// and element-wise head/tail, when the gradient pointer is aligned for vector loads.
struct GSpan {
    int64_t vb, ve, start, nh, tail0, nt;
};

__device__ __forceinline__ GSpan grad_span(const Seg& sg, int64_t start, int64_t len)
{
    const int64_t end = start + len;
    const uintptr_t al = sg.gdtype == DT_F32 ? 15 : 7;
    int64_t b = end, e = end;
    if ((reinterpret_cast<uintptr_t>(sg.grad) & al) == 0) {
        b = (start + 3) & ~int64_t(3);
        e = end & ~int64_t(3);
        if (b > end) b = end;
        if (e < b) e = b;
    }
    GSpan s;
    s.vb = b >> 2;
    s.ve = e >> 2;
    s.start = start;
    s.nh = b - start;
    s.tail0 = e;
    s.nt = end - e;
    return s;
}

// Absmax over a span by `stride` threads, this one being `tid` (per-thread partial; the
// caller reduces).
__device__ __forceinline__ float span_absmax(const Seg& sg, const GSpan& sp, int tid, int stride)
{
    float a = 0.0f;
#pragma unroll 2
    for (int64_t v = sp.vb + tid; v < sp.ve; v += stride) {
        float g[4];
        grad4_at(sg, v, g);
        a = fmaxf(a, fmaxf(fmaxf(fabsf(g[0]), fabsf(g[1])), fmaxf(fabsf(g[2]), fabsf(g[3]))));
    }
    for (int64_t i = tid; i < sp.nh + sp.nt; i += stride) {
        const int64_t e = i < sp.nh ? sp.start + i : sp.tail0 + (i - sp.nh);
        a = fmaxf(a, fabsf(grad_at(sg, e)));
    }
    return a;
}

__device__ __forceinline__ void span_bins(const Seg& sg, const GSpan& sp, float a, double half_nb,
                                          int nbins, uint32_t* h, int tid, int stride)
{
#pragma unroll 2
    for (int64_t v = sp.vb + tid; v < sp.ve; v += stride) {
        float g[4];
        grad4_at(sg, v, g);
#pragma unroll
        for (int c = 0; c < 4; ++c) atomicAdd(&h[bin_of(g[c], a, half_nb, nbins)], 1u);
    }
    for (int64_t i = tid; i < sp.nh + sp.nt; i += stride) {
        const int64_t e = i < sp.nh ? sp.start + i : sp.tail0 + (i - sp.nh);
        atomicAdd(&h[bin_of(grad_at(sg, e), a, half_nb, nbins)], 1u);
    }
}

__device__ __forceinline__ void tile_block(const Seg& sg, const Tile& tl, int bi, int64_t& start,
                                           int64_t& len)
{
    if (sg.period > 0) {
        start = tl.elem0 + static_cast<int64_t>(bi) * sg.period;
        len = sg.period;
    } else {
        const int64_t local = tl.blk0 + bi - sg.blk_begin;
        start = sg.csr[local];
        len = sg.csr[local + 1] - start;
    }
}

// Absolute maximum of |g| over one chunk of a huge block.
__global__ __launch_bounds__(kThreads) void k_hist_h_absmax(const Tile* __restrict__ tiles,
                                                            const HTile* __restrict__ htiles,
                                                            const Seg* __restrict__ segs,
                                                            float* __restrict__ am_partials)
{
    __shared__ float red[kThreads / 64];
    const Tile tl = tiles[blockIdx.x];
    const HTile ht = htiles[blockIdx.x];
    const Seg sg = segs[tl.seg];
    float a = span_absmax(sg, grad_span(sg, tl.elem0, tl.nelem), threadIdx.x, kThreads);
    for (int off = 1; off < 64; off <<= 1) a = fmaxf(a, __shfl_xor(a, off));
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int w = 1; w < kThreads / 64; ++w) a = fmaxf(a, red[w]);
        am_partials[ht.first + ht.chunk] = fmaxf(a, red[0]);
    }
}

__global__ __launch_bounds__(kThreads) void k_histogram(const Tile* __restrict__ tiles,
                                                        int64_t n_tiles,
                                                        const int32_t* __restrict__ tile_kind,
                                                        const HTile* __restrict__ htiles,
                                                        const float* __restrict__ am_partials,
                                                        const Seg* __restrict__ segs,
                                                        int32_t nbins,
                                                        uint64_t* __restrict__ hist)
{
    __shared__ uint32_t h[kMaxBins];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    for (int i = tid; i < nbins; i += kThreads) h[i] = 0;
    __syncthreads();
    const double half_nb = 0.5 * static_cast<double>(nbins);

    // Every wave takes its own tiles (wave-strided persistent loop) and reduces within
    // itself, so no barrier is needed until the flush.
    constexpr int kWaves = kThreads / 64;
    for (int64_t ti = static_cast<int64_t>(blockIdx.x) * kWaves + wave; ti < n_tiles;
         ti += static_cast<int64_t>(gridDim.x) * kWaves) {
        const Tile tl = tiles[ti];
        const Seg sg = segs[tl.seg];
        const int kind = tile_kind[ti];
        if (kind == KIND_L) {
            // one lane per small block
            for (int bi = lane; bi < tl.nblk; bi += 64) {
                int64_t start, len;
                tile_block(sg, tl, bi, start, len);
                float a = 0.0f;
                for (int64_t i = 0; i < len; ++i) a = fmaxf(a, fabsf(grad_at(sg, start + i)));
                if (a > 0.0f)
                    for (int64_t i = 0; i < len; ++i)
                        atomicAdd(&h[bin_of(grad_at(sg, start + i), a, half_nb, nbins)], 1u);
            }
        } else if (kind == KIND_H) {
            // one chunk of a huge block: block absmax from the chunk maxima
            const HTile ht = htiles[ti];
            float a = 0.0f;
            for (int c = lane; c < ht.nchunk; c += 64) a = fmaxf(a, am_partials[ht.first + c]);
            for (int off = 1; off < 64; off <<= 1) a = fmaxf(a, __shfl_xor(a, off));
            if (a > 0.0f)
                span_bins(sg, grad_span(sg, tl.elem0, tl.nelem), a, half_nb, nbins, h, lane, 64);
        } else {
            // the tile's blocks one after another, each by the whole wave
            for (int bi = 0; bi < tl.nblk; ++bi) {
                int64_t start, len;
                tile_block(sg, tl, bi, start, len);
                const GSpan sp = grad_span(sg, start, len);
                float a = span_absmax(sg, sp, lane, 64);
                for (int off = 1; off < 64; off <<= 1) a = fmaxf(a, __shfl_xor(a, off));
                if (a > 0.0f) span_bins(sg, sp, a, half_nb, nbins, h, lane, 64);
            }
        }
    }
    __syncthreads();
    for (int i = tid; i < nbins; i += kThreads) {
        const uint32_t c = h[i];
        if (c) atomicAdd(reinterpret_cast<unsigned long long*>(&hist[i]),
                         static_cast<unsigned long long>(c));
    }
}

// ---------------------------------------------------------------------------------
// DP workspace layout (offsets in bytes, all 256-byte aligned):
//   hdr    int32[16]: [0] b (non-empty bins), [1] keff (entries the DP solves for),
//          [2] status
//   Z0,Z1,Z2,cnt,ctr   double[NB + 1] each (1-based, index 0 = 0)
//   D      double[(k + 1) * (NB + 1)]   D[j][r]
//   split  uint16[(k + 1) * (NB + 1)]
//   pv, pa double / int32 [2][NB + 1][kDpMaxChunks]: per-chunk partial minima of a level
// ---------------------------------------------------------------------------------
struct DpLayout {
    size_t hdr, z0, z1, z2, cnt, ctr, d, split, pv, pa, total;
};

constexpr int kDpThreads = 1024;
constexpr int kDpRows = kDpThreads / 64;                        // rows r per workgroup
constexpr int kDpChunk = 1024;                                  // l values per workgroup
constexpr int kDpMaxChunks = (kMaxBins + kDpChunk - 1) / kDpChunk;

__host__ __device__ inline size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

__host__ __device__ inline DpLayout dp_layout(int32_t nbins, int32_t k)
{
    DpLayout L;
    const size_t row = static_cast<size_t>(nbins) + 1;
    size_t o = 0;
    L.hdr = o; o += align256(16 * sizeof(int32_t));
    L.z0 = o; o += align256(row * sizeof(double));
    L.z1 = o; o += align256(row * sizeof(double));
    L.z2 = o; o += align256(row * sizeof(double));
    L.cnt = o; o += align256(row * sizeof(double));
    L.ctr = o; o += align256(row * sizeof(double));
    L.d = o; o += align256(static_cast<size_t>(k + 1) * row * sizeof(double));
    L.split = o; o += align256(static_cast<size_t>(k + 1) * row * sizeof(uint16_t));
    L.pv = o; o += align256(2 * row * kDpMaxChunks * sizeof(double));
    L.pa = o; o += align256(2 * row * kDpMaxChunks * sizeof(int32_t));
    L.total = o;
    return L;
}

template <typename T>
__device__ __forceinline__ T* at(void* ws, size_t off)
{
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Compaction of non-empty bins and prefix sums, in increasing bin order. The workgroup
// compacts the non-empty bins (a prefix count over 16-bin runs) and forms each one's
// centre, count and the two products c m and (c m) m in LDS; one thread then takes the
// three running sums in increasing bin order, so the summation order is the
// definition's, with nothing but three additions per bin on its path. The sums are
// copied out by the whole workgroup. Also clears row 0 of D.
constexpr int kPrepRun = kMaxBins / kThreads;   // bins per thread in the compaction

__global__ __launch_bounds__(kThreads) void k_dp_prep(const uint64_t* __restrict__ hist,
                                                      int32_t nbins, int32_t k, void* ws)
{
    __shared__ double t0[kMaxBins + 1], t1[kMaxBins + 1], t2[kMaxBins + 1];   // c, c m, c m m
    __shared__ int runs[kThreads];
    __shared__ int nr;
    const int tid = threadIdx.x;
    const DpLayout L = dp_layout(nbins, k);
    double* D = at<double>(ws, L.d);
    double* Z0 = at<double>(ws, L.z0);
    double* Z1 = at<double>(ws, L.z1);
    double* Z2 = at<double>(ws, L.z2);
    double* cnt = at<double>(ws, L.cnt);
    double* ctr = at<double>(ws, L.ctr);
    const size_t row = static_cast<size_t>(nbins) + 1;
    for (size_t r = tid; r < row; r += blockDim.x) D[r] = r == 0 ? 0.0 : INFINITY;
    const double w = 2.0 / static_cast<double>(nbins);
    // thread tid owns bins [tid * kPrepRun, + kPrepRun): count, then scan the counts
    const int i0 = tid * kPrepRun;
    int mine = 0;
    for (int i = i0; i < i0 + kPrepRun && i < nbins; ++i) mine += hist[i] != 0;
    runs[tid] = mine;
    __syncthreads();
    if (tid == 0) {
        int acc = 0;
        for (int q = 0; q < kThreads; ++q) {
            const int c = runs[q];
            runs[q] = acc;
            acc += c;
        }
        nr = acc;
    }
    __syncthreads();
    int r = runs[tid];   // compacted slots before this thread's bins (0-based)
    for (int i = i0; i < i0 + kPrepRun && i < nbins; ++i) {
        const uint64_t hv = hist[i];
        if (hv == 0) continue;
        const double c = static_cast<double>(hv);
        const double m = -1.0 + (static_cast<double>(i) + 0.5) * w;
        ++r;
        const double cm = c * m;
        t0[r] = c;
        t1[r] = cm;
        t2[r] = cm * m;
        ctr[r] = m;
        cnt[r] = c;
    }
    __syncthreads();
    const int b = nr;
    if (tid == 0) {
        double z0 = 0.0, z1 = 0.0, z2 = 0.0;
        t0[0] = 0.0;
        t1[0] = 0.0;
        t2[0] = 0.0;
        for (int q = 1; q <= b; ++q) {
            z0 = z0 + t0[q];
            z1 = z1 + t1[q];
            z2 = z2 + t2[q];
            t0[q] = z0;
            t1[q] = z1;
            t2[q] = z2;
        }
        int32_t* hdr = at<int32_t>(ws, L.hdr);
        hdr[0] = b;
        hdr[1] = b >= k ? k : (b >= 2 ? b : 0);
        hdr[2] = b >= k ? 0 : 1;
    }
    __syncthreads();
    for (int q = tid; q <= b; q += blockDim.x) {
        Z0[q] = t0[q];
        Z1[q] = t1[q];
        Z2[q] = t2[q];
    }
}

// ---------------------------------------------------------------------------------
// DP level j: D[j][r] = min over l of D[j-1][l-1] + C(l, r), argmin to the smallest l.
// Workgroup (x, y) takes rows r0 .. r0 + 15 (one wave each) and the candidates l of
// chunk y, [j + 1024 y, j + 1024 y + 1023], staging Z[l-1] and D[j-1][l-1] for that
// chunk in LDS (32 KB), so every workgroup does at most 16 x 1024 evaluations. It writes
// a partial (min, argmin) per row and chunk (double-buffered by level parity); level
// j + 1 rebuilds D[j][.] from them while staging, in chunk order with ties to the
// smaller l, and its last row of workgroups (whose chunks cover every l) stores the
// final D[j][.] and split[j][.] rows for the backtrack. k_dp_final reduces the last
// level. Level j < keff takes only the rows r <= b - (keff - j): a longer prefix leaves
// too few bins for the entries still to come, so no path to D[keff][b] passes through
// it (the rows it does take, and their candidates, are the ones the full scan has).
// ---------------------------------------------------------------------------------
__device__ __forceinline__ int dp_chunks(int jj, int r)
{
    const int hi = jj == 1 ? 1 : r;
    return hi < jj ? 0 : (hi - jj) / kDpChunk + 1;
}

__device__ __forceinline__ void dp_reduce(const double* __restrict__ pv,
                                          const int32_t* __restrict__ pa, int jj, int r,
                                          double& v, int& a)
{
    v = INFINITY;
    a = 0x7fffffff;
    const int nc = dp_chunks(jj, r);
    for (int c = 0; c < nc; ++c) {
        const double x = pv[static_cast<size_t>(r) * kDpMaxChunks + c];
        const int y = pa[static_cast<size_t>(r) * kDpMaxChunks + c];
        if (x < v || (x == v && y < a)) {
            v = x;
            a = y;
        }
    }
}

__global__ __launch_bounds__(kDpThreads) void k_dp_level(int32_t nbins, int32_t k, int32_t j,
                                                         void* ws)
{
    __shared__ double sZ0[kDpChunk], sZ1[kDpChunk], sZ2[kDpChunk], sD[kDpChunk];
    const DpLayout L = dp_layout(nbins, k);
    const int32_t* hdr = at<int32_t>(ws, L.hdr);
    const int b = hdr[0];
    const int keff = hdr[1];
    if (j > keff) return;
    int r0, r1;
    if (j == keff) {
        if (blockIdx.x != 0) return;
        r0 = r1 = b;
    } else {
        const int rmax = b - keff + j;
        r0 = j + static_cast<int>(blockIdx.x) * kDpRows;
        if (r0 > rmax) return;
        r1 = r0 + kDpRows - 1 < rmax ? r0 + kDpRows - 1 : rmax;
    }
    const int hi_max = j == 1 ? 1 : r1;
    const int l0 = j + static_cast<int>(blockIdx.y) * kDpChunk;
    if (l0 > hi_max) return;
    const int l1 = l0 + kDpChunk - 1 < hi_max ? l0 + kDpChunk - 1 : hi_max;
    const double* Z0 = at<double>(ws, L.z0);
    const double* Z1 = at<double>(ws, L.z1);
    const double* Z2 = at<double>(ws, L.z2);
    const size_t row = static_cast<size_t>(nbins) + 1;
    double* D = at<double>(ws, L.d);
    uint16_t* split = at<uint16_t>(ws, L.split);
    const size_t pstride = row * kDpMaxChunks;
    const double* pv_prev = at<double>(ws, L.pv) + ((j - 1) & 1) * pstride;
    const int32_t* pa_prev = at<int32_t>(ws, L.pa) + ((j - 1) & 1) * pstride;
    double* pv_cur = at<double>(ws, L.pv) + (j & 1) * pstride;
    int32_t* pa_cur = at<int32_t>(ws, L.pa) + (j & 1) * pstride;
    const bool last_rows = j == keff || static_cast<int>(blockIdx.x) == (b - keff) / kDpRows;
    for (int i = threadIdx.x; i <= l1 - l0; i += kDpThreads) {
        const int l = l0 + i;
        sZ0[i] = Z0[l - 1];
        sZ1[i] = Z1[l - 1];
        sZ2[i] = Z2[l - 1];
        double dv;
        if (j == 1) {
            dv = l == 1 ? 0.0 : INFINITY;   // D[0][l-1]
        } else {
            int da;
            dp_reduce(pv_prev, pa_prev, j - 1, l - 1, dv, da);
            if (last_rows) {
                D[static_cast<size_t>(j - 1) * row + (l - 1)] = dv;
                split[static_cast<size_t>(j - 1) * row + (l - 1)] = static_cast<uint16_t>(da);
            }
        }
        sD[i] = dv;
    }
    __syncthreads();
    const int r = r0 + static_cast<int>(threadIdx.x >> 6);
    if (r > r1) return;
    const int lane = threadIdx.x & 63;
    const double zr0 = Z0[r], zr1 = Z1[r], zr2 = Z2[r];
    const int hi = j == 1 ? 1 : r;
    double best = INFINITY;
    int arg = 0x7fffffff;
    for (int i = lane; i <= l1 - l0; i += 64) {   // increasing l: first minimum kept
        const int l = l0 + i;
        if (l > hi) break;
        const double S0 = zr0 - sZ0[i];
        const double S1 = zr1 - sZ1[i];
        const double S2 = zr2 - sZ2[i];
        double c;
        if (j == 1 || j == keff) {
            const double a = j == 1 ? -1.0 : 1.0;
            c = S2 - 2.0 * a * S1 + a * a * S0;
        } else {
            c = S2 - S1 * S1 / S0;
        }
        const double cand = sD[i] + c;
        if (cand < best) {
            best = cand;
            arg = l;
        }
    }
    for (int off = 1; off < 64; off <<= 1) {
        const double ob = __shfl_xor(best, off);
        const int oa = __shfl_xor(arg, off);
        if (ob < best || (ob == best && oa < arg)) {
            best = ob;
            arg = oa;
        }
    }
    if (lane == 0) {
        pv_cur[static_cast<size_t>(r) * kDpMaxChunks + blockIdx.y] = best;
        pa_cur[static_cast<size_t>(r) * kDpMaxChunks + blockIdx.y] = arg;
    }
}

// The last level's result for r = b.
__global__ void k_dp_final(int32_t nbins, int32_t k, void* ws)
{
    if (threadIdx.x != 0) return;
    const DpLayout L = dp_layout(nbins, k);
    const int32_t* hdr = at<int32_t>(ws, L.hdr);
    const int b = hdr[0];
    const int keff = hdr[1];
    if (keff < 2) return;
    const size_t row = static_cast<size_t>(nbins) + 1;
    const size_t pstride = row * kDpMaxChunks;
    double v;
    int a;
    dp_reduce(at<double>(ws, L.pv) + (keff & 1) * pstride,
              at<int32_t>(ws, L.pa) + (keff & 1) * pstride, keff, b, v, a);
    at<double>(ws, L.d)[static_cast<size_t>(keff) * row + b] = v;
    at<uint16_t>(ws, L.split)[static_cast<size_t>(keff) * row + b] = static_cast<uint16_t>(a);
}

// Backtracking (one thread): entry j is -1, +1 or the weighted mean of its interval;
// degenerate histograms (b < k) are padded with +1.
__global__ void k_dp_backtrack(int32_t nbins, int32_t k, void* ws, double* codebook,
                               double* cost, int32_t* status)
{
    if (threadIdx.x != 0) return;
    const DpLayout L = dp_layout(nbins, k);
    const int32_t* hdr = at<int32_t>(ws, L.hdr);
    const int b = hdr[0];
    const int keff = hdr[1];
    const double* Z0 = at<double>(ws, L.z0);
    const double* Z1 = at<double>(ws, L.z1);
    const double* cnt = at<double>(ws, L.cnt);
    const double* ctr = at<double>(ws, L.ctr);
    const size_t row = static_cast<size_t>(nbins) + 1;
    const double* D = at<double>(ws, L.d);
    const uint16_t* split = at<uint16_t>(ws, L.split);
    if (keff >= 2) {
        *cost = D[static_cast<size_t>(keff) * row + b];
        int r = b;
        for (int j = keff; j >= 1; --j) {
            const int l = split[static_cast<size_t>(j) * row + r];
            if (j == 1) {
                codebook[j - 1] = -1.0;
            } else if (j == keff) {
                codebook[j - 1] = 1.0;
            } else {
                const double S0 = Z0[r] - Z0[l - 1];
                const double S1 = Z1[r] - Z1[l - 1];
                codebook[j - 1] = S1 / S0;
            }
            r = l - 1;
        }
        for (int j = keff; j < k; ++j) codebook[j] = 1.0;
    } else {
        codebook[0] = -1.0;
        for (int j = 1; j < k; ++j) codebook[j] = 1.0;
        double e = 0.0;
        for (int i = 1; i <= b; ++i) {
            const double dl = ctr[i] + 1.0, dr = 1.0 - ctr[i];
            const double d2 = (dl * dl < dr * dr) ? dl * dl : dr * dr;
            e += cnt[i] * d2;
        }
        *cost = e;
    }
    *status = hdr[2];
}

// ---------------------------------------------------------------------------------
// Codebook installation: fp32 entries, fp64 copy, midpoints and the guide table.
// guide[bk] = number of midpoints whose bucket is < bk, bucket(x) =
// min(ng - 1, (int)((x + 1) * ng / 2)) in fp32 -- the same function the step applies
// to the (clamped) value being encoded, so the lookup is exact for fp32 midpoints.
// ---------------------------------------------------------------------------------
__global__ void k_install(const double* __restrict__ in64, const float* __restrict__ in32,
                          int32_t k, int32_t ng, float* cb32, double* cb64, float* mid,
                          uint8_t* guide)
{
    __shared__ float c[kMaxK];
    __shared__ uint16_t cnt[kMaxBins];
    const int t = threadIdx.x;
    for (int i = t; i < k; i += blockDim.x) {
        const float f = in64 ? static_cast<float>(in64[i]) : in32[i];
        c[i] = f;
        cb32[i] = f;
        cb64[i] = in64 ? in64[i] : static_cast<double>(in32[i]);
    }
    for (int i = t; i < ng; i += blockDim.x) cnt[i] = 0;
    __syncthreads();
    const float half_ng = 0.5f * static_cast<float>(ng);
    for (int i = t; i < k; i += blockDim.x) {
        const float mdp = i + 1 < k ? 0.5f * (c[i] + c[i + 1]) : 2.0f;
        mid[i] = mdp;
    }
    if (t == 0) {
        for (int i = 0; i + 1 < k; ++i) {
            const float mdp = 0.5f * (c[i] + c[i + 1]);
            const float x = fminf(fmaxf(mdp, -1.0f), 1.0f);
            int bk = static_cast<int>((x + 1.0f) * half_ng);
            bk = bk < ng - 1 ? bk : ng - 1;
            cnt[bk] += 1;
        }
        int acc = 0;
        for (int bk = 0; bk < ng; ++bk) {
            guide[bk] = static_cast<uint8_t>(acc);
            acc += cnt[bk];
        }
        guide[ng] = static_cast<uint8_t>(acc);
        for (int bk = ng + 1; bk < ((ng + 1 + 15) & ~15); ++bk) guide[bk] = 0;
    }
}

}  // namespace

size_t dp_workspace_bytes(int32_t nbins, int32_t k) { return dp_layout(nbins, k).total; }

hipError_t launch_hist_h_absmax(const Tile* tiles, const HTile* htiles, int64_t n_tiles,
                                const Seg* segs, float* am_partials, hipStream_t stream)
{
    if (n_tiles <= 0) return hipSuccess;
    if (n_tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_hist_h_absmax, dim3(static_cast<unsigned>(n_tiles)), dim3(kThreads), 0,
                       stream, tiles, htiles, segs, am_partials);
    return hipGetLastError();
}

hipError_t launch_histogram(const Tile* tiles, int64_t n_tiles, const int32_t* tile_kind,
                            const HTile* htiles, const float* am_partials, const Seg* segs,
                            int32_t nbins, uint64_t* hist, hipStream_t stream)
{
    if (n_tiles <= 0) return hipSuccess;
    const int64_t w = (n_tiles + kThreads / 64 - 1) / (kThreads / 64);
    const int64_t g = w < 4096 ? w : 4096;
    hipLaunchKernelGGL(k_histogram, dim3(static_cast<unsigned>(g)), dim3(kThreads), 0, stream,
                       tiles, n_tiles, tile_kind, htiles, am_partials, segs, nbins, hist);
    return hipGetLastError();
}

hipError_t launch_dp(const uint64_t* hist, int32_t nbins, int32_t k, void* ws,
                     double* codebook_out, double* cost_out, int32_t* status_out,
                     hipStream_t stream)
{
    hipLaunchKernelGGL(k_dp_prep, dim3(1), dim3(kThreads), 0, stream, hist, nbins, k, ws);
    const dim3 grid((static_cast<unsigned>(nbins) + kDpRows - 1) / kDpRows,
                    (static_cast<unsigned>(nbins) + kDpChunk - 1) / kDpChunk);
    for (int j = 1; j <= k; ++j)
        hipLaunchKernelGGL(k_dp_level, grid, dim3(kDpThreads), 0, stream, nbins, k, j, ws);
    hipLaunchKernelGGL(k_dp_final, dim3(1), dim3(64), 0, stream, nbins, k, ws);
    hipLaunchKernelGGL(k_dp_backtrack, dim3(1), dim3(64), 0, stream, nbins, k, ws,
                       codebook_out, cost_out, status_out);
    return hipGetLastError();
}

hipError_t launch_install_codebook(const double* cb64_in, int32_t k, int32_t ng, float* cb32,
                                   double* cb64, float* mid, uint8_t* guide, hipStream_t stream)
{
    hipLaunchKernelGGL(k_install, dim3(1), dim3(kThreads), 0, stream, cb64_in,
                       static_cast<const float*>(nullptr), k, ng, cb32, cb64, mid, guide);
    return hipGetLastError();
}

hipError_t launch_install_codebook_f32(const float* cb32_in, int32_t k, int32_t ng, float* cb32,
                                       double* cb64, float* mid, uint8_t* guide,
                                       hipStream_t stream)
{
    hipLaunchKernelGGL(k_install, dim3(1), dim3(kThreads), 0, stream,
                       static_cast<const double*>(nullptr), cb32_in, k, ng, cb32, cb64, mid,
                       guide);
    return hipGetLastError();
}

}  // namespace gefen
