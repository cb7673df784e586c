// Automatic Block Partitioning (Sec. 5.1, Alg. 2) for gfx950.
//
// For every tensor of n elements and every divisor p of n:
//   z_j  = log(g_j^2 + eps)                     (float64)
//   mu_i = (sum of z over block i of p elements) / p
//   S(p) = sum_{i < n/p - 1} |mu_{i+1} - mu_i| / (n/p - 1),   S(n) = 0
// then the strict local maxima of S over the sorted divisors (1 < p < n), and the one
// with the largest S (ties: smallest p), else 1.
//
// Work items (one workgroup each) are described per (tensor, divisor) pair:
//   mode 0 (p <= kPBig): an item owns `rpi` consecutive pairs of blocks; it computes the
//          means of the rpi + 1 blocks involved (the last one is recomputed by the next
//          item) and writes the item's sum of |mu_{i+1} - mu_i|.
//   mode 1 (p >  kPBig): an item sums z over one sub-chunk of kChunk elements of one
//          block; the finalize kernel assembles block means from the sub-chunk sums.
// All sums run in a fixed order, so the scores are deterministic.
#include "gefen_internal.h"

#include <math.h>

namespace gefen {
namespace {

constexpr int64_t kChunk = 65536;
constexpr int kMaxPairs = 2048;

__device__ __forceinline__ double z_at(const void* g, int gdt, int64_t i, double eps)
{
    double x;
    if (gdt == DT_F32)
        x = static_cast<double>(static_cast<const float*>(g)[i]);
    else
        x = static_cast<double>(
            __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(g)[i]) << 16));
    return log(x * x + eps);
}

__device__ __forceinline__ double wave_sum(double v)
{
    for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off);
    return v;
}

// Fixed-order workgroup sum (wave butterflies, then waves 0..3 in order).
__device__ __forceinline__ double block_sum(double v, double* red)
{
    v = wave_sum(v);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) red[wave] = v;
    __syncthreads();
    double t = red[0];
    for (int w = 1; w < kThreads / 64; ++w) t += red[w];
    __syncthreads();
    return t;
}

__device__ __forceinline__ int find_desc(const PartDesc* descs, int32_t n_desc, int64_t item)
{
    int lo = 0, hi = n_desc - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (descs[mid].item0 <= item) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__global__ __launch_bounds__(kThreads) void k_part_items(const PartDesc* __restrict__ descs,
                                                         int32_t n_desc, double eps,
                                                         double* __restrict__ partials)
{
    __shared__ double mu[kMaxPairs + 1];
    __shared__ double red[kThreads / 64];
    const int64_t item = blockIdx.x;
    const PartDesc d = descs[find_desc(descs, n_desc, item)];
    const int64_t it = item - d.item0;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t p = d.p;

    if (d.mode == 1) {
        const int64_t blk = it / d.rpi;
        const int64_t c = it % d.rpi;
        const int64_t start = blk * p + c * kChunk;
        const int64_t stop = start + kChunk < (blk + 1) * p ? start + kChunk : (blk + 1) * p;
        double acc = 0.0;
        for (int64_t i = start + tid; i < stop; i += kThreads) acc += z_at(d.grad, d.gdtype, i, eps);
        const double t = block_sum(acc, red);
        if (tid == 0) partials[d.out0 + it] = t;
        return;
    }

    const int64_t nb = d.n / p;
    const int64_t b0 = it * d.rpi;
    const int64_t npairs = (b0 + d.rpi < nb - 1 ? b0 + d.rpi : nb - 1) - b0;
    const int nbk = static_cast<int>(npairs) + 1;
    const double inv_p_den = static_cast<double>(p);
    if (p <= 16) {
        for (int i = tid; i < nbk; i += kThreads) {
            const int64_t s0 = (b0 + i) * p;
            double acc = 0.0;
            for (int64_t e = 0; e < p; ++e) acc += z_at(d.grad, d.gdtype, s0 + e, eps);
            mu[i] = acc / inv_p_den;
        }
    } else {
        for (int i = wave; i < nbk; i += kThreads / 64) {
            const int64_t s0 = (b0 + i) * p;
            double acc = 0.0;
            for (int64_t e = lane; e < p; e += 64) acc += z_at(d.grad, d.gdtype, s0 + e, eps);
            acc = wave_sum(acc);
            if (lane == 0) mu[i] = acc / inv_p_den;
        }
    }
    __syncthreads();
    double acc = 0.0;
    for (int i = tid; i < npairs; i += kThreads) acc += fabs(mu[i + 1] - mu[i]);
    const double t = block_sum(acc, red);
    if (tid == 0) partials[d.out0 + it] = t;
}

__global__ __launch_bounds__(kThreads) void k_part_finalize(const PartDesc* __restrict__ descs,
                                                            const double* __restrict__ partials,
                                                            double* __restrict__ scores)
{
    __shared__ double red[kThreads / 64];
    const PartDesc d = descs[blockIdx.x];
    const int tid = threadIdx.x;
    const int64_t nb = d.n / d.p;
    if (nb < 2) {
        if (tid == 0) scores[blockIdx.x] = 0.0;
        return;
    }
    double acc = 0.0;
    if (d.mode == 0) {
        for (int64_t i = tid; i < d.n_items; i += kThreads) acc += partials[d.out0 + i];
    } else {
        // block means from sub-chunk sums (in chunk order), then adjacent contrasts
        const double pd = static_cast<double>(d.p);
        for (int64_t i = tid; i + 1 < nb; i += kThreads) {
            double s0 = 0.0, s1 = 0.0;
            for (int c = 0; c < d.rpi; ++c) s0 += partials[d.out0 + i * d.rpi + c];
            for (int c = 0; c < d.rpi; ++c) s1 += partials[d.out0 + (i + 1) * d.rpi + c];
            acc += fabs(s1 / pd - s0 / pd);
        }
    }
    const double t = block_sum(acc, red);
    if (tid == 0) scores[blockIdx.x] = t / static_cast<double>(nb - 1);
}

// Strict local maxima over the sorted divisor list (1 and n included as neighbours),
// then the largest score (first on ties), else period 1.
__global__ void k_part_select(const PartDesc* __restrict__ descs,
                              const double* __restrict__ scores,
                              const int32_t* __restrict__ first, const int32_t* __restrict__ count,
                              int32_t n_tensors, int64_t* __restrict__ periods)
{
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= n_tensors) return;
    const int f = first[t];
    const int c = count[t];
    int64_t best = 1;
    double best_s = 0.0;
    bool have = false;
    for (int i = 1; i + 1 < c; ++i) {
        const double s = scores[f + i];
        if (s > scores[f + i - 1] && s > scores[f + i + 1]) {
            if (!have || s > best_s) {
                best = descs[f + i].p;
                best_s = s;
                have = true;
            }
        }
    }
    periods[t] = best;
}

}  // namespace

hipError_t launch_partition(const PartDesc* descs, int32_t n_desc, int64_t n_items, double eps,
                            double* partials, double* scores, const int32_t* tensor_first_desc,
                            const int32_t* tensor_n_desc, int32_t n_tensors, int64_t* periods,
                            hipStream_t stream)
{
    if (n_items > 0x7fffffffLL) return hipErrorInvalidValue;
    if (n_items > 0)
        hipLaunchKernelGGL(k_part_items, dim3(static_cast<unsigned>(n_items)), dim3(kThreads), 0,
                           stream, descs, n_desc, eps, partials);
    if (n_desc > 0)
        hipLaunchKernelGGL(k_part_finalize, dim3(static_cast<unsigned>(n_desc)), dim3(kThreads),
                           0, stream, descs, partials, scores);
    if (n_tensors > 0)
        hipLaunchKernelGGL(k_part_select, dim3((n_tensors + 63) / 64), dim3(64), 0, stream,
                           descs, scores, tensor_first_desc, tensor_n_desc, n_tensors, periods);
    return hipGetLastError();
}

}  // namespace gefen
