// Gefen-Muon (appendix "Gefen-Muon"), the parts around the orthogonalisation: the
// Frobenius norm of each momentum matrix, its normalised bfloat16 copy in the wide
// orientation (the Newton-Schulz input), and the parameter update from the result.
// The momentum codec itself lives with the step kernels; the Newton-Schulz matrix
// products are plain bfloat16 GEMMs (rocBLAS), driven from the host.
#include "gefen_internal.h"

namespace gefen {
namespace {

__device__ __forceinline__ float bf16_val(uint16_t b)
{
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

__device__ __forceinline__ uint16_t to_bf16(float x)
{
    const uint32_t b = __float_as_uint(x);
    return static_cast<uint16_t>((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

// One workgroup per tensor: norm = bf16(sqrt(sum of u^2 over its tiles [tile_range[2t],
// tile_range[2t+1]))), clamped below by bf16(eps), summed in a fixed order (float64).
__global__ __launch_bounds__(256) void k_muon_norm(const float* __restrict__ tile_ss,
                                                   const int64_t* __restrict__ tile_range,
                                                   float eps_bf16, float* __restrict__ norm)
{
    __shared__ double red[256];
    const int t = blockIdx.x;
    const int64_t a = tile_range[2 * t], b = tile_range[2 * t + 1];
    double acc = 0.0;
    for (int64_t i = a + threadIdx.x; i < b; i += 256) acc += static_cast<double>(tile_ss[i]);
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int w = 128; w > 0; w >>= 1) {
        if (static_cast<int>(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const float nv = bf16_val(to_bf16(static_cast<float>(sqrt(red[0]))));
        norm[t] = fmaxf(nv, eps_bf16);
    }
}

constexpr int kT = 64;   // transpose tile edge

// X[batch] (m x n row-major, m = min(R, C)) = bf16(U_t / norm_t), with U_t the tensor's
// R x C momentum matrix; transposed when R > C. 64 x 64 tiles through LDS so both the
// read and the write are coalesced.
__global__ __launch_bounds__(256) void k_muon_prep(const uint16_t* __restrict__ u,
                                                   const Seg* __restrict__ segs,
                                                   const int32_t* __restrict__ tensor_of,
                                                   const float* __restrict__ norm, int64_t R,
                                                   int64_t C, int transposed,
                                                   uint16_t* __restrict__ x)
{
    __shared__ uint16_t tile[kT][kT + 2];
    const int b = blockIdx.z;
    const int t = tensor_of[b];
    const uint16_t* __restrict__ src = u + segs[t].code_off;
    uint16_t* __restrict__ dst = x + static_cast<int64_t>(b) * R * C;
    const float nrm = norm[t];
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kT;
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kT;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < kT; i += 4) {
        const int64_t r = r0 + i, c = c0 + tx;
        uint16_t v = 0;
        if (r < R && c < C) v = to_bf16(bf16_val(src[r * C + c]) / nrm);
        tile[i][tx] = v;
    }
    __syncthreads();
    if (!transposed) {
        for (int i = ty; i < kT; i += 4) {
            const int64_t r = r0 + i, c = c0 + tx;
            if (r < R && c < C) dst[r * C + c] = tile[i][tx];
        }
    } else {
        // X is C x R: X[c][r] = U[r][c]
        for (int i = ty; i < kT; i += 4) {
            const int64_t c = c0 + i, r = r0 + tx;
            if (r < R && c < C) dst[c * R + r] = tile[tx][i];
        }
    }
}

// Untransposed orientation (R <= C): the same copy and update as flat element loops,
// eight bfloat16 (prep) or four parameters (update) per thread where sizes and pointers
// are aligned, element by element otherwise.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void k_muon_prep_flat(const uint16_t* __restrict__ u,
                                                        const Seg* __restrict__ segs,
                                                        const int32_t* __restrict__ tensor_of,
                                                        const float* __restrict__ norm,
                                                        int64_t n, uint16_t* __restrict__ x)
{
    const int b = blockIdx.y;
    const int t = tensor_of[b];
    const uint16_t* __restrict__ src = u + segs[t].code_off;
    uint16_t* __restrict__ dst = x + static_cast<int64_t>(b) * n;
    const float nrm = norm[t];
    const int64_t stride = 256LL * gridDim.x;
    if ((n & 7) == 0) {
        for (int64_t v = blockIdx.x * 256LL + threadIdx.x; v < n / 8; v += stride) {
            const u32x4 w = reinterpret_cast<const u32x4*>(src)[v];
            u32x4 o;
            for (int c = 0; c < 4; ++c) {
                const uint32_t lo = to_bf16(bf16_val(static_cast<uint16_t>(w[c] & 0xffffu)) / nrm);
                const uint32_t hi = to_bf16(bf16_val(static_cast<uint16_t>(w[c] >> 16)) / nrm);
                o[c] = lo | (hi << 16);
            }
            reinterpret_cast<u32x4*>(dst)[v] = o;
        }
    } else {
        for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < n; i += stride)
            dst[i] = to_bf16(bf16_val(src[i]) / nrm);
    }
}

__global__ __launch_bounds__(256) void k_muon_update_flat(const uint16_t* __restrict__ o,
                                                          const Seg* __restrict__ segs,
                                                          const int32_t* __restrict__ tensor_of,
                                                          int64_t n, float decay, float step)
{
    const int b = blockIdx.y;
    const int t = tensor_of[b];
    float* __restrict__ th = segs[t].theta;
    const uint16_t* __restrict__ src = o + static_cast<int64_t>(b) * n;
    const int64_t stride = 256LL * gridDim.x;
    if ((n & 3) == 0 && (reinterpret_cast<uintptr_t>(th) & 15) == 0) {
        for (int64_t v = blockIdx.x * 256LL + threadIdx.x; v < n / 4; v += stride) {
            const u32x2v w = reinterpret_cast<const u32x2v*>(src)[v];
            f32x4v tv = reinterpret_cast<const f32x4v*>(th)[v];
            tv.x = fmaf(-step, bf16_val(static_cast<uint16_t>(w.x & 0xffffu)), tv.x * decay);
            tv.y = fmaf(-step, bf16_val(static_cast<uint16_t>(w.x >> 16)), tv.y * decay);
            tv.z = fmaf(-step, bf16_val(static_cast<uint16_t>(w.y & 0xffffu)), tv.z * decay);
            tv.w = fmaf(-step, bf16_val(static_cast<uint16_t>(w.y >> 16)), tv.w * decay);
            reinterpret_cast<f32x4v*>(th)[v] = tv;
        }
    } else {
        for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < n; i += stride)
            th[i] = fmaf(-step, bf16_val(src[i]), th[i] * decay);
    }
}

// theta_t (R x C) = theta_t * decay - step * O, O the orthogonalised matrix of batch
// entry b (m x n row-major, transposed back when R > C).
__global__ __launch_bounds__(256) void k_muon_update(const uint16_t* __restrict__ o,
                                                     const Seg* __restrict__ segs,
                                                     const int32_t* __restrict__ tensor_of,
                                                     int64_t R, int64_t C, int transposed,
                                                     float decay, float step)
{
    __shared__ uint16_t tile[kT][kT + 2];
    const int b = blockIdx.z;
    const int t = tensor_of[b];
    float* __restrict__ th = segs[t].theta;
    const uint16_t* __restrict__ src = o + static_cast<int64_t>(b) * R * C;
    const int64_t r0 = static_cast<int64_t>(blockIdx.y) * kT;
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kT;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    if (transposed) {
        // O is C x R: stage O[c0 .. c0 + 64)[r0 .. r0 + 64) with coalesced reads along r
        for (int i = ty; i < kT; i += 4) {
            const int64_t c = c0 + i, r = r0 + tx;
            tile[i][tx] = (r < R && c < C) ? src[c * R + r] : 0;
        }
        __syncthreads();
    }
    for (int i = ty; i < kT; i += 4) {
        const int64_t r = r0 + i, c = c0 + tx;
        if (r < R && c < C) {
            const uint16_t ob = transposed ? tile[tx][i] : src[r * C + c];
            const int64_t e = r * C + c;
            th[e] = fmaf(-step, bf16_val(ob), th[e] * decay);
        }
    }
}

// Split-K Gram: A = bf16(sum over s of P[s]), the float32 partial products of K-chunks,
// added in chunk order.
__global__ __launch_bounds__(256) void k_muon_splitk_sum(const float* __restrict__ partial,
                                                         int32_t splits, int64_t mm,
                                                         uint16_t* __restrict__ a)
{
    for (int64_t i = blockIdx.x * 256LL + threadIdx.x; i < mm; i += 256LL * gridDim.x) {
        float acc = partial[i];
        for (int32_t s = 1; s < splits; ++s) acc += partial[s * mm + i];
        a[i] = to_bf16(acc);
    }
}

// Newton-Schulz on 1 x n matrices (one workgroup per batch entry): the Gram matrix is
// the scalar s = x x^T, so every iteration is x <- bf16(a x + bf16(b s + c s^2) x), with
// s = bf16(x x^T) accumulated in float32 -- the same rounding points as the GEMM form.
__global__ __launch_bounds__(256) void k_muon_ns_vec(uint16_t* __restrict__ x, int64_t n,
                                                     int32_t steps, float ca, float cb,
                                                     float cc)
{
    __shared__ float red[256];
    uint16_t* __restrict__ v = x + static_cast<int64_t>(blockIdx.x) * n;
    for (int32_t it = 0; it < steps; ++it) {
        float acc = 0.0f;
        for (int64_t i = threadIdx.x; i < n; i += 256) {
            const float e = bf16_val(v[i]);
            acc = fmaf(e, e, acc);
        }
        red[threadIdx.x] = acc;
        __syncthreads();
        for (int w = 128; w > 0; w >>= 1) {
            if (static_cast<int>(threadIdx.x) < w) red[threadIdx.x] += red[threadIdx.x + w];
            __syncthreads();
        }
        const float gram = bf16_val(to_bf16(red[0]));
        const float poly = bf16_val(to_bf16(fmaf(cc, gram * gram, cb * gram)));
        __syncthreads();   // red[0] is read by every thread before the next iteration
        for (int64_t i = threadIdx.x; i < n; i += 256) {
            const float e = bf16_val(v[i]);
            v[i] = to_bf16(fmaf(poly, e, ca * e));
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_muon_norm(const float* tile_ss, const int64_t* tile_range, int32_t n_tensors,
                            float eps_bf16, float* norm, hipStream_t stream)
{
    if (n_tensors <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_muon_norm, dim3(n_tensors), dim3(256), 0, stream, tile_ss, tile_range,
                       eps_bf16, norm);
    return hipGetLastError();
}

static dim3 tile_grid(int64_t R, int64_t C, int batch)
{
    return dim3(static_cast<unsigned>((C + kT - 1) / kT), static_cast<unsigned>((R + kT - 1) / kT),
                static_cast<unsigned>(batch));
}

static dim3 flat_grid(int64_t n, int batch)
{
    int64_t g = (n + 2047) / 2048;
    if (g > 4096) g = 4096;
    if (g < 1) g = 1;
    return dim3(static_cast<unsigned>(g), static_cast<unsigned>(batch));
}

hipError_t launch_muon_prep(const uint16_t* u, const Seg* segs, const int32_t* tensor_of,
                            int32_t batch, const float* norm, int64_t R, int64_t C,
                            uint16_t* x, hipStream_t stream)
{
    if (batch <= 0) return hipSuccess;
    if (batch > 65535) return hipErrorInvalidValue;
    if (R <= C) {
        hipLaunchKernelGGL(k_muon_prep_flat, flat_grid(R * C, batch), dim3(256), 0, stream, u,
                           segs, tensor_of, norm, R * C, x);
        return hipGetLastError();
    }
    if ((R + kT - 1) / kT > 65535 || batch > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_muon_prep, tile_grid(R, C, batch), dim3(256), 0, stream, u, segs,
                       tensor_of, norm, R, C, R > C ? 1 : 0, x);
    return hipGetLastError();
}

hipError_t launch_muon_update(const uint16_t* o, const Seg* segs, const int32_t* tensor_of,
                              int32_t batch, int64_t R, int64_t C, float decay, float step,
                              hipStream_t stream)
{
    if (batch <= 0) return hipSuccess;
    if (batch > 65535) return hipErrorInvalidValue;
    if (R <= C) {
        hipLaunchKernelGGL(k_muon_update_flat, flat_grid(R * C, batch), dim3(256), 0, stream, o,
                           segs, tensor_of, R * C, decay, step);
        return hipGetLastError();
    }
    if ((R + kT - 1) / kT > 65535 || batch > 65535) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_muon_update, tile_grid(R, C, batch), dim3(256), 0, stream, o, segs,
                       tensor_of, R, C, R > C ? 1 : 0, decay, step);
    return hipGetLastError();
}

hipError_t launch_muon_splitk_sum(const float* partial, int32_t splits, int64_t mm,
                                  uint16_t* a, hipStream_t stream)
{
    if (mm <= 0) return hipSuccess;
    int64_t g = (mm + 255) / 256;
    if (g > 65536) g = 65536;
    hipLaunchKernelGGL(k_muon_splitk_sum, dim3(static_cast<unsigned>(g)), dim3(256), 0, stream,
                       partial, splits, mm, a);
    return hipGetLastError();
}

hipError_t launch_muon_ns_vec(uint16_t* x, int32_t batch, int64_t n, int32_t steps, float a,
                              float b, float c, hipStream_t stream)
{
    if (batch <= 0 || steps <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_muon_ns_vec, dim3(static_cast<unsigned>(batch)), dim3(256), 0, stream,
                       x, n, steps, a, b, c);
    return hipGetLastError();
}

}  // namespace gefen
