// Gefen-Muon (appendix "Gefen-Muon") on the device: the codec that keeps Muon's
// momentum in Gefen's quantized form, the Frobenius norm of each momentum matrix, its
// and the Newton-Schulz iterations of 1 x n matrices. The matrix products of the other
// shapes, and the kernels around them, are in ns_gemm.hip.
#include "muon_internal.h"
#include "step_device.h"

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

// ---------------------------------------------------------------------------------
// Gefen-Muon codec (appendix "Gefen-Muon"): Muon's momentum held in Gefen's quantized
// form. Per block: m = mu * c_dec[q] * s + (1 - mu) * g, s' = max |m|,
// q' = nearest(c_enc, m / s'); the matrix handed to the orthogonalisation is
// u = nesterov ? (1 - mu) * g + mu * m : m, written as bfloat16 at the code index of
// each element, and each tile's sum of u^2 (of the bfloat16 values) goes to tile_ss.
// Tile mode in Tile::vpl: 0 = the workgroup on one block, 1 = one lane per block,
// 2 = one wave per block.
// ---------------------------------------------------------------------------------
struct MuonOut {
    uint16_t* u;
    float mu, one_minus_mu;
    int nesterov;
};

// One element of the output pass: encode, write u, return u^2 (of the bfloat16 value).
template <int CB>
__device__ __forceinline__ float muon_elem_out(const LdsTables& L, uint8_t* __restrict__ codes,
                                               int64_t j, float g, float s_old, float s_new,
                                               float inv_s, const StepScalars& sc,
                                               const MuonOut& mo, float half_ng, int ng_m1)
{
    const int q0 = code_ld<CB>(codes, j);
    const float mm = momentum(L, q0, s_old, g, sc);
    const int q = s_new > 0.0f ? encode(L, mm * inv_s, half_ng, ng_m1) : 0;
    code_st<CB>(codes, j, q0, q);
    const float uu = mo.nesterov ? fmaf(mo.mu, mm, mo.one_minus_mu * g) : mm;
    const uint16_t ub = to_bf16(uu);
    mo.u[j] = ub;
    const float ur = __uint_as_float(static_cast<uint32_t>(ub) << 16);
    return ur * ur;
}

// Both passes of a block by BS threads (a wave or the workgroup; tid = index among them)
// over the Span layout of the streamed step: 4-element vectors over the aligned body
// (16- or 8-byte gradient loads, one code word, one 8-byte store of four bfloat16 u),
// elements at the head and tail. absmax_pass returns the thread's max |m|.
template <int GDT, int BS, int CB>
__device__ __forceinline__ float muon_absmax_pass(const LdsTables& L, const Seg& sg,
                                                  const uint8_t* __restrict__ codes,
                                                  const Span& sp, float s_old,
                                                  const StepScalars& sc, int tid)
{
    const int64_t cj = sg.code_off;
    float am = 0.0f;
#pragma unroll 2
    for (int64_t v = sp.vb + tid; v < sp.ve; v += BS) {
        float g[4];
        load_grad4<GDT>(sg, v, g);
        const uint32_t q4 = code_ld4<CB>(codes, cj + 4 * v);
#pragma unroll
        for (int c = 0; c < 4; ++c)
            am = fmaxf(am, fabsf(momentum(L, code_get<CB>(q4, c), s_old, g[c], sc)));
    }
    for (int64_t i = tid; i < sp.nh + sp.nt; i += BS) {
        const int64_t e = i < sp.nh ? sp.start + i : sp.tail0 + (i - sp.nh);
        const float g = load_grad(sg.grad, e, GDT);
        am = fmaxf(am, fabsf(momentum(L, code_ld<CB>(codes, cj + e), s_old, g, sc)));
    }
    return am;
}

template <int GDT, int BS, int CB>
__device__ __forceinline__ float muon_out_pass(const LdsTables& L, const Seg& sg,
                                               uint8_t* __restrict__ codes, const Span& sp,
                                               float s_old, float s_new, const StepScalars& sc,
                                               const MuonOut& mo, float half_ng, int ng_m1,
                                               int tid)
{
    const int64_t cj = sg.code_off;
    const float inv_s = s_new > 0.0f ? 1.0f / s_new : 0.0f;
    float uss = 0.0f;
#pragma unroll 2
    for (int64_t v = sp.vb + tid; v < sp.ve; v += BS) {
        float g[4];
        load_grad4<GDT>(sg, v, g);
        const uint32_t q4 = code_ld4<CB>(codes, cj + 4 * v);
        uint32_t packed = 0;
        uint32_t ub[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float mm = momentum(L, code_get<CB>(q4, c), s_old, g[c], sc);
            const int q = s_new > 0.0f ? encode(L, mm * inv_s, half_ng, ng_m1) : 0;
            packed |= static_cast<uint32_t>(q) << (CB * c);
            const float uu = mo.nesterov ? fmaf(mo.mu, mm, mo.one_minus_mu * g[c]) : mm;
            ub[c] = to_bf16(uu);
            const float ur = __uint_as_float(ub[c] << 16);
            uss = fmaf(ur, ur, uss);
        }
        code_st4<CB>(codes, cj + 4 * v, packed);
        const u32x2 w = {ub[0] | (ub[1] << 16), ub[2] | (ub[3] << 16)};
        *glw<u32x2>(mo.u + cj + 4 * v) = w;
    }
    for (int64_t i = tid; i < sp.nh + sp.nt; i += BS) {
        const int64_t e = i < sp.nh ? sp.start + i : sp.tail0 + (i - sp.nh);
        uss += muon_elem_out<CB>(L, codes, cj + e, load_grad(sg.grad, e, GDT), s_old, s_new,
                                 inv_s, sc, mo, half_ng, ng_m1);
    }
    return uss;
}

template <int GDT, int CB>
__global__ __launch_bounds__(kThreads) void k_muon_codec(const Tile* __restrict__ tiles,
                                                         const Seg* __restrict__ segs,
                                                         uint8_t* __restrict__ codes,
                                                         float* __restrict__ scale,
                                                         CodebookDev cbd, StepScalars sc,
                                                         MuonOut mo, float* __restrict__ tile_ss)
{
    __shared__ LdsTables L;
    const Tile tl = tiles[blockIdx.x];
    const Seg sg = segs[tl.seg];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    // Register path for a block of whole, aligned 4-element vectors: the workgroup
    // (mode 0, up to 4 * kRegV * kThreads elements) or one wave (mode 2, up to
    // 4 * kRegV * 64) holds it, every load issued before the tables are staged, so the
    // gradient and the codes are read once. Other blocks take the two streaming passes.
    constexpr int kRegV = 4;
    const bool wg_mode = tl.vpl == 0;
    const int bi = wg_mode ? 0 : wave;
    const int ti = wg_mode ? tid : lane;      // index within the block's threads
    const int bs = wg_mode ? kThreads : 64;   // threads per block
    int64_t start = 0, len = 0;
    bool reg = false;
    if ((wg_mode || tl.vpl == 2) && bi < tl.nblk) {
        block_range(sg, tl, bi, start, len);
        reg = ((start | len) & 3) == 0 && len <= 4LL * kRegV * bs && vector_ok<GDT>(sg);
    }
    float g[kRegV][4];
    uint32_t cq[kRegV];
    const int64_t v0 = start >> 2;
    const int nv = static_cast<int>(len >> 2);
    if (reg) {
#pragma unroll
        for (int j = 0; j < kRegV; ++j) {
            const int v = ti + j * bs;
            cq[j] = 0;
            g[j][0] = g[j][1] = g[j][2] = g[j][3] = 0.0f;
            if (v < nv) {
                load_grad4<GDT>(sg, v0 + v, g[j]);
                cq[j] = code_ld4<CB>(codes, sg.code_off + 4 * (v0 + v));
            }
        }
    }
    load_tables<kThreads>(L, cbd);
    __syncthreads();
    const float half_ng = 0.5f * static_cast<float>(cbd.ng);
    const int ng_m1 = cbd.ng - 1;
    float uss = 0.0f;
    if (reg) {   // uniform over the workgroup in mode 0, over the wave in mode 2
        const int64_t blk = tl.blk0 + bi;
        const float s_old = scale[blk];
        // momentum (kept in g), u = nesterov ? mu m + (1 - mu) g : m as packed bfloat16
        // (it does not depend on the new scale), and the block's max |m|
        uint32_t up[kRegV][2];
        float am = 0.0f;
#pragma unroll
        for (int j = 0; j < kRegV; ++j) {
            const bool ok = ti + j * bs < nv;
            uint32_t ub[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float mm = ok ? momentum(L, code_get<CB>(cq[j], c), s_old, g[j][c], sc)
                                    : 0.0f;
                const float uu = mo.nesterov ? fmaf(mo.mu, mm, mo.one_minus_mu * g[j][c]) : mm;
                ub[c] = ok ? to_bf16(uu) : 0u;
                const float ur = __uint_as_float(ub[c] << 16);
                uss = fmaf(ur, ur, uss);
                am = fmaxf(am, fabsf(mm));
                g[j][c] = mm;
            }
            up[j][0] = ub[0] | (ub[1] << 16);
            up[j][1] = ub[2] | (ub[3] << 16);
        }
        for (int off = 1; off < 64; off <<= 1) am = fmaxf(am, __shfl_xor(am, off));
        if (wg_mode) {
            if (lane == 0) L.red_am[wave] = am;
            __syncthreads();
            am = L.red_am[0];
            for (int w = 1; w < kThreads / 64; ++w) am = fmaxf(am, L.red_am[w]);
        }
        if (ti == 0) scale[blk] = am;
        const float inv_s = am > 0.0f ? 1.0f / am : 0.0f;
#pragma unroll
        for (int j = 0; j < kRegV; ++j) {
            const int v = ti + j * bs;
            if (v < nv) {
                uint32_t packed = 0;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int q = am > 0.0f ? encode(L, g[j][c] * inv_s, half_ng, ng_m1) : 0;
                    packed |= static_cast<uint32_t>(q) << (CB * c);
                }
                code_st4<CB>(codes, sg.code_off + 4 * (v0 + v), packed);
                const u32x2 w = {up[j][0], up[j][1]};
                *glw<u32x2>(mo.u + sg.code_off + 4 * (v0 + v)) = w;
            }
        }
    } else if (wg_mode) {
        const float s_old = scale[tl.blk0];
        const Span sp = make_span<GDT>(sg, start, len);
        float am = muon_absmax_pass<GDT, kThreads, CB>(L, sg, codes, sp, s_old, sc, tid);
        for (int off = 1; off < 64; off <<= 1) am = fmaxf(am, __shfl_xor(am, off));
        if (lane == 0) L.red_am[wave] = am;
        __syncthreads();
        am = L.red_am[0];
        for (int w = 1; w < kThreads / 64; ++w) am = fmaxf(am, L.red_am[w]);
        if (tid == 0) scale[tl.blk0] = am;
        uss = muon_out_pass<GDT, kThreads, CB>(L, sg, codes, sp, s_old, am, sc, mo, half_ng,
                                               ng_m1, tid);
    } else if (tl.vpl == 1) {
        if (tid < tl.nblk) {
            int64_t start, len;
            block_range(sg, tl, tid, start, len);
            const int64_t blk = tl.blk0 + tid;
            const float s_old = scale[blk];
            const int64_t cj = sg.code_off + start;
            float am = 0.0f;
            for (int64_t i = 0; i < len; ++i) {
                const float g = load_grad(sg.grad, start + i, GDT);
                am = fmaxf(am, fabsf(momentum(L, code_ld<CB>(codes, cj + i), s_old, g, sc)));
            }
            scale[blk] = am;
            const float inv_s = am > 0.0f ? 1.0f / am : 0.0f;
            for (int64_t i = 0; i < len; ++i)
                uss += muon_elem_out<CB>(L, codes, cj + i, load_grad(sg.grad, start + i, GDT),
                                         s_old, am, inv_s, sc, mo, half_ng, ng_m1);
        }
    } else if (tl.vpl == 2) {
        if (wave < tl.nblk) {
            const int64_t blk = tl.blk0 + wave;
            const float s_old = scale[blk];
            const Span sp = make_span<GDT>(sg, start, len);
            float am = muon_absmax_pass<GDT, 64, CB>(L, sg, codes, sp, s_old, sc, lane);
            for (int off = 1; off < 64; off <<= 1) am = fmaxf(am, __shfl_xor(am, off));
            if (lane == 0) scale[blk] = am;
            uss = muon_out_pass<GDT, 64, CB>(L, sg, codes, sp, s_old, am, sc, mo, half_ng, ng_m1,
                                             lane);
        }
    }
    // the tile's sum of u^2, fixed order (red_ss is not used above)
    for (int off = 1; off < 64; off <<= 1) uss += __shfl_xor(uss, off);
    if (lane == 0) L.red_ss[wave] = uss;
    __syncthreads();
    if (tid == 0) {
        float t = L.red_ss[0];
        for (int w = 1; w < kThreads / 64; ++w) t += L.red_ss[w];
        tile_ss[blockIdx.x] = t;
    }
}

// Newton-Schulz on 1 x n matrices (one workgroup per batch entry): the Gram matrix is
// the scalar s = x x^T, so every iteration is x <- bf16(a x + bf16(b s + c s^2) x), with
// s = bf16(x x^T) accumulated in float32 -- the same rounding points as the GEMM form.
__global__ __launch_bounds__(256) void k_muon_ns_vec(uint16_t* __restrict__ x, int64_t n,
                                                     int64_t stride, int32_t steps, float ca,
                                                     float cb, float cc)
{
    __shared__ float red[256];
    uint16_t* __restrict__ v = x + static_cast<int64_t>(blockIdx.x) * stride;
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

hipError_t launch_muon_ns_vec(uint16_t* x, int32_t batch, int64_t n, int64_t stride, int32_t steps,
                              float a, float b, float c, hipStream_t stream)
{
    if (batch <= 0 || steps <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_muon_ns_vec, dim3(static_cast<unsigned>(batch)), dim3(256), 0, stream,
                       x, n, stride, steps, a, b, c);
    return hipGetLastError();
}

hipError_t launch_muon_codec(int code_bits, int gdtype, const Tile* tiles, int64_t n_tiles,
                             const Seg* segs,
                             uint8_t* codes, float* scale, CodebookDev cb, float mu,
                             float one_minus_mu, int nesterov, uint16_t* u, float* tile_ss,
                             hipStream_t stream)
{
    if (n_tiles <= 0) return hipSuccess;
    if (n_tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    StepScalars sc{};
    sc.beta1 = mu;
    sc.one_minus_beta1 = one_minus_mu;
    MuonOut mo{u, mu, one_minus_mu, nesterov};
    const dim3 grid(static_cast<unsigned>(n_tiles));
#define GEFEN_MC(G, C)                                                                      \
    hipLaunchKernelGGL((k_muon_codec<G, C>), grid, dim3(kThreads), 0, stream, tiles, segs,  \
                       codes, scale, cb, sc, mo, tile_ss)
    if (code_bits != 8 && code_bits != 4) return hipErrorInvalidValue;
    if (gdtype == DT_F32) {
        if (code_bits == 8) GEFEN_MC(DT_F32, 8); else GEFEN_MC(DT_F32, 4);
    } else {
        if (code_bits == 8) GEFEN_MC(DT_BF16, 8); else GEFEN_MC(DT_BF16, 4);
    }
#undef GEFEN_MC
    return hipGetLastError();
}

}  // namespace gefen
