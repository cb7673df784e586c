// Gefen optimizer step (Alg. 1, loop body) for gfx950.
//
// For every block B of a tensor (consecutive `period` elements, or an explicit range):
//   m_i  = beta1 * (c_dec[q_i] * s_B) + (1 - beta1) * g_i       dequantize + momentum
//   s_B' = max |m_i|,  q_i' = nearest(c_enc, m_i / s_B')         requantize, new absmax
//   v_B' = beta2 * v_B + (1 - beta2) * mean(g_i^2)               shared second moment
//   theta_i = theta_i * (1 - lr*wd) - (lr / (1 - beta1^t)) * m_i / (sqrt(v_B' / (1 - beta2^t)) + eps)
// The bias-corrected momentum uses the unquantized m_i of the same step.
//
// The step is bound by HBM bandwidth (12-14 bytes per element against ~30 FP32
// operations), so the kernels stream every array once, keep the momentum of a block in
// registers, and reduce each block with wavefront shuffles (plus LDS across waves).
// The codebook sits in LDS: decoding is one LDS read; encoding is a guide-table lookup
// (one byte per bucket of [-1, 1] giving the number of midpoints below the bucket) plus
// a short scan over the midpoints that fall inside the bucket (at most one for codebooks
// whose entries are at least a bucket apart, as the DP's are).
#include "tile_plan.h"
#include "step_device.h"

namespace gefen {
namespace {

// ---------------------------------------------------------------------------------
// KIND_U: uniform blocks of p elements (p % 4 == 0, p <= 8192). A group of
// LPB = 2^lpb_log2 lanes owns one block; lane li holds vectors v = j * LPB + li,
// j < VPL, of 4 consecutive elements each. A workgroup of BS threads holds BS / LPB
// blocks. Small tiles (one block per workgroup, one or two vectors per lane) keep
// the most independent streams in flight, which is what saturates HBM here.
// ---------------------------------------------------------------------------------
template <int GDT, int VPL, int BS, bool ALIGNED, int CB>
__device__ __forceinline__ void step_u_body(LdsTables& L, const Tile& tl, const Seg& sg,
                                            uint8_t* __restrict__ codes,
                                            float* __restrict__ scale,
                                            float* __restrict__ vmom, const CodebookDev& cbd,
                                            const StepScalars& sc)
{
    const int lpb_log2 = tl.lpb_log2;
    const int lpb = 1 << lpb_log2;
    const int tid = threadIdx.x;
    const int gi = tid >> lpb_log2;
    const int li = tid & (lpb - 1);
    const bool active = gi < tl.nblk;
    const int64_t p = sg.period;
    const int nv = static_cast<int>(p >> 2);
    const int64_t e0 = tl.elem0 + static_cast<int64_t>(gi) * p;
    const int64_t blk = tl.blk0 + gi;

    float* __restrict__ th_base = sg.theta + e0;
    const int64_t cj0 = sg.code_off + e0;   // code index of the block's first element

    float th[VPL][4];
    float gv[VPL][4];
    uint32_t cq[VPL];
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
        const int v = j * lpb + li;
        cq[j] = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) { th[j][c] = 0.0f; gv[j][c] = 0.0f; }
        if (active && v < nv) {
            const int64_t o = 4 * static_cast<int64_t>(v);
            if (ALIGNED) {
                const f32x4 t4 = __builtin_nontemporal_load(gl<f32x4>(th_base + o));
                th[j][0] = t4.x; th[j][1] = t4.y; th[j][2] = t4.z; th[j][3] = t4.w;
                if (GDT == DT_F32) {
                    const f32x4 g4 = __builtin_nontemporal_load(
                        gl<f32x4>(static_cast<const float*>(sg.grad) + e0 + o));
                    gv[j][0] = g4.x; gv[j][1] = g4.y; gv[j][2] = g4.z; gv[j][3] = g4.w;
                } else {
                    const u32x2 g2 = __builtin_nontemporal_load(
                        gl<u32x2>(static_cast<const uint16_t*>(sg.grad) + e0 + o));
                    gv[j][0] = bf16_lo(g2.x); gv[j][1] = bf16_hi(g2.x);
                    gv[j][2] = bf16_lo(g2.y); gv[j][3] = bf16_hi(g2.y);
                }
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    th[j][c] = th_base[o + c];
                    gv[j][c] = load_grad(sg.grad, e0 + o + c, GDT);
                }
            }
            if (CB == 8)
                cq[j] = __builtin_nontemporal_load(gl<uint32_t>(codes + cj0 + o));
            else
                cq[j] = __builtin_nontemporal_load(gl<uint16_t>(codes + ((cj0 + o) >> 1)));
        }
    }
    float s_old = 0.0f, v_old = 0.0f;
    if (active) {
        s_old = scale[blk];
        v_old = vmom[blk];
    }
    load_tables<BS>(L, cbd);
    __syncthreads();

    // phase 1: dequantize + momentum, block reductions of sum g^2 and max |m|
    // (lanes past the end of their block, or without a block, contribute 0 to both)
    float m[VPL][4];
    float ss = 0.0f, am = 0.0f;
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
        const bool ok = active && (j * lpb + li) < nv;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int q = code_get<CB>(cq[j], c);
            const float mm = ok ? momentum(L, q, s_old, gv[j][c], sc) : 0.0f;
            m[j][c] = mm;
            ss = fmaf(gv[j][c], gv[j][c], ss);
            am = fmaxf(am, fabsf(mm));
        }
    }
    const int wl = lpb < 64 ? lpb : 64;
    for (int off = 1; off < wl; off <<= 1) {
        ss += __shfl_xor(ss, off);
        am = fmaxf(am, __shfl_xor(am, off));
    }
    if (lpb > 64) {
        const int wave = tid >> 6;
        if ((tid & 63) == 0) {
            L.red_ss[wave] = ss;
            L.red_am[wave] = am;
        }
        __syncthreads();
        const int wpb = lpb >> 6;
        const int w0 = (wave / wpb) * wpb;
        ss = L.red_ss[w0];
        am = L.red_am[w0];
        for (int w = 1; w < wpb; ++w) {
            ss += L.red_ss[w0 + w];
            am = fmaxf(am, L.red_am[w0 + w]);
        }
    }
    if (!active) return;

    const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(p), sc);
    if (li == 0) {
        scale[blk] = bo.s_new;
        vmom[blk] = bo.v_new;
    }
    const float half_ng = 0.5f * static_cast<float>(cbd.ng);
    const int ng_m1 = cbd.ng - 1;
#pragma unroll
    for (int j = 0; j < VPL; ++j) {
        const int v = j * lpb + li;
        if (v < nv) {
            uint32_t packed = 0;
            float out[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float mm = m[j][c];
                const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
                packed |= static_cast<uint32_t>(q) << (CB * c);
                out[c] = fmaf(-bo.r, mm, th[j][c] * sc.decay);
            }
            const int64_t o = 4 * static_cast<int64_t>(v);
            if (ALIGNED) {
                const f32x4 o4 = {out[0], out[1], out[2], out[3]};
                __builtin_nontemporal_store(o4, glw<f32x4>(th_base + o));
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) th_base[o + c] = out[c];
            }
            code_st4<CB>(codes, cj0 + o, packed);
        }
    }
}

// ---------------------------------------------------------------------------------
// KIND_ANY: the leftover small tiles of every shape in one launch (generic path, kept
// out of the KIND_U kernel, whose fast path measurably slows down when this code is
// compiled into it): two streaming passes per block, by the whole workgroup for a
// single block, one lane per block for blocks of at most 32 elements, else one wave
// per block.
// ---------------------------------------------------------------------------------
template <int BS, int CB>
__device__ void foreign_tile(LdsTables& L, const Tile& tl, const Seg& sg,
                             uint8_t* __restrict__ codes, float* __restrict__ scale,
                             float* __restrict__ vmom, const CodebookDev& cbd,
                             const StepScalars& sc)
{
    load_tables<BS>(L, cbd);
    __syncthreads();
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int gdt = sg.gdtype;
    const float half_ng = 0.5f * static_cast<float>(cbd.ng);
    const int ng_m1 = cbd.ng - 1;
    if (tl.nblk == 1) {
        int64_t start, len;
        block_range(sg, tl, 0, start, len);
        const int64_t blk = tl.blk0;
        const float s_old = scale[blk];
        const float v_old = vmom[blk];
        float* __restrict__ th = sg.theta + start;
        const int64_t cj = sg.code_off + start;
        float ss = 0.0f, am = 0.0f;
        for (int64_t i = tid; i < len; i += BS) {
            const float g = load_grad(sg.grad, start + i, gdt);
            const float mm = momentum(L, code_ld<CB>(codes, cj + i), s_old, g, sc);
            ss = fmaf(g, g, ss);
            am = fmaxf(am, fabsf(mm));
        }
        for (int off = 1; off < 64; off <<= 1) {
            ss += __shfl_xor(ss, off);
            am = fmaxf(am, __shfl_xor(am, off));
        }
        if (lane == 0) {
            L.red_ss[wave] = ss;
            L.red_am[wave] = am;
        }
        __syncthreads();
        ss = L.red_ss[0];
        am = L.red_am[0];
        for (int w = 1; w < BS / 64; ++w) {
            ss += L.red_ss[w];
            am = fmaxf(am, L.red_am[w]);
        }
        const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(len), sc);
        if (tid == 0) {
            scale[blk] = bo.s_new;
            vmom[blk] = bo.v_new;
        }
        for (int64_t i = tid; i < len; i += BS) {
            const float g = load_grad(sg.grad, start + i, gdt);
            const int q0 = code_ld<CB>(codes, cj + i);
            const float mm = momentum(L, q0, s_old, g, sc);
            const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
            th[i] = fmaf(-bo.r, mm, th[i] * sc.decay);
            code_st<CB>(codes, cj + i, q0, q);
        }
        return;
    }
    if (sg.period > 0 && sg.period <= kSmallBlock) {
        // small uniform blocks: a group of lpb = 2^ceil(log2 p) consecutive lanes per
        // block, one element per lane, so every access of a wave is contiguous; block
        // sums by shuffles inside the group. The planner sizes these tiles to one pass
        // (nblk * lpb <= BS); longer tiles take several.
        const int p = static_cast<int>(sg.period);
        int lpb = 1;
        while (lpb < p) lpb <<= 1;
        const int li = tid & (lpb - 1);
        for (int b0 = 0; b0 < tl.nblk; b0 += BS / lpb) {
            const int bi = b0 + tid / lpb;
            const bool okb = bi < tl.nblk;
            const bool ok = okb && li < p;
            const int64_t e = tl.elem0 + static_cast<int64_t>(bi) * p + li;
            const int64_t blk = tl.blk0 + bi;
            float g = 0.0f, tv = 0.0f, s_old = 0.0f, v_old = 0.0f;
            int q0 = 0;
            if (ok) {
                g = load_grad(sg.grad, e, gdt);
                q0 = code_ld<CB>(codes, sg.code_off + e);
                tv = sg.theta[e];
            }
            if (okb) {
                s_old = scale[blk];
                v_old = vmom[blk];
            }
            const float mm = ok ? momentum(L, q0, s_old, g, sc) : 0.0f;
            float ss = g * g, am = fabsf(mm);
            for (int off = 1; off < lpb; off <<= 1) {
                ss += __shfl_xor(ss, off);
                am = fmaxf(am, __shfl_xor(am, off));
            }
            const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(p), sc);
            if (okb && li == 0) {
                scale[blk] = bo.s_new;
                vmom[blk] = bo.v_new;
            }
            if (ok) {
                const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
                sg.theta[e] = fmaf(-bo.r, mm, tv * sc.decay);
                code_st<CB>(codes, sg.code_off + e, q0, q);
            }
        }
        return;
    }
    if (sg.period == 0) {
        // explicit small-block tile: lane per block
        for (int bi = tid; bi < tl.nblk; bi += BS) {
            int64_t start, len;
            block_range(sg, tl, bi, start, len);
            const int64_t blk = tl.blk0 + bi;
            const float s_old = scale[blk];
            const float v_old = vmom[blk];
            float* __restrict__ th = sg.theta + start;
            const int64_t cj = sg.code_off + start;
            // len <= kSmallBlock: the block stays in registers. Every load is issued
            // unconditionally (past the block's end it re-reads its first element), so
            // the loads of a pass go out together instead of one guarded load at a time.
            float g[kSmallBlock], m[kSmallBlock], tv[kSmallBlock];
            int q0[kSmallBlock];
#pragma unroll
            for (int i = 0; i < kSmallBlock; ++i) {
                const int64_t ii = i < len ? i : 0;
                g[i] = load_grad(sg.grad, start + ii, gdt);
                q0[i] = code_ld<CB>(codes, cj + ii);
                tv[i] = th[ii];
            }
            float ss = 0.0f, am = 0.0f;
#pragma unroll
            for (int i = 0; i < kSmallBlock; ++i) {
                const bool ok = i < len;
                m[i] = ok ? momentum(L, q0[i], s_old, g[i], sc) : 0.0f;
                ss = ok ? fmaf(g[i], g[i], ss) : ss;
                am = fmaxf(am, fabsf(m[i]));
            }
            const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(len), sc);
            scale[blk] = bo.s_new;
            vmom[blk] = bo.v_new;
#pragma unroll
            for (int i = 0; i < kSmallBlock; ++i) {
                if (i < len) {
                    const int q = bo.s_new > 0.0f ? encode(L, m[i] * bo.inv_s, half_ng, ng_m1)
                                                  : 0;
                    th[i] = fmaf(-bo.r, m[i], tv[i] * sc.decay);
                    code_st<CB>(codes, cj + i, q0[i], q);
                }
            }
        }
        return;
    }
    for (int bi = wave; bi < tl.nblk; bi += BS / 64) {
        int64_t start, len;
        block_range(sg, tl, bi, start, len);
        const int64_t blk = tl.blk0 + bi;
        const float s_old = scale[blk];
        const float v_old = vmom[blk];
        float* __restrict__ th = sg.theta + start;
        const int64_t cj = sg.code_off + start;
        float ss = 0.0f, am = 0.0f;
        for (int64_t i = lane; i < len; i += 64) {
            const float g = load_grad(sg.grad, start + i, gdt);
            const float mm = momentum(L, code_ld<CB>(codes, cj + i), s_old, g, sc);
            ss = fmaf(g, g, ss);
            am = fmaxf(am, fabsf(mm));
        }
        for (int off = 1; off < 64; off <<= 1) {
            ss += __shfl_xor(ss, off);
            am = fmaxf(am, __shfl_xor(am, off));
        }
        const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(len), sc);
        if (lane == 0) {
            scale[blk] = bo.s_new;
            vmom[blk] = bo.v_new;
        }
        for (int64_t i = lane; i < len; i += 64) {
            const float g = load_grad(sg.grad, start + i, gdt);
            const int q0 = code_ld<CB>(codes, cj + i);
            const float mm = momentum(L, q0, s_old, g, sc);
            const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
            th[i] = fmaf(-bo.r, mm, th[i] * sc.decay);
            code_st<CB>(codes, cj + i, q0, q);
        }
    }
}

template <int CB>
__global__ __launch_bounds__(kThreads) void k_step_any(const Tile* __restrict__ tiles,
                                                       const Seg* __restrict__ segs,
                                                       uint8_t* __restrict__ codes,
                                                       float* __restrict__ scale,
                                                       float* __restrict__ vmom, CodebookDev cbd,
                                                       StepScalars sc)
{
    __shared__ LdsTables L;
    const Tile tl = tiles[blockIdx.x];
    const Seg sg = segs[tl.seg];
    foreign_tile<kThreads, CB>(L, tl, sg, codes, scale, vmom, cbd, sc);
}

// XCD-aware tile order. Workgroups are dispatched round-robin over the 8 XCDs, so
// workgroup b runs on XCD b % 8. Within every group of 8 * kXcdRun workgroups, XCD x
// takes kXcdRun consecutive tiles instead of every 8th one: four 32-byte descriptors
// share an L2 line and each XCD streams longer contiguous runs, while the round-robin
// over groups keeps every XCD's share of the work balanced. The trailing partial
// group keeps the identity order. A bijection on [0, n).
constexpr uint32_t kXcdRun = 8;
__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t n)
{
    constexpr uint32_t G = 8 * kXcdRun;
    if (b >= (n / G) * G) return b;
    const uint32_t base = (b / G) * G, r = b - base;
    return base + (r % 8) * kXcdRun + r / 8;
}

template <int GDT, int VPL, int BS, int CB>
__global__ __launch_bounds__(BS) void k_step_u(const Tile* __restrict__ tiles,
                                                     const Seg* __restrict__ segs,
                                                     uint8_t* __restrict__ codes,
                                                     float* __restrict__ scale,
                                                     float* __restrict__ vmom, CodebookDev cbd,
                                                     StepScalars sc)
{
    __shared__ LdsTables L;
    const Tile tl = tiles[xcd_tile(blockIdx.x, gridDim.x)];
    const Seg sg = segs[tl.seg];
    const uintptr_t galign = GDT == DT_F32 ? 15 : 7;
    const bool aligned = ((reinterpret_cast<uintptr_t>(sg.theta) & 15) == 0) &&
                         ((reinterpret_cast<uintptr_t>(sg.grad) & galign) == 0);
    if (aligned)
        step_u_body<GDT, VPL, BS, true, CB>(L, tl, sg, codes, scale, vmom, cbd, sc);
    else
        step_u_body<GDT, VPL, BS, false, CB>(L, tl, sg, codes, scale, vmom, cbd, sc);
}

// Streaming passes over the Span of one block (KIND_G: the whole block; KIND_H: one
// chunk). The reduce pass uses ordinary loads so that the update pass finds gradient and
// code lines in cache. Both passes evaluate the momentum with the same operations, so
// they agree bit for bit.
// HG: also the block's max |g| into *ag (for the histogram).
template <int GDT, int BS, int CB, int UNR = 2, bool HG = false>
__device__ __forceinline__ void pass_reduce(const LdsTables& L, const Seg& sg,
                                            const uint8_t* __restrict__ codes, const Span& sp,
                                            float s_old, const StepScalars& sc, float& ss,
                                            float& am, float* ag = nullptr)
{
    const int tid = threadIdx.x;
    const int64_t cj = sg.code_off;
    // batches of UNR vectors per thread, every load of a batch issued before its use
    for (int64_t v0 = sp.vb + tid; v0 < sp.ve; v0 += static_cast<int64_t>(BS) * UNR) {
        float g[UNR][4];
        uint32_t q4[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t v = v0 + static_cast<int64_t>(u) * BS;
            q4[u] = 0;
            g[u][0] = g[u][1] = g[u][2] = g[u][3] = 0.0f;
            if (v < sp.ve) {
                load_grad4<GDT>(sg, v, g[u]);
                q4[u] = code_ld4<CB>(codes, cj + 4 * v);
            }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const bool ok = v0 + static_cast<int64_t>(u) * BS < sp.ve;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float mm = ok ? momentum(L, code_get<CB>(q4[u], c), s_old, g[u][c], sc)
                                    : 0.0f;
                ss = fmaf(g[u][c], g[u][c], ss);
                am = fmaxf(am, fabsf(mm));
                if constexpr (HG) *ag = fmaxf(*ag, fabsf(g[u][c]));
            }
        }
    }
    for (int64_t i = tid; i < sp.nh + sp.nt; i += BS) {
        const int64_t e = i < sp.nh ? sp.start + i : sp.tail0 + (i - sp.nh);
        const float g = load_grad(sg.grad, e, GDT);
        const float mm = momentum(L, code_ld<CB>(codes, cj + e), s_old, g, sc);
        ss = fmaf(g, g, ss);
        am = fmaxf(am, fabsf(mm));
        if constexpr (HG) *ag = fmaxf(*ag, fabsf(g));
    }
}

// HG: also adds every element to the LDS histogram hl (block max |g| = ag; a block with
// ag = 0 adds nothing).
template <int GDT, int BS, int CB, int UNR = 2, bool HG = false>
__device__ __forceinline__ void pass_update(const LdsTables& L, const Seg& sg,
                                            uint8_t* __restrict__ codes, const Span& sp,
                                            float s_old, const BlockOut& bo,
                                            const StepScalars& sc, float half_ng, int ng_m1,
                                            uint32_t* hl = nullptr, float ag = 0.0f,
                                            double half_nb = 0.0, int nbins = 0)
{
    const int tid = threadIdx.x;
    float* __restrict__ th = sg.theta;
    const int64_t cj = sg.code_off;
    for (int64_t v0 = sp.vb + tid; v0 < sp.ve; v0 += static_cast<int64_t>(BS) * UNR) {
        float g[UNR][4];
        uint32_t q4[UNR];
        f32x4 t4[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t v = v0 + static_cast<int64_t>(u) * BS;
            if (v < sp.ve) {
                load_grad4<GDT>(sg, v, g[u]);
                q4[u] = code_ld4<CB>(codes, cj + 4 * v);
                t4[u] = __builtin_nontemporal_load(gl<f32x4>(th) + v);
            }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int64_t v = v0 + static_cast<int64_t>(u) * BS;
            if (v < sp.ve) {
                const float tv[4] = {t4[u].x, t4[u].y, t4[u].z, t4[u].w};
                float out[4];
                uint32_t packed = 0;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const float mm = momentum(L, code_get<CB>(q4[u], c), s_old, g[u][c], sc);
                    const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
                    packed |= static_cast<uint32_t>(q) << (CB * c);
                    out[c] = fmaf(-bo.r, mm, tv[c] * sc.decay);
                    if constexpr (HG)
                        if (ag > 0.0f) atomicAdd(&hl[hist_bin(g[u][c], ag, half_nb, nbins)], 1u);
                }
                const f32x4 o4 = {out[0], out[1], out[2], out[3]};
                __builtin_nontemporal_store(o4, glw<f32x4>(th) + v);
                code_st4<CB>(codes, cj + 4 * v, packed);
            }
        }
    }
    for (int64_t i = tid; i < sp.nh + sp.nt; i += BS) {
        const int64_t e = i < sp.nh ? sp.start + i : sp.tail0 + (i - sp.nh);
        const float g = load_grad(sg.grad, e, GDT);
        const int q0 = code_ld<CB>(codes, cj + e);
        const float mm = momentum(L, q0, s_old, g, sc);
        const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
        th[e] = fmaf(-bo.r, mm, th[e] * sc.decay);
        code_st<CB>(codes, cj + e, q0, q);
        if constexpr (HG)
            if (ag > 0.0f) atomicAdd(&hl[hist_bin(g, ag, half_nb, nbins)], 1u);
    }
}

// HG: *ag (max |g|) is reduced too.
template <int BS, bool HG = false>
__device__ __forceinline__ void wg_reduce(float& ss, float& am, LdsTables& L, float* ag = nullptr)
{
    for (int off = 1; off < 64; off <<= 1) {
        ss += __shfl_xor(ss, off);
        am = fmaxf(am, __shfl_xor(am, off));
        if constexpr (HG) *ag = fmaxf(*ag, __shfl_xor(*ag, off));
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        L.red_ss[wave] = ss;
        L.red_am[wave] = am;
        if constexpr (HG) L.red_ag[wave] = *ag;
    }
    __syncthreads();
    ss = L.red_ss[0];
    am = L.red_am[0];
    if constexpr (HG) *ag = L.red_ag[0];
    for (int w = 1; w < BS / 64; ++w) {
        ss += L.red_ss[w];
        am = fmaxf(am, L.red_am[w]);
        if constexpr (HG) *ag = fmaxf(*ag, L.red_ag[w]);
    }
    __syncthreads();
}

// Register runs inside the KIND_G launch (tile.vpl == 1): consecutive explicit blocks of
// kRunMinBlock .. kRunMaxElems elements, at most kRunMaxElems in all, taken by one
// workgroup with every element in registers (two 4-element vectors per thread, loaded
// before anything else), so nothing is read twice. A vector meets at most two blocks, so
// it keeps one partial (sum g^2, max |m|) for the block of its first element and one
// for the next; one wave per block then reduces them in a fixed order. Edge vectors
// (shared with neighbouring tiles) are loaded and stored element by element.
// HG (the step that also takes the histogram): the partials carry max |g| of both blocks
// as well, and every element goes into the LDS histogram hl at the end.
template <bool HG>
struct RunLdsT {
    int64_t start[kRunMaxBlocks + 1];   // tensor-relative block starts; start[nblk] = end
    float s_old[kRunMaxBlocks], v_old[kRunMaxBlocks];
    float s_new[kRunMaxBlocks], r[kRunMaxBlocks], inv_s[kRunMaxBlocks];
    float ag[HG ? kRunMaxBlocks : 1];
    float part[kRunMaxVec][HG ? 6 : 4];
};

template <int GDT, bool HG = false>
__device__ __forceinline__ void run_tile(LdsTables& L, RunLdsT<HG>& R, const Tile& tl,
                                         const Seg& sg, uint8_t* __restrict__ codes,
                                         float* __restrict__ scale, float* __restrict__ vmom,
                                         const CodebookDev& cbd, const StepScalars& sc,
                                         uint32_t* hl = nullptr, double half_nb = 0.0,
                                         int nbins = 0)
{
    const int tid = threadIdx.x;
    const int64_t e_lo = tl.elem0, e_hi = tl.elem0 + tl.nelem;
    const int64_t va = e_lo >> 2;
    const int nvec = static_cast<int>(((e_hi + 3) >> 2) - va);   // <= kRunMaxVec (planner)
    const int nb = tl.nblk;                                       // <= kRunMaxBlocks
    const bool aligned = vector_ok<GDT>(sg);
    float* __restrict__ th = sg.theta;
    const int64_t cj = sg.code_off;
    float tv[kRunVpl][4], gv[kRunVpl][4];
    uint32_t cq[kRunVpl];
#pragma unroll
    for (int j = 0; j < kRunVpl; ++j) {
        const int i = tid + j * kThreads;
        cq[j] = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) { tv[j][c] = 0.0f; gv[j][c] = 0.0f; }
        if (i < nvec) {
            const int64_t v = va + i;
            const int64_t e = 4 * v;
            if (aligned && e >= e_lo && e + 4 <= e_hi) {
                const f32x4 t4 = __builtin_nontemporal_load(gl<f32x4>(th) + v);
                tv[j][0] = t4.x; tv[j][1] = t4.y; tv[j][2] = t4.z; tv[j][3] = t4.w;
                load_grad4<GDT>(sg, v, gv[j]);
                cq[j] = *gl<uint32_t>(codes + cj + e);
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int64_t x = e + c;
                    if (x >= e_lo && x < e_hi) {
                        tv[j][c] = th[x];
                        gv[j][c] = load_grad(sg.grad, x, GDT);
                        cq[j] |= static_cast<uint32_t>(codes[cj + x]) << (8 * c);
                    }
                }
            }
        }
    }
    const int64_t local0 = tl.blk0 - sg.blk_begin;
    for (int k = tid; k <= nb; k += kThreads) R.start[k] = sg.csr[local0 + k];
    for (int k = tid; k < nb; k += kThreads) {
        R.s_old[k] = scale[tl.blk0 + k];
        R.v_old[k] = vmom[tl.blk0 + k];
    }
    load_tables(L, cbd);
    __syncthreads();
    int kb[kRunVpl];
    float gk[HG ? kRunVpl : 1][4];   // the gradients (gv becomes the momentum)
#pragma unroll
    for (int j = 0; j < kRunVpl; ++j) {
        const int i = tid + j * kThreads;
        kb[j] = 0;
        if constexpr (HG) {
#pragma unroll
            for (int c = 0; c < 4; ++c) gk[j][c] = gv[j][c];
        }
        if (i < nvec) {
            const int64_t e = 4 * (va + i);
            const int64_t first = e > e_lo ? e : e_lo;
            int lo = 0, hi = nb - 1;   // last block whose start <= first
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (R.start[mid] <= first) lo = mid; else hi = mid - 1;
            }
            kb[j] = lo;
            const int64_t next = R.start[lo + 1];
            float ssa = 0.0f, ama = 0.0f, ssb = 0.0f, amb = 0.0f, aga = 0.0f, agb = 0.0f;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t x = e + c;
                if (x >= e_lo && x < e_hi) {
                    const bool second = x >= next;   // then lo + 1 < nb
                    const float g = gv[j][c];
                    const float m = momentum(L, code_get<8>(cq[j], c),
                                             R.s_old[lo + (second ? 1 : 0)], g, sc);
                    gv[j][c] = m;
                    if (second) {
                        ssb = fmaf(g, g, ssb);
                        amb = fmaxf(amb, fabsf(m));
                        agb = fmaxf(agb, fabsf(g));
                    } else {
                        ssa = fmaf(g, g, ssa);
                        ama = fmaxf(ama, fabsf(m));
                        aga = fmaxf(aga, fabsf(g));
                    }
                }
            }
            R.part[i][0] = ssa;
            R.part[i][1] = ama;
            R.part[i][2] = ssb;
            R.part[i][3] = amb;
            if constexpr (HG) {
                R.part[i][4] = aga;
                R.part[i][5] = agb;
            }
        }
    }
    __syncthreads();
    const int wave = tid >> 6, lane = tid & 63;
    for (int k = wave; k < nb; k += kThreads / 64) {
        const int64_t bs = R.start[k], be = R.start[k + 1];
        const int i0 = static_cast<int>((bs >> 2) - va);
        const int i1 = static_cast<int>(((be - 1) >> 2) - va);
        float ss = 0.0f, am = 0.0f, ag = 0.0f;
        for (int i = i0 + lane; i <= i1; i += 64) {
            const int64_t e = 4 * (va + i);
            const bool own_first = (e > e_lo ? e : e_lo) >= bs;
            ss += own_first ? R.part[i][0] : R.part[i][2];
            am = fmaxf(am, own_first ? R.part[i][1] : R.part[i][3]);
            if constexpr (HG) ag = fmaxf(ag, own_first ? R.part[i][4] : R.part[i][5]);
        }
        for (int off = 1; off < 64; off <<= 1) {
            ss += __shfl_xor(ss, off);
            am = fmaxf(am, __shfl_xor(am, off));
            if constexpr (HG) ag = fmaxf(ag, __shfl_xor(ag, off));
        }
        if (lane == 0) {
            if constexpr (HG) R.ag[k] = ag;
            const BlockOut bo = finish_block(ss, am, R.v_old[k], static_cast<float>(be - bs), sc);
            scale[tl.blk0 + k] = bo.s_new;
            vmom[tl.blk0 + k] = bo.v_new;
            R.s_new[k] = bo.s_new;
            R.r[k] = bo.r;
            R.inv_s[k] = bo.inv_s;
        }
    }
    __syncthreads();
    const float half_ng = 0.5f * static_cast<float>(cbd.ng);
    const int ng_m1 = cbd.ng - 1;
#pragma unroll
    for (int j = 0; j < kRunVpl; ++j) {
        const int i = tid + j * kThreads;
        if (i >= nvec) continue;
        const int64_t v = va + i;
        const int64_t e = 4 * v;
        const int lo = kb[j];
        const int64_t next = R.start[lo + 1];
        uint32_t packed = 0;
        float out[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int k = lo + (e + c >= next ? 1 : 0);
            const int kk = k < nb ? k : nb - 1;   // lanes outside the run: any valid block
            const float m = gv[j][c];
            const int q = R.s_new[kk] > 0.0f ? encode(L, m * R.inv_s[kk], half_ng, ng_m1) : 0;
            packed |= static_cast<uint32_t>(q) << (8 * c);
            out[c] = fmaf(-R.r[kk], m, tv[j][c] * sc.decay);
            if constexpr (HG) {
                const int64_t x = e + c;
                if (x >= e_lo && x < e_hi && R.ag[k] > 0.0f)
                    atomicAdd(&hl[hist_bin(gk[j][c], R.ag[k], half_nb, nbins)], 1u);
            }
        }
        if (aligned && e >= e_lo && e + 4 <= e_hi) {
            const f32x4 o4 = {out[0], out[1], out[2], out[3]};
            __builtin_nontemporal_store(o4, glw<f32x4>(th) + v);
            code_st4<8>(codes, cj + e, packed);
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t x = e + c;
                if (x >= e_lo && x < e_hi) {
                    th[x] = out[c];
                    codes[cj + x] = static_cast<uint8_t>(packed >> (8 * c));
                }
            }
        }
    }
}

// KIND_G: one block per workgroup, any size and alignment: reduce pass, update pass;
// or a register run of short explicit blocks (tile.vpl == 1, 8-bit codes).
// HIST: the step that also takes the histogram of this step's gradients (Alg. 3): a
// persistent grid walks the tiles (tile blockIdx.x, + gridDim.x, ...), every element goes
// into an LDS histogram once its block's max |g| is known, and each workgroup adds its
// histogram to `hist` at the end (integer atomics: the sum does not depend on the order).
template <int GDT, int CB, bool HIST = false>
__global__ __launch_bounds__(kThreads) void k_step_g(const Tile* __restrict__ tiles,
                                                     const Seg* __restrict__ segs,
                                                     uint8_t* __restrict__ codes,
                                                     float* __restrict__ scale,
                                                     float* __restrict__ vmom, CodebookDev cbd,
                                                     StepScalars sc, int64_t n_tiles,
                                                     uint64_t* __restrict__ hist, int32_t nbins)
{
    __shared__ LdsTables L;
    __shared__ RunLdsT<HIST> R;
    __shared__ uint32_t H[HIST ? 16 * kMaxK : 1];
    const double half_nb = 0.5 * static_cast<double>(nbins);
    auto one = [&](const Tile& tl) {
        const Seg sg = segs[tl.seg];
        if (CB == 8 && tl.vpl == 1) {   // a register run (8-bit codes only)
            run_tile<GDT, HIST>(L, R, tl, sg, codes, scale, vmom, cbd, sc, H, half_nb, nbins);
            return;
        }
        const int64_t blk = tl.blk0;
        const Span sp = make_span<GDT>(sg, tl.elem0, tl.nelem);
        const float s_old = scale[blk];
        const float v_old = vmom[blk];
        load_tables(L, cbd);
        __syncthreads();
        float ss = 0.0f, am = 0.0f, ag = 0.0f;
        pass_reduce<GDT, kThreads, CB, 2, HIST>(L, sg, codes, sp, s_old, sc, ss, am, &ag);
        wg_reduce<kThreads, HIST>(ss, am, L, &ag);
        const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(tl.nelem), sc);
        if (threadIdx.x == 0) {
            scale[blk] = bo.s_new;
            vmom[blk] = bo.v_new;
        }
        pass_update<GDT, kThreads, CB, 2, HIST>(L, sg, codes, sp, s_old, bo, sc,
                                                0.5f * static_cast<float>(cbd.ng), cbd.ng - 1,
                                                H, ag, half_nb, nbins);
    };
    if constexpr (!HIST) {
        one(tiles[blockIdx.x]);
    } else {
        for (int i = threadIdx.x; i < nbins; i += kThreads) H[i] = 0;
        __syncthreads();
        for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
            one(tiles[t]);
            __syncthreads();   // the next tile reuses the LDS
        }
        for (int i = threadIdx.x; i < nbins; i += kThreads) {
            const uint32_t c = H[i];
            if (c) atomicAdd(reinterpret_cast<unsigned long long*>(&hist[i]),
                             static_cast<unsigned long long>(c));
        }
    }
}

// ---------------------------------------------------------------------------------
// KIND_L: up to 256 small blocks (<= 32 elements) per workgroup, one lane per block.
// ---------------------------------------------------------------------------------
template <int GDT, int CB>
__global__ __launch_bounds__(kThreads) void k_step_l(const Tile* __restrict__ tiles,
                                                     const Seg* __restrict__ segs,
                                                     uint8_t* __restrict__ codes,
                                                     float* __restrict__ scale,
                                                     float* __restrict__ vmom, CodebookDev cbd,
                                                     StepScalars sc)
{
    __shared__ LdsTables L;
    const Tile tl = tiles[blockIdx.x];
    const Seg sg = segs[tl.seg];
    load_tables(L, cbd);
    __syncthreads();
    const int bi = threadIdx.x;
    if (bi >= tl.nblk) return;
    int64_t start, len;
    block_range(sg, tl, bi, start, len);
    const int64_t blk = tl.blk0 + bi;
    float* __restrict__ th = sg.theta + start;
    const int64_t cj = sg.code_off + start;
    const void* gp =
        GDT == DT_F32 ? static_cast<const void*>(static_cast<const float*>(sg.grad) + start)
                      : static_cast<const void*>(static_cast<const uint16_t*>(sg.grad) + start);
    const float s_old = scale[blk];
    const float v_old = vmom[blk];
    float m[kSmallBlock];
    float ss = 0.0f, am = 0.0f;
#pragma unroll
    for (int i = 0; i < kSmallBlock; ++i) {
        m[i] = 0.0f;
        if (i < len) {
            const float g = load_grad(gp, i, GDT);
            m[i] = momentum(L, code_ld<CB>(codes, cj + i), s_old, g, sc);
            ss = fmaf(g, g, ss);
            am = fmaxf(am, fabsf(m[i]));
        }
    }
    const BlockOut bo = finish_block(ss, am, v_old, static_cast<float>(len), sc);
    scale[blk] = bo.s_new;
    vmom[blk] = bo.v_new;
    const float half_ng = 0.5f * static_cast<float>(cbd.ng);
    const int ng_m1 = cbd.ng - 1;
#pragma unroll
    for (int i = 0; i < kSmallBlock; ++i) {
        if (i < len) {
            const float mm = m[i];
            const int q = bo.s_new > 0.0f ? encode(L, mm * bo.inv_s, half_ng, ng_m1) : 0;
            th[i] = fmaf(-bo.r, mm, th[i] * sc.decay);
            code_st<CB>(codes, cj + i, code_ld<CB>(codes, cj + i), q);
        }
    }
}

// ---------------------------------------------------------------------------------
// KIND_H: chunks of huge blocks. Reduce: per-chunk (sum g^2, max |m|); chunk 0 also
// saves the block's old (s, v) so the update kernel can decode while chunk 0 of the
// update overwrites the state. Update: every chunk combines all partials of its block
// in chunk order (identical result in every chunk), recomputes m bit-identically and
// updates its chunk.
// ---------------------------------------------------------------------------------
template <int GDT, int CB>
__global__ __launch_bounds__(kThreads) void k_step_h_reduce(
    const Tile* __restrict__ tiles, const HTile* __restrict__ htiles, const Seg* __restrict__ segs,
    const uint8_t* __restrict__ codes, const float* __restrict__ scale,
    const float* __restrict__ vmom, CodebookDev cbd, StepScalars sc, float2* __restrict__ partials,
    float2* __restrict__ ws_old)
{
    __shared__ LdsTables L;
    const Tile tl = tiles[blockIdx.x];
    const HTile ht = htiles[blockIdx.x];
    const Seg sg = segs[tl.seg];
    const Span sp = make_span<GDT>(sg, tl.elem0, tl.nelem);
    const float s_old = scale[tl.blk0];
    load_tables(L, cbd);
    __syncthreads();
    float ss = 0.0f, am = 0.0f;
    pass_reduce<GDT, kThreads, CB>(L, sg, codes, sp, s_old, sc, ss, am);
    wg_reduce<kThreads>(ss, am, L);
    if (threadIdx.x == 0) {
        partials[ht.first + ht.chunk] = make_float2(ss, am);
        if (ht.chunk == 0) ws_old[ht.hb] = make_float2(s_old, vmom[tl.blk0]);
    }
}

template <int GDT, int CB>
__global__ __launch_bounds__(kThreads) void k_step_h_update(
    const Tile* __restrict__ tiles, const HTile* __restrict__ htiles, const Seg* __restrict__ segs,
    uint8_t* __restrict__ codes, float* __restrict__ scale, float* __restrict__ vmom,
    CodebookDev cbd, StepScalars sc, const float2* __restrict__ partials,
    const float2* __restrict__ ws_old)
{
    __shared__ LdsTables L;
    const Tile tl = tiles[blockIdx.x];
    const HTile ht = htiles[blockIdx.x];
    const Seg sg = segs[tl.seg];
    const int tid = threadIdx.x;
    const Span sp = make_span<GDT>(sg, tl.elem0, tl.nelem);
    const float2 old = ws_old[ht.hb];
    load_tables(L, cbd);
    // partials of the whole block, fixed order: thread t takes chunks t, t + 256, ...
    float ss = 0.0f, am = 0.0f;
    for (int c = tid; c < ht.nchunk; c += kThreads) {
        const float2 pa = partials[ht.first + c];
        ss += pa.x;
        am = fmaxf(am, pa.y);
    }
    __syncthreads();
    wg_reduce<kThreads>(ss, am, L);
    const BlockOut bo = finish_block(ss, am, old.y, static_cast<float>(ht.blk_len), sc);
    if (tid == 0 && ht.chunk == 0) {
        scale[tl.blk0] = bo.s_new;
        vmom[tl.blk0] = bo.v_new;
    }
    pass_update<GDT, kThreads, CB>(L, sg, codes, sp, old.x, bo, sc,
                                   0.5f * static_cast<float>(cbd.ng), cbd.ng - 1);
}

template <int GDT, int CB>
hipError_t launch_u(int vpl, int bs, dim3 grid, const Tile* tiles, const Seg* segs,
                    uint8_t* codes, float* scale, float* vmom, CodebookDev cb, StepScalars sc,
                    hipStream_t s)
{
#define GEFEN_U_CASE(V, B)                                                                  \
    if (vpl == V && bs == B) {                                                              \
        hipLaunchKernelGGL((k_step_u<GDT, V, B, CB>), grid, dim3(B), 0, s, tiles, segs,     \
                           codes, scale, vmom, cb, sc);                                     \
        return hipGetLastError();                                                           \
    }
    GEFEN_U_CASE(1, 256)
    GEFEN_U_CASE(2, 256)
    GEFEN_U_CASE(3, 256)
    GEFEN_U_CASE(4, 256)
    GEFEN_U_CASE(5, 256)
    GEFEN_U_CASE(6, 256)
    GEFEN_U_CASE(7, 256)
    GEFEN_U_CASE(8, 256)
    GEFEN_U_CASE(1, 512)
    GEFEN_U_CASE(2, 512)
    GEFEN_U_CASE(3, 512)
    GEFEN_U_CASE(4, 512)
    GEFEN_U_CASE(1, 1024)
    GEFEN_U_CASE(2, 1024)
    GEFEN_U_CASE(3, 1024)
    GEFEN_U_CASE(4, 1024)
#undef GEFEN_U_CASE
    return hipErrorInvalidValue;
}


template <int GDT, int CB>
hipError_t launch_h(dim3 grid, const Tile* tiles, const HTile* htiles, const Seg* segs,
                    uint8_t* codes, float* scale, float* vmom, CodebookDev cb, StepScalars sc,
                    float2* partials, float2* ws_old, hipStream_t stream)
{
    hipLaunchKernelGGL((k_step_h_reduce<GDT, CB>), grid, dim3(kThreads), 0, stream, tiles,
                       htiles, segs, codes, scale, vmom, cb, sc, partials, ws_old);
    hipLaunchKernelGGL((k_step_h_update<GDT, CB>), grid, dim3(kThreads), 0, stream, tiles,
                       htiles, segs, codes, scale, vmom, cb, sc, partials, ws_old);
    return hipGetLastError();
}

template <int GDT, int CB>
hipError_t launch_kind(int kind, int vpl, int bs, dim3 grid, const Tile* tiles,
                       const Seg* segs, uint8_t* codes, float* scale, float* vmom,
                       CodebookDev cb, StepScalars sc, hipStream_t stream)
{
    switch (kind) {
    case KIND_U:
        return launch_u<GDT, CB>(vpl, bs, grid, tiles, segs, codes, scale, vmom, cb, sc, stream);
    case KIND_G:
        hipLaunchKernelGGL((k_step_g<GDT, CB>), grid, dim3(kThreads), 0, stream, tiles, segs,
                           codes, scale, vmom, cb, sc, int64_t(grid.x),
                           static_cast<uint64_t*>(nullptr), 0);
        return hipGetLastError();
    case KIND_L:
        hipLaunchKernelGGL((k_step_l<GDT, CB>), grid, dim3(kThreads), 0, stream, tiles, segs,
                           codes, scale, vmom, cb, sc);
        return hipGetLastError();
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_step_h(int gdtype, int code_bits, const Tile* tiles, const HTile* htiles,
                         int64_t n_tiles, const Seg* segs, uint8_t* codes, float* scale,
                         float* vmom, CodebookDev cb, StepScalars sc, float2* partials,
                         float2* ws_old, hipStream_t stream)
{
    if (n_tiles <= 0) return hipSuccess;
    if (n_tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(n_tiles));
    if (code_bits == 8)
        return gdtype == DT_F32
                   ? launch_h<DT_F32, 8>(grid, tiles, htiles, segs, codes, scale, vmom, cb, sc,
                                         partials, ws_old, stream)
                   : launch_h<DT_BF16, 8>(grid, tiles, htiles, segs, codes, scale, vmom, cb, sc,
                                          partials, ws_old, stream);
    if (code_bits == 4)
        return gdtype == DT_F32
                   ? launch_h<DT_F32, 4>(grid, tiles, htiles, segs, codes, scale, vmom, cb, sc,
                                         partials, ws_old, stream)
                   : launch_h<DT_BF16, 4>(grid, tiles, htiles, segs, codes, scale, vmom, cb, sc,
                                          partials, ws_old, stream);
    return hipErrorInvalidValue;
}

hipError_t launch_step_g_hist(int gdtype, int code_bits, const Tile* tiles, int64_t n_tiles,
                              const Seg* segs, uint8_t* codes, float* scale, float* vmom,
                              CodebookDev cb, StepScalars sc, uint64_t* hist, int32_t nbins,
                              hipStream_t stream)
{
    if (n_tiles <= 0) return hipSuccess;
    if (nbins < 1 || nbins > 16 * kMaxK || (code_bits != 8 && code_bits != 4))
        return hipErrorInvalidValue;
    // as many workgroups as are resident at once (each adds its 16 k bins at its end)
#define GEFEN_GH(G, C)                                                                        \
    do {                                                                                      \
        static int resident = 0;                                                              \
        if (resident == 0) {                                                                  \
            int per_cu = 0, dev = 0, cus = 0;                                                 \
            if (hipOccupancyMaxActiveBlocksPerMultiprocessor(                                 \
                    &per_cu, k_step_g<G, C, true>, kThreads, 0) != hipSuccess ||              \
                hipGetDevice(&dev) != hipSuccess ||                                           \
                hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=    \
                    hipSuccess)                                                               \
                return hipErrorInvalidValue;                                                  \
            resident = std::max(1, per_cu) * std::max(1, cus);                                \
        }                                                                                     \
        const dim3 grid(static_cast<unsigned>(std::min<int64_t>(n_tiles, resident)));         \
        hipLaunchKernelGGL((k_step_g<G, C, true>), grid, dim3(kThreads), 0, stream, tiles,    \
                           segs, codes, scale, vmom, cb, sc, n_tiles, hist, nbins);           \
    } while (0)
    if (code_bits == 8) {
        if (gdtype == DT_F32) GEFEN_GH(DT_F32, 8); else GEFEN_GH(DT_BF16, 8);
    } else {
        if (gdtype == DT_F32) GEFEN_GH(DT_F32, 4); else GEFEN_GH(DT_BF16, 4);
    }
#undef GEFEN_GH
    return hipGetLastError();
}

hipError_t launch_step(int kind, int gdtype, int code_bits, int vpl, int bs, const Tile* tiles,
                       int64_t n_tiles, const Seg* segs, uint8_t* codes, float* scale,
                       float* vmom, CodebookDev cb, StepScalars sc, hipStream_t stream)
{
    if (n_tiles <= 0) return hipSuccess;
    if (n_tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    if (code_bits != 8 && code_bits != 4) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(n_tiles));
    if (kind == KIND_ANY) {
        if (code_bits == 8)
            hipLaunchKernelGGL(k_step_any<8>, grid, dim3(kThreads), 0, stream, tiles, segs,
                               codes, scale, vmom, cb, sc);
        else
            hipLaunchKernelGGL(k_step_any<4>, grid, dim3(kThreads), 0, stream, tiles, segs,
                               codes, scale, vmom, cb, sc);
        return hipGetLastError();
    }
    if (code_bits == 8)
        return gdtype == DT_F32
                   ? launch_kind<DT_F32, 8>(kind, vpl, bs, grid, tiles, segs, codes, scale, vmom,
                                            cb, sc, stream)
                   : launch_kind<DT_BF16, 8>(kind, vpl, bs, grid, tiles, segs, codes, scale,
                                             vmom, cb, sc, stream);
    return gdtype == DT_F32
               ? launch_kind<DT_F32, 4>(kind, vpl, bs, grid, tiles, segs, codes, scale, vmom, cb,
                                        sc, stream)
               : launch_kind<DT_BF16, 4>(kind, vpl, bs, grid, tiles, segs, codes, scale, vmom,
                                         cb, sc, stream);
}


}  // namespace gefen
