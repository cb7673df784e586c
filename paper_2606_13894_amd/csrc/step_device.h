// Device helpers shared by the Gefen step kernels and the Gefen-Muon codec: the
// codebook tables in LDS (decode entries, encode midpoints, guide table), nearest-entry
// encoding, access to 8- and 4-bit momentum codes, the momentum and per-block scalar
// formulas of Alg. 1, block ranges and the vector/element split of a streamed range.
// Everything sits in an unnamed namespace: each translation unit gets its own copy.
#pragma once
#include "gefen_internal.h"

namespace gefen {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Pointers read from the tensor table are generic to the compiler, which then emits
// flat accesses (counted against both the memory and the LDS wait counters); these
// casts state that they point to global memory.
#define GEFEN_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const GEFEN_GLOBAL T* gl(const void* p)
{
    return (const GEFEN_GLOBAL T*)p;
}
template <typename T>
__device__ __forceinline__ GEFEN_GLOBAL T* glw(void* p)
{
    return (GEFEN_GLOBAL T*)p;
}

struct LdsTables {
    float cb[kMaxK];                  // decode entries
    float mid[kMaxK];                 // encode midpoints
    uint8_t guide[16 * kMaxK + 16];   // ng + 1 bytes (padded)
    float red_ss[kMaxThreads / 64];
    float red_am[kMaxThreads / 64];
    float red_ag[kMaxThreads / 64];   // max |g| (the step that also takes the histogram)
};

template <int BS = kThreads>
__device__ __forceinline__ void load_tables(LdsTables& L, const CodebookDev& cb)
{
    const int t = threadIdx.x;
    if (t < cb.k) {
        L.cb[t] = cb.dec[t];
        L.mid[t] = cb.enc_mid[t];
    }
    const int words = (cb.ng + 1 + 3) >> 2;   // the global guide is padded to 16 bytes
    const uint32_t* src = reinterpret_cast<const uint32_t*>(cb.enc_guide);
    uint32_t* dst = reinterpret_cast<uint32_t*>(L.guide);
    for (int i = t; i < words; i += BS) dst[i] = src[i];
}

// Nearest codebook entry of x (ties to the lower index) = number of midpoints < x.
__device__ __forceinline__ int encode(const LdsTables& L, float x, float half_ng, int ng_m1)
{
    x = fminf(fmaxf(x, -1.0f), 1.0f);
    int b = static_cast<int>((x + 1.0f) * half_ng);
    b = min(b, ng_m1);
    int q = L.guide[b];
    const int hi = L.guide[b + 1];
    while (q < hi && L.mid[q] < x) ++q;
    return q;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Momentum codes of CB bits (8 or 4), addressed by code index j = the tensor's code
// offset + element index. CB = 8: byte j. CB = 4: nibble j, i.e. byte j / 2, low half
// for even j, so four consecutive codes from j % 4 == 0 form one 16-bit word.
template <int CB>
__device__ __forceinline__ int code_ld(const uint8_t* codes, int64_t j)
{
    if (CB == 8) return codes[j];
    return (codes[j >> 1] >> (4 * (j & 1))) & 0xf;
}

// Scalar store of code j whose current value is `old`. With 4-bit codes the byte can be
// shared with a neighbouring block that another lane or workgroup updates at the same
// time, so the nibble changes by one atomic XOR (old ^ q) of its 32-bit word, which
// leaves every other nibble of the word as it is.
template <int CB>
__device__ __forceinline__ void code_st(uint8_t* codes, int64_t j, int old, int q)
{
    if (CB == 8) {
        codes[j] = static_cast<uint8_t>(q);
    } else if (old != q) {
        atomicXor(reinterpret_cast<unsigned int*>(codes) + (j >> 3),
                  static_cast<unsigned int>(old ^ q) << (4 * (j & 7)));
    }
}

// Codes j .. j + 3 (j % 4 == 0) packed CB bits apiece, lowest index in the lowest bits.
template <int CB>
__device__ __forceinline__ uint32_t code_ld4(const uint8_t* codes, int64_t j)
{
    if (CB == 8) return *gl<uint32_t>(codes + j);
    return *gl<uint16_t>(codes + (j >> 1));
}

template <int CB>
__device__ __forceinline__ void code_st4(uint8_t* codes, int64_t j, uint32_t w)
{
    if (CB == 8)
        __builtin_nontemporal_store(w, glw<uint32_t>(codes + j));
    else
        __builtin_nontemporal_store(static_cast<uint16_t>(w), glw<uint16_t>(codes + (j >> 1)));
}

template <int CB>
__device__ __forceinline__ int code_get(uint32_t w, int c)
{
    return static_cast<int>((w >> (CB * c)) & ((1u << CB) - 1));
}

__device__ __forceinline__ float momentum(const LdsTables& L, int q, float s_old, float g,
                                          const StepScalars& sc)
{
    return fmaf(sc.beta1, L.cb[q] * s_old, sc.one_minus_beta1 * g);
}

__device__ __forceinline__ float load_grad(const void* base, int64_t i, int gdt)
{
    if (gdt == DT_F32) return static_cast<const float*>(base)[i];
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(base)[i]) << 16);
}

// Block-local scalars after the reductions.
struct BlockOut {
    float s_new, v_new, r, inv_s;
};

__device__ __forceinline__ BlockOut finish_block(float ss, float am, float v_old, float count,
                                                 const StepScalars& sc)
{
    BlockOut o;
    o.s_new = am;
    o.v_new = fmaf(sc.beta2, v_old, sc.one_minus_beta2 * (ss / count));
    const float denom = sqrtf(o.v_new * sc.inv_bc2) + sc.eps;
    o.r = sc.step_size / denom;
    o.inv_s = am > 0.0f ? 1.0f / am : 0.0f;
    return o;
}

// ---------------------------------------------------------------------------------
// Block range of block `bi` of a tile (tensor-relative start, length).
// ---------------------------------------------------------------------------------
__device__ __forceinline__ void block_range(const Seg& sg, const Tile& tl, int bi,
                                            int64_t& start, int64_t& len)
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

// ---------------------------------------------------------------------------------
// Span of a streamed element range [start, start + len) of one block. When the tensor's
// parameter and gradient pointers allow it, the 4-element-aligned body of the range
// moves with 128-bit (parameters, fp32 gradients), 64-bit (bf16 gradients) and 32-bit
// (4 codes) accesses; the head and tail (at most 3 elements each) go element by element.
// ---------------------------------------------------------------------------------
template <int GDT>
__device__ __forceinline__ bool vector_ok(const Seg& sg)
{
    const uintptr_t galign = GDT == DT_F32 ? 15 : 7;
    return ((reinterpret_cast<uintptr_t>(sg.theta) & 15) == 0) &&
           ((reinterpret_cast<uintptr_t>(sg.grad) & galign) == 0);
}

template <int GDT>
__device__ __forceinline__ void load_grad4(const Seg& sg, int64_t v, float g[4])
{
    if (GDT == DT_F32) {
        const f32x4 x = gl<f32x4>(sg.grad)[v];
        g[0] = x.x; g[1] = x.y; g[2] = x.z; g[3] = x.w;
    } else {
        const u32x2 x = gl<u32x2>(sg.grad)[v];
        g[0] = bf16_lo(x.x); g[1] = bf16_hi(x.x); g[2] = bf16_lo(x.y); g[3] = bf16_hi(x.y);
    }
}

struct Span {
    int64_t vb, ve;   // vector body [vb, ve) in vector units (4 elements)
    int64_t start, nh, hb_end, tail0, nt;
};

template <int GDT>
__device__ __forceinline__ Span make_span(const Seg& sg, int64_t start, int64_t len)
{
    const int64_t end = start + len;
    int64_t b = end, e = end;
    if (vector_ok<GDT>(sg)) {
        b = (start + 3) & ~int64_t(3);
        e = end & ~int64_t(3);
        if (b > end) b = end;
        if (e < b) e = b;
    }
    Span sp;
    sp.vb = b >> 2;
    sp.ve = e >> 2;
    sp.start = start;
    sp.nh = b - start;
    sp.tail0 = e;
    sp.nt = end - e;
    sp.hb_end = b;
    return sp;
}

}  // namespace
}  // namespace gefen
