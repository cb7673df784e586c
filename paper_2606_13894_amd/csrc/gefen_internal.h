// Internal declarations shared by the HIP sources of libgefen (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gefen {

// Gradient element types.
enum : int32_t { DT_F32 = 0, DT_BF16 = 1 };

// Work classes of the step kernels. Every tile belongs to exactly one class.
//  KIND_U  uniform blocks, p % 4 == 0, 16-byte aligned rows: groups of 2^lpb_log2 lanes
//          own one block each, every lane holds `vpl` 4-element vectors in registers.
//  KIND_G  any single block (irregular, unaligned, odd or very large p): the whole
//          workgroup streams it twice (reduce pass, then update pass).
//  KIND_L  up to 256 small blocks (<= 32 elements): one lane per block.
//  KIND_H  one chunk of a huge block: a reduce kernel writes per-chunk partials, an
//          update kernel combines the partials of the block (same fixed order in every
//          chunk) and updates its chunk, so a huge block spreads over many workgroups.
//  KIND_ANY small leftover tiles of any of the shapes above, one generic launch.
enum : int32_t { KIND_U = 0, KIND_G = 1, KIND_L = 2, KIND_H = 3, KIND_ANY = 4 };

constexpr int kThreads = 256;         // workgroup size of the streaming kernels
constexpr int kMaxThreads = 1024;     // largest KIND_U workgroup
constexpr int kMaxVpl = 8;            // max 4-element vectors per lane (KIND_U)
constexpr int kMaxLpbLog2 = 10;       // KIND_U lanes per block up to 1024
constexpr int kSmallBlock = 32;       // KIND_L blocks hold at most this many elements
constexpr int kMaxK = 256;            // max codebook entries
constexpr int64_t kHChunk = 8192;     // KIND_H chunk length

// One tile = the work of one workgroup (32 bytes).
struct Tile {
    int64_t elem0;      // first element of the tile, relative to its tensor
    int64_t blk0;       // global index of the tile's first block
    int64_t nelem;      // elements in the tile
    int32_t seg;        // tensor index
    int16_t nblk;       // blocks in the tile
    uint8_t vpl;        // KIND_U: vectors per lane
    uint8_t lpb_log2;   // KIND_U: log2(lanes per block); workgroup size is a class property
};
static_assert(sizeof(Tile) == 32, "Tile layout");

// KIND_H bookkeeping, one entry per tile (parallel to the tile array).
struct HTile {
    int64_t blk_len;     // elements of the whole block
    int64_t first;       // absolute tile index of the block's chunk 0 (chunks are
                         // consecutive tiles; partial arrays are indexed absolutely)
    int32_t nchunk;      // chunks of the block
    int32_t chunk;       // this tile's chunk index
    int32_t hb;          // index of the block among huge blocks (workspace slot)
    int32_t pad;
};
static_assert(sizeof(HTile) == 32, "HTile layout");

// Per-tensor descriptor on device (64 bytes). Pointers are refreshed when the caller
// passes different parameter or gradient buffers.
struct Seg {
    float* theta;             // parameters (fp32)
    const void* grad;         // gradients (fp32 or bf16)
    int64_t code_off;         // code index of the tensor's first code (a multiple of 32)
    int64_t period;           // > 0: uniform blocks of this size; 0: explicit blocks
    int64_t blk_begin;        // global index of the tensor's first block
    const int64_t* csr;       // explicit blocks: tensor-relative starts (n_blocks + 1)
    int64_t numel;
    int32_t gdtype;
    int32_t pad;
};
static_assert(sizeof(Seg) == 64, "Seg layout");

// Scalars of one step, computed on the host in float64 and rounded once.
struct StepScalars {
    float beta1, one_minus_beta1;
    float beta2, one_minus_beta2;
    float step_size;          // lr / (1 - beta1^t)
    float inv_bc2;            // 1 / (1 - beta2^t)
    float eps;
    float decay;              // 1 - lr * weight_decay
};

// Codebook tables used by the step: decode entries (fp32[k]) and, for encoding, the
// midpoints between consecutive entries (fp32[k], last unused) plus a guide table
// (uint8[ng + 1]) giving, per bucket of [-1, 1], the number of midpoints in lower
// buckets.
struct CodebookDev {
    const float* dec;
    const float* enc_mid;
    const uint8_t* enc_guide;
    int32_t k;
    int32_t ng;
};

// Histogram bin (Alg. 3) of gradient g in a block whose largest |g| is a > 0: the bin of
// x = g / a among nbins equal bins of [-1, 1], the last one closed; half_nb = nbins / 2.
// The defining evaluation is in float64, b = trunc((g / a + 1) * half_nb) (these sources
// are built with contraction off). Most elements take a float32 estimate instead,
// t = fma(g * rcp(a), h, h) with h = half_nb: the reciprocal is within 1 ulp and each of
// the two products rounds once, so |t - (g / a + 1) h| <= 2^-21.4 h, and float64 is within
// 2^-50 h. When t lies more than 2^-18 h from every integer (eight times the bound), the
// exact value and the float64 one share t's integer part, so the estimate's floor is
// the bin; otherwise (about 2^-17 h of all elements: 1.6 % at h = 2048), and for tiny
// or non-finite inputs, the float64 evaluation decides. Both histogram paths (the
// histogram kernel and the step kernels that take the histogram on the way) call this.
__device__ __forceinline__ int hist_bin(float g, float a, double half_nb, int nbins)
{
    const float h = static_cast<float>(half_nb);
    if (a >= 0x1p-100f && a <= 0x1p100f) {
        const float t = fmaf(g * __builtin_amdgcn_rcpf(a), h, h);
        const float fl = floorf(t);
        const float fr = t - fl;   // exact: t < 2^24
        const float d = h * 0x1p-18f;
        if (fr > d && fr < 1.0f - d) {
            const int b = static_cast<int>(fl);
            return b < nbins - 1 ? b : nbins - 1;
        }
    }
    const double x = static_cast<double>(g) / static_cast<double>(a);
    const int b = static_cast<int>((x + 1.0) * half_nb);
    return b < nbins - 1 ? b : nbins - 1;
}

// Launchers (all enqueue on `stream` and return the launch status).
// `bs` is the KIND_U workgroup size (256, 512 or 1024); other kinds use kThreads.
// `code_bits` is 8 (one code per byte) or 4 (two codes per byte, low nibble first);
// codes are addressed by code index Seg::code_off + element index.
hipError_t launch_step(int kind, int gdtype, int code_bits, int vpl, int bs, const Tile* tiles,
                       int64_t n_tiles, const Seg* segs, uint8_t* codes, float* scale,
                       float* vmom, CodebookDev cb, StepScalars sc, hipStream_t stream);

// KIND_H needs `htiles` (parallel to `tiles`), `partials` (float2 per tile) and
// `ws_old` (float2 per huge block).
hipError_t launch_step_h(int gdtype, int code_bits, const Tile* tiles, const HTile* htiles,
                         int64_t n_tiles, const Seg* segs, uint8_t* codes, float* scale,
                         float* vmom, CodebookDev cb, StepScalars sc, float2* partials,
                         float2* ws_old, hipStream_t stream);

// The KIND_G step of launch_step that also adds every element of its blocks to `hist`
// (uint64[nbins], accumulated into; Alg. 3 on this step's gradients). Persistent
// workgroups, each flushing one LDS histogram at its end.
hipError_t launch_step_g_hist(int gdtype, int code_bits, const Tile* tiles, int64_t n_tiles,
                              const Seg* segs, uint8_t* codes, float* scale, float* vmom,
                              CodebookDev cb, StepScalars sc, uint64_t* hist, int32_t nbins,
                              hipStream_t stream);

// Histogram over all tiles. KIND_H tiles need their block absmax first:
// launch_hist_h_absmax over each KIND_H class range writes am_partials[first + chunk].
hipError_t launch_hist_h_absmax(const Tile* tiles, const HTile* htiles, int64_t n_tiles,
                                const Seg* segs, float* am_partials, hipStream_t stream);
hipError_t launch_histogram(const Tile* tiles, int64_t n_tiles, const int32_t* tile_kind,
                            const HTile* htiles, const float* am_partials, const Seg* segs,
                            int32_t nbins, uint64_t* hist, hipStream_t stream);

// DP over a device histogram. ws must hold dp_workspace_bytes(nbins, k) bytes.
size_t dp_workspace_bytes(int32_t nbins, int32_t k);
hipError_t launch_dp(const uint64_t* hist, int32_t nbins, int32_t k, void* ws,
                     double* codebook_out, double* cost_out, int32_t* status_out,
                     hipStream_t stream);

// Install a float64 codebook into a slot: fp32 entries, fp64 copy, midpoints, guide.
hipError_t launch_install_codebook(const double* cb64_in, int32_t k, int32_t ng,
                                   float* cb32, double* cb64, float* mid, uint8_t* guide,
                                   hipStream_t stream);
// Same from an fp32 codebook (imports).
hipError_t launch_install_codebook_f32(const float* cb32_in, int32_t k, int32_t ng,
                                       float* cb32, double* cb64, float* mid,
                                       uint8_t* guide, hipStream_t stream);

// Block partitioning (Alg. 2) of several tensors.
struct PartDesc {              // one (tensor, divisor) pair
    const void* grad;
    int64_t n;                 // tensor numel
    int64_t p;                 // divisor
    int64_t item0;             // first work item of this pair
    int64_t n_items;           // work items of this pair
    int64_t out0;              // first partial-output slot
    int32_t gdtype;
    int32_t mode;              // 0: pairs of block means per item; 1: sub-chunk sums
    int32_t rpi;               // mode 0: block pairs per item; mode 1: sub-chunks per block
    int32_t pad;
};
hipError_t launch_partition(const PartDesc* descs, int32_t n_desc, int64_t n_items,
                            double eps, double* partials, double* scores,
                            const int32_t* tensor_first_desc, const int32_t* tensor_n_desc,
                            int32_t n_tensors, int64_t* periods, hipStream_t stream);

}  // namespace gefen
