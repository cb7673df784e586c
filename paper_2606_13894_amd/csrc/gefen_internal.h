// Internal declarations shared by the HIP sources of libgefen (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tile_plan.h"

namespace gefen {

// Kernel classes, tiles and the planner: tile_plan.h (host-only, shared with the
// host tests).


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
// Evaluated in float64 (these sources are built with contraction off), so that the
// histogram kernel and the step kernels that take the histogram on the way bin every
// element identically. (A float32 estimate with a float64 evaluation near bin edges
// measured slower in both kernels: a wave almost always holds some lane near an edge.)
__device__ __forceinline__ int hist_bin(float g, float a, double half_nb, int nbins)
{
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
