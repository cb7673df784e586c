// Gefen-Muon launchers (appendix "Gefen-Muon"): the quantized-momentum codec, the
// per-tensor Frobenius norm, the 1 x n Newton-Schulz kernel, and the matrix-core
// Newton-Schulz products with the kernels that move matrices into and out of their layout.
#pragma once
#include "gefen_internal.h"
#include "ns_plan.h"

namespace gefen {

// Gefen-Muon. Codec tiles carry their mode in Tile::vpl (0: the workgroup on one block,
// 1: one lane per block, 2: one wave per block). u: bfloat16 momentum matrix at each
// element's code index; tile_ss: per-tile sum of u^2.
// All tiles must belong to tensors whose gradients have dtype gdtype.
hipError_t launch_muon_codec(int code_bits, int gdtype, const Tile* tiles, int64_t n_tiles,
                             const Seg* segs,
                             uint8_t* codes, float* scale, CodebookDev cb, float mu,
                             float one_minus_mu, int nesterov, uint16_t* u, float* tile_ss,
                             hipStream_t stream);
// norm[t] = max(bf16(sqrt(sum of tile_ss over [tile_range[2t], tile_range[2t+1]))), eps_bf16)
hipError_t launch_muon_norm(const float* tile_ss, const int64_t* tile_range, int32_t n_tensors,
                            float eps_bf16, float* norm, hipStream_t stream);
// `steps` Newton-Schulz iterations in place on `batch` 1 x n bfloat16 rows, row b at
// x + b * stride
hipError_t launch_muon_ns_vec(uint16_t* x, int32_t batch, int64_t n, int64_t stride, int32_t steps,
                              float a, float b, float c, hipStream_t stream);

// Newton-Schulz on the matrix cores (ns_gemm.hip; layout and products in ns_plan.h).
// One batched product (and, when split over K, the in-order sum of its chunks).
hipError_t launch_ns_gemm(const NsGemmArgs& a, hipStream_t stream);
// Batch entry b takes tensor t = tensor_of ? tensor_of[b] : b, whose R x C matrix starts at
// src + (src_off ? src_off[t] : b * R * C), divided by norm[t] (norm null: 1); writes
// copy[b] (R rows of cs >= C elements) = S / norm and trans[b] (C rows of ts >= R) =
// (S / norm)^T, zero padded, at batch strides copy_stride and trans_stride (elements; all
// four multiples of 8).
hipError_t launch_ns_prep(const uint16_t* src, const int64_t* src_off, const int32_t* tensor_of,
                          const float* norm, int32_t batch, int64_t R, int64_t C, uint16_t* copy,
                          int64_t copy_stride, int64_t cs, uint16_t* trans, int64_t trans_stride,
                          int64_t ts, hipStream_t stream);
// theta of tensor tensor_of[b] (R x C) = theta * decay - step * S[b], S[b] the R x C matrix
// of row stride ss at o + b * stride
hipError_t launch_ns_update(const uint16_t* o, int64_t stride, int64_t ss, const Seg* segs,
                            const int32_t* tensor_of, int32_t batch, int64_t R, int64_t C,
                            float decay, float step, hipStream_t stream);
// dst[b] (R x C, dense) = the R x C matrix of row stride ss at src + b * stride
hipError_t launch_ns_unpad(const uint16_t* src, int64_t stride, int64_t ss, int32_t batch,
                           int64_t R, int64_t C, uint16_t* dst, hipStream_t stream);

}  // namespace gefen
