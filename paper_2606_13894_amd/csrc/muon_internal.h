// Gefen-Muon launchers (appendix "Gefen-Muon"): the quantized-momentum codec, the
// per-tensor Frobenius norm, the normalised bfloat16 Newton-Schulz input, the split-K
// sum, the 1 x n Newton-Schulz kernel and the parameter update.
#pragma once
#include "gefen_internal.h"

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
// x[b] = bf16(u of tensor tensor_of[b] / norm[tensor]), n elements in the tensor's own
// row-major layout
hipError_t launch_muon_prep(const uint16_t* u, const Seg* segs, const int32_t* tensor_of,
                            int32_t batch, const float* norm, int64_t n, uint16_t* x,
                            hipStream_t stream);
// Tall matrices (R > C > 1): x[b] (C x ldx row-major, ldx >= R, ldx % 8 == 0) =
// bf16(U^T / norm), U the R x C momentum matrix of tensor tensor_of[b], zero in
// columns R .. ldx - 1
hipError_t launch_muon_prep_t(const uint16_t* u, const Seg* segs, const int32_t* tensor_of,
                              int32_t batch, const float* norm, int64_t R, int64_t C,
                              int64_t ldx, uint16_t* x, hipStream_t stream);
// theta (R x C) of tensor_of[b] = theta * decay - step * O^T, O = o[b] (C x ldx)
hipError_t launch_muon_update_t(const uint16_t* o, const Seg* segs, const int32_t* tensor_of,
                                int32_t batch, int64_t R, int64_t C, int64_t ldx, float decay,
                                float step, hipStream_t stream);
// a (mm bfloat16) = bf16(sum of `splits` float32 partial products, in order)
hipError_t launch_muon_splitk_sum(const float* partial, int32_t splits, int64_t mm,
                                  uint16_t* a, hipStream_t stream);
// `steps` Newton-Schulz iterations in place on `batch` 1 x n bfloat16 rows
hipError_t launch_muon_ns_vec(uint16_t* x, int32_t batch, int64_t n, int32_t steps, float a,
                              float b, float c, hipStream_t stream);
// theta of tensor_of[b] = theta * decay - step * o[b], n elements, the tensor's layout
hipError_t launch_muon_update(const uint16_t* o, const Seg* segs, const int32_t* tensor_of,
                              int32_t batch, int64_t n, float decay, float step,
                              hipStream_t stream);

}  // namespace gefen
