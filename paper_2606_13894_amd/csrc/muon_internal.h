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
// x[b] = bf16(u of tensor tensor_of[b] / norm), R x C, transposed to C x R when R > C
hipError_t launch_muon_prep(const uint16_t* u, const Seg* segs, const int32_t* tensor_of,
                            int32_t batch, const float* norm, int64_t R, int64_t C,
                            uint16_t* x, hipStream_t stream);
// a (mm bfloat16) = bf16(sum of `splits` float32 partial products, in order)
hipError_t launch_muon_splitk_sum(const float* partial, int32_t splits, int64_t mm,
                                  uint16_t* a, hipStream_t stream);
// `steps` Newton-Schulz iterations in place on `batch` 1 x n bfloat16 rows
hipError_t launch_muon_ns_vec(uint16_t* x, int32_t batch, int64_t n, int32_t steps, float a,
                              float b, float c, hipStream_t stream);
// theta of tensor_of[b] = theta * decay - step * o[b] (o in the orientation of x)
hipError_t launch_muon_update(const uint16_t* o, const Seg* segs, const int32_t* tensor_of,
                              int32_t batch, int64_t R, int64_t C, float decay, float step,
                              hipStream_t stream);

}  // namespace gefen
