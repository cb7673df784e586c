// Streaming ceiling of the step's access mix on this GPU: the bytes of one Gefen step
// (a float32 array read and written, a gradient array read, one code byte read and
// written per element) with none of its arithmetic, in one-shot tiles of 1024 elements
// (256 threads, one 16-byte parameter vector each) with non-temporal accesses -- the
// tile shape that measured fastest for this mix. Measurement support only.
#include "measure_internal.h"

namespace gefen {
namespace {

typedef float f32x4m __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2m __attribute__((ext_vector_type(2)));

template <int GDT>
__global__ __launch_bounds__(256) void k_stream_mix(float* __restrict__ theta,
                                                    const void* __restrict__ grad,
                                                    uint8_t* __restrict__ codes, int64_t n)
{
    const int64_t e = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 4;
    if (e + 4 <= n) {
        f32x4m t = __builtin_nontemporal_load(reinterpret_cast<const f32x4m*>(theta + e));
        float g0, g3;
        if (GDT == DT_F32) {
            const f32x4m g = __builtin_nontemporal_load(
                reinterpret_cast<const f32x4m*>(static_cast<const float*>(grad) + e));
            g0 = g.x;
            g3 = g.w;
        } else {
            const u32x2m g = __builtin_nontemporal_load(
                reinterpret_cast<const u32x2m*>(static_cast<const uint16_t*>(grad) + e));
            g0 = __uint_as_float(g.x << 16);
            g3 = __uint_as_float(g.y & 0xffff0000u);
        }
        const uint32_t c = __builtin_nontemporal_load(reinterpret_cast<const uint32_t*>(codes + e));
        t.x += g0;
        t.w += g3;
        __builtin_nontemporal_store(t, reinterpret_cast<f32x4m*>(theta + e));
        __builtin_nontemporal_store(c ^ 0x01010101u, reinterpret_cast<uint32_t*>(codes + e));
    } else {
        for (int64_t i = e; i < n; ++i) {
            const float g = GDT == DT_F32
                                ? static_cast<const float*>(grad)[i]
                                : __uint_as_float(static_cast<uint32_t>(
                                                      static_cast<const uint16_t*>(grad)[i])
                                                  << 16);
            theta[i] += g;
            codes[i] ^= 1u;
        }
    }
}

}  // namespace

hipError_t launch_stream_mix(float* theta, const void* grad, int gdtype, uint8_t* codes,
                             int64_t n, hipStream_t stream)
{
    if (n <= 0) return hipSuccess;
    const int64_t tiles = (n + 1023) / 1024;
    if (tiles > 0x7fffffffLL) return hipErrorInvalidValue;
    const dim3 grid(static_cast<unsigned>(tiles));
    if (gdtype == DT_F32)
        hipLaunchKernelGGL(k_stream_mix<DT_F32>, grid, dim3(256), 0, stream, theta, grad, codes,
                           n);
    else
        hipLaunchKernelGGL(k_stream_mix<DT_BF16>, grid, dim3(256), 0, stream, theta, grad, codes,
                           n);
    return hipGetLastError();
}

}  // namespace gefen
