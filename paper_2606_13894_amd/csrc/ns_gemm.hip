// Newton-Schulz products of Gefen-Muon (appendix "Gefen-Muon") on the CDNA4 matrix
// cores, and the kernels that bring the momentum matrices into and out of their layout
// (ns_plan.h gives the layout and the three products of an iteration).
//
// The product kernel: one workgroup computes a 128 x 128 or 256 x 256 output tile of one
// batch entry (and one K chunk when split). At 128, four waves (two workgroups per CU)
// own quarters of 2 x 2 v_mfma_f32_32x32x16_bf16 accumulators (float32); at 256, eight
// waves (one workgroup per CU, two waves per SIMD) own eighths of 2 x 4 accumulators, which
// needs 6 fragment reads per 8 matrix-core ops where a quarter of 4 x 4 per wave would
// leave one wave per SIMD (measured 8-14 % slower on the model shapes). Both operands are
// read along contiguous K through buffer resources, 16 bytes per thread, into LDS tiles of
// 64 K per row (rows padded to 72 elements so that the 16-byte fragment reads of 16
// consecutive rows hit distinct banks); two LDS stages in a software pipeline: the next
// stage's global loads are in flight while the current one feeds the matrix cores, each
// K step's fragments are read during the previous step's MFMAs, one barrier per stage.
// The epilogue forms alpha * C + beta * E in float32 and rounds once to bfloat16 (round to
// nearest even, as the float32-accumulating GEMMs of the implementation the paper uses),
// through one LDS tile in the transposed orientation, so that E is read and O and the
// transposed output (or, for the symmetric products, the mirror) are written as 16-byte
// row segments; the 128 tile loads its E rows during the last stage. Work items are dealt
// to the eight XCDs in contiguous runs, so the tiles of one batch entry share an XCD's L2.
#include "muon_internal.h"
#include "ns_plan.h"

namespace gefen {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4v __attribute__((ext_vector_type(4)));

constexpr int BK = kNsBK;
constexpr int kNsBigWaves = 8;   // waves of the 256 x 256 tile's workgroup
constexpr int LDK = BK + 8;      // LDS row stride of the operand tiles (elements)

__device__ __forceinline__ float bf16_val(uint16_t b)
{
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float32 -> bfloat16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t to_bf16(float x)
{
    const uint32_t b = __float_as_uint(x);
    if ((b & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((b >> 16) | 0x40u);
    return static_cast<uint16_t>((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

// Element j (0..7) of eight packed bfloat16.
__device__ __forceinline__ uint32_t bf16_at(const u32x4& w, int j)
{
    const uint32_t v = w[j >> 1];
    return (j & 1) ? (v >> 16) : (v & 0xffffu);
}

// A (64 W) x (64 W) output tile computed by NW waves (4 or 8) in a grid of NW / 2 x 2:
// each wave owns MI x NI accumulator blocks of 32 x 32 (MI = NI = W with four waves;
// MI = W / 2, NI = W with eight, so that a wave's fragment reads per matrix-core op drop
// from 1 to 3/4 of a 16-byte read at the 256 tile and two waves share each SIMD).
template <int W, int NW = 4>
struct NsTileShape {
    static constexpr int T = 64 * W;               // tile rows and columns
    static constexpr int kThreads = 64 * NW;
    static constexpr int WR = NW / 2;              // wave rows (along M); two wave columns
    static constexpr int MI = T / (32 * WR), NI = T / 64;
    static constexpr int LDT = T + 8;              // LDS row stride of the epilogue tiles
    static constexpr int kStage = 2 * T * LDK;     // both operand tiles of one stage
    static constexpr int kLds = 2 * kStage > T * LDT ? 2 * kStage : T * LDT;
    static constexpr int kRowsPerPass = kThreads / 8;   // 64-element rows loaded per pass
    static constexpr int kPasses = T / kRowsPerPass;
    static constexpr int kSRows = kThreads / 16;   // epilogue tile rows per pass
    static constexpr int kEPasses = T / kSRows;
};

// The E^T tile rows a thread moves into the epilogue's LDS tile: pass p of half h is
// tile row p * kSRows + tid / 16, columns h * 128 + (tid % 16) * 8 .. + 7 (zero beyond N
// rows and lde columns; E^T rows are zero beyond M up to lde, a multiple of 8).
template <int W, int NW>
__device__ __forceinline__ void load_et(const NsGemmArgs& a, const NsWork& w, int tid,
                                        u32x4 (&e)[W / 2][NsTileShape<W, NW>::kEPasses])
{
    using S = NsTileShape<W, NW>;
    constexpr int T = S::T;
    const int64_t row0 = int64_t(w.ti) * T, col0 = int64_t(w.tj) * T;
    const uint16_t* __restrict__ Et = a.et + w.b * a.se;
    const int srow = tid >> 4, scol = (tid & 15) * 8;
#pragma unroll
    for (int half = 0; half < T / 128; ++half)
#pragma unroll
        for (int pass = 0; pass < S::kEPasses; ++pass) {
            const int64_t j = col0 + pass * S::kSRows + srow, i = row0 + half * 128 + scol;
            const u32x4 z = {0u, 0u, 0u, 0u};
            e[half][pass] =
                (j < a.N && i < a.lde) ? *reinterpret_cast<const u32x4*>(Et + j * a.lde + i) : z;
        }
}

// Epilogue through one LDS tile in the E^T / O^T orientation (rows j, columns i), so that
// every global access is a 16-byte row segment: (1) the E^T tile as stored; (2) each lane
// turns its accumulators into bfloat16 results in place, over the E^T elements of the
// same positions (8 bytes: four consecutive i); (3) the tile's rows are the rows of O^T
// (or of the mirror); (4) the rows of O come from 8 x 8 blocks of the tile transposed in
// registers. pre: the E^T rows of this thread (load_et), loaded during the last stage;
// null: loaded here.
template <int W, int NW>
__device__ __forceinline__ void epilogue(
    const NsGemmArgs& a, const NsWork& w,
    const f32x16 (&acc)[NsTileShape<W, NW>::MI][NsTileShape<W, NW>::NI], uint16_t* lds,
    int tid, const u32x4 (*pre)[NsTileShape<W, NW>::kEPasses] = nullptr)
{
    using S = NsTileShape<W, NW>;
    constexpr int T = S::T, LDT = S::LDT, MI = S::MI, NI = S::NI;
    const int64_t row0 = int64_t(w.ti) * T, col0 = int64_t(w.tj) * T;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * (32 * MI), wn = (wave & 1) * (32 * NI);
    const int frow = lane & 31, fk = (lane >> 5) * 8;

    const bool Et = a.et != nullptr;
    uint16_t* __restrict__ Ot = a.ot ? a.ot + w.b * a.sot : nullptr;
    const bool mirror = Ot && (!a.sym || w.ti != w.tj);
    const int srow = tid >> 4, scol = (tid & 15) * 8;
    if (Et) {
        u32x4 e[W / 2][S::kEPasses];
        if (pre) {
#pragma unroll
            for (int half = 0; half < T / 128; ++half)
#pragma unroll
                for (int pass = 0; pass < S::kEPasses; ++pass) e[half][pass] = pre[half][pass];
        } else {
            load_et<W, NW>(a, w, tid, e);
        }
#pragma unroll
        for (int half = 0; half < T / 128; ++half)
#pragma unroll
            for (int pass = 0; pass < S::kEPasses; ++pass)
                *reinterpret_cast<u32x4*>(lds + (pass * S::kSRows + srow) * LDT + half * 128 +
                                          scol) = e[half][pass];
        __syncthreads();
    }
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
            const int lc = wn + ni * 32 + frow;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int lr = wm + mi * 32 + g * 8 + fk / 2;
                u32x2* cell = reinterpret_cast<u32x2*>(lds + lc * LDT + lr);
                float e[4] = {0.0f, 0.0f, 0.0f, 0.0f};
                if (Et) {
                    const u32x2 ev = *cell;
                    e[0] = bf16_val(static_cast<uint16_t>(ev.x & 0xffffu));
                    e[1] = bf16_val(static_cast<uint16_t>(ev.x >> 16));
                    e[2] = bf16_val(static_cast<uint16_t>(ev.y & 0xffffu));
                    e[3] = bf16_val(static_cast<uint16_t>(ev.y >> 16));
                }
                uint32_t h[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    h[q] = to_bf16(fmaf(a.alpha, acc[mi][ni][g * 4 + q], a.beta * e[q]));
                u32x2 hv;
                hv.x = h[0] | (h[1] << 16);
                hv.y = h[2] | (h[3] << 16);
                *cell = hv;
            }
        }
    __syncthreads();
    if (mirror) {
#pragma unroll
        for (int half = 0; half < T / 128; ++half)
#pragma unroll
            for (int pass = 0; pass < S::kEPasses; ++pass) {
                const int r = pass * S::kSRows + srow, c = half * 128 + scol;
                const int64_t j = col0 + r, i = row0 + c;
                if (j < a.N && i < a.ot_cols)
                    *reinterpret_cast<u32x4*>(Ot + j * a.ldot + i) =
                        *reinterpret_cast<const u32x4*>(lds + r * LDT + c);
            }
    }
    if (a.o) {
        constexpr int NB = T / 8;   // 8 x 8 blocks along a side
        uint16_t* __restrict__ O = a.o + w.b * a.so;
#pragma unroll
        for (int q = 0; q < NB * NB / S::kThreads; ++q) {
            const int blk = q * S::kThreads + tid;
            const int bj = blk % NB, bi = blk / NB;
            u32x4 rv[8];   // tile rows j = 8 bj .. + 7, columns i = 8 bi .. + 7
#pragma unroll
            for (int jj = 0; jj < 8; ++jj)
                rv[jj] = *reinterpret_cast<const u32x4*>(lds + (bj * 8 + jj) * LDT + bi * 8);
            const int64_t j = col0 + bj * 8;
#pragma unroll
            for (int ii = 0; ii < 8; ++ii) {
                const int64_t i = row0 + bi * 8 + ii;
                if (i < a.M && j < a.o_cols) {
                    u32x4 o;
#pragma unroll
                    for (int p = 0; p < 4; ++p)
                        o[p] = bf16_at(rv[2 * p], ii) | (bf16_at(rv[2 * p + 1], ii) << 16);
                    *reinterpret_cast<u32x4*>(O + i * a.ldo + j) = o;
                }
            }
        }
    }
}

template <int W, bool SPLIT, int NW = 4>
__global__ __launch_bounds__(64 * NW, W == 2 ? 2 : 1) void k_ns_gemm(const NsGemmArgs a)
{
    using S = NsTileShape<W, NW>;
    constexpr int T = S::T, LDT = S::LDT, NP = S::kPasses, MI = S::MI, NI = S::NI;
    constexpr int RP = S::kRowsPerPass;
    __shared__ __attribute__((aligned(16))) uint16_t lds[S::kLds];
    const int64_t total = int64_t(a.batch) * a.splits * a.tiles;
    const int64_t per_xcd = (total + 7) / 8;
    const int64_t wid = static_cast<int64_t>(blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (wid >= total) return;
    const NsWork w = ns_decode(a, wid);
    const int64_t row0 = int64_t(w.ti) * T, col0 = int64_t(w.tj) * T;
    const int64_t kbeg = int64_t(w.s) * a.kchunk;
    const int64_t kend = SPLIT ? min(int64_t(a.K), kbeg + a.kchunk) : int64_t(a.K);

    // Operands through buffer resources over the tile's own rows of this batch entry,
    // ending at row M (N): the hardware returns zero for a load whose vector offset (the
    // lane's row, its row pass and K position) lies past the range, so the loads need no
    // predicates (K is a whole number of stages). The stage's K offset is uniform.
    const int64_t prow = min(int64_t(T), int64_t(a.M) - row0);
    const int64_t qrow = min(int64_t(T), int64_t(a.N) - col0);
    const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.p + w.b * a.sp + row0 * a.ldp), 0,
        static_cast<int>(2 * prow * a.ldp), 0x00020000);
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.q + w.b * a.sq + col0 * a.ldq), 0,
        static_cast<int>(2 * qrow * a.ldq), 0x00020000);
    const int ldp = static_cast<int>(a.ldp), ldq = static_cast<int>(a.ldq);

    const int tid = threadIdx.x;
    const int lrow = tid >> 3, lk = (tid & 7) * 8;   // loader: 8 threads per 64-element row
    const int vp = 2 * (lrow * ldp + lk), vq = 2 * (lrow * ldq + lk);
    u32x4 ra[NP], rb[NP];
    auto gload = [&](int k0) {
#pragma unroll
        for (int r = 0; r < NP; ++r) {
            ra[r] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                  rp, vp + 2 * RP * r * ldp, 2 * k0, 0));
            rb[r] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                  rq, vq + 2 * RP * r * ldq, 2 * k0, 0));
        }
    };
    auto lstore = [&](int buf) {
        uint16_t* sa = lds + buf * S::kStage;
        uint16_t* sb = sa + T * LDK;
#pragma unroll
        for (int r = 0; r < NP; ++r) {
            *reinterpret_cast<u32x4*>(sa + (lrow + RP * r) * LDK + lk) = ra[r];
            *reinterpret_cast<u32x4*>(sb + (lrow + RP * r) * LDK + lk) = rb[r];
        }
    };

    const int lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * (32 * MI), wn = (wave & 1) * (32 * NI);
    const int frow = lane & 31, fk = (lane >> 5) * 8;
    f32x16 acc[MI][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mi][ni][v] = 0.0f;

    // The fragments of one 16-wide K step: rows of the wave's A and B blocks.
    typedef bf16x8 FragA[MI];
    typedef bf16x8 FragB[NI];
    auto frags = [&](FragA& fa, FragB& fb, int buf, int kk) {
        const uint16_t* sa = lds + buf * S::kStage;
        const uint16_t* sb = sa + T * LDK;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
            fa[mi] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(sa + (wm + mi * 32 + frow) * LDK + kk + fk));
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
            fb[ni] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(sb + (wn + ni * 32 + frow) * LDK + kk + fk));
    };
    auto mfmas = [&](const FragA& fa, const FragB& fb, int from, int to) {
#pragma unroll
        for (int q = from; q < to; ++q)
            acc[q / NI][q % NI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                fa[q / NI], fb[q % NI], acc[q / NI][q % NI], 0, 0, 0);
    };
    // Scheduling groups (instruction classes of __builtin_amdgcn_sched_group_barrier):
    // `n` matrix-core ops, each followed by `per` ops of class `mask`.
    constexpr int kMfma = 0x008, kDsRead = 0x100, kDsWrite = 0x200, kVmemRead = 0x020;
    constexpr int kMM = MI * NI;               // MFMAs of one K step
    constexpr int kFr = MI + NI;               // fragment reads of one K step
    constexpr int kWr = 2 * NP;                // LDS writes of one stage

    // One stage in a software pipeline: the next stage's global loads go out first; each
    // K step's matrix-core ops run while the next step's fragments are read from LDS; the
    // next stage goes into the other LDS buffer during the third step, and after a
    // barrier in the middle of the fourth step the next stage's first fragments are read.
    FragA fa, na;
    FragB fb, nb;
    const int nk = static_cast<int>((kend - kbeg) / BK);
    gload(static_cast<int>(kbeg));
    lstore(0);
    __syncthreads();
    frags(fa, fb, 0, 0);
    // Fragment reads against matrix-core ops inside one K step. With W = 2 a step has
    // only four MFMAs, so all of the next step's reads go out before them (their own
    // registers; reads placed between the MFMAs would reuse the current fragments'
    // registers and reach the next step's first MFMA too late); with W = 4 they go out
    // one per MFMA over the first half of the step.
    auto step_groups = [&]() {
        if constexpr (W == 2) {
            __builtin_amdgcn_sched_group_barrier(kDsRead, kFr, 0);
            __builtin_amdgcn_sched_group_barrier(kMfma, kMM, 0);
        } else {
#pragma unroll
            for (int q = 0; q < kFr; ++q) {
                __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kMfma, kMM - kFr, 0);
        }
    };
    auto advance = [&]() {
#pragma unroll
        for (int q = 0; q < MI; ++q) fa[q] = na[q];
#pragma unroll
        for (int q = 0; q < NI; ++q) fb[q] = nb[q];
    };
    for (int it = 0; it + 1 < nk; ++it) {
        const int cur = it & 1;
        gload(static_cast<int>(kbeg) + (it + 1) * BK);
        __builtin_amdgcn_sched_group_barrier(kVmemRead, kWr, 0);
        // steps 0 and 1
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            frags(na, nb, cur, (ks + 1) * 16);
            mfmas(fa, fb, 0, kMM);
            step_groups();
            advance();
        }
        // step 2: the last fragments of this stage, the next stage into LDS
        frags(na, nb, cur, 48);
        lstore(cur ^ 1);
        mfmas(fa, fb, 0, kMM);
        if constexpr (W == 2) {
            __builtin_amdgcn_sched_group_barrier(kDsRead, kFr, 0);
#pragma unroll
            for (int q = 0; q < kMM; ++q) {
                __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kDsWrite, kWr / kMM, 0);
            }
            // step 3: the barrier first, then the next stage's first fragments before
            // this step's MFMAs
            __syncthreads();
            frags(fa, fb, cur ^ 1, 0);
            mfmas(na, nb, 0, kMM);
            __builtin_amdgcn_sched_group_barrier(kDsRead, kFr, 0);
            __builtin_amdgcn_sched_group_barrier(kMfma, kMM, 0);
        } else {
#pragma unroll
            for (int q = 0; q < kMM; ++q) {
                __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
                if (q < kFr) __builtin_amdgcn_sched_group_barrier(kDsRead, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kDsWrite, (kWr + kMM - 1) / kMM, 0);
            }
            // step 3: half its MFMAs, the barrier, then the next stage's first fragments
            // under the other half
            mfmas(na, nb, 0, kMM / 2);
            __builtin_amdgcn_sched_group_barrier(kMfma, kMM / 2, 0);
            __syncthreads();
            frags(fa, fb, cur ^ 1, 0);
            mfmas(na, nb, kMM / 2, kMM);
#pragma unroll
            for (int q = 0; q < kMM / 2; ++q) {
                __builtin_amdgcn_sched_group_barrier(kMfma, 1, 0);
                __builtin_amdgcn_sched_group_barrier(kDsRead, (2 * kFr + kMM - 1) / kMM, 0);
            }
        }
    }
    // The 128 tile loads the epilogue's E^T rows during the last stage, so their latency
    // hides behind its matrix-core ops (the 256 tile has no registers to spare for them).
    constexpr bool kPrefetchE = !SPLIT && W == 2;
    u32x4 epre[W / 2][S::kEPasses];
    {   // the last stage
        const int cur = (nk - 1) & 1;
        if constexpr (kPrefetchE)
            if (a.et) load_et<W, NW>(a, w, tid, epre);
#pragma unroll
        for (int ks = 0; ks < 3; ++ks) {
            frags(na, nb, cur, (ks + 1) * 16);
            mfmas(fa, fb, 0, kMM);
            step_groups();
            advance();
        }
        mfmas(fa, fb, 0, kMM);
    }
    __syncthreads();   // the epilogue reuses the LDS

    // Accumulator element v of block (mi, ni): row (v / 4) * 8 + (lane / 32) * 4 + v % 4,
    // column lane % 32 of the 32 x 32 block.
    if constexpr (SPLIT) {
        float* __restrict__ part = a.partial + ((int64_t(w.s) * a.batch + w.b) * a.M) * a.N;
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
#pragma unroll
            for (int ni = 0; ni < NI; ++ni) {
                const int64_t j = col0 + wn + ni * 32 + frow;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int64_t i = row0 + wm + mi * 32 + (v >> 2) * 8 + fk / 2 + (v & 3);
                    if (i < a.M && j < a.N) part[i * a.N + j] = acc[mi][ni][v];
                }
            }
    } else {
        if constexpr (kPrefetchE)
            epilogue<W, NW>(a, w, acc, lds, tid, a.et ? epre : nullptr);
        else
            epilogue<W, NW>(a, w, acc, lds, tid);
    }
}

// Split-K Gram: O[b][i][j] = bf16(alpha * the sum over the chunks s, in order, of the
// float32 partials of (i, j)), zero in the padding columns N .. o_cols - 1, and the mirror
// O[b][j][i] for tiles above the diagonal. A workgroup takes 16 rows x 128 columns of one
// upper tile: each thread sums 8 consecutive partials of a row (two 16-byte loads per
// chunk) and stores them as one 16-byte row segment; the mirror goes through an LDS
// transpose.
constexpr int kReduceRows = 16;
constexpr int kReduceCols = 128;
constexpr int kReduceLdt = kReduceCols + 8;

__global__ __launch_bounds__(256) void k_ns_reduce(const NsGemmArgs a)
{
    __shared__ __attribute__((aligned(16))) uint16_t t[kReduceRows * kReduceLdt];
    const int64_t slices = int64_t(a.tile / kReduceRows) * (a.tile / kReduceCols);
    const int64_t total = int64_t(a.batch) * a.tiles * slices;
    const int64_t wid = blockIdx.x;
    if (wid >= total) return;
    NsGemmArgs one = a;
    one.splits = 1;
    const NsWork w = ns_decode(one, wid / slices);
    const int slice = static_cast<int>(wid % slices);
    const int rs = slice / (a.tile / kReduceCols), cs = slice % (a.tile / kReduceCols);
    const int64_t row0 = int64_t(w.ti) * a.tile + rs * kReduceRows;
    const int64_t col0 = int64_t(w.tj) * a.tile + cs * kReduceCols;
    const int tid = threadIdx.x, r = tid >> 4, scol = (tid & 15) * 8;
    const int64_t plane = int64_t(a.batch) * a.M * a.N;
    const int64_t i = row0 + r, j0 = col0 + scol;
    float v[8] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    if (i < a.M && j0 < a.N) {
        const float* __restrict__ src = a.partial + (w.b * a.M + i) * a.N + j0;
        // 16-byte loads when the row segment is whole and aligned (N % 4 == 0)
        const bool vec = j0 + 8 <= a.N && (a.N & 3) == 0;
        for (int32_t sp = 0; sp < a.splits; ++sp) {
            const float* row = src + sp * plane;
            if (vec) {
                const f32x4v lo = *reinterpret_cast<const f32x4v*>(row);
                const f32x4v hi = *reinterpret_cast<const f32x4v*>(row + 4);
                v[0] += lo.x; v[1] += lo.y; v[2] += lo.z; v[3] += lo.w;
                v[4] += hi.x; v[5] += hi.y; v[6] += hi.z; v[7] += hi.w;
            } else {
                for (int c = 0; c < 8; ++c)
                    if (j0 + c < a.N) v[c] += row[c];
            }
        }
    }
    u32x4 h;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        h[c] = uint32_t(to_bf16(a.alpha * v[2 * c])) |
               (uint32_t(to_bf16(a.alpha * v[2 * c + 1])) << 16);
    if (i < a.M && j0 < a.o_cols)
        *reinterpret_cast<u32x4*>(a.o + w.b * a.so + i * a.ldo + j0) = h;
    if (w.ti == w.tj) return;
    *reinterpret_cast<u32x4*>(t + r * kReduceLdt + scol) = h;
    __syncthreads();
    // mirror: row j = col0 + jr of O takes this slice's 16 rows as columns
    const int jr = tid >> 1, half = (tid & 1) * 8;
    const int64_t j = col0 + jr, ic = row0 + half;
    if (j < a.N && ic < a.ot_cols) {
        u32x4 m;
#pragma unroll
        for (int c = 0; c < 4; ++c)
            m[c] = uint32_t(t[(half + 2 * c) * kReduceLdt + jr]) |
                   (uint32_t(t[(half + 2 * c + 1) * kReduceLdt + jr]) << 16);
        *reinterpret_cast<u32x4*>(a.ot + w.b * a.sot + j * a.ldot + ic) = m;
    }
}

// ---------------------------------------------------------------------------------
// Into and out of the layout. A lane moves an 8 x 8 block of a source matrix S (R x C,
// row-major, dense): lane l of a wave takes rows 8 (l / 8) .. + 7 and columns
// 8 (l % 8) .. + 7 of a 64 x 64 tile (a workgroup holds 4 tiles along R), so its row
// loads and the row stores of the copy and of the transpose each join seven neighbouring
// lanes' into 128 contiguous bytes.
// ---------------------------------------------------------------------------------
constexpr int kTile = 64;
constexpr int kTilesPerGroup = 4;


// Batch entry b takes tensor t = tensor_of ? tensor_of[b] : b, whose R x C matrix starts at
// src + src_off[t] (src_off null: src + b R C; bfloat16), divided by norm[t] (norm null:
// 1). Writes, zero in the padding, copy[b] (R rows of cs >= C elements) = S / norm and
// trans[b] (C rows of ts >= R elements) = (S / norm)^T; cs and ts are multiples of 8,
// copy_stride / trans_stride the batch strides.
__global__ __launch_bounds__(256) void k_ns_prep(const uint16_t* __restrict__ src,
                                                 const int64_t* __restrict__ src_off,
                                                 const int32_t* __restrict__ tensor_of,
                                                 const float* __restrict__ norm, int64_t R,
                                                 int64_t C, uint16_t* __restrict__ copy,
                                                 int64_t copy_stride, int64_t cs,
                                                 uint16_t* __restrict__ trans,
                                                 int64_t trans_stride, int64_t ts)
{
    const int b = blockIdx.z;
    const int t = tensor_of ? tensor_of[b] : b;
    const uint16_t* __restrict__ s = src + (src_off ? src_off[t] : b * R * C);
    const float nrm = norm ? norm[t] : 1.0f;
    uint16_t* __restrict__ cp = copy + b * copy_stride;
    uint16_t* __restrict__ tp = trans + b * trans_stride;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t r0 = (static_cast<int64_t>(blockIdx.y) * kTilesPerGroup + wave) * kTile +
                       8 * (lane >> 3);
    const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kTile + 8 * (lane & 7);
    if (r0 >= ts || c0 >= cs) return;
    u32x4 w[8];
    const bool vec = r0 + 8 <= R && c0 + 8 <= C && (C & 7) == 0 &&
                     (reinterpret_cast<uintptr_t>(s) & 15) == 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        if (vec) {
            w[j] = *reinterpret_cast<const u32x4*>(s + (r0 + j) * C + c0);
        } else {
            for (int q = 0; q < 4; ++q) {
                const int64_t r = r0 + j, c = c0 + 2 * q;
                const uint32_t lo = (r < R && c < C) ? s[r * C + c] : 0u;
                const uint32_t hi = (r < R && c + 1 < C) ? s[r * C + c + 1] : 0u;
                w[j][q] = lo | (hi << 16);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t lo = to_bf16(bf16_val(static_cast<uint16_t>(w[j][q] & 0xffffu)) / nrm);
            const uint32_t hi = to_bf16(bf16_val(static_cast<uint16_t>(w[j][q] >> 16)) / nrm);
            w[j][q] = lo | (hi << 16);
        }
#pragma unroll
    for (int j = 0; j < 8; ++j)
        if (r0 + j < R) *reinterpret_cast<u32x4*>(cp + (r0 + j) * cs + c0) = w[j];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        if (c0 + k >= C) break;
        u32x4 o;
#pragma unroll
        for (int p = 0; p < 4; ++p) o[p] = bf16_at(w[2 * p], k) | (bf16_at(w[2 * p + 1], k) << 16);
        *reinterpret_cast<u32x4*>(tp + (c0 + k) * ts + r0) = o;
    }
}

// theta of tensor tensor_of[b] (R x C, dense) = theta * decay - step * S[b], where S[b] is
// R x C with row stride ss (a multiple of 8) at o + b * stride.
__global__ __launch_bounds__(256) void k_ns_update(const uint16_t* __restrict__ o, int64_t stride,
                                                   int64_t ss, const Seg* __restrict__ segs,
                                                   const int32_t* __restrict__ tensor_of,
                                                   int64_t R, int64_t C, float decay, float step)
{
    const int b = blockIdx.y;
    float* __restrict__ th = segs[tensor_of[b]].theta;
    const uint16_t* __restrict__ src = o + b * stride;
    const int64_t n = R * C;
    const int64_t gstride = 256LL * gridDim.x;
    if ((C & 3) == 0 && (reinterpret_cast<uintptr_t>(th) & 15) == 0) {
        for (int64_t v = blockIdx.x * 256LL + threadIdx.x; v < n / 4; v += gstride) {
            const int64_t e = 4 * v, r = e / C, c = e - r * C;
            const u32x2 wv = *reinterpret_cast<const u32x2*>(src + r * ss + c);
            f32x4v tv = reinterpret_cast<const f32x4v*>(th)[v];
            tv.x = fmaf(-step, bf16_val(static_cast<uint16_t>(wv.x & 0xffffu)), tv.x * decay);
            tv.y = fmaf(-step, bf16_val(static_cast<uint16_t>(wv.x >> 16)), tv.y * decay);
            tv.z = fmaf(-step, bf16_val(static_cast<uint16_t>(wv.y & 0xffffu)), tv.z * decay);
            tv.w = fmaf(-step, bf16_val(static_cast<uint16_t>(wv.y >> 16)), tv.w * decay);
            reinterpret_cast<f32x4v*>(th)[v] = tv;
        }
    } else {
        for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < n; e += gstride) {
            const int64_t r = e / C, c = e - r * C;
            th[e] = fmaf(-step, bf16_val(src[r * ss + c]), th[e] * decay);
        }
    }
}

// dst[b] (R x C, dense) = S[b] (R x C, row stride ss, at src + b * stride).
__global__ __launch_bounds__(256) void k_ns_unpad(const uint16_t* __restrict__ src, int64_t stride,
                                                  int64_t ss, int64_t R, int64_t C,
                                                  uint16_t* __restrict__ dst)
{
    const int b = blockIdx.y;
    const int64_t n = R * C;
    for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < n; e += 256LL * gridDim.x) {
        const int64_t r = e / C, c = e - r * C;
        dst[b * n + e] = src[b * stride + r * ss + c];
    }
}

}  // namespace

hipError_t launch_ns_gemm(const NsGemmArgs& a, hipStream_t stream)
{
    const int64_t groups = ns_workgroups(a);
    const dim3 grid(static_cast<unsigned>(groups)), block(kNsThreads);
    if (a.tile == kNsTileBig) {
        constexpr int NW = kNsBigWaves;
        const dim3 big(NsTileShape<4, NW>::kThreads);
        if (a.splits > 1)
            hipLaunchKernelGGL((k_ns_gemm<4, true, NW>), grid, big, 0, stream, a);
        else
            hipLaunchKernelGGL((k_ns_gemm<4, false, NW>), grid, big, 0, stream, a);
    } else {
        if (a.splits > 1)
            hipLaunchKernelGGL((k_ns_gemm<2, true>), grid, block, 0, stream, a);
        else
            hipLaunchKernelGGL((k_ns_gemm<2, false>), grid, block, 0, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.splits == 1) return e;
    const int64_t slices = int64_t(a.tile / kReduceRows) * (a.tile / kReduceCols);
    hipLaunchKernelGGL(k_ns_reduce, dim3(static_cast<unsigned>(int64_t(a.batch) * a.tiles * slices)),
                       dim3(256), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_ns_prep(const uint16_t* src, const int64_t* src_off, const int32_t* tensor_of,
                          const float* norm, int32_t batch, int64_t R, int64_t C, uint16_t* copy,
                          int64_t copy_stride, int64_t cs, uint16_t* trans, int64_t trans_stride,
                          int64_t ts, hipStream_t stream)
{
    if (cs < C || ts < R || cs % 8 || ts % 8) return hipErrorInvalidValue;
    const int64_t gx = (cs + kTile - 1) / kTile;
    const int64_t gy = (ts + kTile * kTilesPerGroup - 1) / (kTile * kTilesPerGroup);
    if (gx > 0x7fffffff || gy > 65535 || batch > 65535) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_ns_prep, dim3(static_cast<unsigned>(gx), static_cast<unsigned>(gy), batch),
                       dim3(256), 0, stream, src, src_off, tensor_of, norm, R, C, copy,
                       copy_stride, cs, trans, trans_stride, ts);
    return hipGetLastError();
}

static dim3 ns_flat_grid(int64_t n, int32_t batch)
{
    int64_t g = (n / 4 + 255) / 256;
    g = std::max<int64_t>(1, std::min<int64_t>(g, 4096));
    return dim3(static_cast<unsigned>(g), static_cast<unsigned>(batch));
}

hipError_t launch_ns_update(const uint16_t* o, int64_t stride, int64_t ss, const Seg* segs,
                            const int32_t* tensor_of, int32_t batch, int64_t R, int64_t C,
                            float decay, float step, hipStream_t stream)
{
    if (batch > 65535) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_ns_update, ns_flat_grid(R * C, batch), dim3(256), 0, stream, o, stride, ss,
                       segs, tensor_of, R, C, decay, step);
    return hipGetLastError();
}

hipError_t launch_ns_unpad(const uint16_t* src, int64_t stride, int64_t ss, int32_t batch, int64_t R,
                           int64_t C, uint16_t* dst, hipStream_t stream)
{
    if (batch > 65535) return hipErrorInvalidConfiguration;
    hipLaunchKernelGGL(k_ns_unpad, ns_flat_grid(4 * R * C, batch), dim3(256), 0, stream, src, stride,
                       ss, R, C, dst);
    return hipGetLastError();
}

}  // namespace gefen
