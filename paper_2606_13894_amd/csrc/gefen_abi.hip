// C ABI of libgefen: argument checks, state layout, work planning and kernel launches.
// The arithmetic of the method runs in the kernels (step.hip, codebook.hip,
// partition.hip); this file decides which kernel processes which part of which tensor.
#include "gefen.h"
#include "gefen_internal.h"
#include "muon_internal.h"
#include "measure_internal.h"

#include <algorithm>
#include <cstdlib>
#include <memory>
#include <mutex>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

using namespace gefen;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

#define GEFEN_HIP(call)                                                                  \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess)                                                            \
            return fail(GEFEN_EHIP, "%s failed: %s", #call, hipGetErrorString(e_));      \
    } while (0)

using Class = PlanClass;

constexpr int kSegSlots = 4;                 // device tensor tables cached per state
constexpr int64_t kPartChunk = 65536;     // elements of one partition sub-chunk (mode 1)
constexpr int64_t kPartItemElems = 16384; // elements per partition item (mode 0)
constexpr int kPartMaxPairs = 2048;
constexpr uint32_t kCkptMagic = 0x4e464547u;   // "GEFN"

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

std::vector<int64_t> divisors_of(int64_t n)
{
    std::vector<int64_t> lo, hi;
    for (int64_t d = 1; d <= n / d; ++d) {
        if (n % d == 0) {
            lo.push_back(d);
            if (d != n / d) hi.push_back(n / d);
        }
    }
    for (auto it = hi.rbegin(); it != hi.rend(); ++it) lo.push_back(*it);
    return lo;
}

bool finite_f(double x) { return std::isfinite(x); }

}  // namespace

struct gefen_state {
    int device = 0;
    int32_t n_tensors = 0;
    int32_t k = 256, nbins = 4096, ng = 4096;
    int32_t code_bits = 8;
    bool explicit_blocks = false;
    std::vector<int64_t> numel, period, blk_begin, code_off;   // blk_begin/code_off: n + 1
    std::vector<int32_t> gdtype;
    int64_t total_blocks = 0, code_bytes = 0;

    uint8_t* codes = nullptr;
    float* scale = nullptr;
    float* vmom = nullptr;
    float* cb32[2] = {nullptr, nullptr};
    double* cb64[2] = {nullptr, nullptr};
    float* mid[2] = {nullptr, nullptr};
    uint8_t* guide[2] = {nullptr, nullptr};
    int dec_slot = 0, enc_slot = 0;

    Tile* tiles = nullptr;
    int32_t* tile_kind = nullptr;
    HTile* htiles = nullptr;        // parallel to tiles (KIND_H entries only)
    float2* h_partials = nullptr;   // parallel to tiles: per-chunk (sum g^2, max |m|)
    float* h_absmax = nullptr;      // parallel to tiles: per-chunk max |g| (histogram)
    float2* h_old = nullptr;        // per huge block: (s, v) before the step
    int64_t n_tiles = 0, n_hblocks = 0;
    std::vector<Class> classes;

    // Device tensor tables: kSegSlots of them, each keyed by the buffers it points to, so
    // that a caller cycling through a few parameter/gradient buffer sets uploads nothing
    // in steady state.  `segs` points at the table the next launches read.
    Seg* segs = nullptr;
    Seg* seg_slots = nullptr;
    std::vector<Seg> segs_host;     // the table wanted by the current call
    Seg* segs_pinned = nullptr;     // upload staging, one table per slot
    hipEvent_t seg_evt[kSegSlots] = {};
    bool seg_evt_pending[kSegSlots] = {};
    std::vector<const void*> slot_key[kSegSlots];   // (theta, grad) per tensor; empty = free
    uint64_t slot_used[kSegSlots] = {};
    uint64_t seg_clock = 0;
    int cur_slot = -1;
    int64_t* csr = nullptr;

    uint64_t* hist = nullptr;
    void* dp_ws = nullptr;
    double* fit_cb64 = nullptr;
    double* fit_cost = nullptr;
    int32_t* fit_status = nullptr;

    int64_t persistent_bytes = 0, workspace_bytes = 0;
    std::vector<void*> dev_allocs;

    // Gefen-Muon (gefen_muon_init): codec tiles over every block, the bfloat16 momentum
    // matrix per code index, tensors grouped by shape for batched Newton-Schulz products.
    bool muon_ready = false;
    Tile* muon_tiles = nullptr;
    int64_t muon_n_tiles = 0;
    int64_t* muon_tile_range = nullptr;   // [first, end) tile of each tensor
    int64_t muon_dt_first[2] = {0, 0}, muon_dt_count[2] = {0, 0};   // tiles per grad dtype
    float* muon_tile_ss = nullptr;
    float* muon_norm = nullptr;
    uint16_t* muon_u = nullptr;
    int64_t* muon_u_off = nullptr;        // code index of each tensor's first element
    int32_t* muon_tensor_of = nullptr;
    std::vector<NsGroup> muon_groups;
    // The shape groups are split over lanes that run concurrently: lane 0 on the caller's
    // stream, the others on streams of the library's own (forked after the norms, joined
    // at the end of the step). Each lane has its own Newton-Schulz buffers.
    struct MuonLane {
        NsLaneBuffers buf{};            // X and X^T (ping-pong), A, B, split-K partials
        NsLaneSizes size;
        std::vector<int32_t> groups;    // indices into muon_groups, in launch order
    };
    MuonLane muon_lane[kNsLanes];
    hipStream_t muon_side[kNsLanes - 1] = {};   // lane l >= 1 runs on muon_side[l - 1]
    hipEvent_t muon_fork = nullptr;              // (default priority streams)
    hipEvent_t muon_join[kNsLanes - 1] = {};

    // measurement: events[(step * classes + c) * 2 + {0 start, 1 stop}]
    bool prof_armed = false;
    int32_t prof_max_steps = 0, prof_steps = 0;
    std::vector<hipEvent_t> prof_events;
    // Gefen-Muon steps: per step, events [step start, codec + norms end, step end], all
    // on the caller's stream (the step end follows the joins of the other lanes)
    int32_t muon_prof_steps = 0;
    std::vector<hipEvent_t> muon_prof_events;

    size_t muon_prof_stride() const { return 3; }

    void prof_free()
    {
        for (hipEvent_t e : prof_events) (void)hipEventDestroy(e);
        for (hipEvent_t e : muon_prof_events) (void)hipEventDestroy(e);
        prof_events.clear();
        muon_prof_events.clear();
        prof_armed = false;
        prof_steps = 0;
        muon_prof_steps = 0;
    }

    ~gefen_state()
    {
        prof_free();
        if (muon_fork) (void)hipEventDestroy(muon_fork);
        for (hipEvent_t e : muon_join)
            if (e) (void)hipEventDestroy(e);
        for (hipStream_t s : muon_side)
            if (s) (void)hipStreamDestroy(s);
        for (void* p : dev_allocs) (void)hipFree(p);
        if (segs_pinned) (void)hipHostFree(segs_pinned);
        for (hipEvent_t e : seg_evt)
            if (e) (void)hipEventDestroy(e);
    }

    template <typename T>
    int alloc(T** out, size_t bytes, bool persistent)
    {
        void* p = nullptr;
        hipError_t e = hipMalloc(&p, bytes ? bytes : 16);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(GEFEN_ENOMEM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
        }
        dev_allocs.push_back(p);
        *out = static_cast<T*>(p);
        (persistent ? persistent_bytes : workspace_bytes) += static_cast<int64_t>(bytes);
        return GEFEN_OK;
    }
};

// ------------------------------------------------------------------ helpers
namespace {

int check_tensors(const gefen_tensor* ts, int32_t n, bool params, const char* what)
{
    if (!ts) return fail(GEFEN_EINVAL, "%s is NULL", what);
    for (int32_t i = 0; i < n; ++i) {
        if (!ts[i].ptr && ts[i].numel > 0) return fail(GEFEN_EINVAL, "%s[%d].ptr is NULL", what, i);
        if (ts[i].numel < 1) return fail(GEFEN_EINVAL, "%s[%d].numel must be >= 1", what, i);
        if (params ? ts[i].dtype != GEFEN_F32
                   : (ts[i].dtype != GEFEN_F32 && ts[i].dtype != GEFEN_BF16))
            return fail(GEFEN_EDTYPE, "%s[%d] has unsupported dtype %d", what, i, ts[i].dtype);
    }
    return GEFEN_OK;
}

int check_against_state(const gefen_state* st, const gefen_tensor* ts, int32_t n, bool params,
                        const char* what)
{
    if (!st) return fail(GEFEN_EINVAL, "state is NULL");
    if (n != st->n_tensors)
        return fail(GEFEN_EINVAL, "%s: %d tensors, state has %d", what, n, st->n_tensors);
    int rc = check_tensors(ts, n, params, what);
    if (rc) return rc;
    for (int32_t i = 0; i < n; ++i) {
        if (ts[i].numel != st->numel[i])
            return fail(GEFEN_EINVAL, "%s[%d]: numel %lld, state has %lld", what, i,
                        (long long)ts[i].numel, (long long)st->numel[i]);
        if (!params && ts[i].dtype != st->gdtype[i])
            return fail(GEFEN_EDTYPE, "%s[%d]: dtype %d, state has %d", what, i, ts[i].dtype,
                        st->gdtype[i]);
    }
    return GEFEN_OK;
}

bool slot_matches(const gefen_state* st, int k)
{
    const std::vector<const void*>& key = st->slot_key[k];
    if (key.size() != 2 * static_cast<size_t>(st->n_tensors)) return false;
    for (int32_t i = 0; i < st->n_tensors; ++i)
        if (key[2 * i] != st->segs_host[i].theta || key[2 * i + 1] != st->segs_host[i].grad)
            return false;
    return true;
}

// Point `segs` at a device table holding the caller's buffers: reuse a slot whose table
// already matches, else upload into the least recently used slot.  Overwriting a slot is
// ordered after earlier launches that read it by the stream; calls on one state are
// stream-ordered by the caller.
int refresh_segs(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
                 hipStream_t stream)
{
    for (int32_t i = 0; i < st->n_tensors; ++i) {
        Seg& s = st->segs_host[i];
        if (params) s.theta = static_cast<float*>(params[i].ptr);
        if (grads) s.grad = grads[i].ptr;
    }
    const size_t n = static_cast<size_t>(st->n_tensors);
    int hit = -1;
    if (st->cur_slot >= 0 && slot_matches(st, st->cur_slot)) hit = st->cur_slot;
    for (int k = 0; hit < 0 && k < kSegSlots; ++k)
        if (slot_matches(st, k)) hit = k;
    if (hit < 0) {
        hit = 0;
        for (int k = 1; k < kSegSlots; ++k)
            if (st->slot_used[k] < st->slot_used[hit]) hit = k;
        Seg* staging = st->segs_pinned + hit * n;
        if (st->seg_evt_pending[hit]) GEFEN_HIP(hipEventSynchronize(st->seg_evt[hit]));
        std::memcpy(staging, st->segs_host.data(), sizeof(Seg) * n);
        GEFEN_HIP(hipMemcpyAsync(st->seg_slots + hit * n, staging, sizeof(Seg) * n,
                                 hipMemcpyHostToDevice, stream));
        GEFEN_HIP(hipEventRecord(st->seg_evt[hit], stream));
        st->seg_evt_pending[hit] = true;
        std::vector<const void*>& key = st->slot_key[hit];
        key.resize(2 * n);
        for (size_t i = 0; i < n; ++i) {
            key[2 * i] = st->segs_host[i].theta;
            key[2 * i + 1] = st->segs_host[i].grad;
        }
    }
    st->slot_used[hit] = ++st->seg_clock;
    st->cur_slot = hit;
    st->segs = st->seg_slots + hit * n;
    return GEFEN_OK;
}

__global__ void k_fill_zero(uint32_t* p, size_t words)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < words;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = 0u;
}

// Zero `bytes` (a multiple of 4) of device memory with a kernel (graph-capture safe).
hipError_t fill_zero(void* p, size_t bytes, hipStream_t s)
{
    const size_t words = bytes / 4;
    if (!words) return hipSuccess;
    size_t g = (words + 255) / 256;
    if (g > 65536) g = 65536;
    hipLaunchKernelGGL(k_fill_zero, dim3(static_cast<unsigned>(g)), dim3(256), 0, s,
                       static_cast<uint32_t*>(p), words);
    return hipGetLastError();
}

// Plan the tiles (tile_plan.h), check the plan against the kernels' assumptions and
// upload the tables. starts[t]: tensor t's explicit block starts (n_blocks + 1).
int plan_tiles(gefen_state* st, const std::vector<std::vector<int64_t>>& starts)
{
    PlanCtx ctx;
    ctx.n_tensors = st->n_tensors;
    ctx.code_bits = st->code_bits;
    ctx.explicit_blocks = st->explicit_blocks;
    ctx.numel = st->numel;
    ctx.period = st->period;
    ctx.blk_begin = st->blk_begin;
    ctx.gdtype = st->gdtype;
    Plan plan;
    std::string why = build_plan(&ctx, starts, plan);
    if (why.empty()) why = check_plan(ctx, starts, plan);
    if (!why.empty()) return fail(GEFEN_EINVAL, "internal: tile plan: %s", why.c_str());
    st->n_hblocks = ctx.n_hblocks;
    st->classes = plan.classes;
    st->n_tiles = static_cast<int64_t>(plan.tiles.size());
    int rc = st->alloc(&st->tiles, sizeof(Tile) * plan.tiles.size(), false);
    if (rc) return rc;
    rc = st->alloc(&st->tile_kind, sizeof(int32_t) * plan.kinds.size(), false);
    if (rc) return rc;
    GEFEN_HIP(hipMemcpy(st->tiles, plan.tiles.data(), sizeof(Tile) * plan.tiles.size(),
                        hipMemcpyHostToDevice));
    GEFEN_HIP(hipMemcpy(st->tile_kind, plan.kinds.data(), sizeof(int32_t) * plan.kinds.size(),
                        hipMemcpyHostToDevice));
    if (st->n_hblocks > 0) {
        const size_t nt = plan.tiles.size();
        if ((rc = st->alloc(&st->htiles, sizeof(HTile) * nt, false))) return rc;
        if ((rc = st->alloc(&st->h_partials, sizeof(float2) * nt, false))) return rc;
        if ((rc = st->alloc(&st->h_absmax, sizeof(float) * nt, false))) return rc;
        if ((rc = st->alloc(&st->h_old, sizeof(float2) * st->n_hblocks, false))) return rc;
        GEFEN_HIP(hipMemcpy(st->htiles, plan.htiles.data(), sizeof(HTile) * nt,
                            hipMemcpyHostToDevice));
    }
    return GEFEN_OK;
}

// Alg. 2 for a list of tensors. Writes one period per tensor (host), and optionally the
// scores of every divisor (host, concatenated in tensor order).
int infer_periods(const std::vector<gefen_tensor>& ts, double eps, hipStream_t stream,
                  std::vector<int64_t>& periods, std::vector<int64_t>* divs_out,
                  std::vector<double>* scores_out)
{
    std::vector<PartDesc> descs;
    std::vector<int32_t> first, count;
    std::vector<int64_t> all_divs;
    int64_t items = 0, slots = 0;
    for (const gefen_tensor& g : ts) {
        const int64_t n = g.numel;
        const std::vector<int64_t> dv = divisors_of(n);
        first.push_back(static_cast<int32_t>(descs.size()));
        count.push_back(static_cast<int32_t>(dv.size()));
        for (int64_t p : dv) {
            PartDesc d{};
            d.grad = g.ptr;
            d.n = n;
            d.p = p;
            d.gdtype = g.dtype;
            d.item0 = items;
            d.out0 = slots;
            const int64_t nb = n / p;
            if (nb < 2) {
                d.mode = 0;
                d.rpi = 1;
                d.n_items = 0;
            } else if (p <= kPartChunk) {
                d.mode = 0;
                int64_t rpi = kPartItemElems / p;
                rpi = std::max<int64_t>(1, std::min<int64_t>(rpi, kPartMaxPairs));
                d.rpi = static_cast<int32_t>(rpi);
                d.n_items = (nb - 1 + rpi - 1) / rpi;
                slots += d.n_items;
            } else {
                d.mode = 1;
                d.rpi = static_cast<int32_t>((p + kPartChunk - 1) / kPartChunk);
                d.n_items = nb * d.rpi;
                slots += d.n_items;
            }
            items += d.n_items;
            descs.push_back(d);
            all_divs.push_back(p);
        }
    }
    const int32_t nd = static_cast<int32_t>(descs.size());
    const int32_t nt = static_cast<int32_t>(ts.size());
    void *d_descs = nullptr, *d_partials = nullptr, *d_scores = nullptr, *d_first = nullptr,
         *d_count = nullptr, *d_periods = nullptr;
    auto cleanup = [&]() {
        for (void* p : {d_descs, d_partials, d_scores, d_first, d_count, d_periods})
            if (p) (void)hipFree(p);
    };
#define GEFEN_PART_HIP(call)                                                             \
    do {                                                                                 \
        hipError_t e_ = (call);                                                          \
        if (e_ != hipSuccess) {                                                          \
            cleanup();                                                                   \
            return fail(GEFEN_EHIP, "%s failed: %s", #call, hipGetErrorString(e_));      \
        }                                                                                \
    } while (0)
    GEFEN_PART_HIP(hipMalloc(&d_descs, sizeof(PartDesc) * std::max(nd, 1)));
    GEFEN_PART_HIP(hipMalloc(&d_partials, sizeof(double) * std::max<int64_t>(slots, 1)));
    GEFEN_PART_HIP(hipMalloc(&d_scores, sizeof(double) * std::max(nd, 1)));
    GEFEN_PART_HIP(hipMalloc(&d_first, sizeof(int32_t) * std::max(nt, 1)));
    GEFEN_PART_HIP(hipMalloc(&d_count, sizeof(int32_t) * std::max(nt, 1)));
    GEFEN_PART_HIP(hipMalloc(&d_periods, sizeof(int64_t) * std::max(nt, 1)));
    GEFEN_PART_HIP(hipMemcpyAsync(d_descs, descs.data(), sizeof(PartDesc) * nd,
                                  hipMemcpyHostToDevice, stream));
    GEFEN_PART_HIP(hipMemcpyAsync(d_first, first.data(), sizeof(int32_t) * nt,
                                  hipMemcpyHostToDevice, stream));
    GEFEN_PART_HIP(hipMemcpyAsync(d_count, count.data(), sizeof(int32_t) * nt,
                                  hipMemcpyHostToDevice, stream));
    GEFEN_PART_HIP(launch_partition(static_cast<PartDesc*>(d_descs), nd, items, eps,
                                    static_cast<double*>(d_partials),
                                    static_cast<double*>(d_scores),
                                    static_cast<int32_t*>(d_first),
                                    static_cast<int32_t*>(d_count), nt,
                                    static_cast<int64_t*>(d_periods), stream));
    periods.assign(nt, 1);
    GEFEN_PART_HIP(hipMemcpyAsync(periods.data(), d_periods, sizeof(int64_t) * nt,
                                  hipMemcpyDeviceToHost, stream));
    if (scores_out) {
        scores_out->assign(nd, 0.0);
        GEFEN_PART_HIP(hipMemcpyAsync(scores_out->data(), d_scores, sizeof(double) * nd,
                                      hipMemcpyDeviceToHost, stream));
    }
    GEFEN_PART_HIP(hipStreamSynchronize(stream));
#undef GEFEN_PART_HIP
    cleanup();
    if (divs_out) *divs_out = all_divs;
    return GEFEN_OK;
}

CodebookDev codebook_dev(const gefen_state* st)
{
    CodebookDev c;
    c.dec = st->cb32[st->dec_slot];
    c.enc_mid = st->mid[st->enc_slot];
    c.enc_guide = st->guide[st->enc_slot];
    c.k = st->k;
    c.ng = st->ng;
    return c;
}

// Histogram with the state's blocks into `hist` (already zeroed).
int run_histogram(gefen_state* st, uint64_t* hist, hipStream_t stream)
{
    for (const Class& c : st->classes)
        if (c.kind == KIND_H)
            GEFEN_HIP(launch_hist_h_absmax(st->tiles + c.first, st->htiles + c.first, c.count,
                                           st->segs, st->h_absmax, stream));
    GEFEN_HIP(launch_histogram(st->tiles, st->n_tiles, st->tile_kind, st->htiles, st->h_absmax,
                               st->segs, st->nbins, hist, stream));
    return GEFEN_OK;
}

// Histogram of `grads` with the state's blocks, DP, install into `slot`.
int fit_into_slot(gefen_state* st, int slot, hipStream_t stream)
{
    GEFEN_HIP(fill_zero(st->hist, sizeof(uint64_t) * st->nbins, stream));
    int rc = run_histogram(st, st->hist, stream);
    if (rc) return rc;
    GEFEN_HIP(launch_dp(st->hist, st->nbins, st->k, st->dp_ws, st->fit_cb64, st->fit_cost,
                        st->fit_status, stream));
    GEFEN_HIP(launch_install_codebook(st->fit_cb64, st->k, st->ng, st->cb32[slot],
                                      st->cb64[slot], st->mid[slot], st->guide[slot], stream));
    return GEFEN_OK;
}

struct CkptLayout {
    int64_t header, codes, scale, vmom, cb0, cb1, total;
};

CkptLayout ckpt_layout(const gefen_state* st)
{
    auto a8 = [](int64_t x) { return (x + 7) & ~int64_t(7); };
    CkptLayout L;
    L.header = 0;
    L.codes = 64;
    L.scale = a8(L.codes + st->code_bytes);
    L.vmom = L.scale + 4 * st->total_blocks;
    L.cb0 = a8(L.vmom + 4 * st->total_blocks);
    L.cb1 = L.cb0 + 8 * st->k;
    L.total = L.cb1 + 8 * st->k;
    return L;
}

// A codebook the encode and decode tables accept: finite, first entry -1, last +1, never
// decreasing. A degenerate fit pads its DP solution with repeated +1 entries; equal
// entries give equal midpoints, which the encoder resolves to the lower index.
template <typename T>
bool valid_codebook(const T* cb, int32_t k)
{
    if (k < 2 || cb[0] != T(-1) || cb[k - 1] != T(1)) return false;
    for (int32_t i = 1; i < k; ++i)
        if (!(cb[i] >= cb[i - 1]) || !std::isfinite(static_cast<double>(cb[i]))) return false;
    return true;
}

bool is_host_ptr(const void* p)
{
    hipPointerAttribute_t a;
    if (hipPointerGetAttributes(&a, p) != hipSuccess) {
        (void)hipGetLastError();
        return true;
    }
    return a.type == hipMemoryTypeHost || a.type == hipMemoryTypeUnregistered;
}

}  // namespace

// ------------------------------------------------------------------ fixed DP workspace
// The workspace of gefen_dp_codebook_static: one array per GPU, for the process's
// lifetime, large enough for the largest DP (16 * 256 bins, 256 entries: 11,088,896
// bytes). Host code never passes `scratch` itself to a kernel (in host code it is a
// stand-in, not a device address): the first call on each device asks the runtime for
// that device's copy and keeps the address.
constexpr size_t kDpScratchBytes = size_t(11) << 20;
static __device__ __align__(256) unsigned char scratch[kDpScratchBytes];

namespace {

std::mutex g_scratch_mu;
std::vector<void*> g_scratch_ptr;   // per device ordinal; null until its first call

int dp_scratch(void** out)
{
    int dev = 0;
    GEFEN_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (dev >= static_cast<int>(g_scratch_ptr.size())) g_scratch_ptr.resize(dev + 1, nullptr);
    if (!g_scratch_ptr[dev]) {
        if (dp_workspace_bytes(16 * kMaxK, kMaxK) > kDpScratchBytes)
            return fail(GEFEN_EHIP, "internal: the fixed DP workspace is too small");
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(GEFEN_EHIP, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return GEFEN_OK;
}

}  // namespace

// ------------------------------------------------------------------ ABI
extern "C" {

const char* gefen_last_error(void) { return g_err.c_str(); }

int gefen_init(const gefen_tensor* grads0, int32_t n_tensors, const int64_t* period_override,
               const int64_t* block_offsets, int64_t n_blocks, int32_t code_bits,
               double eps_part, void* stream_, gefen_state** out)
{
    g_err.clear();
    if (!out) return fail(GEFEN_EINVAL, "out is NULL");
    *out = nullptr;
    if (n_tensors < 1) return fail(GEFEN_EINVAL, "n_tensors must be >= 1");
    int rc = check_tensors(grads0, n_tensors, false, "grads0");
    if (rc) return rc;
    if (code_bits != 8 && code_bits != 4)
        return fail(GEFEN_EINVAL, "code_bits must be 8 or 4 (got %d)", code_bits);
    if (!finite_f(eps_part) || eps_part < 0) return fail(GEFEN_EINVAL, "eps_part must be >= 0");
    hipStream_t stream = as_stream(stream_);

    std::unique_ptr<gefen_state> st(new gefen_state());
    GEFEN_HIP(hipGetDevice(&st->device));
    st->n_tensors = n_tensors;
    st->code_bits = code_bits;
    st->k = 1 << code_bits;
    st->nbins = 16 * st->k;
    st->ng = 16 * st->k;
    int64_t total = 0;
    for (int32_t i = 0; i < n_tensors; ++i) {
        st->numel.push_back(grads0[i].numel);
        st->gdtype.push_back(grads0[i].dtype);
        total += grads0[i].numel;
    }

    // blocks
    std::vector<std::vector<int64_t>> starts(n_tensors);
    st->period.assign(n_tensors, 0);
    if (block_offsets) {
        if (n_blocks < 1) return fail(GEFEN_EINVAL, "n_blocks must be >= 1");
        if (block_offsets[0] != 0) return fail(GEFEN_EINVAL, "block_offsets[0] must be 0");
        if (block_offsets[n_blocks] != total)
            return fail(GEFEN_EINVAL, "block_offsets[n_blocks] must equal the total numel");
        st->explicit_blocks = true;
        int64_t b = 0, base = 0;
        for (int32_t t = 0; t < n_tensors; ++t) {
            const int64_t end = base + st->numel[t];
            starts[t].push_back(0);
            while (b < n_blocks && block_offsets[b + 1] <= end) {
                if (block_offsets[b + 1] <= block_offsets[b])
                    return fail(GEFEN_EINVAL, "block_offsets must increase strictly (at %lld)",
                                (long long)b);
                starts[t].push_back(block_offsets[b + 1] - base);
                ++b;
            }
            if (starts[t].back() != st->numel[t])
                return fail(GEFEN_EINVAL, "tensor %d does not end on a block boundary", t);
            base = end;
        }
    } else {
        std::vector<gefen_tensor> infer;
        std::vector<int32_t> which;
        for (int32_t t = 0; t < n_tensors; ++t) {
            const int64_t ov = period_override ? period_override[t] : 0;
            if (ov < 0) return fail(GEFEN_EINVAL, "period_override[%d] < 0", t);
            if (ov > 0) {
                if (st->numel[t] % ov != 0)
                    return fail(GEFEN_EINVAL, "period_override[%d] = %lld does not divide %lld",
                                t, (long long)ov, (long long)st->numel[t]);
                st->period[t] = ov;
            } else {
                infer.push_back(grads0[t]);
                which.push_back(t);
            }
        }
        if (!infer.empty()) {
            std::vector<int64_t> per;
            rc = infer_periods(infer, eps_part, stream, per, nullptr, nullptr);
            if (rc) return rc;
            for (size_t i = 0; i < which.size(); ++i) st->period[which[i]] = per[i];
        }
    }

    // state layout
    st->blk_begin.assign(n_tensors + 1, 0);
    st->code_off.assign(n_tensors + 1, 0);
    for (int32_t t = 0; t < n_tensors; ++t) {
        const int64_t nb = st->explicit_blocks ? static_cast<int64_t>(starts[t].size()) - 1
                                               : st->numel[t] / st->period[t];
        st->blk_begin[t + 1] = st->blk_begin[t] + nb;
        // every tensor's codes start on a 16-byte boundary (32 codes at 4 bits)
        st->code_off[t + 1] = st->code_off[t] + ((st->numel[t] + 31) & ~int64_t(31));
    }
    st->total_blocks = st->blk_begin[n_tensors];
    st->code_bytes = st->code_off[n_tensors] * code_bits / 8;

    if ((rc = st->alloc(&st->codes, st->code_bytes, true))) return rc;
    if ((rc = st->alloc(&st->scale, 4 * st->total_blocks, true))) return rc;
    if ((rc = st->alloc(&st->vmom, 4 * st->total_blocks, true))) return rc;
    const size_t guide_bytes = ((st->ng + 1 + 15) / 16) * 16;
    for (int s = 0; s < 2; ++s) {
        if ((rc = st->alloc(&st->cb32[s], 4 * st->k, true))) return rc;
        if ((rc = st->alloc(&st->cb64[s], 8 * st->k, true))) return rc;
        if ((rc = st->alloc(&st->mid[s], 4 * st->k, true))) return rc;
        if ((rc = st->alloc(&st->guide[s], guide_bytes, true))) return rc;
    }
    if ((rc = st->alloc(&st->seg_slots, sizeof(Seg) * n_tensors * kSegSlots, false))) return rc;
    if ((rc = st->alloc(&st->hist, sizeof(uint64_t) * st->nbins, false))) return rc;
    if ((rc = st->alloc(&st->dp_ws, dp_workspace_bytes(st->nbins, st->k), false))) return rc;
    if ((rc = st->alloc(&st->fit_cb64, 8 * st->k, false))) return rc;
    if ((rc = st->alloc(&st->fit_cost, 8, false))) return rc;
    if ((rc = st->alloc(&st->fit_status, 8, false))) return rc;
    void* pinned = nullptr;
    GEFEN_HIP(hipHostMalloc(&pinned, sizeof(Seg) * n_tensors * kSegSlots, hipHostMallocDefault));
    st->segs_pinned = static_cast<Seg*>(pinned);
    for (hipEvent_t& e : st->seg_evt) GEFEN_HIP(hipEventCreateWithFlags(&e, hipEventDisableTiming));

    if (st->explicit_blocks) {
        int64_t entries = 0;
        for (int32_t t = 0; t < n_tensors; ++t) entries += static_cast<int64_t>(starts[t].size());
        if ((rc = st->alloc(&st->csr, sizeof(int64_t) * entries, false))) return rc;
        std::vector<int64_t> flat;
        flat.reserve(entries);
        for (int32_t t = 0; t < n_tensors; ++t) flat.insert(flat.end(), starts[t].begin(), starts[t].end());
        GEFEN_HIP(hipMemcpy(st->csr, flat.data(), sizeof(int64_t) * entries, hipMemcpyHostToDevice));
    }

    st->segs_host.assign(n_tensors, Seg{});
    int64_t csr_base = 0;
    for (int32_t t = 0; t < n_tensors; ++t) {
        Seg& s = st->segs_host[t];
        s.theta = nullptr;
        s.grad = grads0[t].ptr;
        s.code_off = st->code_off[t];
        s.period = st->period[t];
        s.blk_begin = st->blk_begin[t];
        s.csr = st->explicit_blocks ? st->csr + csr_base : nullptr;
        s.numel = st->numel[t];
        s.gdtype = st->gdtype[t];
        if (st->explicit_blocks) csr_base += static_cast<int64_t>(starts[t].size());
    }
    if ((rc = refresh_segs(st.get(), nullptr, nullptr, stream))) return rc;

    if ((rc = plan_tiles(st.get(), starts))) return rc;

    // zero state (Alg. 1: codes 0, scales 0, second moments 0)
    GEFEN_HIP(fill_zero(st->codes, st->code_bytes, stream));
    GEFEN_HIP(fill_zero(st->scale, 4 * st->total_blocks, stream));
    GEFEN_HIP(fill_zero(st->vmom, 4 * st->total_blocks, stream));

    // codebook from the first gradients (Alg. 3)
    if ((rc = fit_into_slot(st.get(), 0, stream))) return rc;
    st->dec_slot = st->enc_slot = 0;
    GEFEN_HIP(hipStreamSynchronize(stream));
    *out = st.release();
    return GEFEN_OK;
}

namespace {

// One step (Alg. 1); with `fit`, the codebook fit (Alg. 3) on this step's gradients as
// well: the KIND_G launches bin every element of their blocks on the way (the blocks'
// max |g| come out of the same reduction as sum g^2), the other classes' tiles go through
// the histogram kernel after their step launch, then the DP installs the new codebook
// into the slot the next step encodes with -- the same result as gefen_step followed by
// gefen_fit_codebook on the same gradients.
int step_impl(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
              int32_t n_tensors, double lr, double beta1, double beta2, double eps,
              double weight_decay, int64_t t, void* stream_, bool fit)
{
    int rc = check_against_state(st, params, n_tensors, true, "params");
    if (rc) return rc;
    if ((rc = check_against_state(st, grads, n_tensors, false, "grads"))) return rc;
    if (t < 1) return fail(GEFEN_EINVAL, "t must be >= 1 (got %lld)", (long long)t);
    if (!(beta1 >= 0.0 && beta1 < 1.0)) return fail(GEFEN_EINVAL, "beta1 must be in [0, 1)");
    if (!(beta2 >= 0.0 && beta2 < 1.0)) return fail(GEFEN_EINVAL, "beta2 must be in [0, 1)");
    if (!finite_f(lr) || !finite_f(weight_decay)) return fail(GEFEN_EINVAL, "lr and weight_decay must be finite");
    if (!finite_f(eps) || eps < 0.0) return fail(GEFEN_EINVAL, "eps must be finite and >= 0");
    hipStream_t stream = as_stream(stream_);
    if ((rc = refresh_segs(st, params, grads, stream))) return rc;

    const double bc1 = 1.0 - std::pow(beta1, static_cast<double>(t));
    const double bc2 = 1.0 - std::pow(beta2, static_cast<double>(t));
    StepScalars sc;
    sc.beta1 = static_cast<float>(beta1);
    sc.one_minus_beta1 = static_cast<float>(1.0 - beta1);
    sc.beta2 = static_cast<float>(beta2);
    sc.one_minus_beta2 = static_cast<float>(1.0 - beta2);
    sc.step_size = static_cast<float>(lr / bc1);
    sc.inv_bc2 = static_cast<float>(1.0 / bc2);
    sc.eps = static_cast<float>(eps);
    sc.decay = static_cast<float>(1.0 - lr * weight_decay);
    const CodebookDev cb = codebook_dev(st);
    const bool prof = st->prof_armed && st->prof_steps < st->prof_max_steps;
    const size_t ncls = st->classes.size();
    if (fit) GEFEN_HIP(fill_zero(st->hist, sizeof(uint64_t) * st->nbins, stream));
    for (size_t ci = 0; ci < ncls; ++ci) {
        const Class& c = st->classes[ci];
        const Tile* tiles = st->tiles + c.first;
        if (prof) GEFEN_HIP(hipEventRecord(st->prof_events[(st->prof_steps * ncls + ci) * 2], stream));
        hipError_t e =
            c.kind == KIND_H
                ? launch_step_h(c.gdtype, st->code_bits, tiles, st->htiles + c.first, c.count,
                                st->segs, st->codes, st->scale, st->vmom, cb, sc,
                                st->h_partials, st->h_old, stream)
            : fit && c.kind == KIND_G
                ? launch_step_g_hist(c.gdtype, st->code_bits, tiles, c.count, st->segs,
                                     st->codes, st->scale, st->vmom, cb, sc, st->hist,
                                     st->nbins, stream)
                : launch_step(c.kind, c.gdtype, st->code_bits, c.vpl, c.bs, tiles, c.count,
                              st->segs, st->codes, st->scale, st->vmom, cb, sc, stream);
        if (e != hipSuccess)
            return fail(GEFEN_EHIP, "step launch (kind %d) failed: %s", c.kind, hipGetErrorString(e));
        if (prof) GEFEN_HIP(hipEventRecord(st->prof_events[(st->prof_steps * ncls + ci) * 2 + 1], stream));
        if (fit && c.kind != KIND_G) {   // the gradients are read-only: any order is fine
            if (c.kind == KIND_H)
                GEFEN_HIP(launch_hist_h_absmax(tiles, st->htiles + c.first, c.count, st->segs,
                                               st->h_absmax, stream));
            GEFEN_HIP(launch_histogram(tiles, c.count, st->tile_kind + c.first,
                                       st->htiles + c.first, st->h_absmax, st->segs, st->nbins,
                                       st->hist, stream));
        }
    }
    if (prof) ++st->prof_steps;
    st->dec_slot = st->enc_slot;
    if (fit) {
        const int slot = 1 - st->dec_slot;
        GEFEN_HIP(launch_dp(st->hist, st->nbins, st->k, st->dp_ws, st->fit_cb64, st->fit_cost,
                            st->fit_status, stream));
        GEFEN_HIP(launch_install_codebook(st->fit_cb64, st->k, st->ng, st->cb32[slot],
                                          st->cb64[slot], st->mid[slot], st->guide[slot], stream));
        st->enc_slot = slot;
    }
    if (std::getenv("GEFEN_DEBUG_SYNC")) {
        GEFEN_HIP(hipStreamSynchronize(stream));
        GEFEN_HIP(hipGetLastError());
    }
    return GEFEN_OK;
}

}  // namespace

int gefen_step(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
               int32_t n_tensors, double lr, double beta1, double beta2, double eps,
               double weight_decay, int64_t t, void* stream)
{
    return step_impl(st, params, grads, n_tensors, lr, beta1, beta2, eps, weight_decay, t,
                     stream, false);
}

int gefen_step_fit(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
                   int32_t n_tensors, double lr, double beta1, double beta2, double eps,
                   double weight_decay, int64_t t, void* stream)
{
    return step_impl(st, params, grads, n_tensors, lr, beta1, beta2, eps, weight_decay, t,
                     stream, true);
}

int gefen_fit_codebook(gefen_state* st, const gefen_tensor* grads, int32_t n_tensors,
                       void* stream_)
{
    int rc = check_against_state(st, grads, n_tensors, false, "grads");
    if (rc) return rc;
    hipStream_t stream = as_stream(stream_);
    if ((rc = refresh_segs(st, nullptr, grads, stream))) return rc;
    const int slot = 1 - st->dec_slot;
    if ((rc = fit_into_slot(st, slot, stream))) return rc;
    st->enc_slot = slot;
    return GEFEN_OK;
}

int gefen_partition_scores(const gefen_tensor* grad, double eps_part, int64_t* divisors_out,
                           double* scores_out, int32_t cap, int32_t* n_div, int64_t* period_out,
                           void* stream_)
{
    g_err.clear();
    int rc = check_tensors(grad, 1, false, "grad");
    if (rc) return rc;
    if (!n_div || !period_out) return fail(GEFEN_EINVAL, "n_div and period_out must not be NULL");
    if (!finite_f(eps_part) || eps_part < 0) return fail(GEFEN_EINVAL, "eps_part must be >= 0");
    std::vector<int64_t> per, divs;
    std::vector<double> scores;
    rc = infer_periods(std::vector<gefen_tensor>{*grad}, eps_part, as_stream(stream_), per,
                       &divs, &scores);
    if (rc) return rc;
    *n_div = static_cast<int32_t>(divs.size());
    *period_out = per[0];
    if (static_cast<int64_t>(divs.size()) > cap)
        return fail(GEFEN_EINVAL, "cap %d < %zu divisors", cap, divs.size());
    if (divisors_out) std::memcpy(divisors_out, divs.data(), sizeof(int64_t) * divs.size());
    if (scores_out) std::memcpy(scores_out, scores.data(), sizeof(double) * scores.size());
    return GEFEN_OK;
}

int gefen_histogram(gefen_state* st, const gefen_tensor* grads, int32_t n_tensors,
                    uint64_t* hist_out, void* stream_)
{
    int rc = check_against_state(st, grads, n_tensors, false, "grads");
    if (rc) return rc;
    if (!hist_out) return fail(GEFEN_EINVAL, "hist_out is NULL");
    hipStream_t stream = as_stream(stream_);
    if ((rc = refresh_segs(st, nullptr, grads, stream))) return rc;
    GEFEN_HIP(fill_zero(hist_out, sizeof(uint64_t) * st->nbins, stream));
    return run_histogram(st, hist_out, stream);
}

int gefen_dp_codebook(const uint64_t* hist, int32_t nbins, int32_t k, double* codebook_out,
                      double* cost_out, int32_t* status_out, void* stream_)
{
    g_err.clear();
    if (!hist || !codebook_out || !cost_out || !status_out)
        return fail(GEFEN_EINVAL, "NULL argument");
    if (k < 2 || k > kMaxK) return fail(GEFEN_EINVAL, "k must be in [2, %d]", kMaxK);
    if (nbins < 1 || nbins > 16 * kMaxK) return fail(GEFEN_EINVAL, "nbins must be in [1, %d]", 16 * kMaxK);
    hipStream_t stream = as_stream(stream_);
    void* ws = nullptr;
    GEFEN_HIP(hipMallocAsync(&ws, dp_workspace_bytes(nbins, k), stream));
    hipError_t e = launch_dp(hist, nbins, k, ws, codebook_out, cost_out, status_out, stream);
    (void)hipFreeAsync(ws, stream);
    if (e != hipSuccess) return fail(GEFEN_EHIP, "DP launch failed: %s", hipGetErrorString(e));
    return GEFEN_OK;
}

int gefen_dp_codebook_static(const uint64_t* hist, int32_t nbins, int32_t k, double* codebook_out,
                             double* cost_out, int32_t* status_out, void* stream_)
{
    g_err.clear();
    if (!hist || !codebook_out || !cost_out || !status_out)
        return fail(GEFEN_EINVAL, "NULL argument");
    if (k < 2 || k > kMaxK) return fail(GEFEN_EINVAL, "k must be in [2, %d]", kMaxK);
    if (nbins < 1 || nbins > 16 * kMaxK) return fail(GEFEN_EINVAL, "nbins must be in [1, %d]", 16 * kMaxK);
    const size_t need = dp_workspace_bytes(nbins, k);
    if (need > kDpScratchBytes)
        return fail(GEFEN_EINVAL, "a DP of %d bins and %d entries needs %zu bytes of workspace; "
                    "the fixed workspace holds %zu", nbins, k, need, kDpScratchBytes);
    void* ws = nullptr;
    int rc = dp_scratch(&ws);
    if (rc) return rc;
    hipError_t e = launch_dp(hist, nbins, k, ws, codebook_out, cost_out, status_out,
                             as_stream(stream_));
    if (e != hipSuccess) return fail(GEFEN_EHIP, "DP launch failed: %s", hipGetErrorString(e));
    return GEFEN_OK;
}

int gefen_get_periods(const gefen_state* st, int64_t* periods_out)
{
    if (!st || !periods_out) return fail(GEFEN_EINVAL, "NULL argument");
    for (int32_t i = 0; i < st->n_tensors; ++i) periods_out[i] = st->period[i];
    return GEFEN_OK;
}

int gefen_get_layout(const gefen_state* st, int64_t* code_offsets, int64_t* block_index,
                     int64_t* total_code_bytes, int64_t* total_blocks, int32_t* k)
{
    if (!st) return fail(GEFEN_EINVAL, "state is NULL");
    if (code_offsets) std::memcpy(code_offsets, st->code_off.data(), 8 * (st->n_tensors + 1));
    if (block_index) std::memcpy(block_index, st->blk_begin.data(), 8 * (st->n_tensors + 1));
    if (total_code_bytes) *total_code_bytes = st->code_bytes;
    if (total_blocks) *total_blocks = st->total_blocks;
    if (k) *k = st->k;
    return GEFEN_OK;
}

static int state_array(const gefen_state* st, int32_t which, void** ptr, int64_t* bytes)
{
    switch (which) {
    case 0: *ptr = st->codes; *bytes = st->code_bytes; return GEFEN_OK;
    case 1: *ptr = st->scale; *bytes = 4 * st->total_blocks; return GEFEN_OK;
    case 2: *ptr = st->vmom; *bytes = 4 * st->total_blocks; return GEFEN_OK;
    case 3: *ptr = st->cb32[st->dec_slot]; *bytes = 4 * st->k; return GEFEN_OK;
    case 4: *ptr = st->cb32[st->enc_slot]; *bytes = 4 * st->k; return GEFEN_OK;
    case 5: *ptr = st->cb64[st->dec_slot]; *bytes = 8 * st->k; return GEFEN_OK;
    case 7: *ptr = st->hist; *bytes = 8 * int64_t(st->nbins); return GEFEN_OK;
    case 6:
        if (!st->muon_ready) return fail(GEFEN_EINVAL, "array 6 needs gefen_muon_init");
        *ptr = st->muon_u;
        *bytes = 2 * st->code_off[st->n_tensors];
        return GEFEN_OK;
    default: return fail(GEFEN_EINVAL, "unknown state array %d", which);
    }
}

int gefen_read_state(const gefen_state* st, int32_t which, void* dst, int64_t bytes,
                     void* stream_)
{
    if (!st || !dst) return fail(GEFEN_EINVAL, "NULL argument");
    void* src;
    int64_t need;
    int rc = state_array(st, which, &src, &need);
    if (rc) return rc;
    if (bytes != need) return fail(GEFEN_EINVAL, "bytes = %lld, array has %lld", (long long)bytes, (long long)need);
    hipStream_t stream = as_stream(stream_);
    GEFEN_HIP(hipMemcpyAsync(dst, src, need, hipMemcpyDefault, stream));
    if (is_host_ptr(dst)) GEFEN_HIP(hipStreamSynchronize(stream));
    return GEFEN_OK;
}

int gefen_write_state(gefen_state* st, int32_t which, const void* src, int64_t bytes,
                      void* stream_)
{
    if (!st || !src) return fail(GEFEN_EINVAL, "NULL argument");
    if (which >= 5) return fail(GEFEN_EINVAL, "array %d is read-only", which);
    void* dst;
    int64_t need;
    int rc = state_array(st, which, &dst, &need);
    if (rc) return rc;
    if (bytes != need) return fail(GEFEN_EINVAL, "bytes = %lld, array has %lld", (long long)bytes, (long long)need);
    hipStream_t stream = as_stream(stream_);
    if (which == 3 || which == 4) {
        std::vector<float> cb(st->k);
        GEFEN_HIP(hipMemcpyAsync(cb.data(), src, need, hipMemcpyDefault, stream));
        GEFEN_HIP(hipStreamSynchronize(stream));
        if (!valid_codebook(cb.data(), st->k))
            return fail(GEFEN_EINVAL, "a codebook must be finite, start at -1, end at +1 and "
                        "never decrease");
        const int slot = which == 3 ? st->dec_slot : st->enc_slot;
        float* staging = nullptr;
        GEFEN_HIP(hipMallocAsync(reinterpret_cast<void**>(&staging), need, stream));
        GEFEN_HIP(hipMemcpyAsync(staging, cb.data(), need, hipMemcpyHostToDevice, stream));
        hipError_t e = launch_install_codebook_f32(staging, st->k, st->ng, st->cb32[slot],
                                                   st->cb64[slot], st->mid[slot],
                                                   st->guide[slot], stream);
        (void)hipFreeAsync(staging, stream);
        GEFEN_HIP(e);
        GEFEN_HIP(hipStreamSynchronize(stream));
        return GEFEN_OK;
    }
    GEFEN_HIP(hipMemcpyAsync(dst, src, need, hipMemcpyDefault, stream));
    if (is_host_ptr(src)) GEFEN_HIP(hipStreamSynchronize(stream));
    return GEFEN_OK;
}

int gefen_get_fit_info(const gefen_state* st, double* cost_out, int32_t* status_out,
                       void* stream_)
{
    if (!st) return fail(GEFEN_EINVAL, "state is NULL");
    hipStream_t stream = as_stream(stream_);
    double c = 0;
    int32_t s = 0;
    GEFEN_HIP(hipMemcpyAsync(&c, st->fit_cost, 8, hipMemcpyDeviceToHost, stream));
    GEFEN_HIP(hipMemcpyAsync(&s, st->fit_status, 4, hipMemcpyDeviceToHost, stream));
    GEFEN_HIP(hipStreamSynchronize(stream));
    if (cost_out) *cost_out = c;
    if (status_out) *status_out = s;
    return GEFEN_OK;
}

int gefen_state_bytes(const gefen_state* st, int64_t* persistent, int64_t* workspace)
{
    if (!st) return fail(GEFEN_EINVAL, "state is NULL");
    if (persistent) *persistent = st->persistent_bytes;
    if (workspace) *workspace = st->workspace_bytes;
    return GEFEN_OK;
}

int gefen_checkpoint_bytes(const gefen_state* st, int64_t* bytes)
{
    if (!st || !bytes) return fail(GEFEN_EINVAL, "NULL argument");
    *bytes = ckpt_layout(st).total;
    return GEFEN_OK;
}

int gefen_export(const gefen_state* st, void* dst, int64_t bytes, void* stream_)
{
    if (!st || !dst) return fail(GEFEN_EINVAL, "NULL argument");
    const CkptLayout L = ckpt_layout(st);
    if (bytes != L.total) return fail(GEFEN_EINVAL, "checkpoint needs %lld bytes", (long long)L.total);
    hipStream_t stream = as_stream(stream_);
    char* d = static_cast<char*>(dst);
    int64_t hdr[8] = {kCkptMagic | (int64_t(1) << 32), st->n_tensors, st->k, st->code_bytes,
                      st->total_blocks, st->dec_slot, st->enc_slot, 0};
    GEFEN_HIP(hipMemcpyAsync(d + L.header, hdr, sizeof hdr, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(d + L.codes, st->codes, st->code_bytes, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(d + L.scale, st->scale, 4 * st->total_blocks, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(d + L.vmom, st->vmom, 4 * st->total_blocks, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(d + L.cb0, st->cb64[0], 8 * st->k, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(d + L.cb1, st->cb64[1], 8 * st->k, hipMemcpyDefault, stream));
    GEFEN_HIP(hipStreamSynchronize(stream));   // the header lives on this host stack
    return GEFEN_OK;
}

int gefen_import(gefen_state* st, const void* src, int64_t bytes, void* stream_)
{
    if (!st || !src) return fail(GEFEN_EINVAL, "NULL argument");
    const CkptLayout L = ckpt_layout(st);
    if (bytes != L.total) return fail(GEFEN_EINVAL, "checkpoint needs %lld bytes", (long long)L.total);
    hipStream_t stream = as_stream(stream_);
    const char* s = static_cast<const char*>(src);
    // header and both codebooks are checked before anything of the state is touched
    int64_t hdr[8];
    std::vector<double> cbs(2 * static_cast<size_t>(st->k));
    GEFEN_HIP(hipMemcpyAsync(hdr, s + L.header, sizeof hdr, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(cbs.data(), s + L.cb0, 16 * st->k, hipMemcpyDefault, stream));
    GEFEN_HIP(hipStreamSynchronize(stream));
    if (hdr[0] != (kCkptMagic | (int64_t(1) << 32)) || hdr[1] != st->n_tensors ||
        hdr[2] != st->k || hdr[3] != st->code_bytes || hdr[4] != st->total_blocks ||
        hdr[5] < 0 || hdr[5] > 1 || hdr[6] < 0 || hdr[6] > 1)
        return fail(GEFEN_EINVAL, "checkpoint does not match this state");
    // the slots in use: decode and encode (one slot until the first refit; the other
    // holds whatever it was allocated with)
    for (int64_t slot : {hdr[5], hdr[6]})
        if (!valid_codebook(cbs.data() + slot * st->k, st->k))
            return fail(GEFEN_EINVAL, "checkpoint codebook %d is not valid (finite, -1 first, "
                        "+1 last, never decreasing)", static_cast<int>(slot));
    GEFEN_HIP(hipMemcpyAsync(st->codes, s + L.codes, st->code_bytes, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(st->scale, s + L.scale, 4 * st->total_blocks, hipMemcpyDefault, stream));
    GEFEN_HIP(hipMemcpyAsync(st->vmom, s + L.vmom, 4 * st->total_blocks, hipMemcpyDefault, stream));
    double* staging = nullptr;
    GEFEN_HIP(hipMallocAsync(reinterpret_cast<void**>(&staging), 16 * st->k, stream));
    GEFEN_HIP(hipMemcpyAsync(staging, cbs.data(), 16 * st->k, hipMemcpyHostToDevice, stream));
    for (int slot = 0; slot < 2; ++slot) {
        hipError_t e = launch_install_codebook(staging + slot * st->k, st->k, st->ng,
                                               st->cb32[slot], st->cb64[slot], st->mid[slot],
                                               st->guide[slot], stream);
        if (e != hipSuccess) {
            (void)hipFreeAsync(staging, stream);
            return fail(GEFEN_EHIP, "codebook install failed: %s", hipGetErrorString(e));
        }
    }
    (void)hipFreeAsync(staging, stream);
    GEFEN_HIP(hipStreamSynchronize(stream));
    st->dec_slot = static_cast<int>(hdr[5]);
    st->enc_slot = static_cast<int>(hdr[6]);
    return GEFEN_OK;
}

int gefen_profile_begin(gefen_state* st, int32_t max_steps)
{
    if (!st || max_steps < 1) return fail(GEFEN_EINVAL, "bad arguments");
    st->prof_free();
    const size_t n = static_cast<size_t>(max_steps) * st->classes.size() * 2;
    st->prof_events.resize(n, nullptr);
    for (size_t i = 0; i < n; ++i) GEFEN_HIP(hipEventCreate(&st->prof_events[i]));
    if (st->muon_ready) {
        const size_t nm = static_cast<size_t>(max_steps) * st->muon_prof_stride();
        st->muon_prof_events.resize(nm, nullptr);
        for (size_t i = 0; i < nm; ++i) GEFEN_HIP(hipEventCreate(&st->muon_prof_events[i]));
    }
    st->prof_max_steps = max_steps;
    st->prof_steps = 0;
    st->prof_armed = true;
    return GEFEN_OK;
}

int gefen_profile_end(gefen_state* st, int32_t cap, int32_t* n_classes, int32_t* kind,
                      int32_t* vpl, int32_t* threads, int32_t* gdtype, int64_t* launches,
                      double* total_ms, int64_t* elems_per_launch, int64_t* bytes_per_launch)
{
    if (!st || !n_classes) return fail(GEFEN_EINVAL, "bad arguments");
    const size_t ncls = st->classes.size();
    *n_classes = static_cast<int32_t>(ncls);
    if (static_cast<int64_t>(ncls) > cap) return fail(GEFEN_EINVAL, "cap < %zu classes", ncls);
    std::vector<double> ms(ncls, 0.0);
    if (st->prof_armed && st->prof_steps > 0) {
        GEFEN_HIP(hipEventSynchronize(st->prof_events[(st->prof_steps * ncls - 1) * 2 + 1]));
        for (int32_t s = 0; s < st->prof_steps; ++s)
            for (size_t c = 0; c < ncls; ++c) {
                float m = 0.0f;
                GEFEN_HIP(hipEventElapsedTime(&m, st->prof_events[(s * ncls + c) * 2],
                                              st->prof_events[(s * ncls + c) * 2 + 1]));
                ms[c] += m;
            }
    }
    for (size_t c = 0; c < ncls; ++c) {
        const Class& k = st->classes[c];
        if (kind) kind[c] = k.kind;
        if (vpl) vpl[c] = k.vpl;
        if (threads) threads[c] = k.bs;
        if (gdtype) gdtype[c] = k.gdtype;
        if (launches) launches[c] = st->prof_steps;
        if (total_ms) total_ms[c] = ms[c];
        if (elems_per_launch) elems_per_launch[c] = k.elems;
        if (bytes_per_launch) bytes_per_launch[c] = k.bytes;
    }
    st->prof_free();
    return GEFEN_OK;
}

int gefen_stream_mix(float* theta, const void* grad, int32_t grad_dtype, uint8_t* codes,
                     int64_t n, void* stream)
{
    g_err.clear();
    if (n < 0) return fail(GEFEN_EINVAL, "n must be >= 0");
    if (grad_dtype != GEFEN_F32 && grad_dtype != GEFEN_BF16)
        return fail(GEFEN_EDTYPE, "grad_dtype %d is not F32 or BF16", grad_dtype);
    if (n == 0) return GEFEN_OK;
    if (!theta || !grad || !codes) return fail(GEFEN_EINVAL, "NULL array");
    const uintptr_t ga = grad_dtype == GEFEN_F32 ? 15 : 7;
    if ((reinterpret_cast<uintptr_t>(theta) & 15) || (reinterpret_cast<uintptr_t>(grad) & ga) ||
        (reinterpret_cast<uintptr_t>(codes) & 3))
        return fail(GEFEN_EINVAL, "theta must be 16-byte, grad %d-byte, codes 4-byte aligned",
                    static_cast<int>(ga + 1));
    const hipError_t e = launch_stream_mix(theta, grad, grad_dtype == GEFEN_F32 ? DT_F32 : DT_BF16,
                                           codes, n, as_stream(stream));
    if (e != hipSuccess) return fail(GEFEN_EHIP, "stream mix launch: %s", hipGetErrorString(e));
    return GEFEN_OK;
}

void gefen_destroy(gefen_state* st) { delete st; }


// ------------------------------------------------------------------ Gefen-Muon
namespace {

uint16_t host_bf16(float x)
{
    uint32_t b;
    std::memcpy(&b, &x, 4);
    return static_cast<uint16_t>((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

float host_bf16_value(float x)
{
    const uint32_t b = static_cast<uint32_t>(host_bf16(x)) << 16;
    float f;
    std::memcpy(&f, &b, 4);
    return f;
}

// One Newton-Schulz iteration of a shape group on a lane's buffers (ns_plan.h):
// A = X X^T, B = b A + c A A, X' = a X + B X, each a bfloat16 product with float32
// accumulation; `cur` selects the ping-pong buffers that hold X and X^T.
int ns_iteration(const NsLaneBuffers& lb, const NsLaneSizes& z, const NsShape& sh, int cur,
                 float a, float b, float c, hipStream_t stream)
{
    NsGemmArgs prods[3];
    int64_t avail[3][6];
    ns_iteration_products(sh, lb, z, cur, a, b, c, prods, avail);
    for (const NsGemmArgs& p : prods) GEFEN_HIP(launch_ns_gemm(p, stream));
    return GEFEN_OK;
}

// Gefen-Muon codec tiles over every block (host side), in launch order: fp32-gradient
// tensors first, then bf16 (one codec launch per gradient dtype). Tile mode in
// Tile::vpl: 1 (lane per block) for blocks of <= 32 elements, 2 (wave per block, up to
// 4) for <= 2048, else 0 (the workgroup on one block). tile_range[2t, 2t + 1) are
// tensor t's tiles.
int muon_codec_tiles(gefen_state* st, std::vector<Tile>& tiles, std::vector<int64_t>& tile_range)
{
    const int32_t n = st->n_tensors;
    tile_range.assign(2 * static_cast<size_t>(n), 0);
    // block starts on the host (explicit blocks: from the device table)
    std::vector<int64_t> csr_host;
    if (st->explicit_blocks) {
        csr_host.resize(static_cast<size_t>(st->total_blocks + n));
        GEFEN_HIP(hipMemcpy(csr_host.data(), st->csr, 8 * csr_host.size(), hipMemcpyDeviceToHost));
    }
    std::vector<int64_t> csr_at(n + 1, 0);
    for (int32_t t = 0; t < n; ++t)
        csr_at[t + 1] = csr_at[t] + (st->explicit_blocks
                                          ? st->blk_begin[t + 1] - st->blk_begin[t] + 1 : 0);
    for (int32_t pass = 0; pass < 2; ++pass)
    for (int32_t t = 0; t < n; ++t) {
        if (st->gdtype[t] != (pass == 0 ? DT_F32 : DT_BF16)) continue;
        const int64_t csr_base = csr_at[t];
        tile_range[2 * t] = static_cast<int64_t>(tiles.size());
        const int64_t nb = st->blk_begin[t + 1] - st->blk_begin[t];
        const int64_t bb = st->blk_begin[t];
        auto start = [&](int64_t b) {
            return st->explicit_blocks ? csr_host[csr_base + b] : b * st->period[t];
        };
        auto mode_of = [](int64_t len) { return len <= kSmallBlock ? 1 : (len <= 2048 ? 2 : 0); };
        int64_t b = 0;
        while (b < nb) {
            const int mode = mode_of(start(b + 1) - start(b));
            const int cap = mode == 1 ? kThreads : (mode == 2 ? kThreads / 64 : 1);
            Tile tl{};
            tl.elem0 = start(b);
            tl.blk0 = bb + b;
            tl.seg = t;
            int cnt = 0;
            while (b < nb && cnt < cap && mode_of(start(b + 1) - start(b)) == mode) {
                ++cnt;
                ++b;
            }
            tl.nblk = static_cast<int16_t>(cnt);
            tl.nelem = start(b) - tl.elem0;
            tl.vpl = static_cast<uint8_t>(mode);
            tiles.push_back(tl);
        }
        tile_range[2 * t + 1] = static_cast<int64_t>(tiles.size());
        st->muon_dt_count[pass] = static_cast<int64_t>(tiles.size()) - st->muon_dt_first[pass];
        if (pass == 0) st->muon_dt_first[1] = static_cast<int64_t>(tiles.size());
    }

    return GEFEN_OK;
}

// Per-lane Newton-Schulz buffers (sized for the lane's largest group), the host check of
// every product and prep/update extent the steps will run, and the side stream.
int muon_lane_resources(gefen_state* st)
{
    int rc;
    for (int l = 0; l < kNsLanes; ++l) {
        gefen_state::MuonLane& ln = st->muon_lane[l];
        if (ln.groups.empty()) continue;
        ln.size = ns_lane_sizes(st->muon_groups, ln.groups);
        NsLaneBuffers& lb = ln.buf;
        for (int k = 0; k < 2; ++k) {
            if ((rc = st->alloc(&lb.x[k], 2 * static_cast<size_t>(ln.size.x_elems), false))) return rc;
            if ((rc = st->alloc(&lb.xt[k], 2 * static_cast<size_t>(ln.size.x_elems), false))) return rc;
        }
        if ((rc = st->alloc(&lb.a, 2 * static_cast<size_t>(ln.size.a_elems), false))) return rc;
        if ((rc = st->alloc(&lb.b, 2 * static_cast<size_t>(ln.size.a_elems), false))) return rc;
        if ((rc = st->alloc(&lb.partial, 4 * static_cast<size_t>(ln.size.partial_elems), false)))
            return rc;
        for (int32_t gi : ln.groups) {
            const std::string why = ns_check_group(st->muon_groups[gi], lb, ln.size);
            if (!why.empty()) return fail(GEFEN_EINVAL, "internal: %s", why.c_str());
        }
    }
    for (int l = 1; l < kNsLanes; ++l) {
        if (st->muon_lane[l].groups.empty()) continue;
        if (!st->muon_fork)
            GEFEN_HIP(hipEventCreateWithFlags(&st->muon_fork, hipEventDisableTiming));
        GEFEN_HIP(hipStreamCreateWithFlags(&st->muon_side[l - 1], hipStreamNonBlocking));
        GEFEN_HIP(hipEventCreateWithFlags(&st->muon_join[l - 1], hipEventDisableTiming));
    }
    return GEFEN_OK;
}

// One shape group on a lane's buffers runs in phases, each a few launches on the lane's
// stream: 0 normalises its momentum matrices into the layout (prep), 1 .. the
// Newton-Schulz iterations (the vector kernel does all of them in phase 1), the last
// writes the updates.
int muon_group_phases(const NsGroup& g, int32_t ns_steps)
{
    return 2 + (g.shape.m == 1 ? 1 : ns_steps);
}

struct MuonGroupRun {
    float ca, cb, cc, decay;
    double lr;
    int32_t ns_steps;
};

// Enqueues phase `phase` of group g; cur (the buffer parity of X, X^T) advances with the
// iterations.
int muon_group_phase(gefen_state* st, const gefen_state::MuonLane& lane, const NsGroup& g,
                     const MuonGroupRun& r, int phase, int& cur, hipStream_t ls)
{
    const NsShape& sh = g.shape;
    const NsLaneBuffers& ln = lane.buf;
    const int64_t xs = sh.m * sh.ldx, ts = sh.ldx * sh.ldm;   // batch strides of X, X^T
    const int last = muon_group_phases(g, r.ns_steps) - 1;
    if (phase == 0) {
        cur = 0;
        for (const auto& pt : g.parts) {
            const int32_t* tof = st->muon_tensor_of + g.first + pt.first;
            uint16_t* x0 = ln.x[0] + pt.first * xs;
            uint16_t* t0 = ln.xt[0] + pt.first * ts;
            if (sh.m == 1)
                GEFEN_HIP(launch_ns_prep(st->muon_u, st->muon_u_off, tof, st->muon_norm, pt.count,
                                         1, pt.rows * pt.cols, x0, xs, sh.ldx, t0, ts, sh.ldm, ls));
            else if (!pt.transposed)
                GEFEN_HIP(launch_ns_prep(st->muon_u, st->muon_u_off, tof, st->muon_norm, pt.count,
                                         pt.rows, pt.cols, x0, xs, sh.ldx, t0, ts, sh.ldm, ls));
            else
                GEFEN_HIP(launch_ns_prep(st->muon_u, st->muon_u_off, tof, st->muon_norm, pt.count,
                                         pt.rows, pt.cols, t0, ts, sh.ldm, x0, xs, sh.ldx, ls));
        }
    } else if (phase < last) {
        if (sh.m == 1) {
            GEFEN_HIP(launch_muon_ns_vec(ln.x[0], static_cast<int32_t>(sh.count), sh.n, sh.ldx,
                                         r.ns_steps, r.ca, r.cb, r.cc, ls));
        } else {
            const int rc = ns_iteration(ln, lane.size, sh, cur, r.ca, r.cb, r.cc, ls);
            if (rc) return rc;
            cur ^= 1;
        }
    } else {
        for (const auto& pt : g.parts) {
            const int32_t* tof = st->muon_tensor_of + g.first + pt.first;
            const double scale = std::sqrt(std::max(1.0, static_cast<double>(pt.rows) / pt.cols));
            const float step = static_cast<float>(r.lr * scale);
            if (sh.m == 1)
                GEFEN_HIP(launch_ns_update(ln.x[cur] + pt.first * xs, xs, sh.ldx, st->segs, tof,
                                           pt.count, 1, pt.rows * pt.cols, r.decay, step, ls));
            else if (!pt.transposed)   // theta = X' (m x n)
                GEFEN_HIP(launch_ns_update(ln.x[cur] + pt.first * xs, xs, sh.ldx, st->segs, tof,
                                           pt.count, pt.rows, pt.cols, r.decay, step, ls));
            else                       // theta = X'^T (n x m)
                GEFEN_HIP(launch_ns_update(ln.xt[cur] + pt.first * ts, ts, sh.ldm, st->segs, tof,
                                           pt.count, pt.rows, pt.cols, r.decay, step, ls));
        }
    }
    return GEFEN_OK;
}

}  // namespace

int gefen_muon_init(gefen_state* st, const int64_t* rows, int32_t n_tensors, void* stream_)
{
    if (!st || !rows) return fail(GEFEN_EINVAL, "NULL argument");
    if (n_tensors != st->n_tensors)
        return fail(GEFEN_EINVAL, "n_tensors = %d, state has %d", n_tensors, st->n_tensors);
    if (st->muon_ready) return fail(GEFEN_EINVAL, "gefen_muon_init was already called");
    const int32_t n = n_tensors;
    for (int32_t t = 0; t < n; ++t)
        if (rows[t] < 1 || st->numel[t] % rows[t] != 0)
            return fail(GEFEN_EINVAL, "rows[%d] = %lld does not divide numel %lld", t,
                        (long long)rows[t], (long long)st->numel[t]);
    hipStream_t stream = as_stream(stream_);

    int rc;
    std::vector<Tile> tiles;
    std::vector<int64_t> tile_range;
    if ((rc = muon_codec_tiles(st, tiles, tile_range))) return rc;
    std::vector<int32_t> order;
    const std::string why = ns_plan_groups(n, rows, st->numel.data(), st->muon_groups, order);
    if (!why.empty()) return fail(GEFEN_EINVAL, "%s", why.c_str());
    {
        std::vector<int32_t> lanes[kNsLanes];
        ns_assign_lanes(st->muon_groups, lanes);
        for (int l = 0; l < kNsLanes; ++l) st->muon_lane[l].groups = lanes[l];
    }

    st->muon_n_tiles = static_cast<int64_t>(tiles.size());
    if ((rc = st->alloc(&st->muon_tiles, sizeof(Tile) * tiles.size(), false))) return rc;
    if ((rc = st->alloc(&st->muon_tile_range, 8 * tile_range.size(), false))) return rc;
    if ((rc = st->alloc(&st->muon_tile_ss, 4 * tiles.size(), false))) return rc;
    if ((rc = st->alloc(&st->muon_norm, 4 * static_cast<size_t>(n), false))) return rc;
    if ((rc = st->alloc(&st->muon_tensor_of, 4 * order.size(), false))) return rc;
    if ((rc = st->alloc(&st->muon_u, 2 * static_cast<size_t>(st->code_off[n]), false))) return rc;
    GEFEN_HIP(hipMemcpy(st->muon_tiles, tiles.data(), sizeof(Tile) * tiles.size(), hipMemcpyHostToDevice));
    GEFEN_HIP(hipMemcpy(st->muon_tile_range, tile_range.data(), 8 * tile_range.size(), hipMemcpyHostToDevice));
    GEFEN_HIP(hipMemcpy(st->muon_tensor_of, order.data(), 4 * order.size(), hipMemcpyHostToDevice));
    if ((rc = st->alloc(&st->muon_u_off, 8 * static_cast<size_t>(n), false))) return rc;
    GEFEN_HIP(hipMemcpy(st->muon_u_off, st->code_off.data(), 8 * static_cast<size_t>(n),
                        hipMemcpyHostToDevice));
    if ((rc = muon_lane_resources(st))) return rc;
    GEFEN_HIP(hipStreamSynchronize(stream));
    st->muon_ready = true;
    return GEFEN_OK;
}

int gefen_muon_step(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
                    int32_t n_tensors, double lr, double momentum, double weight_decay,
                    int32_t nesterov, int32_t ns_steps, double ns_a, double ns_b, double ns_c,
                    double ns_eps, void* stream_)
{
    int rc = check_against_state(st, params, n_tensors, true, "params");
    if (rc) return rc;
    if ((rc = check_against_state(st, grads, n_tensors, false, "grads"))) return rc;
    if (!st->muon_ready) return fail(GEFEN_EINVAL, "call gefen_muon_init first");
    if (!(momentum >= 0.0 && momentum < 1.0)) return fail(GEFEN_EINVAL, "momentum must be in [0, 1)");
    if (!finite_f(lr) || !finite_f(weight_decay)) return fail(GEFEN_EINVAL, "lr and weight_decay must be finite");
    if (ns_steps < 0 || ns_steps > 100) return fail(GEFEN_EINVAL, "ns_steps must be in [0, 100]");
    if (!finite_f(ns_a) || !finite_f(ns_b) || !finite_f(ns_c))
        return fail(GEFEN_EINVAL, "Newton-Schulz coefficients must be finite");
    if (!finite_f(ns_eps) || ns_eps <= 0.0) return fail(GEFEN_EINVAL, "ns_eps must be finite and > 0");
    hipStream_t stream = as_stream(stream_);
    if ((rc = refresh_segs(st, params, grads, stream))) return rc;
    const bool prof = st->prof_armed && st->muon_prof_steps < st->prof_max_steps &&
                      !st->muon_prof_events.empty();
    hipEvent_t* ev = prof ? &st->muon_prof_events[st->muon_prof_steps * st->muon_prof_stride()]
                          : nullptr;
    if (prof) GEFEN_HIP(hipEventRecord(ev[0], stream));

    for (int d = 0; d < 2; ++d)
        GEFEN_HIP(launch_muon_codec(st->code_bits, d == 0 ? DT_F32 : DT_BF16,
                                    st->muon_tiles + st->muon_dt_first[d], st->muon_dt_count[d],
                                    st->segs, st->codes, st->scale, codebook_dev(st),
                                    static_cast<float>(momentum),
                                    static_cast<float>(1.0 - momentum), nesterov ? 1 : 0,
                                    st->muon_u, st->muon_tile_ss + st->muon_dt_first[d], stream));
    GEFEN_HIP(launch_muon_norm(st->muon_tile_ss, st->muon_tile_range, st->n_tensors,
                               host_bf16_value(static_cast<float>(ns_eps)), st->muon_norm, stream));
    if (prof) GEFEN_HIP(hipEventRecord(ev[1], stream));
    const float decay = static_cast<float>(1.0 - lr * weight_decay);
    const float ca = static_cast<float>(ns_a), cb = static_cast<float>(ns_b),
                cc = static_cast<float>(ns_c);
    const MuonGroupRun run{ca, cb, cc, decay, lr, ns_steps};
    // The lanes' phases are enqueued in turn, so that every stream holds work from the
    // start (enqueueing one lane whole first would leave the others idle for as long as
    // the host takes to launch the first one's kernels).
    if (st->muon_fork) GEFEN_HIP(hipEventRecord(st->muon_fork, stream));
    struct Cursor {
        const gefen_state::MuonLane* lane;
        hipStream_t s;
        size_t gi;
        int phase, cur;
    } cursors[kNsLanes];
    for (int l = 1; l <= kNsLanes; ++l) {   // the side lanes, then lane 0
        const int li = l % kNsLanes;
        hipStream_t s = li == 0 ? stream : st->muon_side[li - 1];
        if (li != 0 && !st->muon_lane[li].groups.empty())
            GEFEN_HIP(hipStreamWaitEvent(s, st->muon_fork, 0));
        cursors[l - 1] = Cursor{&st->muon_lane[li], s, 0, 0, 0};
    }
    for (bool more = true; more;) {
        more = false;
        for (Cursor& c : cursors) {
            if (c.gi >= c.lane->groups.size()) continue;
            const NsGroup& g = st->muon_groups[c.lane->groups[c.gi]];
            if ((rc = muon_group_phase(st, *c.lane, g, run, c.phase, c.cur, c.s))) return rc;
            if (++c.phase == muon_group_phases(g, ns_steps)) {
                c.phase = 0;
                ++c.gi;
            }
            more = more || c.gi < c.lane->groups.size();
        }
    }
    for (int l = 1; l < kNsLanes; ++l) {
        if (st->muon_lane[l].groups.empty()) continue;
        GEFEN_HIP(hipEventRecord(st->muon_join[l - 1], st->muon_side[l - 1]));
        GEFEN_HIP(hipStreamWaitEvent(stream, st->muon_join[l - 1], 0));
    }
    if (prof) {
        GEFEN_HIP(hipEventRecord(ev[st->muon_prof_stride() - 1], stream));
        ++st->muon_prof_steps;
    }
    st->dec_slot = st->enc_slot;
    return GEFEN_OK;
}

int gefen_muon_profile_end(gefen_state* st, int32_t* steps, double* codec_ms, double* ortho_ms)
{
    if (!st || !steps || !codec_ms || !ortho_ms) return fail(GEFEN_EINVAL, "NULL argument");
    *steps = 0;
    *codec_ms = *ortho_ms = 0.0;
    const size_t k = st->muon_prof_stride();
    if (st->prof_armed && st->muon_prof_steps > 0) {
        GEFEN_HIP(hipEventSynchronize(st->muon_prof_events[st->muon_prof_steps * k - 1]));
        for (int32_t s = 0; s < st->muon_prof_steps; ++s) {
            hipEvent_t* ev = &st->muon_prof_events[s * k];
            float a = 0.0f, o = 0.0f;
            GEFEN_HIP(hipEventElapsedTime(&a, ev[0], ev[1]));
            GEFEN_HIP(hipEventElapsedTime(&o, ev[1], ev[2]));
            *codec_ms += a;
            *ortho_ms += o;
        }
        *steps = st->muon_prof_steps;
    }
    st->prof_free();
    return GEFEN_OK;
}

int gefen_newton_schulz(const uint16_t* x_in, uint16_t* x_out, int32_t batch, int64_t m,
                        int64_t n, int32_t steps, double a, double b, double c, void* stream_)
{
    if (!x_in || !x_out) return fail(GEFEN_EINVAL, "NULL argument");
    if (batch < 1 || batch > 65535) return fail(GEFEN_EINVAL, "batch must be in [1, 65535]");
    if (m < 1 || m > n || n > 0x7ffff000LL)
        return fail(GEFEN_EINVAL, "need 1 <= m <= n <= 2^31 - 4096 (m = %lld, n = %lld)",
                    (long long)m, (long long)n);
    if (steps < 0 || steps > 100) return fail(GEFEN_EINVAL, "steps must be in [0, 100]");
    if (!finite_f(a) || !finite_f(b) || !finite_f(c))
        return fail(GEFEN_EINVAL, "Newton-Schulz coefficients must be finite");
    hipStream_t stream = as_stream(stream_);
    NsGroup g{};
    g.shape = ns_shape(batch, m, n);
    g.parts.push_back(NsPart{m, n, 0, batch, false});
    const NsShape& sh = g.shape;
    const NsLaneSizes z = ns_lane_sizes(std::vector<NsGroup>{g}, std::vector<int32_t>{0});
    if (z.x_elems > (int64_t(1) << 40)) return fail(GEFEN_EINVAL, "matrices too large");
    NsLaneBuffers lb{};
    std::vector<void*> bufs;
    auto release = [&]() {
        for (void* p : bufs) (void)hipFreeAsync(p, stream);
    };
    auto get = [&](void** p, int64_t bytes) -> int {
        hipError_t e = hipMallocAsync(p, static_cast<size_t>(std::max<int64_t>(bytes, 16)), stream);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            release();
            return fail(GEFEN_ENOMEM, "hipMallocAsync(%lld) failed: %s", (long long)bytes,
                        hipGetErrorString(e));
        }
        bufs.push_back(*p);
        return GEFEN_OK;
    };
    int rc;
    for (int k = 0; k < 2; ++k) {
        if ((rc = get(reinterpret_cast<void**>(&lb.x[k]), 2 * z.x_elems))) return rc;
        if ((rc = get(reinterpret_cast<void**>(&lb.xt[k]), 2 * z.x_elems))) return rc;
    }
    if ((rc = get(reinterpret_cast<void**>(&lb.a), 2 * z.a_elems))) return rc;
    if ((rc = get(reinterpret_cast<void**>(&lb.b), 2 * z.a_elems))) return rc;
    if ((rc = get(reinterpret_cast<void**>(&lb.partial), 4 * z.partial_elems))) return rc;
    {
        const std::string why = ns_check_group(g, lb, z);
        if (!why.empty()) {
            release();
            return fail(GEFEN_EINVAL, "internal: %s", why.c_str());
        }
    }
    const int64_t xs = sh.m * sh.ldx, ts = sh.ldx * sh.ldm;
    auto run = [&]() -> int {
        GEFEN_HIP(launch_ns_prep(x_in, nullptr, nullptr, nullptr, batch, m, n, lb.x[0], xs,
                                 sh.ldx, lb.xt[0], ts, sh.ldm, stream));
        int cur = 0;
        if (m == 1) {
            GEFEN_HIP(launch_muon_ns_vec(lb.x[0], batch, n, sh.ldx, steps, static_cast<float>(a),
                                         static_cast<float>(b), static_cast<float>(c), stream));
        } else {
            for (int32_t it = 0; it < steps; ++it) {
                const int r = ns_iteration(lb, z, sh, cur, static_cast<float>(a),
                                           static_cast<float>(b), static_cast<float>(c), stream);
                if (r) return r;
                cur ^= 1;
            }
        }
        GEFEN_HIP(launch_ns_unpad(lb.x[cur], xs, sh.ldx, batch, m, n, x_out, stream));
        return GEFEN_OK;
    };
    rc = run();
    release();
    return rc;
}

}  // extern "C"
