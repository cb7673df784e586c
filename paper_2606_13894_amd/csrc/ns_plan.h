// Planning of the Newton-Schulz products of Gefen-Muon (appendix "Gefen-Muon": Muon's
// orthogonalisation X <- a X + (b A + c A A) X, A = X X^T, on bfloat16 matrices).
// Plain C++ with no HIP types, so that host-only tests can build and check it.
//
// Layout of one shape group of `count` wide matrices (m rows <= n columns):
//   X   count x m x ldx   row-major, ldx = n rounded up to 64 (whole K stages), zero in
//       columns n .. ldx-1
//   Xt  count x ldx x ldm row-major X^T, ldm = m rounded up to 64 (8 for a vector), zero
//       in columns m .. ldm-1 (rows n .. ldx-1 are never read)
//   A   count x m x ldm   (A = X X^T, symmetric), zero in columns m .. ldm-1
//   B   count x m x ldm   (B = b A + c A A, symmetric), same padding
// Every product reads both operands along contiguous K:
//   Gram     A = X X^T     P = X, Q = X, K = ldx, symmetric (upper tiles, mirrored)
//   Poly     B = c A A + b A   P = Q = A (A A = A A^T), K = ldm, E = A, symmetric
//   Combine  X' = B X + a X    P = B, Q = Xt (X[k][j] = Xt[j][k]), K = ldm, E^T = Xt;
//            writes X' and X'^T (the next iteration's Xt)
#pragma once

#include <stdint.h>

#include <algorithm>
#include <cstdio>
#include <string>
#include <vector>

#if defined(__HIPCC__)
#define NS_HOST_DEVICE __host__ __device__
#else
#define NS_HOST_DEVICE
#endif

namespace gefen {

// Output tiles of one workgroup: 128 x 128 (four waves of 64 x 64, two workgroups per
// compute unit) or 256 x 256 (eight waves of 64 x 128, one workgroup per compute unit:
// twice the flops per loaded byte and four times the matrix-core work per K stage, to
// cover memory latency on the large products). kNsThreads is the 128 tile's workgroup.
constexpr int kNsTileSmall = 128;
constexpr int kNsTileBig = 256;
constexpr int kNsBK = 64;      // K of one pipeline stage
constexpr int kNsThreads = 256;
constexpr int kNsCUs = 256;
constexpr int kNsBand = 4;     // tile rows per band of a non-symmetric product

// One batched product C[i][j] = sum_k P[i][k] Q[j][k] (i < M, j < N, k < K), then
//   value(i, j) = bf16(alpha * C[i][j] + beta * E[i][j]),  E[i][j] = et[j * lde + i]
// (E absent: beta ignored; E^T rows are read up to lde and must be zero from M on),
// written to O[i][j] (i < M, j < o_cols; columns N .. o_cols-1 are zero) and to Ot[j][i]
// (j < N, i < ot_cols; zero for i >= M). Symmetric mode (M == N, P == Q): only the tiles
// on and above the diagonal run, and each tile above it also writes its mirror through
// Ot (= O, ot_cols = o_cols). Every E load and O or Ot store is a 16-byte row segment:
// the column counts, leading dimensions and batch strides are multiples of 8. Split-K (splits > 1,
// symmetric, no E): workgroup s of a tile sums K range [s * kchunk, (s+1) * kchunk) and
// writes float32 partial[((s * batch + b) * M + i) * N + j]; ns_reduce adds the chunks in
// order and writes O.
struct NsGemmArgs {
    const uint16_t* p;
    int64_t ldp, sp;
    const uint16_t* q;
    int64_t ldq, sq;
    const uint16_t* et;
    int64_t lde, se;
    uint16_t* o;
    int64_t ldo, so;
    uint16_t* ot;
    int64_t ldot, sot;
    float* partial;
    int32_t tile;         // kNsTileSmall or kNsTileBig
    int32_t M, N, K;
    int32_t o_cols, ot_cols;
    int32_t batch, sym, splits;
    int32_t tm, tn;       // tiles along M and along N
    int32_t tiles;        // tiles per batch entry (symmetric: tm (tm + 1) / 2)
    int32_t kchunk;       // split-K chunk (a multiple of kNsBK); K when splits == 1
    float alpha, beta;
};

inline int64_t ns_round64(int64_t v) { return (v + 63) / 64 * 64; }
inline int32_t ns_tiles_along(int64_t v, int tile)
{
    return static_cast<int32_t>((v + tile - 1) / tile);
}

// Workgroups resident on the GPU at once, and the share of their rounds that `groups`
// workgroups fill.
inline int64_t ns_slots(int tile) { return tile == kNsTileBig ? kNsCUs : 2 * kNsCUs; }
inline double ns_fill(int64_t groups, int tile)
{
    const int64_t slots = ns_slots(tile);
    return double(groups) / double((groups + slots - 1) / slots * slots);
}

// Sizes of one shape group.
struct NsShape {
    int64_t count, m, n, ldx, ldm;
    int32_t splits;   // K chunks of the Gram product
    int32_t kchunk;   // their length (a multiple of kNsBK; ldx when splits == 1)
    int32_t tile_gram, tile_poly, tile_comb;
};

// Split the Gram product over K so that its workgroups (count x t (t + 1) / 2 upper
// tiles, times the split) fill their rounds on the GPU: the smallest split whose rounds
// are at least 90 % full, else the fullest, with chunks of at least 8 stages and at most
// 32 chunks. A lone tall-skinny matrix (a token embedding: 21 small tiles at m = 768)
// splits 22 ways; a batch that fills its rounds (the GPT-2 MLP group: 504 small tiles)
// does not split.
inline int32_t ns_gram_splits(int64_t count, int64_t m, int64_t ldx, int tile)
{
    const int64_t t = ns_tiles_along(m, tile);
    const int64_t work = count * t * (t + 1) / 2;
    const int64_t smax = std::max<int64_t>(1, std::min<int64_t>(32, ldx / (8 * kNsBK)));
    int64_t best = 1;
    double best_fill = 0.0;
    for (int64_t s = 1; s <= smax; ++s) {
        const double fill = ns_fill(work * s, tile);
        if (fill >= 0.9) return static_cast<int32_t>(s);
        if (fill > best_fill + 1e-12) {
            best = s;
            best_fill = fill;
        }
    }
    return static_cast<int32_t>(best);
}

// The big tile for a product of M x N outputs (upper tiles only when symmetric) when both
// sides hold at least four big tiles and its workgroups fill at least 75 % of their
// rounds; else the small tile. (Measured on the model shapes: at M = 768 the small tile
// is faster for every product -- the MLP combine 186 against 231 us, the Gram 72 against
// 154 us with its split -- and at M = 2048 the big one by about 8 %.)
inline int ns_pick_tile(int64_t count, int64_t M, int64_t N, bool sym, int32_t splits = 1)
{
    if (M < 4 * kNsTileBig || N < 4 * kNsTileBig) return kNsTileSmall;
    const int64_t tm = ns_tiles_along(M, kNsTileBig), tn = ns_tiles_along(N, kNsTileBig);
    const int64_t tiles = sym ? tm * (tm + 1) / 2 : tm * tn;
    return ns_fill(count * tiles * splits, kNsTileBig) >= 0.75 ? kNsTileBig : kNsTileSmall;
}

inline NsShape ns_shape(int64_t count, int64_t m, int64_t n)
{
    NsShape s{count, m, n, ns_round64(n), m > 1 ? ns_round64(m) : 8, 1, 0, kNsTileSmall,
              kNsTileSmall, kNsTileSmall};
    s.kchunk = static_cast<int32_t>(s.ldx);
    if (m < 2) return s;   // vectors have no matrix products
    // the Gram product: the big tile when it fills the GPU with its own best split
    const int32_t sb = ns_gram_splits(count, m, s.ldx, kNsTileBig);
    s.tile_gram = ns_pick_tile(count, m, m, true, sb);
    s.splits = s.tile_gram == kNsTileBig ? sb : ns_gram_splits(count, m, s.ldx, kNsTileSmall);
    if (s.splits > 1) {
        // equal chunks of whole stages; the last one may be shorter, none is empty
        const int64_t chunk = (s.ldx + s.splits - 1) / s.splits;
        s.kchunk = static_cast<int32_t>((chunk + kNsBK - 1) / kNsBK * kNsBK);
        s.splits = static_cast<int32_t>((s.ldx + s.kchunk - 1) / s.kchunk);
        if (s.splits < 2) s.kchunk = static_cast<int32_t>(s.ldx);
    }
    s.tile_poly = ns_pick_tile(count, m, m, true);
    s.tile_comb = ns_pick_tile(count, m, n, false);
    return s;
}

// Elements each lane buffer needs for a group.
inline int64_t ns_x_elems(const NsShape& s) { return s.count * s.ldx * s.ldm; }   // X, Xt
inline int64_t ns_a_elems(const NsShape& s) { return s.count * s.m * s.ldm; }     // A, B
inline int64_t ns_partial_elems(const NsShape& s)
{
    return s.splits > 1 ? int64_t(s.splits) * s.count * s.m * s.m : 0;
}

inline void ns_fill_tiles(NsGemmArgs& a, int tile)
{
    a.tile = tile;
    a.tm = ns_tiles_along(a.M, tile);
    a.tn = ns_tiles_along(a.N, tile);
    a.tiles = a.sym ? a.tm * (a.tm + 1) / 2 : a.tm * a.tn;
}

// Work item `wid` of a product: batch entry, K chunk and output tile (row and column
// tile). Work items run batch-major, then chunk, then tile; symmetric products number
// their upper tiles row by row. Other products number their tiles in bands of up to
// kNsBand tile rows, column by column inside a band, so that the workgroups that run at
// once on an XCD (its 32 compute units take consecutive work items) share a few row and
// column slabs of the operands in its L2: 4 x 8 tiles read 12 slabs where a row of 32
// tiles reads 33.
struct NsWork {
    int64_t b;
    int32_t s, ti, tj;
};

inline NS_HOST_DEVICE NsWork ns_decode(const NsGemmArgs& a, int64_t wid)
{
    NsWork w;
    const int64_t per_b = int64_t(a.splits) * a.tiles;
    w.b = wid / per_b;
    const int32_t r = static_cast<int32_t>(wid - w.b * per_b);
    w.s = r / a.tiles;
    int32_t t = r - w.s * a.tiles;
    if (a.sym) {
        int32_t ti = 0;
        while (t >= a.tm - ti) {
            t -= a.tm - ti;
            ++ti;
        }
        w.ti = ti;
        w.tj = ti + t;
    } else {
        const int32_t band = t / (kNsBand * a.tn);
        const int32_t r = t - band * (kNsBand * a.tn);
        const int32_t rows = a.tm - band * kNsBand < kNsBand ? a.tm - band * kNsBand : kNsBand;
        w.ti = band * kNsBand + r % rows;
        w.tj = r / rows;
    }
    return w;
}

inline NsGemmArgs ns_gram_args(const NsShape& s, const uint16_t* x, uint16_t* a_out,
                               float* partial)
{
    NsGemmArgs a{};
    a.p = a.q = x;
    a.ldp = a.ldq = s.ldx;
    a.sp = a.sq = s.m * s.ldx;
    a.o = a.ot = a_out;
    a.ldo = a.ldot = s.ldm;
    a.so = a.sot = s.m * s.ldm;
    a.M = a.N = static_cast<int32_t>(s.m);
    a.K = static_cast<int32_t>(s.ldx);
    a.o_cols = static_cast<int32_t>(s.ldm);
    a.ot_cols = static_cast<int32_t>(s.ldm);
    a.batch = static_cast<int32_t>(s.count);
    a.sym = 1;
    a.splits = s.splits;
    a.alpha = 1.0f;
    a.beta = 0.0f;
    a.kchunk = s.kchunk;
    if (s.splits > 1) a.partial = partial;
    ns_fill_tiles(a, s.tile_gram);
    return a;
}

inline NsGemmArgs ns_poly_args(const NsShape& s, const uint16_t* a_in, uint16_t* b_out, float b,
                               float c)
{
    NsGemmArgs a{};
    a.p = a.q = a.et = a_in;
    a.ldp = a.ldq = a.lde = s.ldm;
    a.sp = a.sq = a.se = s.m * s.ldm;
    a.o = a.ot = b_out;
    a.ldo = a.ldot = s.ldm;
    a.so = a.sot = s.m * s.ldm;
    a.M = a.N = static_cast<int32_t>(s.m);
    a.K = static_cast<int32_t>(s.ldm);
    a.o_cols = static_cast<int32_t>(s.ldm);
    a.ot_cols = static_cast<int32_t>(s.ldm);
    a.batch = static_cast<int32_t>(s.count);
    a.sym = 1;
    a.splits = 1;
    a.kchunk = a.K;
    a.alpha = c;
    a.beta = b;
    ns_fill_tiles(a, s.tile_poly);
    return a;
}

// x_out / xt_out may be null (not needed after the last iteration).
inline NsGemmArgs ns_combine_args(const NsShape& s, const uint16_t* b_in, const uint16_t* xt,
                                  uint16_t* x_out, uint16_t* xt_out, float a_coef)
{
    NsGemmArgs a{};
    a.p = b_in;
    a.ldp = s.ldm;
    a.sp = s.m * s.ldm;
    a.q = a.et = xt;
    a.ldq = a.lde = s.ldm;
    a.sq = a.se = s.ldx * s.ldm;
    a.o = x_out;
    a.ldo = s.ldx;
    a.so = s.m * s.ldx;
    a.ot = xt_out;
    a.ldot = s.ldm;
    a.sot = s.ldx * s.ldm;
    a.M = static_cast<int32_t>(s.m);
    a.N = static_cast<int32_t>(s.n);
    a.K = static_cast<int32_t>(s.ldm);
    a.o_cols = static_cast<int32_t>(s.ldx);
    a.ot_cols = static_cast<int32_t>(s.ldm);
    a.batch = static_cast<int32_t>(s.count);
    a.sym = 0;
    a.splits = 1;
    a.kchunk = a.K;
    a.alpha = 1.0f;
    a.beta = a_coef;
    ns_fill_tiles(a, s.tile_comb);
    return a;
}

// Workgroups of a product: tiles x splits x batch, rounded up to a multiple of 8 (the
// kernel deals contiguous runs of work items to the eight XCDs).
inline int64_t ns_workgroups(const NsGemmArgs& a)
{
    const int64_t w = int64_t(a.batch) * a.splits * a.tiles;
    return (w + 7) / 8 * 8;
}

// Furthest element (exclusive) that a batched row-major operand touches, relative to its
// pointer: rows [0, rows) of cols elements each, leading dimension ld, batch stride st.
inline int64_t ns_extent(int64_t batch, int64_t st, int64_t rows, int64_t ld, int64_t cols)
{
    if (batch <= 0 || rows <= 0 || cols <= 0) return 0;
    return (batch - 1) * st + (rows - 1) * ld + cols;
}

// Checks a product against the kernel's assumptions and against the elements available
// behind each pointer (to the end of its allocation). Returns an empty string when the
// product is valid, else the reason.
inline std::string ns_check(const NsGemmArgs& a, int64_t p_avail, int64_t q_avail,
                            int64_t e_avail, int64_t o_avail, int64_t ot_avail,
                            int64_t partial_avail)
{
    char buf[256];
    auto bad = [&](const char* what) {
        std::snprintf(buf, sizeof buf, "Newton-Schulz product: %s (M %d N %d K %d batch %d)",
                      what, a.M, a.N, a.K, a.batch);
        return std::string(buf);
    };
    if (a.M < 1 || a.N < 1 || a.K < 1 || a.batch < 1) return bad("empty product");
    if (a.K % kNsBK || a.ldp % 8 || a.ldq % 8 || a.sp % 8 || a.sq % 8)
        return bad("K or operand alignment");
    if (a.K > a.ldp || a.K > a.ldq) return bad("K beyond a leading dimension");
    // each tile reads its operand rows through buffer resources with 32-bit byte ranges
    // and offsets: a tile's rows must span less than 2 GiB (rows of < 4 Mi elements)
    if (2 * int64_t(a.tile) * a.ldp >= (int64_t(1) << 31) ||
        2 * int64_t(a.tile) * a.ldq >= (int64_t(1) << 31))
        return bad("a tile's operand rows span 2 GiB");
    if (!a.p || !a.q) return bad("missing operand");
    if (a.tile != kNsTileSmall && a.tile != kNsTileBig) return bad("tile size");
    const int64_t tm = ns_tiles_along(a.M, a.tile), tn = ns_tiles_along(a.N, a.tile);
    if (a.tm != tm || a.tn != tn || a.tiles != (a.sym ? tm * (tm + 1) / 2 : tm * tn))
        return bad("tile counts");
    if (a.sym && (a.M != a.N || a.p != a.q)) return bad("symmetric product of unequal operands");
    if (a.splits < 1 || a.splits > 64) return bad("split count");
    if (a.splits > 1) {
        if (!a.sym || a.et || !a.partial) return bad("split-K needs a symmetric product without E");
        if (a.kchunk % kNsBK || int64_t(a.kchunk) * a.splits < a.K ||
            int64_t(a.kchunk) * (a.splits - 1) >= a.K)
            return bad("split-K chunks");
        if (int64_t(a.splits) * a.batch * a.M * a.N > partial_avail) return bad("partial buffer");
    } else if (a.kchunk != a.K) {
        return bad("K chunk");
    }
    if (ns_extent(a.batch, a.sp, a.M, a.ldp, a.K) > p_avail) return bad("P beyond its buffer");
    if (ns_extent(a.batch, a.sq, a.N, a.ldq, a.K) > q_avail) return bad("Q beyond its buffer");
    if (a.et) {
        if (a.lde % 8 || a.se % 8 || a.lde < a.M) return bad("E layout");
        if (ns_extent(a.batch, a.se, a.N, a.lde, a.lde) > e_avail) return bad("E beyond its buffer");
    }
    if (a.o) {
        if (a.ldo % 8 || a.so % 8 || a.o_cols % 8 || a.o_cols < a.N || a.o_cols > a.ldo)
            return bad("O layout");
        if (ns_extent(a.batch, a.so, a.M, a.ldo, a.o_cols) > o_avail) return bad("O beyond its buffer");
    }
    if (a.ot) {
        if (a.ldot % 8 || a.sot % 8 || a.ot_cols % 8 || a.ot_cols < a.M || a.ot_cols > a.ldot)
            return bad("Ot layout");
        if (a.sym && (a.ot != a.o || a.ot_cols != a.o_cols)) return bad("mirror layout");
        if (ns_extent(a.batch, a.sot, a.N, a.ldot, a.ot_cols) > ot_avail)
            return bad("Ot beyond its buffer");
    }
    if (!a.o && !a.ot && a.splits == 1) return bad("no output");
    if (ns_workgroups(a) > int64_t(1) << 31) return bad("grid");
    return std::string();
}

// ------------------------------------------------------------------ groups and lanes
// Tensors of one wide shape share a batch of products (a tall R x C tensor joins the
// C x R ones); inside a group, tensors of one R x C shape form a part (batch entries
// [first, first + count)) with its own prep and update launches. A vector (one row or one
// column) is the 1 x numel matrix and takes the vector kernel.
struct NsPart {
    int64_t rows, cols;
    int32_t first, count;
    bool transposed;   // rows > cols, not a vector: X = U^T
};
struct NsGroup {
    NsShape shape;
    int32_t first;     // tensors order[first .. first + shape.count)
    std::vector<NsPart> parts;
};

// Groups and parts in order of first appearance; order lists the tensors batch by batch.
// Returns an empty string, or the reason the shapes are refused.
inline std::string ns_plan_groups(int32_t n, const int64_t* rows, const int64_t* numel,
                                  std::vector<NsGroup>& groups, std::vector<int32_t>& order)
{
    groups.clear();
    order.clear();
    struct Shape {
        int64_t rows, cols, m, n;
        bool transposed;
    };
    std::vector<Shape> shp(static_cast<size_t>(n));
    for (int32_t t = 0; t < n; ++t) {
        Shape& sh = shp[t];
        if (rows[t] < 1 || numel[t] < 1 || numel[t] % rows[t] != 0)
            return "rows[" + std::to_string(t) + "] does not divide the tensor's size";
        sh.rows = rows[t];
        sh.cols = numel[t] / rows[t];
        const bool vec = sh.rows == 1 || sh.cols == 1;
        sh.m = vec ? 1 : std::min(sh.rows, sh.cols);
        sh.n = vec ? numel[t] : std::max(sh.rows, sh.cols);
        if (sh.n > 0x7ffff000LL) return "a matrix side exceeds 2^31 - 4096";
        sh.transposed = !vec && sh.rows > sh.cols;
    }
    std::vector<char> placed(static_cast<size_t>(n), 0);
    for (int32_t t = 0; t < n; ++t) {
        if (placed[t]) continue;
        NsGroup g{};
        g.first = static_cast<int32_t>(order.size());
        int32_t count = 0;
        for (int32_t u = t; u < n; ++u) {
            if (placed[u] || shp[u].m != shp[t].m || shp[u].n != shp[t].n) continue;
            NsPart pt{shp[u].rows, shp[u].cols, count, 0, shp[u].transposed};
            for (int32_t v = u; v < n; ++v)
                if (!placed[v] && shp[v].rows == pt.rows && shp[v].cols == pt.cols) {
                    placed[v] = 1;
                    order.push_back(v);
                    ++pt.count;
                    ++count;
                }
            g.parts.push_back(pt);
        }
        if (count > 65535) return "more than 65535 tensors share one shape";
        g.shape = ns_shape(count, shp[t].m, shp[t].n);
        groups.push_back(g);
    }
    return std::string();
}

// Estimated time of a group's Newton-Schulz iterations relative to the others': each
// product launch costs its flops at the products' measured rate, but at least the
// latency of a small launch (a product of a few dozen workgroups takes 10-50 us whatever
// its flops), so that latency-bound groups such as a position embedding count for the
// time they hold a lane rather than for their flops.
constexpr double kNsLaunchUs = 15.0;

inline double ns_group_cost(const NsShape& sh)
{
    constexpr double kFlopsPerUs = 6.0e8;   // ~600 TFLOP/s on the model shapes
    constexpr double kLaunchUs = kNsLaunchUs;
    const double m = static_cast<double>(sh.m), n = static_cast<double>(sh.ldx);
    const double c = static_cast<double>(sh.count);
    if (sh.m < 2) return kLaunchUs;   // one vector kernel for all iterations
    auto launch = [&](double flops) { return std::max(flops / kFlopsPerUs, kLaunchUs); };
    double t = launch(c * 2.0 * m * m * n) + launch(c * 2.0 * m * m * m) +
               launch(c * 2.0 * m * m * n);
    if (sh.splits > 1) t += kLaunchUs;   // the Gram's split-K reduction
    return t;
}

// The estimated time of a group whose every launch takes the latency of a small launch:
// the one vector kernel, or three products (four with the split-K reduction).
inline double ns_group_floor(const NsShape& sh)
{
    if (sh.m < 2) return kNsLaunchUs;
    return kNsLaunchUs * (sh.splits > 1 ? 4.0 : 3.0);
}

// Three lanes (streams that run concurrently). The latency-bound groups (estimated time
// at the floor of their launches: vectors, small matrices such as a position embedding)
// share lane 2, so that they run beside the long products from the start and hold
// neither long lane; the others, in decreasing order of estimated time, each go to lane 0
// or 1, whichever has less so far, and every lane runs its groups longest first. With
// no long group at all, the latency-bound ones are split over lanes 0 and 1 the same way.
// (Measured on the GPT-2 125M shapes: with two lanes, the short groups sharing a lane
// with the MLP group waited for workgroup slots behind the other lane's long products
// and held the MLP group back until the end of the phase.)
constexpr int kNsLanes = 3;

inline void ns_assign_lanes(const std::vector<NsGroup>& groups,
                            std::vector<int32_t> (&lanes)[kNsLanes])
{
    std::vector<int32_t> byw(groups.size());
    std::vector<double> cost(groups.size());
    bool any_long = false;
    for (size_t gi = 0; gi < groups.size(); ++gi) {
        byw[gi] = static_cast<int32_t>(gi);
        cost[gi] = ns_group_cost(groups[gi].shape);
        any_long = any_long || cost[gi] > ns_group_floor(groups[gi].shape);
    }
    std::stable_sort(byw.begin(), byw.end(),
                     [&](int32_t a, int32_t b) { return cost[a] > cost[b]; });
    double load[2] = {0.0, 0.0};
    for (auto& l : lanes) l.clear();
    for (int32_t gi : byw) {
        if (any_long && cost[gi] <= ns_group_floor(groups[gi].shape)) {
            lanes[2].push_back(gi);
            continue;
        }
        const int l = load[1] < load[0] ? 1 : 0;
        lanes[l].push_back(gi);
        load[l] += cost[gi];
    }
}

// Elements of one lane's buffers: X and X^T (two of each), the two m x m products, the
// split-K partials; the largest over the lane's groups.
struct NsLaneSizes {
    int64_t x_elems = 0, a_elems = 0, partial_elems = 0;
};

inline NsLaneSizes ns_lane_sizes(const std::vector<NsGroup>& groups,
                                 const std::vector<int32_t>& lane)
{
    NsLaneSizes z;
    for (int32_t gi : lane) {
        const NsShape& sh = groups[gi].shape;
        z.x_elems = std::max(z.x_elems, ns_x_elems(sh));
        z.a_elems = std::max(z.a_elems, sh.m > 1 ? ns_a_elems(sh) : int64_t(0));
        z.partial_elems = std::max(z.partial_elems, ns_partial_elems(sh));
    }
    return z;
}

// The three products of an iteration on a lane's buffers (x[cur], xt[cur] hold X and
// X^T), and the elements available behind each of their pointers (P, Q, E, O, Ot,
// partial), for ns_check.
struct NsLaneBuffers {
    uint16_t* x[2];
    uint16_t* xt[2];
    uint16_t* a;
    uint16_t* b;
    float* partial;
};

inline void ns_iteration_products(const NsShape& sh, const NsLaneBuffers& lb,
                                  const NsLaneSizes& z, int cur, float ca, float cb, float cc,
                                  NsGemmArgs prods[3], int64_t avail[3][6])
{
    prods[0] = ns_gram_args(sh, lb.x[cur], lb.a, lb.partial);
    prods[1] = ns_poly_args(sh, lb.a, lb.b, cb, cc);
    prods[2] = ns_combine_args(sh, lb.b, lb.xt[cur], lb.x[1 - cur], lb.xt[1 - cur], ca);
    const int64_t av[3][6] = {
        {z.x_elems, z.x_elems, 0, z.a_elems, z.a_elems, z.partial_elems},
        {z.a_elems, z.a_elems, z.a_elems, z.a_elems, z.a_elems, 0},
        {z.a_elems, z.x_elems, z.x_elems, z.x_elems, z.x_elems, 0}};
    for (int k = 0; k < 3; ++k)
        for (int j = 0; j < 6; ++j) avail[k][j] = av[k][j];
}

// Every product of a group, both ping-pong parities, checked (ns_check); the prep and
// update writes of its parts checked against the lane's X and X^T. Empty string: valid.
inline std::string ns_check_group(const NsGroup& g, const NsLaneBuffers& lb, const NsLaneSizes& z)
{
    const NsShape& sh = g.shape;
    const int64_t xs = sh.m * sh.ldx, ts = sh.ldx * sh.ldm;
    for (const NsPart& pt : g.parts) {
        // prep: copy R rows of cs >= C and transpose C rows of tr >= R elements at the
        // part's batch entries (cs, tr: the group's row strides); the update reads the same
        const int64_t R = sh.m == 1 ? 1 : pt.rows, C = sh.m == 1 ? pt.rows * pt.cols : pt.cols;
        const bool wide = sh.m == 1 || !pt.transposed;
        const int64_t cs = wide ? sh.ldx : sh.ldm, tr = wide ? sh.ldm : sh.ldx;
        if (cs < C || tr < R || cs % 8 || tr % 8) return "prep strides do not hold the matrix";
        const int64_t copy_end = (pt.first + pt.count - 1) * (wide ? xs : ts) + R * cs;
        const int64_t trans_end = (pt.first + pt.count - 1) * (wide ? ts : xs) + C * tr;
        if (copy_end > z.x_elems || trans_end > z.x_elems) return "prep beyond the lane buffers";
    }
    if (sh.m < 2) return std::string();   // vector kernel: X rows of ldx elements
    for (int cur = 0; cur < 2; ++cur) {
        NsGemmArgs prods[3];
        int64_t avail[3][6];
        ns_iteration_products(sh, lb, z, cur, 1.0f, 1.0f, 1.0f, prods, avail);
        for (int k = 0; k < 3; ++k) {
            const std::string why = ns_check(prods[k], avail[k][0], avail[k][1], avail[k][2],
                                             avail[k][3], avail[k][4], avail[k][5]);
            if (!why.empty()) return why;
        }
    }
    return std::string();
}

}  // namespace gefen
