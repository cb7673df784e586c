// Work classes and tiles of the Gefen step kernels, and the host planner that cuts every
// tensor's blocks into tiles (one workgroup's work each) and groups the tiles into
// launch classes. Plain C++ with no HIP types, so that host-only tests can build the
// planner with sanitizers and check every plan it makes (check_plan).
#pragma once

#include <stdint.h>

#include <algorithm>
#include <cstdio>
#include <string>
#include <utility>
#include <vector>

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

// Register runs of explicit blocks inside the KIND_G launch (tile.vpl = 1), shared by
// the planner and the kernel.
constexpr int kRunVpl = 2;                               // 4-element vectors per thread
constexpr int kRunMaxVec = kThreads * kRunVpl;           // vectors a run may touch
// A run of T elements starting anywhere touches at most (T + 6) / 4 vectors.
constexpr int64_t kRunMaxElems = 4 * int64_t(kRunMaxVec) - 6;
constexpr int kRunMaxBlocks = 64;
constexpr int64_t kRunMinBlock = 33;                     // so a vector meets at most 2 blocks


constexpr int64_t kUMaxPeriod = 8192;          // longest period held in registers (KIND_U)
constexpr int64_t kHugeBlock = 65536;         // longer blocks are always split (KIND_H)
constexpr int64_t kMinStreamedBlocks = 4096;  // fewer blocks > kUMaxPeriod: split them too

// What the planner needs to know about the tensors.
struct PlanCtx {
    int32_t n_tensors = 0;
    int32_t code_bits = 8;
    bool explicit_blocks = false;
    std::vector<int64_t> numel, period, blk_begin;   // blk_begin: n_tensors + 1 entries
    std::vector<int32_t> gdtype;
    int64_t n_hblocks = 0;                           // out: blocks split over workgroups
};

// One launch: a kernel class (kind, gradient type, KIND_U shape) over a range of tiles.
struct PlanClass {
    int32_t kind, gdtype, vpl, bs;
    int64_t first, count;
    int64_t elems, bytes;   // per launch: elements and algorithmic HBM bytes
};

// The tiles in launch order, each tile's kernel class (tile_kind: the folded tiles of the
// generic launch keep their own), the KIND_H bookkeeping parallel to the tiles (zero for
// the others), and the classes.
struct Plan {
    std::vector<Tile> tiles;
    std::vector<int32_t> kinds;
    std::vector<HTile> htiles;
    std::vector<PlanClass> classes;
};

// KIND_U shape for period p (p % 4 == 0, p <= kUMaxPeriod): vectors per lane v and a
// power-of-two lane group per block leaving at most 1/8 of the lanes idle, in a
// workgroup of `threads` lanes (threads / lanes blocks per workgroup). Measured on the
// MI355X for the Llama-3 1.5B shape (p = 2048 and 8192, bf16 gradients): 1024 threads
// with v = 2 (about 8K elements per workgroup) reach 5.76 TB/s; v = 1 (4K elements)
// 4.82 TB/s, v = 4 (16K elements) 4.11 TB/s, 512 threads 4.55 TB/s, 256 threads
// 4.38 TB/s -- the per-workgroup start (descriptor loads, LDS tables, barrier) needs
// ~8K elements to amortise, while larger tiles lose memory-level parallelism. So v = 2
// is tried first, then 1, 3, 4; 256-thread workgroups (up to 8 vectors) are the
// fallback.
struct UShape {
    int lpb_log2, vpl, bs;
};

inline UShape choose_u(int64_t p)
{
    const int64_t nv = p / 4;
    constexpr int pref = 1024;
    constexpr int kMaxVplBig = 4;   // instances of the 512/1024-thread kernels
    static const int kOrderBig[kMaxVplBig] = {2, 1, 3, 4};
    static const int kOrderSmall[kMaxVpl] = {2, 1, 3, 4, 5, 6, 7, 8};
    for (int pass = 0; pass < 2; ++pass) {
        const int bs = pass == 0 ? pref : 256;
        const int vmax = bs > 256 ? kMaxVplBig : kMaxVpl;
        for (int vi = 0; vi < vmax; ++vi) {
            const int v = bs > 256 ? kOrderBig[vi] : kOrderSmall[vi];
            const int64_t need = (nv + v - 1) / v;
            int l2 = 0;
            while ((int64_t(1) << l2) < need) ++l2;
            if ((1 << l2) > bs) continue;
            const int64_t waste = (int64_t(1) << l2) * v - nv;
            if (8 * waste <= nv || v == vmax || (pass == 1 && v == kMaxVpl))
                return UShape{l2, v, bs};
        }
    }
    // not reached for p <= 8192: 256 lanes x 8 vectors x 4 = 8192
    return UShape{8, kMaxVpl, 256};
}

// Tiles per kernel class while planning: one list per class key, with the split-block
// bookkeeping and the kind of every tile (the histogram's view of it) kept parallel.
struct TilePlan {
    struct Key {
        int32_t kind, gdtype, vpl, bs;
    };
    std::vector<Key> keys;
    std::vector<std::vector<Tile>> lists;
    std::vector<std::vector<HTile>> hlists;
    std::vector<std::vector<int32_t>> kinds;

    size_t index(int32_t kind, int32_t gdt, int32_t vpl, int32_t bs = kThreads)
    {
        for (size_t i = 0; i < keys.size(); ++i)
            if (keys[i].kind == kind && keys[i].gdtype == gdt && keys[i].vpl == vpl &&
                keys[i].bs == bs)
                return i;
        keys.push_back({kind, gdt, vpl, bs});
        lists.emplace_back();
        hlists.emplace_back();
        kinds.emplace_back();
        return keys.size() - 1;
    }
    void add(size_t i, const Tile& tl)
    {
        lists[i].push_back(tl);
        kinds[i].push_back(keys[i].kind);
    }
    int64_t elems(size_t i) const
    {
        int64_t e = 0;
        for (const Tile& tl : lists[i]) e += tl.nelem;
        return e;
    }
};

// Register-resident shapes: each eligible tensor's own best shape, then every tensor
// that fits the dominant shape's kernel (its vectors per lane and workgroup size; the
// kernel masks vectors past a block's end and reads lanes-per-block from the tile) is
// re-planned onto it, so one launch covers them on the fast path. lpb_log2 < 0: not
// register-resident.
inline std::vector<UShape> plan_u_shapes(const PlanCtx* st)
{
    std::vector<UShape> ushape(st->n_tensors, UShape{-1, 0, 0});
    std::vector<std::pair<std::pair<int, int>, int64_t>> tally;
    for (int32_t t = 0; t < st->n_tensors; ++t) {
        const int64_t p = st->period[t];
        if (st->explicit_blocks || p % 4 != 0 || p > kUMaxPeriod) continue;
        ushape[t] = choose_u(p);
        const std::pair<int, int> key{ushape[t].vpl, ushape[t].bs};
        bool found = false;
        for (auto& e : tally)
            if (e.first == key) {
                e.second += st->numel[t];
                found = true;
            }
        if (!found) tally.push_back({key, st->numel[t]});
    }
    int dom_vpl = 0, dom_bs = 0;
    int64_t best = -1;
    for (auto& e : tally)
        if (e.second > best) {
            best = e.second;
            dom_vpl = e.first.first;
            dom_bs = e.first.second;
        }
    if (best >= 0) {
        for (int32_t t = 0; t < st->n_tensors; ++t) {
            if (ushape[t].lpb_log2 < 0) continue;
            if (ushape[t].vpl == dom_vpl && ushape[t].bs == dom_bs) continue;
            const int64_t nv = st->period[t] / 4;
            const int64_t need = (nv + dom_vpl - 1) / dom_vpl;
            int l2 = 0;
            while ((int64_t(1) << l2) < need) ++l2;
            if ((1 << l2) <= dom_bs) ushape[t] = UShape{l2, dom_vpl, dom_bs};
        }
    }
    return ushape;
}

// A huge block as chunk tiles (KIND_H); the chunk bookkeeping is made absolute when
// the classes are concatenated.
inline void plan_huge(PlanCtx* st, TilePlan& P, int32_t t, int32_t gdt, int64_t start,
               int64_t len, int64_t blk)
{
    const size_t li = P.index(KIND_H, gdt, 0);
    const int64_t nchunk = (len + kHChunk - 1) / kHChunk;
    const int64_t first_rel = static_cast<int64_t>(P.lists[li].size());
    for (int64_t c = 0; c < nchunk; ++c) {
        Tile tl{};
        tl.elem0 = start + c * kHChunk;
        tl.blk0 = blk;
        tl.nelem = std::min(kHChunk, len - c * kHChunk);
        tl.seg = t;
        tl.nblk = 1;
        P.add(li, tl);
        HTile ht{};
        ht.blk_len = len;
        ht.first = first_rel;
        ht.nchunk = static_cast<int32_t>(nchunk);
        ht.chunk = static_cast<int32_t>(c);
        ht.hb = static_cast<int32_t>(st->n_hblocks);
        P.hlists[li].push_back(ht);
    }
    ++st->n_hblocks;
}

// One block per workgroup (KIND_G).
inline void plan_single(TilePlan& P, int32_t t, int32_t gdt, int64_t start, int64_t len, int64_t blk)
{
    Tile tl{};
    tl.elem0 = start;
    tl.blk0 = blk;
    tl.nelem = len;
    tl.seg = t;
    tl.nblk = 1;
    P.add(P.index(KIND_G, gdt, 0), tl);
}

// The tiles of tensor t: explicit blocks by their length; uniform blocks by the period
// (registers, lane per block, split, or streamed).
inline void plan_tensor(PlanCtx* st, TilePlan& P, int32_t t, const UShape& u,
                 const std::vector<int64_t>& s)
{
    const int32_t gdt = st->gdtype[t];
    const int64_t bb = st->blk_begin[t];
    if (st->explicit_blocks) {
        const int64_t nb = static_cast<int64_t>(s.size()) - 1;
        auto run_block = [](int64_t len) { return len >= kRunMinBlock && len <= kRunMaxElems; };
        int64_t b = 0;
        while (b < nb) {
            const int64_t len = s[b + 1] - s[b];
            if (st->code_bits == 8 && run_block(len)) {
                // consecutive short blocks held in registers by one KIND_G workgroup
                const int64_t b0 = b;
                int cnt = 0;
                while (b < nb && cnt < kRunMaxBlocks && run_block(s[b + 1] - s[b]) &&
                       s[b + 1] - s[b0] <= kRunMaxElems) {
                    ++cnt;
                    ++b;
                }
                Tile tl{};
                tl.elem0 = s[b0];
                tl.blk0 = bb + b0;
                tl.nelem = s[b] - s[b0];
                tl.seg = t;
                tl.nblk = static_cast<int16_t>(cnt);
                tl.vpl = 1;
                P.add(P.index(KIND_G, gdt, 0), tl);
            } else if (len > kHugeBlock) {
                plan_huge(st, P, t, gdt, s[b], len, bb + b);
                ++b;
            } else if (len <= kSmallBlock) {
                Tile tl{};
                tl.elem0 = s[b];
                tl.blk0 = bb + b;
                tl.seg = t;
                int n = 0;
                while (b < nb && n < kThreads && s[b + 1] - s[b] <= kSmallBlock) {
                    ++n;
                    ++b;
                }
                tl.nblk = static_cast<int16_t>(n);
                tl.nelem = s[b] - tl.elem0;
                P.add(P.index(KIND_L, gdt, 0), tl);
            } else {
                plan_single(P, t, gdt, s[b], len, bb + b);
                ++b;
            }
        }
        return;
    }
    const int64_t p = st->period[t];
    const int64_t nb = st->numel[t] / p;
    if (u.lpb_log2 >= 0) {
        const int64_t bpw = u.bs >> u.lpb_log2;
        const size_t li = P.index(KIND_U, gdt, u.vpl, u.bs);
        for (int64_t b = 0; b < nb; b += bpw) {
            Tile tl{};
            const int64_t n = std::min(bpw, nb - b);
            tl.elem0 = b * p;
            tl.blk0 = bb + b;
            tl.nelem = n * p;
            tl.seg = t;
            tl.nblk = static_cast<int16_t>(n);
            tl.vpl = static_cast<uint8_t>(u.vpl);
            tl.lpb_log2 = static_cast<uint8_t>(u.lpb_log2);
            P.add(li, tl);
        }
    } else if (p <= kSmallBlock) {
        const size_t li = P.index(KIND_L, gdt, 0);
        for (int64_t b = 0; b < nb; b += kThreads) {
            Tile tl{};
            const int64_t n = std::min<int64_t>(kThreads, nb - b);
            tl.elem0 = b * p;
            tl.blk0 = bb + b;
            tl.nelem = n * p;
            tl.seg = t;
            tl.nblk = static_cast<int16_t>(n);
            P.add(li, tl);
        }
    } else if (p > kHugeBlock || (p > kUMaxPeriod && nb < kMinStreamedBlocks)) {
        for (int64_t b = 0; b < nb; ++b) plan_huge(st, P, t, gdt, b * p, p, bb + b);
    } else {
        for (int64_t b = 0; b < nb; ++b) plan_single(P, t, gdt, b * p, p, bb + b);
    }
}

// Fold the small classes other than the largest register-resident one (and the split
// huge-block classes, which need two kernels) into one generic launch (KIND_ANY,
// tile.vpl = 0); a folded tile runs the slower generic path, so only small classes go.
// The folded tiles keep their kinds for the histogram kernel.
inline void fold_small_classes(const PlanCtx* st, TilePlan& P)
{
    int dom = -1;
    int64_t dom_elems = -1;
    for (size_t i = 0; i < P.lists.size(); ++i) {
        if (P.keys[i].kind != KIND_U) continue;
        const int64_t e = P.elems(i);
        if (e > dom_elems) {
            dom_elems = e;
            dom = static_cast<int>(i);
        }
    }
    if (dom < 0) return;
    const int64_t fold_max = std::max<int64_t>(int64_t(1) << 21, dom_elems / 64);
    std::vector<Tile> front;
    std::vector<int32_t> front_kinds;
    int32_t any_dtype = -1;
    for (size_t i = 0; i < P.lists.size(); ++i) {
        if (static_cast<int>(i) == dom || P.keys[i].kind == KIND_H || P.lists[i].empty())
            continue;
        if (P.elems(i) > fold_max) continue;
        // Uniform small-block tiles are cut to kThreads / lpb blocks, lpb = p rounded up
        // to a power of two: the generic kernel gives each block a group of lpb lanes and
        // covers such a tile in one pass.
        for (size_t j = 0; j < P.lists[i].size(); ++j) {
            Tile tl = P.lists[i][j];
            const int32_t kd = P.kinds[i][j];
            tl.vpl = 0;
            tl.lpb_log2 = 0;
            const int64_t p = st->explicit_blocks ? 0 : st->period[tl.seg];
            if (kd == KIND_L && p > 0) {
                int64_t lpb = 1;
                while (lpb < p) lpb <<= 1;
                const int64_t per = kThreads / lpb;
                for (int64_t b = 0; b < tl.nblk; b += per) {
                    Tile sub = tl;
                    const int64_t nb = std::min<int64_t>(per, tl.nblk - b);
                    sub.elem0 = tl.elem0 + b * p;
                    sub.blk0 = tl.blk0 + b;
                    sub.nblk = static_cast<int16_t>(nb);
                    sub.nelem = nb * p;
                    front.push_back(sub);
                    front_kinds.push_back(kd);
                }
            } else {
                front.push_back(tl);
                front_kinds.push_back(kd);
            }
        }
        any_dtype = P.keys[i].gdtype;
        P.lists[i].clear();
        P.kinds[i].clear();
    }
    if (front.empty()) return;
    const size_t ai = P.index(KIND_ANY, any_dtype, 0);
    P.lists[ai].insert(P.lists[ai].end(), front.begin(), front.end());
    P.kinds[ai].insert(P.kinds[ai].end(), front_kinds.begin(), front_kinds.end());
}


// Concatenate the classes (the small generic class first: it is short and leaves the
// machine to the long launches after it, which measured faster than running it beside
// them on a second stream, whose fork and join cost more than it saves) and record each
// class's launch range and algorithmic bytes. Empty string, or the reason the plan is
// refused.
inline std::string concat_plan(const PlanCtx* st, TilePlan& P, Plan& out)
{
    out = Plan{};
    std::vector<size_t> order;
    for (size_t i = 0; i < P.lists.size(); ++i)
        if (P.keys[i].kind == KIND_ANY) order.push_back(i);
    for (size_t i = 0; i < P.lists.size(); ++i)
        if (P.keys[i].kind != KIND_ANY) order.push_back(i);
    for (size_t i : order) {
        if (P.lists[i].empty()) continue;
        const int64_t base = static_cast<int64_t>(out.tiles.size());
        if (P.keys[i].kind == KIND_H) {
            for (HTile h : P.hlists[i]) {
                h.first += base;
                out.htiles.push_back(h);
            }
        } else {
            out.htiles.insert(out.htiles.end(), P.lists[i].size(), HTile{});
        }
        PlanClass c{P.keys[i].kind, P.keys[i].gdtype, P.keys[i].vpl, P.keys[i].bs, base,
                    static_cast<int64_t>(P.lists[i].size()), 0, 0};
        for (size_t j = 0; j < P.lists[i].size(); ++j) {
            const Tile& tl = P.lists[i][j];
            const int64_t per_elem =
                8 + (st->gdtype[tl.seg] == DT_F32 ? 4 : 2) + (st->code_bits == 4 ? 1 : 2);
            c.elems += tl.nelem;
            c.bytes += tl.nelem * per_elem + 16 * int64_t(tl.nblk);
            if (P.kinds[i][j] == KIND_L && st->explicit_blocks) c.bytes += 8 * int64_t(tl.nblk);
            if (P.kinds[i][j] == KIND_G && tl.vpl == 1) {
                // a register run: the kernel's fixed register and LDS capacity
                const int64_t nvec = ((tl.elem0 + tl.nelem + 3) >> 2) - (tl.elem0 >> 2);
                if (nvec > kRunMaxVec || tl.nblk < 1 || tl.nblk > kRunMaxBlocks)
                    return "run tile of " + std::to_string(nvec) + " vectors, " +
                           std::to_string(tl.nblk) + " blocks";
            }
        }
        out.classes.push_back(c);
        out.tiles.insert(out.tiles.end(), P.lists[i].begin(), P.lists[i].end());
        out.kinds.insert(out.kinds.end(), P.kinds[i].begin(), P.kinds[i].end());
    }
    // Workspace slots of the huge blocks in tile order: the planner numbered them tensor
    // by tensor, but each gradient type's huge blocks form a class of their own, so with
    // both types the classes' concatenation interleaves that numbering.
    int32_t hb = 0;
    for (size_t t = 0; t < out.tiles.size(); ++t)
        if (out.kinds[t] == KIND_H) {
            HTile& h = out.htiles[t];
            h.hb = h.chunk == 0 ? hb++ : out.htiles[static_cast<size_t>(h.first)].hb;
        }
    return std::string();
}

// The plan of every tensor (starts[t]: tensor t's explicit block starts, n_blocks + 1
// entries, when st->explicit_blocks; else unused).
inline std::string build_plan(PlanCtx* st, const std::vector<std::vector<int64_t>>& starts,
                              Plan& out)
{
    st->n_hblocks = 0;
    const std::vector<UShape> ushape = plan_u_shapes(st);
    TilePlan P;
    static const std::vector<int64_t> kNone;
    for (int32_t t = 0; t < st->n_tensors; ++t)
        plan_tensor(st, P, t, ushape[t], st->explicit_blocks ? starts[t] : kNone);
    fold_small_classes(st, P);
    return concat_plan(st, P, out);
}

// Checks a plan against what the kernels assume: the classes are consecutive ranges
// covering every tile once, each with launchable grid sizes; every tile lies inside its
// tensor and covers whole consecutive blocks (a huge block: consecutive chunk tiles of
// kHChunk elements, their bookkeeping consistent), every block of every tensor exactly
// once; and each kind's limits hold (register shapes, lane-per-block sizes, run
// capacities). Empty string: valid.
inline std::string check_plan(const PlanCtx& st, const std::vector<std::vector<int64_t>>& starts,
                              const Plan& p)
{
    char buf[320];
    auto bad = [&](int64_t i, const char* what) {
        std::snprintf(buf, sizeof buf, "tile %lld: %s", static_cast<long long>(i), what);
        return std::string(buf);
    };
    const int64_t n = static_cast<int64_t>(p.tiles.size());
    if (static_cast<int64_t>(p.kinds.size()) != n || static_cast<int64_t>(p.htiles.size()) != n)
        return "tile, kind and huge-block arrays differ in length";
    if (static_cast<int32_t>(st.blk_begin.size()) != st.n_tensors + 1 || st.blk_begin[0] != 0)
        return "block index table";
    int64_t next = 0;
    std::vector<uint8_t> generic(static_cast<size_t>(n), 0);   // tile in the KIND_ANY launch
    for (const PlanClass& c : p.classes) {
        if (c.first != next || c.count < 1 || c.count > 0x7fffffffLL) return "class ranges";
        int64_t elems = 0;
        for (int64_t i = c.first; i < c.first + c.count; ++i) {
            const int32_t kd = p.kinds[i];
            if (c.kind == KIND_ANY ? (kd == KIND_H || kd == KIND_ANY) : kd != c.kind)
                return bad(i, "kind differs from its class");
            if (c.kind != KIND_ANY && st.gdtype[p.tiles[i].seg] != c.gdtype)
                return bad(i, "gradient type differs from its class");
            elems += p.tiles[i].nelem;
            generic[i] = c.kind == KIND_ANY;
        }
        if (elems != c.elems) return "class element count";
        next += c.count;
    }
    if (next != n) return "classes do not cover the tiles";
    const int64_t total_blocks = st.blk_begin[st.n_tensors];
    std::vector<uint8_t> seen(static_cast<size_t>(total_blocks), 0);
    auto block_at = [&](int32_t t, int64_t b, int64_t& s0, int64_t& s1) {   // b tensor-relative
        if (st.explicit_blocks) {
            s0 = starts[t][b];
            s1 = starts[t][b + 1];
        } else {
            s0 = b * st.period[t];
            s1 = s0 + st.period[t];
        }
    };
    int64_t hb_count = 0;
    for (int64_t i = 0; i < n; ++i) {
        const Tile& tl = p.tiles[i];
        const int32_t kd = p.kinds[i];
        if (tl.seg < 0 || tl.seg >= st.n_tensors) return bad(i, "tensor index");
        const int32_t t = tl.seg;
        const int64_t bb = st.blk_begin[t], be = st.blk_begin[t + 1];
        if (tl.nblk < 1 || tl.blk0 < bb || tl.blk0 + tl.nblk > be) return bad(i, "blocks");
        if (tl.elem0 < 0 || tl.nelem < 1 || tl.elem0 + tl.nelem > st.numel[t])
            return bad(i, "elements outside the tensor");
        int64_t s0, s1;
        if (kd == KIND_H) {
            const HTile& h = p.htiles[i];
            block_at(t, tl.blk0 - bb, s0, s1);
            if (tl.nblk != 1 || h.blk_len != s1 - s0 || h.blk_len <= 0) return bad(i, "huge block length");
            const int64_t nchunk = (h.blk_len + kHChunk - 1) / kHChunk;
            if (h.nchunk != nchunk || h.chunk < 0 || h.chunk >= h.nchunk || h.first + h.chunk != i)
                return bad(i, "chunk bookkeeping");
            if (tl.elem0 != s0 + int64_t(h.chunk) * kHChunk ||
                tl.nelem != std::min<int64_t>(kHChunk, h.blk_len - int64_t(h.chunk) * kHChunk))
                return bad(i, "chunk range");
            if (h.chunk == 0) {
                if (h.hb != hb_count) return bad(i, "huge block slot");
                ++hb_count;
                if (seen[tl.blk0]++) return bad(i, "a block covered twice");
                if (h.first + h.nchunk > n) return bad(i, "chunks past the tiles");
                for (int32_t c = 1; c < h.nchunk; ++c)
                    if (p.kinds[h.first + c] != KIND_H || p.tiles[h.first + c].blk0 != tl.blk0)
                        return bad(i, "chunks not consecutive");
            }
            continue;
        }
        // whole consecutive blocks
        block_at(t, tl.blk0 - bb, s0, s1);
        if (tl.elem0 != s0) return bad(i, "tile does not start at its first block");
        int64_t end = s0, longest = 0, shortest = INT64_MAX;
        for (int64_t b = tl.blk0; b < tl.blk0 + tl.nblk; ++b) {
            if (seen[b]++) return bad(i, "a block covered twice");
            block_at(t, b - bb, s0, s1);
            if (s0 != end || s1 <= s0) return bad(i, "blocks not consecutive");
            end = s1;
            longest = std::max(longest, s1 - s0);
            shortest = std::min(shortest, s1 - s0);
        }
        if (end != tl.elem0 + tl.nelem) return bad(i, "tile length");
        if (generic[i]) {   // the generic kernel takes any whole blocks
            if (tl.vpl != 0) return bad(i, "generic tile with a register shape");
            continue;
        }
        if (kd == KIND_U) {
            const int64_t per = st.period[t];
            if (st.explicit_blocks || per % 4 || per > kUMaxPeriod) return bad(i, "register block");
            if (tl.vpl < 1 || tl.vpl > kMaxVpl || tl.lpb_log2 > kMaxLpbLog2)
                return bad(i, "register shape");
            if ((int64_t(1) << tl.lpb_log2) * tl.vpl * 4 < per) return bad(i, "block exceeds its lanes");
        } else if (kd == KIND_L) {
            if (longest > kSmallBlock || tl.nblk > kThreads) return bad(i, "small blocks");
        } else if (kd == KIND_G && tl.vpl == 1) {
            const int64_t nvec = ((tl.elem0 + tl.nelem + 3) >> 2) - (tl.elem0 >> 2);
            if (st.code_bits != 8 || tl.nblk > kRunMaxBlocks || nvec > kRunMaxVec ||
                tl.nelem > kRunMaxElems || shortest < kRunMinBlock || longest > kRunMaxElems)
                return bad(i, "register run");
        } else if (kd == KIND_G) {
            if (tl.nblk != 1 || tl.nelem > kHugeBlock) return bad(i, "single block");
        }
    }
    if (hb_count != st.n_hblocks) return "huge block count";
    for (int64_t b = 0; b < total_blocks; ++b)
        if (seen[b] != 1) {
            std::snprintf(buf, sizeof buf, "block %lld covered %d times", static_cast<long long>(b),
                          int(seen[b]));
            return std::string(buf);
        }
    return std::string();
}

}  // namespace gefen
