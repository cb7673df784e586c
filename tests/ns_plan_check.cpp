// Host-only check of the Gefen-Muon Newton-Schulz plan (paper_2606_13894_amd/csrc/ns_plan.h),
// built with address and undefined-behaviour sanitizers by tests/test_ns_plan_cpu.py.
//
// Input (stdin): a tensor count, then one "rows numel" line per tensor. The program plans
// the shape groups and the lanes exactly as gefen_muon_init does, sizes each lane's
// buffers, runs the library's own checks (ns_check_group), and then walks every work item
// of every product of both ping-pong parities: the item's decoded batch entry, K chunk and
// tile must be in range, every (b, s, tile) must be decoded exactly once, and the furthest
// element the kernel's predicates let it touch in each operand must lie inside the
// buffer behind that pointer. Prints one line per group and "ok", or the first failure.
#include "ns_plan.h"

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <set>
#include <string>
#include <tuple>
#include <vector>

using namespace gefen;

namespace {

// Distinct fake base addresses: only identities (p == q, ot == o) and offsets are used.
uint16_t* fake16(int k) { return reinterpret_cast<uint16_t*>(static_cast<uintptr_t>(k + 1) << 44); }
float* fake32(int k) { return reinterpret_cast<float*>(static_cast<uintptr_t>(k + 1) << 44); }

int64_t last(int64_t start, int64_t len, int64_t limit)   // last index of [start, start+len) below limit
{
    return std::min(start + len, limit) - 1;
}

std::string walk(const NsGemmArgs& a, const int64_t avail[6], const char* what)
{
    char buf[256];
    const int64_t total = int64_t(a.batch) * a.splits * a.tiles;
    const int64_t groups = ns_workgroups(a);
    const int64_t per_xcd = (total + 7) / 8;
    std::set<std::tuple<int64_t, int32_t, int32_t, int32_t>> seen;
    for (int64_t blk = 0; blk < groups; ++blk) {
        const int64_t wid = (blk % 8) * per_xcd + blk / 8;   // the kernel's XCD deal
        if (wid >= total) continue;
        const NsWork w = ns_decode(a, wid);
        if (w.b < 0 || w.b >= a.batch || w.s < 0 || w.s >= a.splits || w.ti < 0 ||
            w.ti >= a.tm || w.tj < 0 || w.tj >= a.tn || (a.sym && w.tj < w.ti)) {
            std::snprintf(buf, sizeof buf, "%s: work item %lld decodes out of range", what,
                          (long long)wid);
            return buf;
        }
        if (!seen.insert(std::make_tuple(w.b, w.s, w.ti, w.tj)).second) {
            std::snprintf(buf, sizeof buf, "%s: work item %lld repeats a tile", what, (long long)wid);
            return buf;
        }
        const int64_t row0 = int64_t(w.ti) * a.tile, col0 = int64_t(w.tj) * a.tile;
        if (row0 >= a.M || col0 >= a.N) return std::string(what) + ": an empty tile";
        const int64_t kbeg = int64_t(w.s) * a.kchunk;
        const int64_t kend = a.splits > 1 ? std::min<int64_t>(a.K, kbeg + a.kchunk) : a.K;
        if (kbeg >= kend || kbeg % kNsBK || kend % kNsBK)
            return std::string(what) + ": an empty or ragged K chunk";
        const int64_t im = last(row0, a.tile, a.M), jn = last(col0, a.tile, a.N);
        auto over = [&](int64_t end, int k, const char* op) -> bool {
            if (end > avail[k]) {
                std::snprintf(buf, sizeof buf, "%s: item %lld reads or writes %s up to %lld of %lld",
                              what, (long long)wid, op, (long long)end, (long long)avail[k]);
                return true;
            }
            return false;
        };
        // operand loads: buffer resources from the tile's first row to row M (N); the
        // loads that land inside are rows below M (N), 16-byte vectors of K below kend
        if (over(w.b * a.sp + im * a.ldp + kend, 0, "P")) return buf;
        if (over(w.b * a.sq + jn * a.ldq + kend, 1, "Q")) return buf;
        if ((a.ldp % 8) || (a.ldq % 8)) return std::string(what) + ": misaligned load";
        // 32-bit byte offsets: lane row (< 32) and K position, plus row pass and stage
        const int64_t off_p = 2 * ((a.tile - 1) * a.ldp + kend);
        const int64_t off_q = 2 * ((a.tile - 1) * a.ldq + kend);
        if (off_p >= (int64_t(1) << 31) || off_q >= (int64_t(1) << 31) ||
            2 * std::min<int64_t>(a.tile, a.M - row0) * a.ldp >= (int64_t(1) << 31) ||
            2 * std::min<int64_t>(a.tile, a.N - col0) * a.ldq >= (int64_t(1) << 31))
            return std::string(what) + ": a buffer offset or range beyond 31 bits";
        if (a.splits > 1) {
            const int64_t end = ((int64_t(w.s) * a.batch + w.b) * a.M + im) * a.N + jn + 1;
            if (over(end, 5, "the partials")) return buf;
            continue;
        }
        if (a.et && over(w.b * a.se + jn * a.lde + last(row0, a.tile, a.lde) + 1, 2, "E"))
            return buf;
        const bool mirror = a.ot && (!a.sym || w.ti != w.tj);
        if (mirror && over(w.b * a.sot + jn * a.ldot + last(row0, a.tile, a.ot_cols) + 1, 4, "Ot"))
            return buf;
        if (a.o && over(w.b * a.so + im * a.ldo + last(col0, a.tile, a.o_cols) + 1, 3, "O"))
            return buf;
    }
    if (static_cast<int64_t>(seen.size()) != total) return std::string(what) + ": tiles missed";
    if (a.splits > 1) {   // the reduce: 16 rows x 128 columns of an upper tile per workgroup
        const int64_t slices = int64_t(a.tile / 16) * (a.tile / 128);
        for (int64_t wid = 0; wid < int64_t(a.batch) * a.tiles * slices; ++wid) {
            NsGemmArgs one = a;
            one.splits = 1;
            const NsWork w = ns_decode(one, wid / slices);
            const int64_t sl = wid % slices, rs = sl / (a.tile / 128), cs = sl % (a.tile / 128);
            const int64_t row0 = int64_t(w.ti) * a.tile + 16 * rs;
            const int64_t col0 = int64_t(w.tj) * a.tile + 128 * cs;
            if (row0 >= a.M || col0 >= a.o_cols) continue;   // the kernel writes nothing there
            const int64_t im = last(row0, 16, a.M);
            if (w.b * a.so + im * a.ldo + last(col0, 128, a.o_cols) + 1 > avail[3])
                return std::string(what) + ": reduce beyond O";
            if (col0 < a.N && ((int64_t(a.splits) - 1) * a.batch * a.M + w.b * a.M + im) * a.N +
                                      last(col0, 128, a.N) + 1 > avail[5])
                return std::string(what) + ": reduce beyond the partials";
            if (w.ti != w.tj && col0 < a.N &&
                w.b * a.sot + last(col0, 128, a.N) * a.ldot + last(row0, 16, a.ot_cols) + 1 >
                    avail[4])
                return std::string(what) + ": reduce mirror beyond O";
        }
    }
    return std::string();
}

}  // namespace

int main()
{
    int32_t n = 0;
    if (std::scanf("%d", &n) != 1 || n < 1) {
        std::puts("bad input");
        return 2;
    }
    std::vector<int64_t> rows(n), numel(n);
    for (int32_t t = 0; t < n; ++t)
        if (std::scanf("%lld %lld", reinterpret_cast<long long*>(&rows[t]),
                       reinterpret_cast<long long*>(&numel[t])) != 2) {
            std::puts("bad input");
            return 2;
        }
    std::vector<NsGroup> groups;
    std::vector<int32_t> order;
    std::string why = ns_plan_groups(n, rows.data(), numel.data(), groups, order);
    if (!why.empty()) {
        std::printf("refused: %s\n", why.c_str());
        return 1;
    }
    if (static_cast<int32_t>(order.size()) != n) {
        std::puts("the groups do not cover every tensor once");
        return 1;
    }
    std::vector<int32_t> lanes[kNsLanes];
    ns_assign_lanes(groups, lanes);
    size_t on_lanes = 0;
    for (const auto& l : lanes) on_lanes += l.size();
    if (on_lanes != groups.size()) {
        std::puts("the lanes do not cover every group once");
        return 1;
    }
    int64_t products = 0, items = 0;
    for (int l = 0; l < kNsLanes; ++l) {
        const NsLaneSizes z = ns_lane_sizes(groups, lanes[l]);
        NsLaneBuffers lb{{fake16(8 * l + 0), fake16(8 * l + 1)},
                         {fake16(8 * l + 2), fake16(8 * l + 3)},
                         fake16(8 * l + 4), fake16(8 * l + 5), fake32(8 * l + 6)};
        for (int32_t gi : lanes[l]) {
            const NsGroup& g = groups[gi];
            const NsShape& sh = g.shape;
            why = ns_check_group(g, lb, z);
            if (!why.empty()) {
                std::printf("group %d: %s\n", gi, why.c_str());
                return 1;
            }
            std::printf("lane %d group %d: %lld x (%lld x %lld), ldx %lld ldm %lld, %d parts, "
                        "Gram splits %d (chunk %d), tiles %d / %d / %d, floor %.3f, cost %.3f\n", l, gi,
                        (long long)sh.count, (long long)sh.m, (long long)sh.n, (long long)sh.ldx,
                        (long long)sh.ldm, static_cast<int>(g.parts.size()), sh.splits, sh.kchunk,
                        sh.tile_gram, sh.tile_poly, sh.tile_comb, ns_group_floor(sh),
                        ns_group_cost(sh));
            if (sh.m < 2) continue;
            for (int cur = 0; cur < 2; ++cur) {
                NsGemmArgs prods[3];
                int64_t avail[3][6];
                ns_iteration_products(sh, lb, z, cur, 3.4445f, -4.775f, 2.0315f, prods, avail);
                const char* names[3] = {"Gram", "poly", "combine"};
                for (int k = 0; k < 3; ++k) {
                    why = walk(prods[k], avail[k], names[k]);
                    if (!why.empty()) {
                        std::printf("group %d: %s\n", gi, why.c_str());
                        return 1;
                    }
                    ++products;
                    items += int64_t(prods[k].batch) * prods[k].splits * prods[k].tiles;
                }
            }
        }
    }
    std::printf("ok: %zu groups, %lld products, %lld work items\n", groups.size(),
                (long long)products, (long long)items);
    return 0;
}
