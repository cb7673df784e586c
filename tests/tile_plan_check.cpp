// Host-only check of the Gefen step's tile planner (paper_2606_13894_amd/csrc/tile_plan.h),
// built with address and undefined-behaviour sanitizers by tests/test_tile_plan_cpu.py.
//
// Usage: tile_plan_check FILE [CORRUPTION]
// FILE (little-endian binary): int32 n_tensors, int32 code_bits, int32 explicit_blocks,
// int32 pad; per tensor int64 numel, int64 period (0 with explicit blocks), int32
// gradient dtype, int32 pad; with explicit blocks, per tensor int64 n_blocks then
// n_blocks + 1 int64 block starts. The program plans the tiles as gefen_init does
// (build_plan) and runs the library's own plan check (check_plan); prints one line per
// launch class and "ok", or the reason. CORRUPTION > 0 plants one mistake in the finished
// plan first (a repeated tile, a shifted tile, a dropped tile, a broken chunk index, an
// oversized register run) and the check must then refuse it (exit status 3 if it does
// not).
#include "tile_plan.h"

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

using namespace gefen;

namespace {

template <typename T>
bool rd(FILE* f, T& v)
{
    return std::fread(&v, sizeof(T), 1, f) == 1;
}

// Plants mistake `k` (1-based) into the plan; false if the plan has nothing to corrupt.
bool corrupt(Plan& p, int k)
{
    const size_t n = p.tiles.size();
    if (n == 0) return false;
    switch (k) {
    case 1:   // a tile repeated in place of its neighbour
        if (n < 2) return false;
        p.tiles[1] = p.tiles[0];
        p.kinds[1] = p.kinds[0];
        p.htiles[1] = p.htiles[0];
        return true;
    case 2:   // a tile one element late
        p.tiles[n / 2].elem0 += 1;
        return true;
    case 3:   // the last tile dropped (its class one shorter)
        p.tiles.pop_back();
        p.kinds.pop_back();
        p.htiles.pop_back();
        p.classes.back().count -= 1;
        p.classes.back().elems = 0;
        for (int64_t i = p.classes.back().first;
             i < p.classes.back().first + p.classes.back().count; ++i)
            p.classes.back().elems += p.tiles[i].nelem;
        if (p.classes.back().count == 0) p.classes.pop_back();
        return true;
    case 4:   // a chunk of a huge block with the wrong index
        for (size_t i = 0; i < n; ++i)
            if (p.kinds[i] == KIND_H && p.htiles[i].nchunk > 1) {
                p.htiles[i].chunk = (p.htiles[i].chunk + 1) % p.htiles[i].nchunk;
                return true;
            }
        return false;
    case 5:   // a register run longer than the kernel holds
        for (size_t i = 0; i < n; ++i)
            if (p.kinds[i] == KIND_G && p.tiles[i].vpl == 1) {
                p.tiles[i].nblk = static_cast<int16_t>(kRunMaxBlocks + 1);
                return true;
            }
        return false;
    default:
        return false;
    }
}

}  // namespace

int main(int argc, char** argv)
{
    if (argc < 2) {
        std::puts("usage: tile_plan_check FILE [CORRUPTION]");
        return 2;
    }
    const int corruption = argc > 2 ? std::atoi(argv[2]) : 0;
    FILE* f = std::fopen(argv[1], "rb");
    if (!f) {
        std::puts("cannot open input");
        return 2;
    }
    int32_t n = 0, bits = 0, expl = 0, pad = 0;
    if (!rd(f, n) || !rd(f, bits) || !rd(f, expl) || !rd(f, pad) || n < 1) {
        std::puts("bad input header");
        return 2;
    }
    PlanCtx ctx;
    ctx.n_tensors = n;
    ctx.code_bits = bits;
    ctx.explicit_blocks = expl != 0;
    ctx.numel.resize(n);
    ctx.period.resize(n);
    ctx.gdtype.resize(n);
    for (int32_t t = 0; t < n; ++t) {
        int32_t dt = 0, pd = 0;
        if (!rd(f, ctx.numel[t]) || !rd(f, ctx.period[t]) || !rd(f, dt) || !rd(f, pd)) {
            std::puts("bad tensor record");
            return 2;
        }
        ctx.gdtype[t] = dt;
    }
    std::vector<std::vector<int64_t>> starts(ctx.explicit_blocks ? n : 0);
    ctx.blk_begin.assign(n + 1, 0);
    for (int32_t t = 0; t < n; ++t) {
        int64_t nb = 0;
        if (ctx.explicit_blocks) {
            if (!rd(f, nb) || nb < 1) {
                std::puts("bad block count");
                return 2;
            }
            starts[t].resize(static_cast<size_t>(nb) + 1);
            if (std::fread(starts[t].data(), sizeof(int64_t), starts[t].size(), f) !=
                starts[t].size()) {
                std::puts("short block table");
                return 2;
            }
            if (starts[t].front() != 0 || starts[t].back() != ctx.numel[t]) {
                std::puts("block table does not span the tensor");
                return 2;
            }
        } else {
            if (ctx.period[t] < 1 || ctx.numel[t] % ctx.period[t]) {
                std::puts("period does not divide the tensor");
                return 2;
            }
            nb = ctx.numel[t] / ctx.period[t];
        }
        ctx.blk_begin[t + 1] = ctx.blk_begin[t] + nb;
    }
    std::fclose(f);

    Plan plan;
    std::string why = build_plan(&ctx, starts, plan);
    if (!why.empty()) {
        std::printf("refused: %s\n", why.c_str());
        return 1;
    }
    if (corruption > 0) {
        if (!corrupt(plan, corruption)) {
            std::puts("nothing to corrupt");
            return 4;
        }
        why = check_plan(ctx, starts, plan);
        if (why.empty()) {
            std::printf("corruption %d was not caught\n", corruption);
            return 3;
        }
        std::printf("caught: %s\n", why.c_str());
        return 0;
    }
    why = check_plan(ctx, starts, plan);
    if (!why.empty()) {
        std::printf("check failed: %s\n", why.c_str());
        return 1;
    }
    static const char* kNames[] = {"U", "G", "L", "H", "ANY"};
    for (const PlanClass& c : plan.classes)
        std::printf("class %s dtype %d vpl %d bs %d: %lld tiles, %lld elements\n",
                    kNames[c.kind], c.gdtype, c.vpl, c.bs, static_cast<long long>(c.count),
                    static_cast<long long>(c.elems));
    std::printf("ok: %zu tiles, %lld blocks, %lld split blocks\n", plan.tiles.size(),
                static_cast<long long>(ctx.blk_begin[n]), static_cast<long long>(ctx.n_hblocks));
    return 0;
}
