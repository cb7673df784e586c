// Limits of the register runs of explicit blocks inside the KIND_G launch (tile.vpl = 1),
// shared by the planner and the kernel.
#pragma once
#include "gefen_internal.h"

namespace gefen {

constexpr int kRunVpl = 2;                               // 4-element vectors per thread
constexpr int kRunMaxVec = kThreads * kRunVpl;           // vectors a run may touch
// A run of T elements starting anywhere touches at most (T + 6) / 4 vectors.
constexpr int64_t kRunMaxElems = 4 * int64_t(kRunMaxVec) - 6;
constexpr int kRunMaxBlocks = 64;
constexpr int64_t kRunMinBlock = 33;                     // so a vector meets at most 2 blocks

}  // namespace gefen
