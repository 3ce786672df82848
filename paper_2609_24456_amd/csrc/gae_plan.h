// Which kernels a time-major GAE call takes (host code only).
#pragma once
#include <cstdint>

namespace conduit {

// The values of conduit_gae_plan's *path.
enum GaePath : int32_t {
    GAE_ONE_PASS = 0,        // one environment per lane, all T steps per workgroup
    GAE_ONE_PASS_V4 = 1,     // four environments per lane, all T steps per workgroup
    GAE_SHORT = 2,           // T <= 64: one tile of 32 environments per workgroup
    GAE_LOOK_BACK = 3,       // split along T, one launch, look-back over segment maps
    GAE_THREE_LAUNCHES = 4,  // split along T, fold / carry / replay launches
};

struct GaePlan {
    int32_t path;      // GaePath
    int32_t chunk;     // steps per lane of a tile (0 for the one-pass kernels)
    int64_t groups;    // tiles across E (32 environments each)
    int64_t segments;  // tiles along T
};

// `vec`: E % 4 == 0 and every row 16-byte aligned.
GaePlan plan_gae(int64_t T, int64_t E, bool vec);

// Tiles the per-GPU look-back table holds (the look-back path's limit).
constexpr int64_t kLookMaxTiles = 4096;

}  // namespace conduit
