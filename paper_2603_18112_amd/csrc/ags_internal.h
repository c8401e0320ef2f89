// Internal declarations shared by the host runtime and the gfx950 kernels of
// libags.  Not part of the public C-ABI (include/ags.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ags.h"

namespace ags {

// One tile block = 256 threads = four wave64s; each thread owns groups of
// 8 consecutive elements (one 16-byte bf16 load or two 16-byte fp32 loads
// per replica).  A tile is at most kTileElems elements of ONE layer, so a
// tile's partial sums belong to exactly one layer.
constexpr int kBlock = 256;
constexpr int kVec = 8;
constexpr int kTileElems = 8192;  // 4 groups of 8 per thread
constexpr int kFinalizeThreads = 1024;

struct Tile {
    int64_t begin;  // first element (flat index), a multiple of kVec
    int32_t count;  // elements in the tile, 1..kTileElems
    int32_t layer;
};

struct LayerDev {
    int32_t tile_begin, tile_end;  // tiles [tile_begin, tile_end) cover the layer
    uint32_t flags;
    int32_t pad_;
};

// Device-resident AGS state, updated by the finalize kernel.
struct DevState {
    double g_prev;  // ||G||^2 of the last committed step (0 before the first)
    int64_t step;   // steps completed
};

// Per-tile fp32 partial sums: W (sum w^2), G (sum gbar^2), D (sum over
// elements of sum_k (g_k - gbar)^2, not yet divided by K), S (small-batch
// sum of squares).
struct Partial {
    float w, g, d, s;
};

struct StatsArgs {
    const void* grads;
    int64_t stride;
    const float* w;
    float* gbar;          // nullptr: do not store the replica mean
    const Tile* tiles;
    Partial* partials;
    int K;
    float invK;
    int small_replica;    // -1, or 0..K-1
};

struct FinalizeArgs {
    const Partial* partials;
    const LayerDev* layers;
    int n_layers;
    int K;
    int mode;
    int small_replica;
    int refresh_every;
    int commit;
    double delta, eps, s_max, trust_coef, weight_decay;
    double* gradscale;     // [n_layers]
    DevState* state;
    float2* coef;          // [n_layers] (a_l, b_l)
    ags_layer_stats* lstats;
    ags_global_stats* gstats;
};

struct UpdateArgs {
    const Tile* tiles;
    const float* gbar;    // materialised replica mean, or nullptr to recompute
    const void* grads;
    int64_t stride;
    int K;
    float invK;
    float* w;
    float* m;
    const float2* coef;
    float lr;
    float momentum;
};

// Launchers (ags_kernels.hip).  They only enqueue; the return value is the
// launch status.
hipError_t launch_stats(const StatsArgs& a, ags_dtype dt, int n_tiles, hipStream_t s);
hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s);
hipError_t launch_update(const UpdateArgs& a, ags_dtype dt, int n_tiles, hipStream_t s);

}  // namespace ags
