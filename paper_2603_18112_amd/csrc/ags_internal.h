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
// tile's partial sums belong to exactly one layer.  The default tile is one
// group per thread: on MI355X (ResNet-50 layout, K = 16 bf16) 2048-element
// tiles ran the step kernel in 186 us against 195 us for 4096 and 202 us
// for 8192 (the many short blocks balance the 256 CUs best).
constexpr int kBlock = 256;
constexpr int kVec = 8;
// Threads of a block of the kernels that walk tiles (step, correction and
// LARS update); a round of such a block covers kTileBlock * kVec elements.
#ifndef AGS_TILE_BLOCK
#define AGS_TILE_BLOCK 256
#endif
constexpr int kTileBlock = AGS_TILE_BLOCK;
static_assert(kTileBlock % 64 == 0 && kTileBlock >= 64 && kTileBlock <= 1024, "whole waves");
#ifndef AGS_TILE_ELEMS
#define AGS_TILE_ELEMS (AGS_TILE_BLOCK * 8)
#endif
constexpr int kTileElems = AGS_TILE_ELEMS;  // a multiple of kTileBlock * kVec
static_assert(kTileElems % (kTileBlock * kVec) == 0, "tile must hold whole block rounds");
// A layer is cut into at most this many tiles (bigger layers get tiles of a
// multiple of kTileElems).
#ifndef AGS_MAX_TILES_PER_LAYER
#define AGS_MAX_TILES_PER_LAYER (1 << 30)
#endif
constexpr int64_t kMaxTilesPerLayer = AGS_MAX_TILES_PER_LAYER;
// The finalize kernel sums at most this many tile partials per block (16 per
// thread); a layer with more tiles is finalized by several blocks whose sums
// the last of them combines.
constexpr int kFinTilesPerChunk = 4096;
// From this many tiles on, the step kernel gives each XCD a contiguous range
// of tiles instead of the hardware's round-robin order.  Measured on MI355X
// (same box, alternating builds): VGG-16, 67,569 tiles, 2.4% faster warm and
// 2.3% cold with it; ResNet-50, 12,560 tiles, 2.4% slower warm and 4% slower
// cold (K = 64: 2% and 1.2%); ResNet-18, 5,493 tiles, 4.5% slower.
constexpr int64_t kXcdMapMinTiles = 32768;

// Element scales: the step kernel loads the scales in force and stores the
// refreshed ones, w and m non-temporally once w, m and the two scale
// buffers (16 bytes per element) pass this size; below it they can stay in
// the 256 MB Infinity Cache from one step to the next and ordinary accesses
// keep them there.  Measured on MI355X, fp32 K = 8, whole step, ordinary
// against streaming: ResNet-18 (11.2M elements) 113.2 / 113.5 us, 16M
// elements 157.8 / 157.1, 20M 195.7 / 186.2, ResNet-50 (25.6M) 272.2 /
// 229.6, VGG-16 (138M) 1400 / 1358.
constexpr int64_t kEwStreamMinBytes = 192ll << 20;
// Once w and m (8 bytes per element) pass this size they cannot stay in the
// Infinity Cache between steps, and every step streams them from HBM with
// the replicas; the fused step kernel then runs best with two blocks per CU
// (fewer concurrent streams, so fewer DRAM row conflicts), which the host
// enforces with an LDS pad.  Measured on MI355X, whole step warm / cold,
// blocks per CU 5 (the kernel's register limit), 4, 3, 2, 1: VGG-16 K = 8
// fp32 1210 / 1177, 1187 / 1155, 1176 / 1147, 1164 / 1140, 1378 / 1375 us;
// the layouts whose w and m fit lose from the cap (ResNet-50 K = 16 bf16
// 193 -> 201 us, ResNet-18 K = 8 fp32 93 -> 100 us at 2 blocks per CU) or
// barely gain (ResNet-50 K = 64 bf16 634 -> 631 us).  LARS's two passes on
// the same layouts: the statistics-only step kernel runs best with three
// blocks per CU (VGG-16 K = 8 fp32: 936 us uncapped, 901 at 3, 916 at 2),
// the update kernel with two (525 -> 484 us); the whole LARS step 1471 ->
// 1381 us.  ResNet-50's first pass loses from a cap (154 -> 160 us at 2).
#ifndef AGS_OCCUPANCY_CAP_MIN_BYTES
#define AGS_OCCUPANCY_CAP_MIN_BYTES (256ll << 20)
#endif
constexpr int64_t kOccupancyCapMinBytes = AGS_OCCUPANCY_CAP_MIN_BYTES;
constexpr int kCappedBlocksPerCu = 2;
constexpr int kCappedBlocksPerCuStats = 3;
constexpr int kCappedBlocksPerCuUpdate = 2;

// Elements per tile of a layer of numel elements.
__host__ __device__ inline int64_t tile_elems_for(int64_t numel) {
    const int64_t per = (int64_t)kTileElems * kMaxTilesPerLayer;
    const int64_t mult = (numel + per - 1) / per;
    return (int64_t)kTileElems * (mult > 0 ? mult : 1);
}
#ifndef AGS_CORRECT_BLOCKS
#define AGS_CORRECT_BLOCKS 512
#endif
// Grid of the correction pass (grid-stride over tiles): small, because on
// most steps the pass only reads its flag and exits.
constexpr int kCorrectBlocks = AGS_CORRECT_BLOCKS;

struct Tile {
    int64_t begin;  // first element (flat index), a multiple of kVec
    int32_t count;  // elements in the tile, 1..kTileElems
    int32_t layer;
};

struct LayerDev {
    int32_t tile_begin, tile_end;    // tiles [tile_begin, tile_end) cover the layer
    uint32_t flags;
    int32_t chunk_begin, chunk_end;  // finalize chunks of the layer
    int32_t pad_;
    int64_t numel;
};

// A finalize block's share: tiles [tile_begin, tile_end) of one layer.
struct FinChunk {
    int32_t layer, tile_begin, tile_end, pad_;
};

struct ChunkSum {
    double w, g, d, s, x;  // x: sum of the refreshed element scales
};

// Device-resident AGS state, updated by the last block of a committed step.
struct DevState {
    double g_prev;      // ||G||^2 of the last committed step (0 before the first)
    int64_t step;       // steps completed
    int32_t last_sens;  // the sensitive bit of the last committed step
    int32_t ew_cur;     // element scales: which of the two buffers is in force
    float lr;           // learning rate in force (ags_set_lr writes it on the handle's
                        // stream, so a step replayed from a graph uses the current one)
    int32_t pad_;
};

// Per-tile fp32 partial sums: W (sum w^2), G (sum gbar^2), D (sum over
// elements of sum_k (g_k - gbar)^2, not yet divided by K), S (small-batch
// sum of squares).
struct Partial {
    float w, g, d, s;
};

// Arguments of the step kernel (statistics of every tile and -- when update
// is on -- the momentum-SGD update with the predicted coefficients) and of
// the finalize kernel (per-layer and global statistics, the decision).
struct StepArgs {
    const void* grads;
    int64_t stride;
    float* w;
    float* m;
    float* gbar;             // store the replica mean here (or nullptr)
    const Tile* tiles;
    Partial* partials;
    const LayerDev* layers;
    int n_layers;
    int K;
    float invK;
    int small_replica;       // -1, or 0..K-1
    int mode;                // ags_mode
    int commit;              // 1: a step (state advances), 0: statistics only
    int refresh_every;
    float momentum;          // used when the kernel updates w and m (lr: state->lr)
    double delta, eps, s_max, trust_coef, weight_decay, static_scale;
    double* gradscale;       // [n_layers]; with element scales, their layer means
    DevState* state;
    double* g_prev_l;        // [n_layers] G_l of the last committed step
    int32_t* last_sens_l;    // [n_layers] the bit that decided each layer then
    int delta_scope;         // ags_delta_scope
    float2* coef;            // [n_layers] (a_l, b_l) as applied, fp32
    float2* corr;            // [n_layers] correction c = x + y * scale_j (fp32)
    int* corr_flag;          // 1 when some layer needs the correction pass
    int updated;             // the step kernel applied predicted coefficients
    int xcd_map;             // step kernel: contiguous tile ranges per XCD
    // Step kernel: tiles in reverse order.  Once w and m outgrow the
    // Infinity Cache the host alternates the direction from step to step,
    // so that a step starts on the lines the step before touched last
    // instead of sweeping a working set larger than the cache in one
    // direction (VGG-16 K = 8 fp32 warm step 1079 -> 1038 us, elementwise
    // 1250 -> 1207 us; layouts that fit the cache gain nothing).
    int reverse;
    unsigned* done_count;    // layers finished (reset by the last block)
    const FinChunk* chunks;  // finalize blocks
    ChunkSum* chunk_sums;    // [n_chunks] sums of multi-chunk layers
    unsigned* layer_chunk_count;  // [n_layers] chunks finished (reset by the last)
    ags_layer_stats* lstats;
    ags_global_stats* gstats;
    // Element scales (elementwise AGS; all null / 0 otherwise).  The buffer
    // in force and whether a step refreshes are read from the device state
    // (state->ew_cur, state->step), so a captured step replays correctly.
    int ew;                  // 0: per layer; per element with 1: ordinary, 2: streaming accesses
    float* ew_buf;           // [2][n_flat] the two scale buffers
    int64_t n_flat;
    float* ew_partials;      // [n_tiles] per-tile sums of the refreshed scales
    // LARS: per-tile sums of w^2 written by the last update pass; when set,
    // the statistics-only step kernel takes W from them and skips w.
    const float* w_norm_in;
    // Bytes of dynamic LDS the step kernel is launched with (it uses none):
    // a pad that caps the blocks resident per CU.  Taken by the fused
    // per-layer-scale variant and the statistics-only ones.
    int lds_pad;
};

struct UpdateArgs {
    const Tile* tiles;
    int n_tiles;
    const float* gbar;    // materialised replica mean, or nullptr to recompute
    const void* grads;
    int64_t stride;
    int K;
    float invK;
    float* w;
    float* m;
    const float2* coef;   // LARS update: (a_l, b_l)
    const float2* corr;   // correction pass: c = x + y * gs_old_j per layer
    const float* ew_buf;  // [2][n_flat] element scales (or null)
    int64_t n_flat;
    const DevState* state;  // after the step: the buffer in force and the step count
    int refresh_every;
    const int* corr_flag;
    float momentum;          // lr: state->lr
    // LARS update: per-tile sums of the new w^2, summed as the statistics
    // pass sums w^2 (or nullptr).
    float* w_norm_out;
    // Dynamic LDS of the LARS update launch (0: none), a cap on its blocks
    // per CU.
    int lds_pad;
    // LARS update: block b takes tile n_tiles - 1 - b (the last tiles
    // first).  The pass then ends on the first tiles, whose replica mean
    // the next statistics pass writes first, and those lines are still in
    // the Infinity Cache: that pass measured 154.4 -> 151.0 us (ResNet-50
    // K = 16 bf16; K = 64 582 -> 574 us) with the update pass unchanged.
    // Used while w and m fit the cache (VGG-16's step lost 0.8% with it).
    int reverse;
};

// Text for ags_last_error(NULL) on this thread (ags_api.hip).
void set_thread_error(const char* why);

// Events a launch records at its kernel's start and end (both null: none).
// They belong to the kernel's own dispatch, so their elapsed time is the
// kernel's execution alone, without the marker packets and cache
// write-backs of a separate hipEventRecord between kernels.
struct KernelEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};

// Launchers (ags_kernels.hip).  They only enqueue; the return value is the
// launch status.  update != 0 makes the step kernel apply the update.
hipError_t launch_step(const StepArgs& a, ags_dtype dt, int n_tiles, bool update, hipStream_t s,
                       KernelEvents ev);
hipError_t launch_finalize(const StepArgs& a, int n_chunks, hipStream_t s, KernelEvents ev);
hipError_t launch_update(const UpdateArgs& a, ags_dtype dt, hipStream_t s, KernelEvents ev);
hipError_t launch_correct(const UpdateArgs& a, ags_dtype dt, hipStream_t s, KernelEvents ev);
// Writes the learning rate in force into the device state (one thread).
hipError_t launch_set_lr(DevState* state, float lr, hipStream_t s);

}  // namespace ags
