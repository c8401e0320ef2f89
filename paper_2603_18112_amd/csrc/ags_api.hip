// Host runtime of libags: argument validation, the tile map, the device
// workspace, kernel launches, statistics read-back, checkpoint state and
// per-kernel timing.  Everything the C-ABI (include/ags.h) promises about
// errors is enforced here: host-side checks first, then device-pointer
// checks, then work.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstddef>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "ags_internal.h"

using ags::DevState;
using ags::LayerDev;
using ags::Partial;
using ags::Tile;

namespace {

thread_local std::string g_thread_error;

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Byte offsets of the pieces of the device workspace.  The statistics
// records, the gradscale array and the state are contiguous at the end so
// that a read-back is one copy.
struct WsLayout {
    size_t gbar = 0, tiles = 0, partials = 0, ldev = 0, coef = 0, corr = 0, counters = 0;
    size_t ew_buf = 0, ew_partials = 0;  // element scales: two [n_flat] fp32 buffers
    size_t w_norm = 0;                    // LARS: [n_tiles] fp32 sums of w^2 carried over
    size_t g_prev_l = 0;                  // [L] fp64 per-layer G_prev
    size_t last_sens_l = 0;               // [L] int32 per-layer last sensitive bit
    size_t chunks = 0, chunk_sums = 0, chunk_count = 0;
    size_t counters_bytes = 0;  // finished-layer counter, correction flag
    size_t lstats = 0, gstats = 0, gradscale = 0, state = 0, end = 0;
    size_t rec_bytes = 0;    // lstats .. gstats end
    size_t state_bytes = 0;  // gradscale .. state end
};

size_t elem_bytes(ags_dtype dt) { return dt == AGS_BF16 ? 2 : 4; }

bool materialize_gbar(const ags_config& c) {
    // Only a LARS step has a second pass over the replica mean.  Keep it when
    // re-reading the replicas there would cost more than writing and reading
    // one fp32 per element.
    return c.mode == AGS_MODE_LARS && (size_t)c.K * elem_bytes(c.grad_dtype) > 8;
}

// stats_only: the pieces a statistics-only call uses (no replica mean kept
// between passes, no element scales, no carried weight norms).
WsLayout ws_layout(const ags_config& c, int64_t n_tiles, int64_t n_chunks, bool stats_only = false) {
    WsLayout w;
    size_t p = 0;
    const size_t L = (size_t)c.n_layers;
    w.gbar = p;
    if (materialize_gbar(c) && !stats_only) p = align_up(p + (size_t)c.n_flat * sizeof(float));
    w.ew_buf = p;
    w.ew_partials = p;
    if (c.elementwise && !stats_only) {
        p = align_up(p + 2 * (size_t)c.n_flat * sizeof(float));
        w.ew_partials = p;
        p = align_up(p + (size_t)n_tiles * sizeof(float));
    }
    w.w_norm = p;
    if (c.reuse_w_norms && !stats_only) p = align_up(p + (size_t)n_tiles * sizeof(float));
    w.tiles = p;
    p = align_up(p + (size_t)n_tiles * sizeof(Tile));
    w.partials = p;
    p = align_up(p + (size_t)n_tiles * sizeof(Partial));
    w.ldev = p;
    p = align_up(p + L * sizeof(LayerDev));
    w.coef = p;
    p = align_up(p + L * sizeof(float2));
    w.chunks = p;
    p = align_up(p + (size_t)n_chunks * sizeof(ags::FinChunk));
    w.chunk_sums = p;
    p = align_up(p + (size_t)n_chunks * sizeof(ags::ChunkSum));
    w.chunk_count = p;
    p = align_up(p + L * sizeof(unsigned));
    w.corr = p;
    p = align_up(p + L * sizeof(float2));
    w.counters = p;
    w.counters_bytes = 2 * sizeof(unsigned);
    p = align_up(p + w.counters_bytes);
    w.g_prev_l = p;
    p = align_up(p + L * sizeof(double));
    w.last_sens_l = p;
    p = align_up(p + L * sizeof(int32_t));
    w.lstats = p;
    p += L * sizeof(ags_layer_stats);
    w.gstats = p;
    p += sizeof(ags_global_stats);
    w.rec_bytes = p - w.lstats;
    p = (p + 7) / 8 * 8;
    w.gradscale = p;
    p += L * sizeof(double);
    w.state = p;
    p += sizeof(DevState);
    w.state_bytes = p - w.gradscale;
    w.end = align_up(p);
    return w;
}

bool finite(double x) { return std::isfinite(x); }

// The 32-bit value of an enum-typed field as the caller stored it: loading
// an enum object that holds a value outside the enumeration is undefined
// behaviour in C++, so fields are validated from their bytes.
template <typename E>
int32_t raw_enum(const E& e) {
    static_assert(sizeof(E) == sizeof(int32_t), "enum fields are 32-bit");
    int32_t v;
    std::memcpy(&v, &e, sizeof v);
    return v;
}

// Host-only validation of a configuration.  Fills why on failure.
ags_status check_config(const ags_config* c, std::string& why) {
    if (!c) { why = "cfg is NULL"; return AGS_E_ARG; }
    if (c->n_layers < 1) { why = "n_layers must be >= 1"; return AGS_E_LAYOUT; }
    if (!c->layers) { why = "layers is NULL"; return AGS_E_ARG; }
    if (c->n_flat < 1) { why = "n_flat must be >= 1"; return AGS_E_LAYOUT; }
    if (c->K < 1 || c->K > AGS_MAX_K) { why = "K out of range 1..AGS_MAX_K"; return AGS_E_ARG; }
    const int32_t dt = raw_enum(c->grad_dtype), mode = raw_enum(c->mode);
    if (dt != AGS_F32 && dt != AGS_BF16) { why = "bad grad_dtype"; return AGS_E_ARG; }
    if (mode != AGS_MODE_SGD && mode != AGS_MODE_AGS && mode != AGS_MODE_LARS &&
        mode != AGS_MODE_STATIC) {
        why = "bad mode";
        return AGS_E_ARG;
    }
    if (!finite(c->lr) || c->lr < 0) { why = "lr must be finite and >= 0"; return AGS_E_ARG; }
    if (!finite(c->momentum) || c->momentum < 0 || c->momentum >= 1) {
        why = "momentum must be in [0, 1)";
        return AGS_E_ARG;
    }
    if (!finite(c->weight_decay) || c->weight_decay < 0) { why = "weight_decay must be >= 0"; return AGS_E_ARG; }
    if (!finite(c->delta) || c->delta < 0) { why = "delta must be finite and >= 0"; return AGS_E_ARG; }
    if (!finite(c->eps) || c->eps < 0) { why = "eps must be finite and >= 0"; return AGS_E_ARG; }
    if (!finite(c->s_max)) { why = "s_max must be finite"; return AGS_E_ARG; }
    if (c->mode == AGS_MODE_LARS && !(finite(c->trust_coef) && c->trust_coef > 0)) {
        why = "trust_coef must be > 0 in LARS mode";
        return AGS_E_ARG;
    }
    if (c->mode == AGS_MODE_STATIC && !(finite(c->static_scale) && c->static_scale > 0)) {
        why = "static_scale must be finite and > 0 in STATIC mode";
        return AGS_E_ARG;
    }
    if (c->elementwise != 0 && c->elementwise != 1) { why = "elementwise must be 0 or 1"; return AGS_E_ARG; }
    if (c->elementwise && c->mode != AGS_MODE_AGS) {
        why = "elementwise scales need AGS_MODE_AGS";
        return AGS_E_ARG;
    }
    if (c->delta_scope != AGS_DELTA_GLOBAL && c->delta_scope != AGS_DELTA_LAYER) {
        why = "bad delta_scope";
        return AGS_E_ARG;
    }
    if (c->reuse_w_norms != 0 && c->reuse_w_norms != 1) {
        why = "reuse_w_norms must be 0 or 1";
        return AGS_E_ARG;
    }
    if (c->reuse_w_norms && c->mode != AGS_MODE_LARS) {
        why = "reuse_w_norms needs AGS_MODE_LARS";
        return AGS_E_ARG;
    }
    if (c->refresh_every < 0) { why = "refresh_every must be >= 0"; return AGS_E_ARG; }
    if (c->small_replica < -1 || c->small_replica >= c->K) {
        why = "small_replica must be -1 or in 0..K-1";
        return AGS_E_ARG;
    }
    int64_t prev_end = 0;
    for (int32_t l = 0; l < c->n_layers; ++l) {
        const ags_layer& L = c->layers[l];
        char buf[160];
        if (L.numel < 1 || L.offset < 0) {
            snprintf(buf, sizeof buf, "layer %d: numel must be > 0 and offset >= 0", l);
            why = buf;
            return AGS_E_LAYOUT;
        }
        if (L.offset % AGS_ALIGN_ELEMS != 0) {
            snprintf(buf, sizeof buf, "layer %d: offset %lld is not a multiple of %d", l,
                     (long long)L.offset, AGS_ALIGN_ELEMS);
            why = buf;
            return AGS_E_ALIGN;
        }
        if (L.offset < prev_end) {
            snprintf(buf, sizeof buf, "layer %d overlaps or precedes the previous layer", l);
            why = buf;
            return AGS_E_LAYOUT;
        }
        if (L.numel > c->n_flat || L.offset > c->n_flat - L.numel) {
            snprintf(buf, sizeof buf, "layer %d ends past n_flat", l);
            why = buf;
            return AGS_E_LAYOUT;
        }
        if ((L.flags & ~(AGS_LAYER_SCALE | AGS_LAYER_DECAY)) != 0 || L.reserved != 0) {
            snprintf(buf, sizeof buf, "layer %d: unknown flags or nonzero reserved field", l);
            why = buf;
            return AGS_E_ARG;
        }
        prev_end = L.offset + L.numel;
    }
    return AGS_OK;
}

int64_t count_tiles(const ags_config& c) {
    int64_t n = 0;
    for (int32_t l = 0; l < c.n_layers; ++l) {
        const int64_t te = ags::tile_elems_for(c.layers[l].numel);
        n += (c.layers[l].numel + te - 1) / te;
    }
    return n;
}

int64_t count_chunks(const ags_config& c) {
    int64_t n = 0;
    for (int32_t l = 0; l < c.n_layers; ++l) {
        const int64_t te = ags::tile_elems_for(c.layers[l].numel);
        const int64_t tiles = (c.layers[l].numel + te - 1) / te;
        n += (tiles + ags::kFinTilesPerChunk - 1) / ags::kFinTilesPerChunk;
    }
    return n;
}

// check_config, then the launch limits: a step kernel launch has one
// 256-thread block per tile, and a launch holds fewer than 2^32 work-items.
ags_status check_config_and_size(const ags_config* c, std::string& why) {
    const ags_status s = check_config(c, why);
    if (s != AGS_OK) return s;
    if (count_tiles(*c) * ags::kTileBlock > (int64_t)0xffffffffLL) {
        why = "the layers need too many tiles for one launch (tiles x 256 must be < 2^32)";
        return AGS_E_LAYOUT;
    }
    return AGS_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Do the byte ranges [a, a + na) and [b, b + nb) share a byte?
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y ? y - x < na : x - y < nb;
}

// Is [p, p + bytes) inside one device allocation of the current device?
ags_status check_device_range(const void* p, size_t bytes, const char* name, std::string& why) {
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof attr);
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        why = std::string(name) + " is not a HIP allocation";
        return AGS_E_ARG;
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) {
        why = std::string(name) + " is not device memory";
        return AGS_E_ARG;
    }
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || attr.device != dev) {
        (void)hipGetLastError();
        why = std::string(name) + " belongs to another device than the current one";
        return AGS_E_ARG;
    }
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<void*>(p));
    if (e != hipSuccess) {
        (void)hipGetLastError();
        why = std::string(name) + ": allocation range unknown";
        return AGS_E_ARG;
    }
    const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
    if (q < b || q - b > size || bytes > size - (q - b)) {
        why = std::string(name) + " is smaller than the layout needs";
        return AGS_E_ARG;
    }
    return AGS_OK;
}

size_t workspace_cap() {
    const char* s = std::getenv("AGS_MAX_WORKSPACE_BYTES");
    if (!s || !*s) return (size_t)-1;
    char* end = nullptr;
    const unsigned long long v = std::strtoull(s, &end, 10);
    if (end == s) return (size_t)-1;
    return (size_t)v;
}

}  // namespace

namespace ags {
void set_thread_error(const char* why) { g_thread_error = why ? why : ""; }
}  // namespace ags

struct ags_handle {
    ags_config cfg{};
    std::vector<ags_layer> layers;
    float* d_w = nullptr;
    float* d_m = nullptr;
    int device = 0;
    int64_t n_tiles = 0;
    int64_t n_chunks = 0;
    // Fused steps launched outside graph capture: their parity sets the
    // step kernel's tile direction for layouts that outgrow the cache.
    int64_t n_fused = 0;
    int64_t grad_extent = 0;  // elements of one replica that are read
    bool materialize = false;
    WsLayout wl;
    char* ws = nullptr;
    char* pinned = nullptr;
    hipStream_t last_stream = nullptr;
    // Orders a call on another stream after the work queued on last_stream.
    hipEvent_t order_ev = nullptr;
    bool has_stats = false;
    // LARS: the last update pass left per-tile sums of w^2 that the next
    // statistics pass may take instead of reading w.
    bool w_norm_valid = false;
    // Dynamic LDS of the fused step kernel's launches, of the statistics-only
    // step kernel's and of the LARS update kernel's (0: none), capping the
    // blocks per CU for layouts whose w and m outgrow the Infinity Cache.
    int lds_pad = 0, lds_pad_stats = 0, lds_pad_update = 0;
    mutable std::string err;
    bool profiling = false;
    // Per timed step: start and stop event of each kernel's dispatch.
    std::vector<std::array<hipEvent_t, 2 * AGS_N_KERNELS>> ev_pending, ev_free;

    Tile* tiles() const { return reinterpret_cast<Tile*>(ws + wl.tiles); }
    Partial* partials() const { return reinterpret_cast<Partial*>(ws + wl.partials); }
    LayerDev* ldev() const { return reinterpret_cast<LayerDev*>(ws + wl.ldev); }
    float2* coef() const { return reinterpret_cast<float2*>(ws + wl.coef); }
    float2* corr() const { return reinterpret_cast<float2*>(ws + wl.corr); }
    float* ew_buf(int i) const {
        return cfg.elementwise ? reinterpret_cast<float*>(ws + wl.ew_buf) + (size_t)i * cfg.n_flat : nullptr;
    }
    float* ew_partials() const {
        return cfg.elementwise ? reinterpret_cast<float*>(ws + wl.ew_partials) : nullptr;
    }
    unsigned* done_count() const { return reinterpret_cast<unsigned*>(ws + wl.counters); }
    int* corr_flag() const { return reinterpret_cast<int*>(done_count() + 1); }
    float* gbar() const { return materialize ? reinterpret_cast<float*>(ws + wl.gbar) : nullptr; }
    float* w_norm() const { return cfg.reuse_w_norms ? reinterpret_cast<float*>(ws + wl.w_norm) : nullptr; }
    ags_layer_stats* lstats() const { return reinterpret_cast<ags_layer_stats*>(ws + wl.lstats); }
    ags_global_stats* gstats() const { return reinterpret_cast<ags_global_stats*>(ws + wl.gstats); }
    double* gradscale() const { return reinterpret_cast<double*>(ws + wl.gradscale); }
    double* g_prev_l() const { return reinterpret_cast<double*>(ws + wl.g_prev_l); }
    int32_t* last_sens_l() const { return reinterpret_cast<int32_t*>(ws + wl.last_sens_l); }
    DevState* state() const { return reinterpret_cast<DevState*>(ws + wl.state); }

    ags_status fail(ags_status s, const std::string& why) const {
        err = why;
        return s;
    }
    ags_status hip_fail(hipError_t e, const char* what) const {
        err = std::string(what) + ": " + hipGetErrorString(e);
        (void)hipGetLastError();
        return AGS_E_DEVICE;
    }
};

namespace {

void free_handle(ags_handle* h) {
    if (!h) return;
    for (auto& q : h->ev_pending)
        for (auto e : q) (void)hipEventDestroy(e);
    for (auto& q : h->ev_free)
        for (auto e : q) (void)hipEventDestroy(e);
    if (h->order_ev) (void)hipEventDestroy(h->order_ev);
    if (h->ws) (void)hipFree(h->ws);
    if (h->pinned) (void)hipHostFree(h->pinned);
    delete h;
}

ags_status check_grads(ags_handle* h, const void* d_grads, int64_t stride) {
    if (!h) return AGS_E_ARG;
    if (!d_grads) return h->fail(AGS_E_ARG, "d_grads is NULL");
    if (!aligned16(d_grads)) return h->fail(AGS_E_ALIGN, "d_grads must be 16-byte aligned");
    if (stride < h->cfg.n_flat) return h->fail(AGS_E_ARG, "replica_stride must be >= n_flat");
    if (stride % AGS_ALIGN_ELEMS != 0)
        return h->fail(AGS_E_ALIGN, "replica_stride must be a multiple of AGS_ALIGN_ELEMS");
    const double total = (double)(h->cfg.K - 1) * (double)stride + (double)h->grad_extent;
    if (total * (double)elem_bytes(h->cfg.grad_dtype) > 9.0e18)
        return h->fail(AGS_E_ARG, "replica_stride too large");
    const size_t bytes = ((size_t)(h->cfg.K - 1) * (size_t)stride + (size_t)h->grad_extent) *
                         elem_bytes(h->cfg.grad_dtype);
    const size_t wm_bytes = (size_t)h->cfg.n_flat * sizeof(float);
    if (overlap(d_grads, bytes, h->d_w, wm_bytes) || overlap(d_grads, bytes, h->d_m, wm_bytes))
        return h->fail(AGS_E_ARG, "d_grads overlaps w or m");
    std::string why;
    const ags_status s = check_device_range(d_grads, bytes, "d_grads", why);
    if (s != AGS_OK) return h->fail(s, why);
    return AGS_OK;
}

// Is s capturing a graph (an error of the query counts as capturing, so no
// cross-stream wait is attempted then)?
bool is_capturing(hipStream_t s) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cs) != hipSuccess) {
        (void)hipGetLastError();
        return true;
    }
    return cs != hipStreamCaptureStatusNone;
}

ags_status launch_step(ags_handle* h, const void* d_grads, int64_t stride, hipStream_t s,
                       bool commit) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess || cur != h->device) {
        (void)hipGetLastError();
        return h->fail(AGS_E_DEVICE, "the current HIP device is not the handle's device");
    }
    // Every step of a handle shares its workspace and state: a call on
    // another stream waits for the work queued on the handle's last one
    // (not during graph capture, whose ordering is the caller's).
    if (s != h->last_stream && !is_capturing(s) && !is_capturing(h->last_stream)) {
        hipError_t e = hipEventRecord(h->order_ev, h->last_stream);
        if (e == hipSuccess) e = hipStreamWaitEvent(s, h->order_ev, 0);
        if (e != hipSuccess) return h->hip_fail(e, "ordering after the handle's last stream");
    }
    constexpr int NE = 2 * AGS_N_KERNELS;
    std::array<hipEvent_t, NE> ev{};
    // Steps enqueued while the stream is being captured into a graph are not
    // timed: a graph replays them without the handle's bookkeeping.
    const bool capturing = is_capturing(s);
    const bool prof = commit && h->profiling && !capturing;
    if (prof) {
        if (!h->ev_free.empty()) {
            ev = h->ev_free.back();
            h->ev_free.pop_back();
        } else {
            for (int i = 0; i < NE; ++i) {
                const hipError_t e = hipEventCreate(&ev[i]);
                if (e != hipSuccess) {
                    for (int j = 0; j < i; ++j) (void)hipEventDestroy(ev[j]);
                    return h->hip_fail(e, "hipEventCreate");
                }
            }
        }
    }
    auto kev = [&](int k) {
        return prof ? ags::KernelEvents{ev[2 * k], ev[2 * k + 1]} : ags::KernelEvents{};
    };
    // A failed launch hands the step's events back to the pool (and the
    // carried weight norms are no longer trusted).
    auto launch_fail = [&](hipError_t err, const char* what) {
        if (prof) h->ev_free.push_back(ev);
        h->w_norm_valid = false;
        return h->hip_fail(err, what);
    };
    const ags_config& c = h->cfg;
    const float invK = (float)(1.0 / (double)c.K);
    // AGS and SGD steps update w and m in the statistics pass with the
    // predicted coefficients; a LARS step needs its layer norms first.
    const bool fused = commit && c.mode != AGS_MODE_LARS;
    // Element scales: the step reads the buffer in force and, when the
    // refresh is due, writes the other one, which is in force afterwards;
    // the old one stays intact for the correction pass.  The kernels take
    // both from the device state.
    const bool ew = c.elementwise != 0;

    ags::StepArgs sa{};
    sa.grads = d_grads;
    sa.stride = stride;
    sa.w = h->d_w;
    sa.m = h->d_m;
    sa.gbar = (commit && !fused) ? h->gbar() : nullptr;
    sa.tiles = h->tiles();
    sa.partials = h->partials();
    sa.layers = h->ldev();
    sa.n_layers = c.n_layers;
    sa.K = c.K;
    sa.invK = invK;
    sa.small_replica = c.small_replica;
    sa.mode = c.mode;
    sa.commit = commit ? 1 : 0;
    sa.refresh_every = c.refresh_every;
    sa.momentum = (float)c.momentum;
    sa.delta = c.delta;
    sa.eps = c.eps;
    sa.s_max = c.s_max;
    sa.trust_coef = c.trust_coef;
    sa.static_scale = c.static_scale;
    sa.weight_decay = c.weight_decay;
    sa.gradscale = h->gradscale();
    sa.state = h->state();
    sa.g_prev_l = h->g_prev_l();
    sa.last_sens_l = h->last_sens_l();
    sa.delta_scope = c.delta_scope;
    sa.coef = h->coef();
    sa.corr = h->corr();
    sa.corr_flag = h->corr_flag();
    sa.updated = fused ? 1 : 0;
    sa.xcd_map = h->n_tiles >= ags::kXcdMapMinTiles ? 1 : 0;
    // A captured step keeps the forward direction (its replays cannot
    // alternate); the results are the same either way, only the order of
    // the tiles differs.
    sa.reverse = (fused && !capturing && 8 * c.n_flat > ags::kOccupancyCapMinBytes && (h->n_fused & 1)) ? 1 : 0;
    sa.done_count = h->done_count();
    sa.chunks = reinterpret_cast<const ags::FinChunk*>(h->ws + h->wl.chunks);
    sa.chunk_sums = reinterpret_cast<ags::ChunkSum*>(h->ws + h->wl.chunk_sums);
    sa.layer_chunk_count = reinterpret_cast<unsigned*>(h->ws + h->wl.chunk_count);
    sa.lstats = h->lstats();
    sa.gstats = h->gstats();
    sa.ew = !ew ? 0 : (16 * c.n_flat > ags::kEwStreamMinBytes ? 2 : 1);
    sa.ew_buf = h->ew_buf(0);
    sa.n_flat = c.n_flat;
    sa.ew_partials = h->ew_partials();
    // A step captured into a graph reads w: a replay cannot see whether the
    // carried weight norms still hold (the caller may have written w, or
    // restored a state, since the capture).
    sa.w_norm_in = (!fused && h->w_norm_valid && !capturing) ? h->w_norm() : nullptr;
    sa.lds_pad = ew ? 0 : (fused ? h->lds_pad : h->lds_pad_stats);
    hipError_t e = ags::launch_step(sa, c.grad_dtype, (int)h->n_tiles, fused, s, kev(0));
    if (e != hipSuccess) return launch_fail(e, "step kernel launch");
    e = ags::launch_finalize(sa, (int)h->n_chunks, s, kev(1));
    if (e != hipSuccess) return launch_fail(e, "finalize kernel launch");

    if (commit && c.mode != AGS_MODE_SGD) {
        ags::UpdateArgs ua{};
        ua.tiles = h->tiles();
        ua.n_tiles = (int)h->n_tiles;
        ua.gbar = h->gbar();
        ua.grads = d_grads;
        ua.stride = stride;
        ua.K = c.K;
        ua.invK = invK;
        ua.w = h->d_w;
        ua.m = h->d_m;
        ua.coef = h->coef();
        ua.corr = h->corr();
        ua.ew_buf = h->ew_buf(0);
        ua.n_flat = c.n_flat;
        ua.state = h->state();
        ua.refresh_every = c.refresh_every;
        ua.corr_flag = h->corr_flag();
        ua.momentum = (float)c.momentum;
        ua.w_norm_out = (c.mode == AGS_MODE_LARS) ? h->w_norm() : nullptr;
        ua.lds_pad = h->lds_pad_update;
        ua.reverse = (8 * c.n_flat <= ags::kOccupancyCapMinBytes) ? 1 : 0;
        e = (c.mode == AGS_MODE_LARS) ? ags::launch_update(ua, c.grad_dtype, s, kev(2))
                                      : ags::launch_correct(ua, c.grad_dtype, s, kev(2));
        if (e != hipSuccess) return launch_fail(e, "second-pass kernel launch");
    }
    if (prof) h->ev_pending.push_back(ev);
    if (fused && !capturing) ++h->n_fused;
    // A captured step has not run: the norms are what the last executed
    // update pass left (every update pass, replayed ones included, writes
    // them for the w it writes).
    if (commit && c.mode == AGS_MODE_LARS && !capturing) h->w_norm_valid = c.reuse_w_norms != 0;
    h->last_stream = s;
    h->has_stats = true;
    return AGS_OK;
}

}  // namespace

extern "C" {

const char* ags_status_string(ags_status s) {
    switch (s) {
        case AGS_OK: return "AGS_OK";
        case AGS_E_ARG: return "AGS_E_ARG: bad argument";
        case AGS_E_LAYOUT: return "AGS_E_LAYOUT: bad layer table";
        case AGS_E_ALIGN: return "AGS_E_ALIGN: misaligned offset, stride or pointer";
        case AGS_E_NOMEM: return "AGS_E_NOMEM: workspace allocation failed";
        case AGS_E_DEVICE: return "AGS_E_DEVICE: HIP error";
        case AGS_E_STATE: return "AGS_E_STATE: handle state mismatch";
    }
    return "unknown ags_status";
}

const char* ags_last_error(const ags_handle* h) {
    return h ? h->err.c_str() : g_thread_error.c_str();
}

ags_status ags_workspace_bytes(const ags_config* cfg, size_t* out_bytes) {
    std::string why;
    ags_status s = check_config_and_size(cfg, why);
    if (s != AGS_OK) {
        g_thread_error = why;
        return s;
    }
    if (!out_bytes) {
        g_thread_error = "out_bytes is NULL";
        return AGS_E_ARG;
    }
    *out_bytes = ws_layout(*cfg, count_tiles(*cfg), count_chunks(*cfg)).end;
    return AGS_OK;
}

ags_status ags_init(const ags_config* cfg, float* d_w, float* d_m, void* hip_stream,
                    ags_handle** out) {
    std::string why;
    if (!out) {
        g_thread_error = "out is NULL";
        return AGS_E_ARG;
    }
    *out = nullptr;
    ags_status st = check_config_and_size(cfg, why);
    if (st != AGS_OK) {
        g_thread_error = why;
        return st;
    }
    if (!d_w || !d_m) {
        g_thread_error = "d_w and d_m must not be NULL";
        return AGS_E_ARG;
    }
    if (!aligned16(d_w) || !aligned16(d_m)) {
        g_thread_error = "d_w and d_m must be 16-byte aligned";
        return AGS_E_ALIGN;
    }
    if (overlap(d_w, (size_t)cfg->n_flat * sizeof(float), d_m, (size_t)cfg->n_flat * sizeof(float))) {
        g_thread_error = "d_w and d_m overlap";
        return AGS_E_ARG;
    }
    const int64_t n_tiles = count_tiles(*cfg);

    // Host-side tables.
    std::vector<Tile> tiles;
    std::vector<LayerDev> ldev(cfg->n_layers);
    std::vector<ags::FinChunk> chunks;
    tiles.reserve((size_t)n_tiles);
    for (int32_t l = 0; l < cfg->n_layers; ++l) {
        const ags_layer& L = cfg->layers[l];
        ldev[l].tile_begin = (int32_t)tiles.size();
        const int64_t te = ags::tile_elems_for(L.numel);
        for (int64_t o = 0; o < L.numel; o += te) {
            Tile t;
            t.begin = L.offset + o;
            t.count = (int32_t)((L.numel - o) < te ? (L.numel - o) : te);
            t.layer = l;
            tiles.push_back(t);
        }
        ldev[l].tile_end = (int32_t)tiles.size();
        ldev[l].flags = L.flags;
        ldev[l].chunk_begin = (int32_t)chunks.size();
        for (int32_t tb = ldev[l].tile_begin; tb < ldev[l].tile_end; tb += ags::kFinTilesPerChunk) {
            ags::FinChunk ch;
            ch.layer = l;
            ch.tile_begin = tb;
            ch.tile_end = std::min<int32_t>(tb + ags::kFinTilesPerChunk, ldev[l].tile_end);
            ch.pad_ = 0;
            chunks.push_back(ch);
        }
        ldev[l].chunk_end = (int32_t)chunks.size();
        ldev[l].pad_ = 0;
        ldev[l].numel = L.numel;
    }
    int64_t extent = 0;
    for (int32_t l = 0; l < cfg->n_layers; ++l)
        extent = std::max<int64_t>(extent, cfg->layers[l].offset + cfg->layers[l].numel);

    // Workspace size and the byte cap, still before any HIP call.
    const WsLayout wl = ws_layout(*cfg, n_tiles, count_chunks(*cfg));
    const size_t cap = workspace_cap();
    if (wl.end > cap) {
        char buf[200];
        snprintf(buf, sizeof buf, "workspace of %zu bytes exceeds AGS_MAX_WORKSPACE_BYTES=%zu",
                 wl.end, cap);
        g_thread_error = buf;
        return AGS_E_NOMEM;
    }

    // Device checks (first HIP calls).
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        g_thread_error = std::string("hipGetDevice: ") + hipGetErrorString(e);
        (void)hipGetLastError();
        return AGS_E_DEVICE;
    }
    st = check_device_range(d_w, (size_t)extent * sizeof(float), "d_w", why);
    if (st == AGS_OK) st = check_device_range(d_m, (size_t)extent * sizeof(float), "d_m", why);
    if (st != AGS_OK) {
        g_thread_error = why;
        return st;
    }

    ags_handle* h = new (std::nothrow) ags_handle();
    if (!h) {
        g_thread_error = "host allocation failed";
        return AGS_E_NOMEM;
    }
    h->cfg = *cfg;
    h->layers.assign(cfg->layers, cfg->layers + cfg->n_layers);
    h->cfg.layers = h->layers.data();
    h->d_w = d_w;
    h->d_m = d_m;
    h->device = dev;
    h->n_tiles = n_tiles;
    h->n_chunks = (int64_t)chunks.size();
    h->grad_extent = extent;
    h->materialize = materialize_gbar(*cfg);
    h->wl = wl;
    e = hipMalloc(reinterpret_cast<void**>(&h->ws), h->wl.end);
    if (e != hipSuccess) {
        h->ws = nullptr;
        (void)hipGetLastError();
        g_thread_error = std::string("hipMalloc of the workspace failed: ") + hipGetErrorString(e);
        free_handle(h);
        return AGS_E_NOMEM;
    }
    const size_t pinned_bytes = h->wl.rec_bytes + h->wl.state_bytes + 64;
    e = hipHostMalloc(reinterpret_cast<void**>(&h->pinned), pinned_bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        h->pinned = nullptr;
        (void)hipGetLastError();
        g_thread_error = std::string("hipHostMalloc of the staging buffer failed: ") + hipGetErrorString(e);
        free_handle(h);
        return AGS_E_NOMEM;
    }
    // Occupancy caps of the fused step kernel, the statistics-only step
    // kernel and the LARS update kernel: LDS pads so that at most the given
    // number of blocks fit on a CU (left off if the device does not report
    // its LDS sizes).  The kernels use at most 1 KiB of static LDS.
    if (8 * cfg->n_flat > ags::kOccupancyCapMinBytes) {
        int lds_cu = 0, lds_block = 0;
        if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
                hipSuccess ||
            hipDeviceGetAttribute(&lds_block, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
                hipSuccess) {
            (void)hipGetLastError();
            lds_cu = lds_block = 0;
        }
        auto pad_for = [&](int blocks) {
            const int pad = lds_cu / (blocks + 1) + 1024;
            return lds_cu > 0 && pad + 1024 <= lds_block && blocks * (pad + 1024) <= lds_cu ? pad : 0;
        };
        h->lds_pad = pad_for(ags::kCappedBlocksPerCu);
        h->lds_pad_stats = pad_for(ags::kCappedBlocksPerCuStats);
        h->lds_pad_update = pad_for(ags::kCappedBlocksPerCuUpdate);
    }
    e = hipEventCreateWithFlags(&h->order_ev, hipEventDisableTiming);
    if (e != hipSuccess) {
        h->order_ev = nullptr;
        g_thread_error = std::string("hipEventCreateWithFlags: ") + hipGetErrorString(e);
        (void)hipGetLastError();
        free_handle(h);
        return AGS_E_DEVICE;
    }

    // Initial device state: tables, gradscale = 1, G_prev = 0, step = 0,
    // the configured learning rate.
    hipStream_t s = static_cast<hipStream_t>(hip_stream);
    std::vector<double> ones(cfg->n_layers, 1.0);
    DevState ds{0.0, 0, 0, 0, (float)cfg->lr, 0};
    const struct {
        size_t off;
        const void* src;
        size_t bytes;
    } up[] = {
        {h->wl.tiles, tiles.data(), tiles.size() * sizeof(Tile)},
        {h->wl.ldev, ldev.data(), ldev.size() * sizeof(LayerDev)},
        {h->wl.chunks, chunks.data(), chunks.size() * sizeof(ags::FinChunk)},
        {h->wl.gradscale, ones.data(), ones.size() * sizeof(double)},
        {h->wl.state, &ds, sizeof ds},
    };
    e = hipMemsetAsync(h->ws + h->wl.lstats, 0, h->wl.rec_bytes, s);
    if (e == hipSuccess) e = hipMemsetAsync(h->ws + h->wl.counters, 0, h->wl.counters_bytes, s);
    if (e == hipSuccess)
        e = hipMemsetAsync(h->ws + h->wl.chunk_count, 0, (size_t)cfg->n_layers * sizeof(unsigned), s);
    if (e == hipSuccess)
        e = hipMemsetAsync(h->ws + h->wl.g_prev_l, 0, (size_t)cfg->n_layers * sizeof(double), s);
    if (e == hipSuccess)
        e = hipMemsetAsync(h->ws + h->wl.last_sens_l, 0, (size_t)cfg->n_layers * sizeof(int32_t), s);
    if (e == hipSuccess && cfg->elementwise)  // element scales start at 1.0f
        e = hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(h->ew_buf(0)), 0x3f800000,
                              2 * (size_t)cfg->n_flat, s);
    for (const auto& u : up) {
        if (e != hipSuccess) break;
        e = hipMemcpyAsync(h->ws + u.off, u.src, u.bytes, hipMemcpyHostToDevice, s);
    }
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        g_thread_error = std::string("initial upload: ") + hipGetErrorString(e);
        (void)hipGetLastError();
        free_handle(h);
        return AGS_E_DEVICE;
    }
    h->last_stream = s;
    *out = h;
    return AGS_OK;
}

ags_status ags_stats(ags_handle* h, const void* d_grads, int64_t replica_stride, void* hip_stream) {
    ags_status s = check_grads(h, d_grads, replica_stride);
    if (s != AGS_OK) return s;
    return launch_step(h, d_grads, replica_stride, static_cast<hipStream_t>(hip_stream), false);
}

ags_status ags_step(ags_handle* h, const void* d_grads, int64_t replica_stride, void* hip_stream) {
    ags_status s = check_grads(h, d_grads, replica_stride);
    if (s != AGS_OK) return s;
    return launch_step(h, d_grads, replica_stride, static_cast<hipStream_t>(hip_stream), true);
}

ags_status ags_read_stats(ags_handle* h, ags_layer_stats* out_layers, ags_global_stats* out_global) {
    if (!h) return AGS_E_ARG;
    if (!h->has_stats) return h->fail(AGS_E_STATE, "no ags_stats / ags_step has run yet");
    hipError_t e = hipMemcpyAsync(h->pinned, h->ws + h->wl.lstats, h->wl.rec_bytes,
                                  hipMemcpyDeviceToHost, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "reading statistics");
    if (out_layers)
        std::memcpy(out_layers, h->pinned, (size_t)h->cfg.n_layers * sizeof(ags_layer_stats));
    if (out_global)
        std::memcpy(out_global, h->pinned + (h->wl.gstats - h->wl.lstats), sizeof(ags_global_stats));
    return AGS_OK;
}

ags_status ags_set_lr(ags_handle* h, double lr) {
    if (!h) return AGS_E_ARG;
    if (!std::isfinite(lr) || lr < 0) return h->fail(AGS_E_ARG, "lr must be finite and >= 0");
    // The rate lives in the device state, written in stream order after the
    // handle's queued work, so that every later step reads it: eager ones
    // and those replayed from a graph captured before.
    const hipError_t e = ags::launch_set_lr(h->state(), (float)lr, h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "setting the learning rate");
    return AGS_OK;
}

ags_status ags_get_state(const ags_handle* h, double* gradscale_L, double* g_sq_prev, int64_t* step) {
    if (!h) return AGS_E_ARG;
    if (!gradscale_L || !g_sq_prev || !step) return h->fail(AGS_E_ARG, "NULL output pointer");
    hipError_t e = hipMemcpyAsync(h->pinned, h->ws + h->wl.gradscale, h->wl.state_bytes,
                                  hipMemcpyDeviceToHost, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "reading state");
    const size_t L = (size_t)h->cfg.n_layers;
    std::memcpy(gradscale_L, h->pinned, L * sizeof(double));
    DevState ds;
    std::memcpy(&ds, h->pinned + (h->wl.state - h->wl.gradscale), sizeof ds);
    *g_sq_prev = ds.g_prev;
    *step = ds.step;
    return AGS_OK;
}

ags_status ags_set_state(ags_handle* h, const double* gradscale_L, double g_sq_prev, int64_t step) {
    if (!h) return AGS_E_ARG;
    const bool ew = h->cfg.elementwise != 0;
    if (!gradscale_L && !ew) return h->fail(AGS_E_ARG, "gradscale_L is NULL");
    if (!std::isfinite(g_sq_prev) || g_sq_prev < 0) return h->fail(AGS_E_ARG, "g_sq_prev must be finite and >= 0");
    if (step < 0) return h->fail(AGS_E_ARG, "step must be >= 0");
    const size_t L = (size_t)h->cfg.n_layers;
    if (!ew)
        for (size_t l = 0; l < L; ++l)
            if (!std::isfinite(gradscale_L[l]) || !(gradscale_L[l] > 0))
                return h->fail(AGS_E_ARG, "gradscale values must be finite and > 0");
    // Wait for queued steps first: the staging buffer and the state are
    // shared with them.
    hipError_t e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "waiting for the last stream");
    h->w_norm_valid = false;  // a restored state comes with weights of its own
    // g_prev and step only: the element-scale buffer index stays.
    DevState ds{g_sq_prev, step, 0, 0, 0.0f, 0};
    const size_t soff = h->wl.state - h->wl.gradscale;
    const size_t head = offsetof(DevState, ew_cur);
    std::memcpy(h->pinned + soff, &ds, head);
    if (!ew) std::memcpy(h->pinned, gradscale_L, L * sizeof(double));
    e = ew ? hipMemcpyAsync(h->ws + h->wl.state, h->pinned + soff, head, hipMemcpyHostToDevice,
                            h->last_stream)
           : hipMemcpyAsync(h->ws + h->wl.gradscale, h->pinned, soff + head,
                            hipMemcpyHostToDevice, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "writing state");
    return AGS_OK;
}

ags_status ags_invalidate_weight_norms(ags_handle* h) {
    if (!h) return AGS_E_ARG;
    if (!h->cfg.reuse_w_norms) return h->fail(AGS_E_STATE, "the handle does not carry weight norms");
    h->w_norm_valid = false;
    return AGS_OK;
}

ags_status ags_get_layer_state(ags_handle* h, double* g_sq_prev_L) {
    if (!h) return AGS_E_ARG;
    if (!g_sq_prev_L) return h->fail(AGS_E_ARG, "g_sq_prev_L is NULL");
    const size_t bytes = (size_t)h->cfg.n_layers * sizeof(double);
    hipError_t e = hipMemcpyAsync(g_sq_prev_L, h->g_prev_l(), bytes, hipMemcpyDeviceToHost,
                                  h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "reading the layer state");
    return AGS_OK;
}

ags_status ags_set_layer_state(ags_handle* h, const double* g_sq_prev_L) {
    if (!h) return AGS_E_ARG;
    if (!g_sq_prev_L) return h->fail(AGS_E_ARG, "g_sq_prev_L is NULL");
    for (int32_t l = 0; l < h->cfg.n_layers; ++l)
        if (!std::isfinite(g_sq_prev_L[l]) || g_sq_prev_L[l] < 0)
            return h->fail(AGS_E_ARG, "g_sq_prev_L values must be finite and >= 0");
    const size_t bytes = (size_t)h->cfg.n_layers * sizeof(double);
    hipError_t e = hipStreamSynchronize(h->last_stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(h->g_prev_l(), g_sq_prev_L, bytes, hipMemcpyHostToDevice, h->last_stream);
    // the layers' last decisions are cleared (ags_set_last_decision restores them)
    if (e == hipSuccess)
        e = hipMemsetAsync(h->last_sens_l(), 0, (size_t)h->cfg.n_layers * sizeof(int32_t),
                           h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "writing the layer state");
    return AGS_OK;
}

ags_status ags_get_last_decision(ags_handle* h, int32_t* sensitive, int32_t* sensitive_L) {
    if (!h) return AGS_E_ARG;
    if (!sensitive) return h->fail(AGS_E_ARG, "sensitive is NULL");
    int32_t g = 0;
    hipError_t e = hipMemcpyAsync(&g, h->ws + h->wl.state + offsetof(DevState, last_sens), sizeof g,
                                  hipMemcpyDeviceToHost, h->last_stream);
    if (e == hipSuccess && sensitive_L)
        e = hipMemcpyAsync(sensitive_L, h->last_sens_l(), (size_t)h->cfg.n_layers * sizeof(int32_t),
                           hipMemcpyDeviceToHost, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "reading the last decision");
    *sensitive = g;
    return AGS_OK;
}

ags_status ags_set_last_decision(ags_handle* h, int32_t sensitive, const int32_t* sensitive_L) {
    if (!h) return AGS_E_ARG;
    if (sensitive != 0 && sensitive != 1) return h->fail(AGS_E_ARG, "sensitive must be 0 or 1");
    const size_t L = (size_t)h->cfg.n_layers;
    if (sensitive_L)
        for (size_t l = 0; l < L; ++l)
            if (sensitive_L[l] != 0 && sensitive_L[l] != 1)
                return h->fail(AGS_E_ARG, "sensitive_L values must be 0 or 1");
    hipError_t e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "waiting for the last stream");
    // through the pinned staging buffer (no step is queued now)
    int32_t* st = reinterpret_cast<int32_t*>(h->pinned);
    st[0] = sensitive;
    e = hipMemcpyAsync(h->ws + h->wl.state + offsetof(DevState, last_sens), st, sizeof(int32_t),
                       hipMemcpyHostToDevice, h->last_stream);
    if (e == hipSuccess && sensitive_L)
        e = hipMemcpyAsync(h->last_sens_l(), sensitive_L, L * sizeof(int32_t), hipMemcpyHostToDevice,
                           h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "writing the last decision");
    return AGS_OK;
}

namespace {

// The element-scale buffer in force (read from the device state).
ags_status ew_current(ags_handle* h, int* cur) {
    int32_t v = 0;
    hipError_t e = hipMemcpyAsync(&v, h->ws + h->wl.state + offsetof(DevState, ew_cur), sizeof v,
                                  hipMemcpyDeviceToHost, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "reading the element-scale buffer index");
    *cur = v ? 1 : 0;
    return AGS_OK;
}

}  // namespace

ags_status ags_get_elementwise_scale(ags_handle* h, float* scale, int64_t n) {
    if (!h) return AGS_E_ARG;
    if (!h->cfg.elementwise) return h->fail(AGS_E_STATE, "the handle has no element scales");
    if (!scale) return h->fail(AGS_E_ARG, "scale is NULL");
    if (n != h->cfg.n_flat) return h->fail(AGS_E_ARG, "n must equal n_flat");
    int cur = 0;
    ags_status st = ew_current(h, &cur);
    if (st != AGS_OK) return st;
    hipError_t e = hipMemcpyAsync(scale, h->ew_buf(cur), (size_t)n * sizeof(float),
                                  hipMemcpyDeviceToHost, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "reading element scales");
    return AGS_OK;
}

ags_status ags_set_elementwise_scale(ags_handle* h, const float* scale, int64_t n) {
    if (!h) return AGS_E_ARG;
    if (!h->cfg.elementwise) return h->fail(AGS_E_STATE, "the handle has no element scales");
    if (!scale) return h->fail(AGS_E_ARG, "scale is NULL");
    if (n != h->cfg.n_flat) return h->fail(AGS_E_ARG, "n must equal n_flat");
    for (int64_t j = 0; j < n; ++j)
        if (!std::isfinite(scale[j]) || scale[j] < 0.0f)
            return h->fail(AGS_E_ARG, "element scales must be finite and >= 0");
    const size_t L = (size_t)h->cfg.n_layers;
    std::vector<double> mean(L);
    for (size_t l = 0; l < L; ++l) {
        const ags_layer& ly = h->layers[l];
        double sum = 0.0;
        for (int64_t j = 0; j < ly.numel; ++j) sum += (double)scale[ly.offset + j];
        mean[l] = sum / (double)ly.numel;
    }
    // The scales go to buffer 0, which is then the one in force.
    const int32_t zero = 0;
    hipError_t e = hipStreamSynchronize(h->last_stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(h->ew_buf(0), scale, (size_t)n * sizeof(float), hipMemcpyHostToDevice,
                           h->last_stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(h->ws + h->wl.gradscale, mean.data(), L * sizeof(double),
                           hipMemcpyHostToDevice, h->last_stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(h->ws + h->wl.state + offsetof(DevState, ew_cur), &zero, sizeof zero,
                           hipMemcpyHostToDevice, h->last_stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->last_stream);
    if (e != hipSuccess) return h->hip_fail(e, "writing element scales");
    return AGS_OK;
}

ags_status ags_set_profiling(ags_handle* h, int enable) {
    if (!h) return AGS_E_ARG;
    h->profiling = enable != 0;
    return AGS_OK;
}

ags_status ags_get_kernel_times(ags_handle* h, double* out_ms, int64_t* out_calls) {
    if (!h) return AGS_E_ARG;
    if (!out_ms || !out_calls) return h->fail(AGS_E_ARG, "NULL output pointer");
    double tot[AGS_N_KERNELS] = {0, 0, 0};
    for (auto& q : h->ev_pending) {
        // An SGD step launches no second pass (its time stays 0).
        const int nk = h->cfg.mode == AGS_MODE_SGD ? AGS_N_KERNELS - 1 : AGS_N_KERNELS;
        hipError_t e = hipEventSynchronize(q[2 * nk - 1]);
        if (e != hipSuccess) return h->hip_fail(e, "hipEventSynchronize");
        for (int k = 0; k < nk; ++k) {
            float ms = 0;
            e = hipEventElapsedTime(&ms, q[2 * k], q[2 * k + 1]);
            if (e != hipSuccess) return h->hip_fail(e, "hipEventElapsedTime");
            tot[k] += ms;
        }
    }
    *out_calls = (int64_t)h->ev_pending.size();
    for (int k = 0; k < AGS_N_KERNELS; ++k) out_ms[k] = tot[k];
    for (auto& q : h->ev_pending) h->ev_free.push_back(q);
    h->ev_pending.clear();
    return AGS_OK;
}

void ags_destroy(ags_handle* h) {
    if (!h) return;
    (void)hipStreamSynchronize(h->last_stream);
    free_handle(h);
}

}  // extern "C"

// ------------------------------------------------ statistics without allocation --
//
// ags_stats_noalloc keeps everything a statistics call needs beyond its
// inputs and outputs (the layer table, the tile map, tile partials, chunk
// sums, counters, the initial state and the records) in one file-scope
// device array, so that it never allocates.  Each GPU holds its own copy of
// the array until the process ends, found once per device through
// hipGetSymbolAddress; host code uses only that address, never the array's
// name.  Every call on a GPU uses the same array, so calls that overlap on
// one GPU race.

namespace {
constexpr size_t kScratchBytes = 6u << 20;
constexpr int kMaxScratchDevices = 64;
}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// The address of this GPU's scratch array (the current device), looked up
// on the first call on the device.
ags_status scratch_address(int dev, unsigned char** out, std::string& why) {
    if (dev < 0 || dev >= kMaxScratchDevices) {
        why = "device index beyond the scratch table";
        return AGS_E_DEVICE;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            why = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
            (void)hipGetLastError();
            return AGS_E_DEVICE;
        }
        g_scratch_ptr[dev] = p;
    }
    *out = static_cast<unsigned char*>(g_scratch_ptr[dev]);
    return AGS_OK;
}

// Pieces of the tables a statistics call builds in the scratch array.
struct NoallocTables {
    const ags_layer* layers;  // copy of the caller's layer table
    int n_layers;
    LayerDev* ldev;
    Tile* tiles;
    ags::FinChunk* chunks;
    DevState* state;
    double* gradscale;
    double* g_prev_l;
    int32_t* last_sens_l;
    unsigned* chunk_count;
    unsigned* counters;  // finished-layer counter, correction flag
};

// One block: every layer's tile and chunk ranges (an exclusive scan of the
// per-layer counts, with ags_init's tiling: tiles of tile_elems_for(numel)
// elements, chunks of ags::kFinTilesPerChunk tiles), and the state of a
// handle that has taken no step (gradscale 1, no previous norms, counters
// at zero).
__global__ __launch_bounds__(256) void noalloc_layers_kernel(NoallocTables t) {
    __shared__ int sh_t[256], sh_c[256];
    const int tid = threadIdx.x;
    const int per = (t.n_layers + 255) / 256;
    const int l0 = min(tid * per, t.n_layers), l1 = min(l0 + per, t.n_layers);
    int nt = 0, nc = 0;
    for (int l = l0; l < l1; ++l) {
        const int64_t n = t.layers[l].numel, te = ags::tile_elems_for(n);
        const int tl = (int)((n + te - 1) / te);
        nt += tl;
        nc += (tl + ags::kFinTilesPerChunk - 1) / ags::kFinTilesPerChunk;
    }
    sh_t[tid] = nt;
    sh_c[tid] = nc;
    __syncthreads();
    if (tid == 0) {
        int rt = 0, rc = 0;
        for (int i = 0; i < 256; ++i) {
            const int a = sh_t[i], b = sh_c[i];
            sh_t[i] = rt;
            sh_c[i] = rc;
            rt += a;
            rc += b;
        }
    }
    __syncthreads();
    int tb = sh_t[tid], cb = sh_c[tid];
    for (int l = l0; l < l1; ++l) {
        const ags_layer ly = t.layers[l];
        const int64_t te = ags::tile_elems_for(ly.numel);
        const int tl = (int)((ly.numel + te - 1) / te);
        const int cl = (tl + ags::kFinTilesPerChunk - 1) / ags::kFinTilesPerChunk;
        LayerDev d;
        d.tile_begin = tb;
        d.tile_end = tb + tl;
        d.flags = ly.flags;
        d.chunk_begin = cb;
        d.chunk_end = cb + cl;
        d.pad_ = 0;
        d.numel = ly.numel;
        t.ldev[l] = d;
        tb += tl;
        cb += cl;
        t.gradscale[l] = 1.0;
        t.g_prev_l[l] = 0.0;
        t.last_sens_l[l] = 0;
        t.chunk_count[l] = 0u;
    }
    if (tid == 0) {
        DevState ds;
        ds.g_prev = 0.0;
        ds.step = 0;
        ds.last_sens = 0;
        ds.ew_cur = 0;
        ds.lr = 0.0f;  // a statistics call updates nothing
        ds.pad_ = 0;
        *t.state = ds;
        t.counters[0] = 0u;
        t.counters[1] = 0u;
    }
}

// One block per layer: its tiles and finalize chunks.
__global__ __launch_bounds__(256) void noalloc_tiles_kernel(NoallocTables t) {
    const int l = blockIdx.x;
    const LayerDev d = t.ldev[l];
    const ags_layer ly = t.layers[l];
    const int64_t te = ags::tile_elems_for(ly.numel);
    for (int i = d.tile_begin + (int)threadIdx.x; i < d.tile_end; i += blockDim.x) {
        const int64_t o = (int64_t)(i - d.tile_begin) * te;
        Tile x;
        x.begin = ly.offset + o;
        x.count = (int32_t)(ly.numel - o < te ? ly.numel - o : te);
        x.layer = l;
        t.tiles[i] = x;
    }
    for (int c = d.chunk_begin + (int)threadIdx.x; c < d.chunk_end; c += blockDim.x) {
        ags::FinChunk ch;
        ch.layer = l;
        ch.tile_begin = d.tile_begin + (c - d.chunk_begin) * ags::kFinTilesPerChunk;
        ch.tile_end = min(ch.tile_begin + ags::kFinTilesPerChunk, d.tile_end);
        ch.pad_ = 0;
        t.chunks[c] = ch;
    }
}

}  // namespace

extern "C" ags_status ags_stats_noalloc(const ags_config* cfg, const float* d_w, const void* d_grads,
                                        int64_t replica_stride, ags_layer_stats* out_layers,
                                        ags_global_stats* out_global, void* hip_stream) {
    std::string why;
    auto fail = [&](ags_status st) {
        g_thread_error = why;
        return st;
    };
    ags_status st = check_config_and_size(cfg, why);
    if (st != AGS_OK) return fail(st);
    if (!d_w || !d_grads) {
        why = "d_w and d_grads must not be NULL";
        return fail(AGS_E_ARG);
    }
    if (!out_layers || !out_global) {
        why = "out_layers and out_global must not be NULL";
        return fail(AGS_E_ARG);
    }
    if (!aligned16(d_w) || !aligned16(d_grads)) {
        why = "d_w and d_grads must be 16-byte aligned";
        return fail(AGS_E_ALIGN);
    }
    if (replica_stride < cfg->n_flat) {
        why = "replica_stride must be >= n_flat";
        return fail(AGS_E_ARG);
    }
    if (replica_stride % AGS_ALIGN_ELEMS != 0) {
        why = "replica_stride must be a multiple of AGS_ALIGN_ELEMS";
        return fail(AGS_E_ALIGN);
    }
    int64_t extent = 0;
    for (int32_t l = 0; l < cfg->n_layers; ++l)
        extent = std::max<int64_t>(extent, cfg->layers[l].offset + cfg->layers[l].numel);
    const double total = (double)(cfg->K - 1) * (double)replica_stride + (double)extent;
    if (total * (double)elem_bytes(cfg->grad_dtype) > 9.0e18) {
        why = "replica_stride too large";
        return fail(AGS_E_ARG);
    }
    const size_t gbytes = ((size_t)(cfg->K - 1) * (size_t)replica_stride + (size_t)extent) *
                          elem_bytes(cfg->grad_dtype);
    if (overlap(d_grads, gbytes, d_w, (size_t)extent * sizeof(float))) {
        why = "d_grads overlaps w";
        return fail(AGS_E_ARG);
    }
    // The scratch array's pieces: the layer table copy, then the workspace
    // of a statistics call.
    const int64_t n_tiles = count_tiles(*cfg), n_chunks = count_chunks(*cfg);
    const size_t lay_bytes = align_up((size_t)cfg->n_layers * sizeof(ags_layer));
    const WsLayout wl = ws_layout(*cfg, n_tiles, n_chunks, true);
    if (lay_bytes + wl.end > kScratchBytes) {
        char buf[240];
        snprintf(buf, sizeof buf,
                 "ags_stats_noalloc needs %zu bytes of scratch for %d layers and %lld tiles; the "
                 "scratch array holds %zu",
                 lay_bytes + wl.end, cfg->n_layers, (long long)n_tiles, kScratchBytes);
        why = buf;
        return fail(AGS_E_NOMEM);
    }
    // Device checks (first HIP calls).
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        why = std::string("hipGetDevice: ") + hipGetErrorString(e);
        (void)hipGetLastError();
        return fail(AGS_E_DEVICE);
    }
    st = check_device_range(d_w, (size_t)extent * sizeof(float), "d_w", why);
    if (st == AGS_OK) st = check_device_range(d_grads, gbytes, "d_grads", why);
    if (st != AGS_OK) return fail(st);
    unsigned char* sp = nullptr;
    st = scratch_address(dev, &sp, why);
    if (st != AGS_OK) return fail(st);
    unsigned char* ws = sp + lay_bytes;
    hipStream_t s = static_cast<hipStream_t>(hip_stream);

    NoallocTables nt{};
    nt.layers = reinterpret_cast<const ags_layer*>(sp);
    nt.n_layers = cfg->n_layers;
    nt.ldev = reinterpret_cast<LayerDev*>(ws + wl.ldev);
    nt.tiles = reinterpret_cast<Tile*>(ws + wl.tiles);
    nt.chunks = reinterpret_cast<ags::FinChunk*>(ws + wl.chunks);
    nt.state = reinterpret_cast<DevState*>(ws + wl.state);
    nt.gradscale = reinterpret_cast<double*>(ws + wl.gradscale);
    nt.g_prev_l = reinterpret_cast<double*>(ws + wl.g_prev_l);
    nt.last_sens_l = reinterpret_cast<int32_t*>(ws + wl.last_sens_l);
    nt.chunk_count = reinterpret_cast<unsigned*>(ws + wl.chunk_count);
    nt.counters = reinterpret_cast<unsigned*>(ws + wl.counters);

    const ags_config& c = *cfg;
    ags::StepArgs sa{};
    sa.grads = d_grads;
    sa.stride = replica_stride;
    sa.w = const_cast<float*>(d_w);  // read only: the statistics kernel never writes w
    sa.m = nullptr;
    sa.gbar = nullptr;
    sa.tiles = nt.tiles;
    sa.partials = reinterpret_cast<Partial*>(ws + wl.partials);
    sa.layers = nt.ldev;
    sa.n_layers = c.n_layers;
    sa.K = c.K;
    sa.invK = (float)(1.0 / (double)c.K);
    sa.small_replica = c.small_replica;
    sa.mode = c.mode;
    sa.commit = 0;
    sa.refresh_every = c.refresh_every;
    sa.momentum = (float)c.momentum;
    sa.delta = c.delta;
    sa.eps = c.eps;
    sa.s_max = c.s_max;
    sa.trust_coef = c.trust_coef;
    sa.static_scale = c.static_scale;
    sa.weight_decay = c.weight_decay;
    sa.gradscale = nt.gradscale;
    sa.state = nt.state;
    sa.g_prev_l = nt.g_prev_l;
    sa.last_sens_l = nt.last_sens_l;
    sa.delta_scope = c.delta_scope;
    sa.coef = reinterpret_cast<float2*>(ws + wl.coef);
    sa.corr = reinterpret_cast<float2*>(ws + wl.corr);
    sa.corr_flag = reinterpret_cast<int*>(nt.counters + 1);
    sa.updated = 0;
    sa.xcd_map = n_tiles >= ags::kXcdMapMinTiles ? 1 : 0;
    sa.done_count = nt.counters;
    sa.chunks = nt.chunks;
    sa.chunk_sums = reinterpret_cast<ags::ChunkSum*>(ws + wl.chunk_sums);
    sa.layer_chunk_count = nt.chunk_count;
    sa.lstats = reinterpret_cast<ags_layer_stats*>(ws + wl.lstats);
    sa.gstats = reinterpret_cast<ags_global_stats*>(ws + wl.gstats);
    sa.ew = 0;
    sa.ew_buf = nullptr;
    sa.n_flat = c.n_flat;
    sa.ew_partials = nullptr;
    sa.w_norm_in = nullptr;

    e = hipMemcpyAsync(sp, c.layers, (size_t)c.n_layers * sizeof(ags_layer), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(noalloc_layers_kernel, dim3(1), dim3(256), 0, s, nt);
        e = hipGetLastError();
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(noalloc_tiles_kernel, dim3(c.n_layers), dim3(256), 0, s, nt);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = ags::launch_step(sa, c.grad_dtype, (int)n_tiles, false, s, ags::KernelEvents{});
    if (e == hipSuccess) e = ags::launch_finalize(sa, (int)n_chunks, s, ags::KernelEvents{});
    if (e == hipSuccess)
        e = hipMemcpyAsync(out_layers, ws + wl.lstats, (size_t)c.n_layers * sizeof(ags_layer_stats),
                           hipMemcpyDeviceToHost, s);
    if (e == hipSuccess)
        e = hipMemcpyAsync(out_global, ws + wl.gstats, sizeof(ags_global_stats), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        why = std::string("ags_stats_noalloc: ") + hipGetErrorString(e);
        (void)hipGetLastError();
        return fail(AGS_E_DEVICE);
    }
    return AGS_OK;
}
