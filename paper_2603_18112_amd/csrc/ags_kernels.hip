// gfx950 kernels of one AGS step.
//
// step_kernel      one block per tile: K replica loads -> replica mean and
//                  spread and the tile's partial statistics, and (AGS / SGD
//                  steps) the momentum-SGD update with the coefficients
//                  predicted before the step.
// finalize_kernel  one block per chunk of a layer's tiles: the layer's
//                  statistics from its tile partials in fp64; the block that
//                  finishes the last layer runs the global decision (Eq. (5),
//                  Algorithm 1), the coefficients and the gradscale refresh.
// correct_kernel   AGS steps whose sensitive bit was mispredicted: adds
//                  (a_true - a_predicted) * gbar to m and -eta times it to w;
//                  exits at once otherwise.
// update_kernel    LARS steps: the trust ratio needs the layer norms first,
//                  so the update is a second pass with the final coefficients.
//
// The streaming kernels are HBM-bound (well under one flop per byte) and use
// no matrix cores.  Element mapping: a block works through its tile in
// rounds of 2048 elements; in a round, wave w owns elements [512w, 512w+512)
// and each lane owns 8 of them.  With fp32 gradients lane l owns two halves
// of 4 elements, [4l, 4l+4) and [256+4l, 256+4l+4), so every 16-byte load
// or store instruction of a wave covers 1 KiB of consecutive elements; with
// bf16 gradients lane l owns [8l, 8l+8), one 16-byte load per replica row.
// Reductions
// run in a fixed order (per thread, wave butterfly, the four waves in index
// order, then per layer in fp64 over tiles in index order); the one atomic
// only counts finished layers, so a step is bitwise reproducible.
#include <math.h>

#include <type_traits>

#include "ags_internal.h"

namespace ags {
namespace {

// Every byte of a step is touched once, so the replica rows are read with
// non-temporal (streaming) loads: measured on MI355X, this cuts the step
// kernel's time by about a quarter against ordinary loads (w and m keep
// ordinary loads and stores, which measured faster than streaming ones).
#ifndef AGS_NT_LOADS
#define AGS_NT_LOADS 1
#endif
// Replicas whose loads are issued together before any is used (a batch):
// 8 bf16 replicas or 2 fp32 replicas per batch measured best.
#ifndef AGS_BATCH_BF16
#define AGS_BATCH_BF16 8
#endif
#ifndef AGS_BATCH_F32
#define AGS_BATCH_F32 2
#endif
// Batches of the element-scale kernels, which hold more per-element state
// (the fp64 replica sums, the scales): with 8 bf16 replicas per batch the
// refresh kernel needs 319 VGPRs (one wave per SIMD), with 4 it needs 121.
// fp32: 4 replicas per batch keep more reads in flight than 2 (step kernel,
// K = 8: ResNet-18 96.4 -> 95.0 us, the ResNet-50 layout 213.6 -> 210.5,
// VGG-16 1357 -> 1348; 8 measured the same as 4).
#ifndef AGS_BATCH_BF16_EW
#define AGS_BATCH_BF16_EW 4
#endif
#ifndef AGS_BATCH_F32_EW
#define AGS_BATCH_F32_EW 4
#endif

// bf16 gradients: a lane's two halves are adjacent (8 consecutive elements,
// one 16-byte load per replica); fp32 gradients: 256 elements apart (every
// 16-byte load instruction of a wave covers 1 KiB of consecutive elements).
// Both measured best for their dtype on MI355X.
#ifndef AGS_BF16_CONTIG
#define AGS_BF16_CONTIG 1
#endif

constexpr int kHalf = 4;                    // elements per half group
constexpr int kWaveSpan = 512;              // elements per wave per round
constexpr int kRound = kTileBlock * kVec;   // elements per tile-kernel block per round
static_assert(kRound == (kTileBlock / 64) * kWaveSpan, "round layout");

// Distance between a lane's two halves for gradients of type GT.
template <typename GT> struct Map {
    static constexpr int HS = (sizeof(GT) == 2 && AGS_BF16_CONTIG) ? kHalf : kWaveSpan / 2;
};

// ---------------------------------------------------------------- loads ---

typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 stream_load(const uint2* p) {
#if AGS_NT_LOADS
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
    return make_uint2(v.x, v.y);
#else
    return *p;
#endif
}

__device__ __forceinline__ uint4 stream_load(const uint4* p) {
#if AGS_NT_LOADS
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
#else
    return *p;
#endif
}

__device__ __forceinline__ float4 stream_load(const float4* p) {
#if AGS_NT_LOADS
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                       __uint_as_float(v.w));
#else
    return *p;
#endif
}

// bf16 -> fp32 is exact: a bf16 value is the upper half of an fp32.
__device__ __forceinline__ float bf16_lo(unsigned int x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(unsigned int x) { return __uint_as_float(x & 0xffff0000u); }

__device__ __forceinline__ float load1(const float* __restrict__ p) { return *p; }
__device__ __forceinline__ float load1(const uint16_t* __restrict__ p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
}

// A group of a lane: halves [p, p+4) and [p+HS, p+HS+4).  FULL groups are
// two 16-byte (fp32) loads; the ragged end of a layer takes element loads
// for the first n0 and n1 elements of the halves, the rest being 0 (which
// adds nothing to any sum).
template <bool FULL, int HS>
__device__ __forceinline__ void load_f32(const float* __restrict__ p, int n0, int n1,
                                         float (&v)[kVec]) {
    if (FULL) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 b = *reinterpret_cast<const float4*>(p + HS);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
#pragma unroll
        for (int e = 0; e < kHalf; ++e) {
            v[e] = (e < n0) ? p[e] : 0.0f;
            v[kHalf + e] = (e < n1) ? p[HS + e] : 0.0f;
        }
    }
}

template <bool FULL, int HS>
__device__ __forceinline__ void store_f32(float* __restrict__ p, int n0, int n1,
                                          const float (&v)[kVec]) {
    if (FULL) {
        *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
        *reinterpret_cast<float4*>(p + HS) = make_float4(v[4], v[5], v[6], v[7]);
    } else {
#pragma unroll
        for (int e = 0; e < kHalf; ++e) {
            if (e < n0) p[e] = v[e];
            if (e < n1) p[HS + e] = v[kHalf + e];
        }
    }
}

// Non-temporal variants of load_f32 / store_f32 (the ragged end keeps
// element accesses).
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <bool FULL, int HS>
__device__ __forceinline__ void load_f32_nt(const float* __restrict__ p, int n0, int n1,
                                            float (&v)[kVec]) {
    if (FULL) {
        const float4 a = stream_load(reinterpret_cast<const float4*>(p));
        const float4 b = stream_load(reinterpret_cast<const float4*>(p + HS));
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
        load_f32<false, HS>(p, n0, n1, v);
    }
}

template <bool FULL, int HS>
__device__ __forceinline__ void store_f32_nt(float* __restrict__ p, int n0, int n1,
                                             const float (&v)[kVec]) {
    if (FULL) {
        const f32x4_t a = {v[0], v[1], v[2], v[3]};
        const f32x4_t b = {v[4], v[5], v[6], v[7]};
        __builtin_nontemporal_store(a, reinterpret_cast<f32x4_t*>(p));
        __builtin_nontemporal_store(b, reinterpret_cast<f32x4_t*>(p + HS));
    } else {
        store_f32<false, HS>(p, n0, n1, v);
    }
}

template <bool NT, bool FULL, int HS>
__device__ __forceinline__ void load_f32_as(const float* __restrict__ p, int n0, int n1,
                                            float (&v)[kVec]) {
    if (NT) load_f32_nt<FULL, HS>(p, n0, n1, v);
    else load_f32<FULL, HS>(p, n0, n1, v);
}

template <bool NT, bool FULL, int HS>
__device__ __forceinline__ void store_f32_as(float* __restrict__ p, int n0, int n1,
                                             const float (&v)[kVec]) {
    if (NT) store_f32_nt<FULL, HS>(p, n0, n1, v);
    else store_f32<FULL, HS>(p, n0, n1, v);
}

template <typename GT, int HS>
__device__ __forceinline__ void load_tail(const GT* __restrict__ p, int n0, int n1,
                                          float (&v)[kVec]) {
#pragma unroll
    for (int e = 0; e < kHalf; ++e) {
        v[e] = (e < n0) ? load1(p + e) : 0.0f;
        v[kHalf + e] = (e < n1) ? load1(p + HS + e) : 0.0f;
    }
}

// A full group of replica values as loaded, before widening to fp32: one
// 16-byte vector (bf16, adjacent halves) or two 8-byte vectors (bf16, split
// halves), two 16-byte vectors for fp32.
template <typename GT> struct RawGroup;
template <> struct RawGroup<uint16_t> {
    static constexpr int kBatch = AGS_BATCH_BF16;
    static constexpr int kBatchEw = AGS_BATCH_BF16_EW;
    static constexpr int HS = Map<uint16_t>::HS;
    uint2 a, b;
    __device__ __forceinline__ void load(const uint16_t* __restrict__ p) {
        if constexpr (HS == kHalf) {
            const uint4 v = stream_load(reinterpret_cast<const uint4*>(p));
            a = make_uint2(v.x, v.y);
            b = make_uint2(v.z, v.w);
        } else {
            a = stream_load(reinterpret_cast<const uint2*>(p));
            b = stream_load(reinterpret_cast<const uint2*>(p + HS));
        }
    }
    __device__ __forceinline__ void widen(float (&o)[kVec]) const {
        o[0] = bf16_lo(a.x); o[1] = bf16_hi(a.x); o[2] = bf16_lo(a.y); o[3] = bf16_hi(a.y);
        o[4] = bf16_lo(b.x); o[5] = bf16_hi(b.x); o[6] = bf16_lo(b.y); o[7] = bf16_hi(b.y);
    }
};
template <> struct RawGroup<float> {
    static constexpr int kBatch = AGS_BATCH_F32;
    static constexpr int kBatchEw = AGS_BATCH_F32_EW;
    static constexpr int HS = Map<float>::HS;
    float4 a, b;
    __device__ __forceinline__ void load(const float* __restrict__ p) {
        a = stream_load(reinterpret_cast<const float4*>(p));
        b = stream_load(reinterpret_cast<const float4*>(p + HS));
    }
    __device__ __forceinline__ void widen(float (&o)[kVec]) const {
        o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
        o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
    }
};

// ------------------------------------------------------ replica moments ---
//
// Replica mean and spread of one group, with replica 0 as the shift: for
// k >= 1, d_k = g_k - g_0, s1 = sum d_k, s2 = sum d_k^2; then
//   gbar = g_0 + s1 / K   and   sum_k (g_k - gbar)^2 = s2 - s1^2 / K.
// Identical replicas give d_k = 0, hence gbar = g_0 and a spread of exactly
// 0; the spread is formed from differences, never as E[g^2] - E[g]^2.
// Every kernel forms gbar with this code, so all of them see the same bits.
//
// RMODE selects the small-batch gradient: 0 = replica 0, 1 = mean over
// replicas (no per-replica value needed), 2 = replica r (runtime).
// EX: also return q = sum_k g_k in fp64 (exact for bf16 replicas and, in
// practice, for fp32 ones), from which an element scale's denominator
// gbar + eps is formed without the cancellation of the fp32 sums.

#ifndef AGS_PIPELINE
#define AGS_PIPELINE 1
#endif
#ifndef AGS_STATS_SPLIT
#define AGS_STATS_SPLIT 1
#endif
#ifndef AGS_STATS_WBARRIER
#define AGS_STATS_WBARRIER 1
#endif
// SPLIT: keep each later batch in its packed form until the batch before
// it is summed (a scheduling barrier after the batch's loads).  Without it
// the statistics-only step kernel widened all K = 16 bf16 replicas as they
// arrived and took 202 VGPRs (two waves per SIMD); the sums are the same.
template <typename GT, int KT, int RMODE, bool FULL, bool EX = false,
          int BATCH = RawGroup<GT>::kBatch, bool SPLIT = false>
__device__ __forceinline__ void moments(const GT* __restrict__ g, int64_t stride, int64_t idx,
                                        int n0, int n1, int K, int r, float invK,
                                        float (&gbar)[kVec], float (&dev)[kVec],
                                        float (&gr)[kVec], double (&q)[kVec]) {
    float g0[kVec], s1[kVec], s2[kVec];
    if (FULL) {
        RawGroup<GT> r0;
        r0.load(g + idx);
        r0.widen(g0);
    } else {
        load_tail<GT, Map<GT>::HS>(g + idx, n0, n1, g0);
    }
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        s1[e] = 0.0f;
        s2[e] = 0.0f;
        gr[e] = g0[e];
        if (EX) q[e] = (double)g0[e];
    }
    auto acc = [&](int k, const float (&x)[kVec]) {
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
            const float d = x[e] - g0[e];
            s1[e] += d;
            s2[e] = fmaf(d, d, s2[e]);
            if (RMODE == 2) gr[e] = (k == r) ? x[e] : gr[e];
            if (EX) q[e] += (double)x[e];
        }
    };
    // bf16 replicas, K >= 16, no fp64 sums: two batches in registers (of 4
    // replicas for K = 16, of 8 above), the next batch's loads in flight
    // while the current one is summed, in the same replica order (so the
    // same bits).  Measured on MI355X against one batch of 8 at a time:
    // ResNet-50 K = 16 step 192.4 / 216.3 -> 192.0 / 213.0 us warm / cold,
    // K = 32 343.7 -> 339.0, K = 64 637.4 -> 631.6, LARS K = 64 678.5 ->
    // 671.5 us.
    constexpr int PB = (sizeof(GT) == 2 && !EX && AGS_PIPELINE) ? (KT >= 32 ? 8 : 4) : 0;
    if constexpr (KT >= 16 && FULL && PB > 0) {
        constexpr int KB = PB;
        static_assert(KT % (2 * KB) == 0, "K must be a multiple of two batches");
        RawGroup<GT> a[KB], b[KB];
#pragma unroll
        for (int j = 1; j < KB; ++j) a[j].load(g + (int64_t)j * stride + idx);
#pragma unroll
        for (int j = 0; j < KB; ++j) b[j].load(g + (int64_t)(KB + j) * stride + idx);
#pragma unroll
        for (int j = 1; j < KB; ++j) {
            float v[kVec];
            a[j].widen(v);
            acc(j, v);
        }
#pragma unroll 1
        for (int kb = KB; kb < KT; kb += 2 * KB) {
            // b holds replicas [kb, kb + KB); a takes the next batch, if any
            const bool more = kb + KB < KT;
            if (more) {
#pragma unroll
                for (int j = 0; j < KB; ++j) a[j].load(g + (int64_t)(kb + KB + j) * stride + idx);
            }
#pragma unroll
            for (int j = 0; j < KB; ++j) {
                float v[kVec];
                b[j].widen(v);
                acc(kb + j, v);
            }
            if (!more) break;
            if (kb + 2 * KB < KT) {
#pragma unroll
                for (int j = 0; j < KB; ++j) b[j].load(g + (int64_t)(kb + 2 * KB + j) * stride + idx);
            }
#pragma unroll
            for (int j = 0; j < KB; ++j) {
                float v[kVec];
                a[j].widen(v);
                acc(kb + KB + j, v);
            }
        }
    } else if constexpr (KT > 0 && FULL) {
        // Every load of a batch is issued before any of its values is used.
        // The first batch holds replicas 1..KB-1 (replica 0 is the shift);
        // later batches run as a loop, one batch in registers at a time.
        constexpr int KB = KT < BATCH ? KT : BATCH;
        static_assert(KT % KB == 0, "K must be a multiple of the batch");
        {
            RawGroup<GT> x[KB];
#pragma unroll
            for (int j = 1; j < KB; ++j) x[j].load(g + (int64_t)j * stride + idx);
#pragma unroll
            for (int j = 1; j < KB; ++j) {
                float v[kVec];
                x[j].widen(v);
                acc(j, v);
            }
        }
#pragma unroll 1
        for (int kb = KB; kb < KT; kb += KB) {
            RawGroup<GT> x[KB];
#pragma unroll
            for (int j = 0; j < KB; ++j) x[j].load(g + (int64_t)(kb + j) * stride + idx);
            if constexpr (SPLIT) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int j = 0; j < KB; ++j) {
                float v[kVec];
                x[j].widen(v);
                acc(kb + j, v);
            }
        }
    } else if constexpr (KT > 0) {
        // The ragged end of a layer (one group per layer at most): one
        // replica at a time, with the full groups' fp32 sums.  A kernel's
        // register allocation is the largest any of its paths needs, so
        // this rare path is kept smaller than the full groups' batches
        // (it had taken the runtime-K loop's fp64 totals, which raised
        // e.g. the fp32 K = 8 step kernel from 78 to 114 VGPRs).
#pragma unroll 1
        for (int k = 1; k < KT; ++k) {
            float x[kVec];
            load_tail<GT, Map<GT>::HS>(g + (int64_t)k * stride + idx, n0, n1, x);
            acc(k, x);
        }
    } else {
        // Runtime K (full groups and the ragged end of a layer).  The fp32
        // sums of every four replicas are added to fp64 totals: each d_k
        // carries replica 0's own deviation, so one fp32 running sum would
        // drift by k times it and gather a rounding error growing like K
        // (about 1e-5 of the mean at K = 1024); with fp64 totals the error
        // stays that of four terms.  Mean and spread are then formed in fp64
        // and rounded once.
        double t1[kVec], t2[kVec];
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
            t1[e] = 0.0;
            t2[e] = 0.0;
        }
        auto flush = [&]() {
#pragma unroll
            for (int e = 0; e < kVec; ++e) {
                t1[e] += (double)s1[e];
                t2[e] += (double)s2[e];
                s1[e] = 0.0f;
                s2[e] = 0.0f;
            }
        };
        int k = 1;
#pragma unroll 1
        for (; k + 3 < K; k += 4) {
            float x[4][kVec];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (FULL) {
                    RawGroup<GT> q;
                    q.load(g + (int64_t)(k + j) * stride + idx);
                    q.widen(x[j]);
                } else {
                    load_tail<GT, Map<GT>::HS>(g + (int64_t)(k + j) * stride + idx, n0, n1, x[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) acc(k + j, x[j]);
            flush();
        }
#pragma unroll 1
        for (; k < K; ++k) {
            float x[kVec];
            if (FULL) {
                RawGroup<GT> q;
                q.load(g + (int64_t)k * stride + idx);
                q.widen(x);
            } else {
                load_tail<GT, Map<GT>::HS>(g + (int64_t)k * stride + idx, n0, n1, x);
            }
            acc(k, x);
        }
        flush();
        const double dK = (double)K;
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
            gbar[e] = (float)((double)g0[e] + t1[e] / dK);
            dev[e] = (float)fmax(t2[e] - t1[e] * (t1[e] / dK), 0.0);
        }
        return;
    }
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        gbar[e] = fmaf(s1[e], invK, g0[e]);
        const float t = s1[e] * invK;
        dev[e] = fmaxf(fmaf(-t, s1[e], s2[e]), 0.0f);
    }
}

// The groups of this thread in a tile of `count` elements starting at
// `begin` (halves HS apart): calls f(idx, n0, n1, full) for every group that
// holds data.
template <int HS, typename F>
__device__ __forceinline__ void for_each_group(int64_t begin, int count, F&& f) {
    const int lane_pos = HS == kHalf ? (int)(threadIdx.x & 63) * kVec : (int)(threadIdx.x & 63) * kHalf;
    const int pos = (int)(threadIdx.x >> 6) * kWaveSpan + lane_pos;
#pragma unroll 1
    for (int r0 = 0; r0 < count; r0 += kRound) {
        const int off = r0 + pos;
        const int n0 = min(max(count - off, 0), kHalf);
        const int n1 = min(max(count - off - HS, 0), kHalf);
        if (n1 == kHalf) f(begin + off, kHalf, kHalf, std::true_type{});
        else if (n0 > 0) f(begin + off, n0, n1, std::false_type{});
    }
}

// -------------------------------------------------------- reductions ---

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ __forceinline__ int wave_sum(int v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// Sum of v over the block, in a fixed order; every thread gets the result.
template <typename T>
__device__ __forceinline__ T block_sum(T v, T* sh /* [kBlock / 64] */) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) sh[wid] = v;
    __syncthreads();
    return (sh[0] + sh[1]) + (sh[2] + sh[3]);
}

struct Sum4 {
    double w, g, d, s;
    double x;  // refreshed element scales (elementwise AGS), else 0
};

// Componentwise block sum with one pair of barriers.
__device__ __forceinline__ Sum4 block_sum4(Sum4 v, Sum4* sh /* [kBlock / 64] */) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    v.w = wave_sum(v.w);
    v.g = wave_sum(v.g);
    v.d = wave_sum(v.d);
    v.s = wave_sum(v.s);
    v.x = wave_sum(v.x);
    __syncthreads();
    if (lane == 0) sh[wid] = v;
    __syncthreads();
    Sum4 r;
    r.w = (sh[0].w + sh[1].w) + (sh[2].w + sh[3].w);
    r.g = (sh[0].g + sh[1].g) + (sh[2].g + sh[3].g);
    r.d = (sh[0].d + sh[1].d) + (sh[2].d + sh[3].d);
    r.s = (sh[0].s + sh[1].s) + (sh[2].s + sh[3].s);
    r.x = (sh[0].x + sh[1].x) + (sh[2].x + sh[3].x);
    return r;
}

// The step's sensitivity is known before the step when Delta is infinite
// by definition: a first step, or no positive finite previous norm.
__device__ __forceinline__ bool surely_sensitive(double g_prev, long long step) {
    return step == 0 || !(g_prev > 0.0) || !isfinite(g_prev);
}

// ------------------------------------------------------- finalize -------

// Sum of the tile partials [tb, te) in fp64, in a fixed order; every
// thread of the block gets the result.
__device__ Sum4 sum_tiles(const StepArgs& a, int tb, int te, Sum4* sh, bool ew_refresh) {
    // Four independent accumulators per thread (tiles i, i + 256, i + 512,
    // i + 768, then the next 1024), combined in a fixed order, so that four
    // loads are in flight per thread.
    constexpr int U = 4;
    const bool ex = ew_refresh;
    Sum4 acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) acc[u] = {0.0, 0.0, 0.0, 0.0, 0.0};
    int i = tb + (int)threadIdx.x;
    for (; i + (U - 1) * kBlock < te; i += U * kBlock) {
        Partial p[U];
        float x[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            p[u] = a.partials[i + u * kBlock];
            x[u] = ex ? a.ew_partials[i + u * kBlock] : 0.0f;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            acc[u].w += (double)p[u].w;
            acc[u].g += (double)p[u].g;
            acc[u].d += (double)p[u].d;
            acc[u].s += (double)p[u].s;
            acc[u].x += (double)x[u];
        }
    }
#pragma unroll
    for (int u = 0; u < U - 1; ++u) {
        const int j = i + u * kBlock;
        if (j < te) {
            const Partial p = a.partials[j];
            acc[u].w += (double)p.w;
            acc[u].g += (double)p.g;
            acc[u].d += (double)p.d;
            acc[u].s += (double)p.s;
            if (ex) acc[u].x += (double)a.ew_partials[j];
        }
    }
    Sum4 v;
    v.w = (acc[0].w + acc[1].w) + (acc[2].w + acc[3].w);
    v.g = (acc[0].g + acc[1].g) + (acc[2].g + acc[3].g);
    v.d = (acc[0].d + acc[1].d) + (acc[2].d + acc[3].d);
    v.s = (acc[0].s + acc[1].s) + (acc[2].s + acc[3].s);
    v.x = (acc[0].x + acc[1].x) + (acc[2].x + acc[3].x);
    return block_sum4(v, sh);
}

__device__ __forceinline__ void write_layer(const StepArgs& a, int l, const Sum4& v,
                                            bool ew_refresh) {
    ags_layer_stats& o = a.lstats[l];
    o.w_sq = v.w;
    o.g_sq = v.g;
    o.var = v.d / (double)a.K;
    o.gsmall_sq = v.s;
    // Mean of the refreshed element scales, taken over by finalize_global.
    if (ew_refresh) o.gradscale = v.x / (double)a.layers[l].numel;
}

// The global decision and every layer's coefficients (one block, after all
// layers are final).  Delta = |G - G_prev| / G_prev, infinite on a first
// step, when G_prev <= 0 or when a value is not finite; sensitive =
// !(Delta < delta); Delta_l likewise from each layer's G_l, and with the
// per-layer scope sensitive_l = !(Delta_l < delta) replaces the global bit
// for that layer.  AGS: a_l = gradscale_l on scaled layers of a
// non-sensitive step, else 1; STATIC: a_l = s likewise (U(s), Eq. (8));
// LARS: a_l = tau ||w|| / (||g|| + lambda ||w||);
// b_l = lambda_l (AGS, SGD) or a_l lambda_l (LARS).  When the refresh is due,
// gradscale_l = min(sqrt(S_l) / (sqrt(G_l) + eps), s_max) (1 if a norm is 0)
// for the steps that follow.  updated: the step kernel has already applied
// the predicted coefficients, so record their difference for the correction.
// With element scales gradscale_l is the layer mean of the element scales
// (so a_l above is the mean coefficient applied), the step kernel has
// refreshed the elements, and a mispredicted scaled layer is corrected per
// element by c_j = 1 - gradscale_j (x = 1, y = -1) when it was applied
// scaled, by c_j = gradscale_j - 1 when it was applied unscaled.  The bits
// that decided the step are kept in the state: the next step predicts
// from them.
// Inputs of the global part that no block of this launch writes before the
// last block reads them, loaded by every block at its start so that the
// last one has them at hand: the state (thread 0) and, for layer
// threadIdx.x, its flags, gradscale and G_l,prev.
struct Prefetch {
    double g_prev, gs, gpl;
    long long step;
    uint32_t flags;
    int ew_cur;
    int last_sens, last_sens_l;  // the last committed step's bits
    bool ew_refresh;  // a committed elementwise step whose refresh is due
};

__device__ __forceinline__ Prefetch prefetch_global(const StepArgs& a) {
    Prefetch p{0.0, 0.0, 0.0, 0, 0u, 0, 0, 0, false};
    p.g_prev = a.state->g_prev;
    p.step = a.state->step;
    p.ew_cur = a.state->ew_cur;
    p.last_sens = a.state->last_sens;
    p.ew_refresh = a.ew && a.commit && a.refresh_every > 0 &&
                   ((p.step + 1) % a.refresh_every) == 0;
    const int l = threadIdx.x;
    if (l < a.n_layers) {
        p.flags = a.layers[l].flags;
        p.gs = a.gradscale[l];
        p.gpl = a.g_prev_l[l];
        p.last_sens_l = a.last_sens_l[l];
    }
    return p;
}

__device__ void finalize_global(const StepArgs& a, bool updated, Sum4* sh, int* shi,
                                const Prefetch& pf) {
    const bool ew_refresh = pf.ew_refresh;
    __shared__ int sh_sens, sh_pred, sh_inf;
    __shared__ long long sh_t;
    Sum4 v = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (int l = threadIdx.x; l < a.n_layers; l += kBlock) {
        const ags_layer_stats& o = a.lstats[l];
        v.g += o.g_sq;
        v.w += (isfinite(o.w_sq) && isfinite(o.g_sq) && isfinite(o.var) && isfinite(o.gsmall_sq)) ? 0.0 : 1.0;
    }
    v = block_sum4(v, sh);
    const double G = v.g;
    int nf = v.w != 0.0;
    if (threadIdx.x == 0) {
        const double Gp = pf.g_prev;
        const long long step = pf.step;
        const long long t = step + 1;
        double delta;
        if (surely_sensitive(Gp, step) || !isfinite(G))
            delta = INFINITY;
        else
            delta = fabs((G - Gp) / Gp);
        const int sens = !(delta < a.delta);
        if (!isfinite(G)) nf = 1;
        ags_global_stats gs;
        gs.step = a.commit ? t : step;
        gs.g_sq = G;
        gs.g_sq_prev = (t == 1) ? 0.0 : Gp;
        gs.delta = delta;
        gs.sensitive = sens;
        gs.nonfinite = nf;
        *a.gstats = gs;
        if (a.commit) {
            a.state->g_prev = G;
            a.state->step = t;
            // A step sensitive by definition (Delta infinite: the first
            // one) says nothing about the next: it predicts not sensitive.
            a.state->last_sens = sens && !surely_sensitive(Gp, step);
            if (ew_refresh) a.state->ew_cur = 1 - pf.ew_cur;  // the refreshed buffer
        }
        sh_sens = sens;
        sh_inf = surely_sensitive(Gp, step);
        sh_pred = sh_inf || pf.last_sens != 0;
        sh_t = t;
    }
    __syncthreads();
    const int sens_g = sh_sens, pred_g = sh_pred;
    const long long t = sh_t;
    const bool refresh = a.commit && a.mode == AGS_MODE_AGS && a.refresh_every > 0 &&
                         (t % a.refresh_every) == 0;
    const double smax = a.s_max > 0.0 ? a.s_max : sqrt((double)a.K);
    int need = 0;
    for (int l = threadIdx.x; l < a.n_layers; l += kBlock) {
        ags_layer_stats& o = a.lstats[l];
        const bool first = l == (int)threadIdx.x;
        const uint32_t f = first ? pf.flags : a.layers[l].flags;
        const bool scaled = (f & AGS_LAYER_SCALE) != 0;
        const double lam = (f & AGS_LAYER_DECAY) ? a.weight_decay : 0.0;
        const double gs_old = first ? pf.gs : a.gradscale[l];
        // The layer's own variability Delta_l (always reported); with the
        // per-layer scope it decides the layer, and the step kernel's
        // prediction was made from the layer's own G_l,prev and last bit.
        const double Gpl = first ? pf.gpl : a.g_prev_l[l];
        const bool inf_l = surely_sensitive(Gpl, t - 1);
        const double dl = (inf_l || !isfinite(o.g_sq)) ? INFINITY : fabs((o.g_sq - Gpl) / Gpl);
        const int sens = a.delta_scope ? !(dl < a.delta) : sens_g;
        const bool last_l = (first ? pf.last_sens_l : a.last_sens_l[l]) != 0;
        const int pred = a.delta_scope ? (inf_l || last_l) : pred_g;
        o.delta = dl;
        o.sensitive = sens;
        o.reserved = 0;
        if (a.commit) {
            a.g_prev_l[l] = o.g_sq;
            a.last_sens_l[l] = sens && !(a.delta_scope ? inf_l : (bool)sh_inf);
        }
        double ca = 1.0, cb = lam;
        if (a.mode == AGS_MODE_AGS) {
            ca = (scaled && !sens) ? gs_old : 1.0;
        } else if (a.mode == AGS_MODE_STATIC) {
            ca = (scaled && !sens) ? a.static_scale : 1.0;
        } else if (a.mode == AGS_MODE_LARS) {
            if (scaled) {
                const double wn = sqrt(o.w_sq), gn = sqrt(o.g_sq);
                ca = (wn > 0.0 && gn > 0.0) ? a.trust_coef * wn / (gn + lam * wn) : 1.0;
            }
            cb = ca * lam;
        }
        o.noise_ratio = (o.g_sq > 0.0) ? o.var / o.g_sq : ((o.var > 0.0) ? INFINITY : 0.0);
        o.coef_a = ca;
        o.coef_b = cb;
        a.coef[l] = make_float2((float)ca, (float)cb);
        if (updated) {
            float2 c = make_float2(0.0f, 0.0f);
            if (a.ew) {
                // c_j = x + y gradscale_j: applied scaled, true unscaled, or
                // the other way round
                if (scaled && !pred && sens) c = make_float2(1.0f, -1.0f);
                else if (scaled && pred && !sens) c = make_float2(-1.0f, 1.0f);
            } else {
                double ap = 1.0;
                if (scaled && !pred) {
                    if (a.mode == AGS_MODE_AGS) ap = gs_old;
                    else if (a.mode == AGS_MODE_STATIC) ap = a.static_scale;
                }
                c.x = (float)ca - (float)ap;
            }
            a.corr[l] = c;
            need |= (c.x != 0.0f || c.y != 0.0f);
        }
        double gsc = gs_old;
        if (a.ew) {
            if (ew_refresh) {
                gsc = o.gradscale;
                a.gradscale[l] = gsc;
            }
        } else if (refresh && scaled) {
            const double S = o.gsmall_sq, Gl = o.g_sq;
            if (S > 0.0 && Gl > 0.0) {
                gsc = sqrt(S) / (sqrt(Gl) + a.eps);
                if (gsc > smax) gsc = smax;
            } else {
                gsc = 1.0;
            }
            a.gradscale[l] = gsc;
        }
        o.gradscale = gsc;
    }
    need = block_sum(need, shi);
    if (threadIdx.x == 0) *a.corr_flag = (updated && need) ? 1 : 0;
}

// ------------------------------------------------- the fused step kernel ---

// Element scale of elementwise AGS (Algorithm 1 read per element):
// |g_small / (gbar + eps)| clipped at smax, 1 for a 0/0 ratio.  q is the
// fp64 replica sum of the element: the denominator q / K + eps is formed in
// fp64 and rounded once, after which the quotient is well conditioned and
// an fp32 division (two roundings in all, 1.2e-7 relative) suffices.
#ifndef AGS_EW_F64_DIV
#define AGS_EW_F64_DIV 0
#endif
__device__ __forceinline__ float element_scale(float gsmall, double q, double invK, double eps,
                                               float smax) {
#if AGS_EW_F64_DIV
    double r = fabs((double)gsmall / fma(q, invK, eps));
    if (isnan(r)) r = 1.0;
    if (r > (double)smax) r = smax;
    return (float)r;
#else
    const float den = (float)fma(q, invK, eps);
    float r = fabsf(gsmall / den);
    if (isnan(r)) r = 1.0f;
    return r > smax ? smax : r;
#endif
}

// One group of a tile.  EW: element scales from gs_old applied (use_gs:
// the layer is scaled and the step is predicted not sensitive) and, when
// refresh, the refreshed scales written to gs_new with their sum over the
// group's elements in sx.  Without EW, per-layer coefficients.
// EW: 0 = one scale per layer; 1 = element scales, ordinary accesses; 2 =
// element scales with non-temporal scale loads and scale, w and m stores
// (the host's choice for working sets the Infinity Cache cannot keep).
// WNC (statistics only): W of the tile comes from the last LARS update
// pass, so w is not read.  GB (statistics only): store the replica mean
// for the LARS update pass.  A compile-time choice: testing the pointer at
// run time had made the K = 16 bf16 statistics kernel keep 183 VGPRs (two
// waves per SIMD) against 95 with the store unconditional.
template <typename GT, int KT, int RMODE, bool UPD, int EW, bool FULL, bool WNC = false,
          bool GB = false>
__device__ __forceinline__ void step_group(const StepArgs& a, const GT* __restrict__ g,
                                           int64_t idx, int n0, int n1, int K, float ca,
                                           float cb, float lr, bool use_gs, bool scaled, bool refresh,
                                           const float* __restrict__ gs_old,
                                           float* __restrict__ gs_new, float smax, float& sw,
                                           float& sg, float& sd, float& ss, float& sx) {
    constexpr int HS = Map<GT>::HS;
    constexpr bool NT = EW == 2;
    constexpr bool ELEM = EW != 0;
    static_assert(!(WNC && UPD), "the update reads w");
    static_assert(!(GB && UPD), "the fused update keeps the mean in registers");
    float wv[kVec], mv[kVec], gb[kVec], dv[kVec], gr[kVec];
    double q[kVec];
    if (!WNC) load_f32<FULL, HS>(a.w + idx, n0, n1, wv);
    if (UPD) load_f32<FULL, HS>(a.m + idx, n0, n1, mv);
    // Keep the w (and m) loads in front of the replica loads: without the
    // barrier the statistics-only variant issued them only after consuming
    // every replica, a second round trip per block.
    if (!UPD && AGS_STATS_WBARRIER) __builtin_amdgcn_sched_barrier(0);
    constexpr int kb = ELEM ? RawGroup<GT>::kBatchEw : RawGroup<GT>::kBatch;
    moments<GT, KT, RMODE, FULL, ELEM, kb, !UPD && AGS_STATS_SPLIT>(g, a.stride, idx, n0, n1, K, a.small_replica,
                                               a.invK, gb, dv, gr, q);
    float gsv[kVec];
    if (ELEM) {
        // Old scales: applied on scaled layers, carried over on the others.
        if (use_gs || (refresh && !scaled)) {
            load_f32_as<NT, FULL, HS>(gs_old + idx, n0, n1, gsv);
        } else {
#pragma unroll
            for (int e = 0; e < kVec; ++e) gsv[e] = 1.0f;
        }
    }
    if (GB) store_f32<FULL, HS>(a.gbar + idx, n0, n1, gb);
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        if (!WNC) sw = fmaf(wv[e], wv[e], sw);
        sg = fmaf(gb[e], gb[e], sg);
        sd += dv[e];
        // (1/K) sum_k g_k^2 = gbar^2 + (1/K) sum_k (g_k - gbar)^2
        if (RMODE == 1) ss += fmaf(gb[e], gb[e], dv[e] * a.invK);
        else ss = fmaf(gr[e], gr[e], ss);
    }
    if (UPD) {
        // d = a gbar + b w ; m <- mu m + d ; w <- w - eta m
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
            const float ae = (ELEM && use_gs) ? gsv[e] : ca;
            const float d = fmaf(ae, gb[e], cb * wv[e]);
            mv[e] = fmaf(a.momentum, mv[e], d);
            wv[e] = fmaf(-lr, mv[e], wv[e]);
        }
        store_f32_as<NT, FULL, HS>(a.w + idx, n0, n1, wv);
        store_f32_as<NT, FULL, HS>(a.m + idx, n0, n1, mv);
    }
    if (ELEM && refresh) {
        float sn[kVec];
        if (scaled) {
            const double invK = 1.0 / (double)K;
#pragma unroll
            for (int e = 0; e < kVec; ++e) {
                const float gs = RMODE == 1 ? sqrtf(fmaf(gb[e], gb[e], dv[e] * a.invK)) : gr[e];
                sn[e] = element_scale(gs, q[e], invK, a.eps, smax);
            }
        } else {
#pragma unroll
            for (int e = 0; e < kVec; ++e) sn[e] = gsv[e];
        }
        store_f32_as<NT, FULL, HS>(gs_new + idx, n0, n1, sn);
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
            const bool valid = FULL || (e < kHalf ? e < n0 : e - kHalf < n1);
            sx += valid ? sn[e] : 0.0f;
        }
    }
}

// Sum of the N wave totals of a block in a fixed pairwise order (for four
// waves: (v0 + v1) + (v2 + v3)).
template <int N>
__device__ __forceinline__ float tree_sum(const float* v) {
    if constexpr (N == 1) return v[0];
    else return tree_sum<N / 2>(v) + tree_sum<N - N / 2>(v + N / 2);
}

// Workgroups are dispatched round-robin over the 8 XCDs.  With xcd_map each
// XCD walks a contiguous range of tiles instead of every 8th tile (a
// bijection of block indices onto tiles).
__device__ __forceinline__ int tile_of_block(int b, int n, int xcd_map) {
    if (!xcd_map) return b;
    constexpr int nx = 8;
    const int q = n / nx, r = n % nx, x = b % nx, i = b / nx;
    return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

template <typename GT, int KT, int RMODE, bool UPD, int EW, bool WNC = false, bool GB = false>
__global__ __launch_bounds__(kTileBlock) void step_kernel(StepArgs a) {
    constexpr bool ELEM = EW != 0;
    __shared__ float red[5][kTileBlock / 64];
    const int tb = tile_of_block(blockIdx.x, gridDim.x, a.xcd_map);
    const int ti = a.reverse ? (int)gridDim.x - 1 - tb : tb;
    const Tile t = a.tiles[ti];
    const int l = t.layer;
    const GT* __restrict__ g = static_cast<const GT*>(a.grads);
    const int K = KT > 0 ? KT : a.K;

    // Coefficients predicted before the step: the unscaled ones when the
    // step is surely sensitive (Delta infinite by definition) or the last
    // committed step was sensitive, otherwise the scaled ones.
    float ca = 1.0f, cb = 0.0f, lr = 0.0f;
    bool use_gs = false, scaled = false, refresh = false;
    const float* gs_old = nullptr;
    float* gs_new = nullptr;
    if (UPD) {
        lr = a.state->lr;
        const uint32_t f = a.layers[l].flags;
        const long long step = a.state->step;
        const bool pred = a.delta_scope
                              ? surely_sensitive(a.g_prev_l[l], step) || a.last_sens_l[l] != 0
                              : surely_sensitive(a.state->g_prev, step) || a.state->last_sens != 0;
        scaled = (f & AGS_LAYER_SCALE) != 0;
        if (ELEM) {
            // The buffer in force and the refresh, from the device state.
            const int cur = a.state->ew_cur;
            gs_old = a.ew_buf + (size_t)cur * (size_t)a.n_flat;
            gs_new = a.ew_buf + (size_t)(1 - cur) * (size_t)a.n_flat;
            refresh = a.refresh_every > 0 && ((step + 1) % a.refresh_every) == 0;
        }
        if (scaled && !pred) {
            if (ELEM) use_gs = true;
            else if (a.mode == AGS_MODE_AGS) ca = (float)a.gradscale[l];
            else if (a.mode == AGS_MODE_STATIC) ca = (float)a.static_scale;
        }
        cb = (f & AGS_LAYER_DECAY) ? (float)a.weight_decay : 0.0f;
    }
    const float smax = (float)(a.s_max > 0.0 ? a.s_max : sqrt((double)K));

    float sw = 0.0f, sg = 0.0f, sd = 0.0f, ss = 0.0f, sx = 0.0f;
    for_each_group<Map<GT>::HS>(t.begin, t.count, [&](int64_t idx, int n0, int n1, auto full) {
        step_group<GT, KT, RMODE, UPD, EW, decltype(full)::value, WNC, GB>(
            a, g, idx, n0, n1, K, ca, cb, lr, use_gs, scaled, refresh, gs_old, gs_new, smax, sw, sg,
            sd, ss, sx);
    });

    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    sw = wave_sum(sw);
    sg = wave_sum(sg);
    sd = wave_sum(sd);
    ss = wave_sum(ss);
    if (ELEM && refresh) sx = wave_sum(sx);
    if (lane == 0) {
        red[0][wid] = sw;
        red[1][wid] = sg;
        red[2][wid] = sd;
        red[3][wid] = ss;
        red[4][wid] = sx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        Partial p;
        p.w = WNC ? a.w_norm_in[ti] : tree_sum<kTileBlock / 64>(red[0]);
        p.g = tree_sum<kTileBlock / 64>(red[1]);
        p.d = tree_sum<kTileBlock / 64>(red[2]);
        p.s = tree_sum<kTileBlock / 64>(red[3]);
        a.partials[ti] = p;
        if (ELEM && refresh) a.ew_partials[ti] = tree_sum<kTileBlock / 64>(red[4]);
    }
}

// Device-scope fences of the finalize's counting protocol: a block makes its
// records visible before it counts itself done (release), and the block
// that counts last sees every record before reading them (acquire).  A full
// __threadfence() would also invalidate the XCD's L2 in every block.
__device__ __forceinline__ void release_fence() { __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent"); }
__device__ __forceinline__ void acquire_fence() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }

// One block per chunk of at most kFinTilesPerChunk tiles of one layer.  A
// layer of several chunks is finished by the block that counts its last
// chunk (one device-scope atomic after a release fence), which adds the
// chunk sums in chunk order; the block that finishes the last layer runs
// the global part.
__global__ __launch_bounds__(kBlock) void finalize_kernel(StepArgs a) {
    __shared__ Sum4 sh4[kBlock / 64];
    __shared__ int shi[kBlock / 64];
    __shared__ int sh_last;
    const Prefetch pf = prefetch_global(a);
    const FinChunk c = a.chunks[blockIdx.x];
    const int l = c.layer;
    const Sum4 v = sum_tiles(a, c.tile_begin, c.tile_end, sh4, pf.ew_refresh);
    const LayerDev ld = a.layers[l];
    const int nch = ld.chunk_end - ld.chunk_begin;
    if (nch == 1) {
        if (threadIdx.x == 0) write_layer(a, l, v, pf.ew_refresh);
    } else {
        if (threadIdx.x == 0) {
            a.chunk_sums[blockIdx.x] = ChunkSum{v.w, v.g, v.d, v.s, v.x};
            release_fence();
            const unsigned prev = atomicAdd(&a.layer_chunk_count[l], 1u);
            sh_last = (prev + 1 == (unsigned)nch);
        }
        __syncthreads();
        if (!sh_last) return;
        acquire_fence();
        if (threadIdx.x == 0) {
            Sum4 t = {0.0, 0.0, 0.0, 0.0, 0.0};
            for (int q = ld.chunk_begin; q < ld.chunk_end; ++q) {
                const ChunkSum cs = a.chunk_sums[q];
                t.w += cs.w;
                t.g += cs.g;
                t.d += cs.d;
                t.s += cs.s;
                t.x += cs.x;
            }
            write_layer(a, l, t, pf.ew_refresh);
            a.layer_chunk_count[l] = 0u;  // ready for the next launch
        }
    }
    if (threadIdx.x == 0) {
        release_fence();
        const unsigned prev = atomicAdd(a.done_count, 1u);
        sh_last = (prev + 1 == (unsigned)a.n_layers);
    }
    __syncthreads();
    if (!sh_last) return;
    acquire_fence();
    finalize_global(a, a.updated != 0, sh4, shi, pf);
    if (threadIdx.x == 0) *a.done_count = 0u;  // ready for the next launch
}

// ----------------------------------------- correction and LARS update ---

// Correction of a mispredicted AGS step: m += c gbar, w -= eta c gbar with
// c = a_true - a_predicted of the layer (0 for most layers); with element
// scales (PE) c_j = x + y * gs_old_j.
template <typename GT, int KT, bool PE, bool FULL>
__device__ __forceinline__ void correct_group(const UpdateArgs& a, const GT* __restrict__ g,
                                              int64_t idx, int n0, int n1, int K, float2 c,
                                              float lr, const float* __restrict__ gs_old) {
    constexpr int HS = Map<GT>::HS;
    float gb[kVec], dv[kVec], gr[kVec], wv[kVec], mv[kVec], cv[kVec];
    double q[kVec];
    load_f32<FULL, HS>(a.w + idx, n0, n1, wv);
    load_f32<FULL, HS>(a.m + idx, n0, n1, mv);
    if (PE) {
        load_f32<FULL, HS>(gs_old + idx, n0, n1, cv);
#pragma unroll
        for (int e = 0; e < kVec; ++e) cv[e] = fmaf(c.y, cv[e], c.x);
    } else {
#pragma unroll
        for (int e = 0; e < kVec; ++e) cv[e] = c.x;
    }
    moments<GT, KT, 0, FULL>(g, a.stride, idx, n0, n1, K, 0, a.invK, gb, dv, gr, q);
    // One rounding each: m + c gbar and w - (eta c) gbar as fused
    // multiply-adds (the applied m already carries the rounding of the
    // predicted step; a second rounding of c gbar would double it).
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        mv[e] = fmaf(cv[e], gb[e], mv[e]);
        wv[e] = fmaf(-lr * cv[e], gb[e], wv[e]);
    }
    store_f32<FULL, HS>(a.w + idx, n0, n1, wv);
    store_f32<FULL, HS>(a.m + idx, n0, n1, mv);
}

template <typename GT, int KT>
__global__ __launch_bounds__(kTileBlock) void correct_kernel(UpdateArgs a) {
    if (*a.corr_flag == 0) return;
    const GT* __restrict__ g = static_cast<const GT*>(a.grads);
    const int K = KT > 0 ? KT : a.K;
    const float lr = a.state->lr;
    // Element scales in force before the step: the other buffer if the
    // step (already counted) refreshed them.
    const float* gs_old = nullptr;
    if (a.ew_buf) {
        const long long t = a.state->step;
        const bool refreshed = a.refresh_every > 0 && (t % a.refresh_every) == 0;
        const int cur = a.state->ew_cur;
        gs_old = a.ew_buf + (size_t)(refreshed ? 1 - cur : cur) * (size_t)a.n_flat;
    }
#pragma unroll 1
    for (int ti = blockIdx.x; ti < a.n_tiles; ti += gridDim.x) {
        const Tile t = a.tiles[ti];
        const float2 c = a.corr[t.layer];
        if (c.x == 0.0f && c.y == 0.0f) continue;
        if (c.y == 0.0f) {
            for_each_group<Map<GT>::HS>(t.begin, t.count, [&](int64_t idx, int n0, int n1, auto full) {
                correct_group<GT, KT, false, decltype(full)::value>(a, g, idx, n0, n1, K, c, lr, gs_old);
            });
        } else {
            for_each_group<Map<GT>::HS>(t.begin, t.count, [&](int64_t idx, int n0, int n1, auto full) {
                correct_group<GT, KT, true, decltype(full)::value>(a, g, idx, n0, n1, K, c, lr, gs_old);
            });
        }
    }
}

// LARS: d = a_l gbar + b_l w ; m <- mu m + d ; w <- w - eta m with the
// final coefficients.  gbar comes from the step kernel's buffer or, when
// re-reading the replicas costs no more than that round trip, is
// recomputed from them by the same code.
// WN: also add the squares of the new w to sw, element by element in the
// order step_group adds the squares of w (a ragged end's missing elements
// are 0 on both sides), so that the tile's sum has the bits the next
// statistics pass would get from reading w.
template <typename GT, int KT, bool RECOMP, bool FULL, bool WN>
__device__ __forceinline__ void update_group(const UpdateArgs& a, const GT* __restrict__ g,
                                             int64_t idx, int n0, int n1, int K, float ca,
                                             float cb, float lr, float& sw) {
    float gb[kVec], wv[kVec], mv[kVec];
    load_f32<FULL, Map<GT>::HS>(a.w + idx, n0, n1, wv);
    load_f32<FULL, Map<GT>::HS>(a.m + idx, n0, n1, mv);
    if (RECOMP) {
        float dv[kVec], gr[kVec];
        double q[kVec];
        moments<GT, KT, 0, FULL>(g, a.stride, idx, n0, n1, K, 0, a.invK, gb, dv, gr, q);
    } else {
        load_f32<FULL, Map<GT>::HS>(a.gbar + idx, n0, n1, gb);
    }
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        const float d = fmaf(ca, gb[e], cb * wv[e]);
        mv[e] = fmaf(a.momentum, mv[e], d);
        wv[e] = fmaf(-lr, mv[e], wv[e]);
    }
    store_f32<FULL, Map<GT>::HS>(a.w + idx, n0, n1, wv);
    store_f32<FULL, Map<GT>::HS>(a.m + idx, n0, n1, mv);
    if (WN) {
#pragma unroll
        for (int e = 0; e < kVec; ++e) sw = fmaf(wv[e], wv[e], sw);
    }
}

template <typename GT, int KT, bool RECOMP, bool WN>
__global__ __launch_bounds__(kTileBlock) void update_kernel(UpdateArgs a) {
    const int ti = a.reverse ? a.n_tiles - 1 - (int)blockIdx.x : (int)blockIdx.x;
    const Tile t = a.tiles[ti];
    const float2 ab = a.coef[t.layer];
    const GT* __restrict__ g = static_cast<const GT*>(a.grads);
    const int K = KT > 0 ? KT : a.K;
    const float lr = a.state->lr;
    float sw = 0.0f;
    for_each_group<Map<GT>::HS>(t.begin, t.count, [&](int64_t idx, int n0, int n1, auto full) {
        update_group<GT, KT, RECOMP, decltype(full)::value, WN>(a, g, idx, n0, n1, K, ab.x, ab.y,
                                                                 lr, sw);
    });
    if (WN) {
        // the step kernel's reduction: wave butterfly, then the waves in a
        // fixed pairwise order
        __shared__ float red[kTileBlock / 64];
        sw = wave_sum(sw);
        if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sw;
        __syncthreads();
        if (threadIdx.x == 0) a.w_norm_out[ti] = tree_sum<kTileBlock / 64>(red);
    }
}

// The learning rate in force, written by one lane (a kernel rather than a
// copy, so that a call made while the stream captures a graph becomes a
// kernel node that sets the same rate on every replay).
__global__ __launch_bounds__(64) void set_lr_kernel(DevState* state, float lr) {
    if (threadIdx.x == 0) state->lr = lr;
}

// ----------------------------------------------------------- dispatch ---

// One launch of a kernel whose single argument is a, with the dispatch's
// own start and stop events when timing is on.
template <typename A>
hipError_t launch(void (*k)(A), dim3 grid, dim3 block, hipStream_t s, const A& a, KernelEvents ev,
                  unsigned lds = 0) {
    if (!ev.start && !ev.stop) {
        hipLaunchKernelGGL(k, grid, block, lds, s, a);
        return hipGetLastError();
    }
    void* args[] = {const_cast<A*>(&a)};
    return hipExtLaunchKernel(reinterpret_cast<const void*>(k), grid, block, args, lds, s, ev.start,
                              ev.stop, 0);
}


template <typename GT, int KT, int RMODE>
hipError_t step_r(const StepArgs& a, int n_tiles, bool update, hipStream_t s, KernelEvents ev) {
    const dim3 grid(n_tiles), block(kTileBlock);
    if (!update) {
        const unsigned lds = (unsigned)a.lds_pad;
        if (a.gbar && a.w_norm_in)
            return launch(step_kernel<GT, KT, RMODE, false, 0, true, true>, grid, block, s, a, ev, lds);
        if (a.gbar)
            return launch(step_kernel<GT, KT, RMODE, false, 0, false, true>, grid, block, s, a, ev, lds);
        if (a.w_norm_in)
            return launch(step_kernel<GT, KT, RMODE, false, 0, true>, grid, block, s, a, ev, lds);
        return launch(step_kernel<GT, KT, RMODE, false, 0>, grid, block, s, a, ev, lds);
    }
    if (a.ew == 2) return launch(step_kernel<GT, KT, RMODE, true, 2>, grid, block, s, a, ev);
    if (a.ew) return launch(step_kernel<GT, KT, RMODE, true, 1>, grid, block, s, a, ev);
    return launch(step_kernel<GT, KT, RMODE, true, 0>, grid, block, s, a, ev, (unsigned)a.lds_pad);
}

template <typename GT, int KT>
hipError_t step_k(const StepArgs& a, int n_tiles, bool update, hipStream_t s, KernelEvents ev) {
    const int rm = a.small_replica == 0 ? 0 : (a.small_replica < 0 ? 1 : 2);
    if (rm == 0) return step_r<GT, KT, 0>(a, n_tiles, update, s, ev);
    if (rm == 1) return step_r<GT, KT, 1>(a, n_tiles, update, s, ev);
    return step_r<GT, KT, 2>(a, n_tiles, update, s, ev);
}

template <typename GT, int KT>
hipError_t update_k(const UpdateArgs& a, hipStream_t s, KernelEvents ev) {
    const dim3 grid(a.n_tiles), block(kTileBlock);
    const unsigned lds = (unsigned)a.lds_pad;
    if (a.w_norm_out) {
        if (a.gbar) return launch(update_kernel<GT, KT, false, true>, grid, block, s, a, ev, lds);
        return launch(update_kernel<GT, KT, true, true>, grid, block, s, a, ev, lds);
    }
    if (a.gbar) return launch(update_kernel<GT, KT, false, false>, grid, block, s, a, ev, lds);
    return launch(update_kernel<GT, KT, true, false>, grid, block, s, a, ev, lds);
}

template <typename GT, int KT>
hipError_t correct_k(const UpdateArgs& a, hipStream_t s, KernelEvents ev) {
    const int nb = a.n_tiles < kCorrectBlocks ? a.n_tiles : kCorrectBlocks;
    return launch(correct_kernel<GT, KT>, dim3(nb), dim3(kTileBlock), s, a, ev);
}

#define AGS_K_DISPATCH(FN, GT, K, ...)           \
    switch (K) {                                 \
        case 1: return FN<GT, 1>(__VA_ARGS__);   \
        case 2: return FN<GT, 2>(__VA_ARGS__);   \
        case 4: return FN<GT, 4>(__VA_ARGS__);   \
        case 8: return FN<GT, 8>(__VA_ARGS__);   \
        case 16: return FN<GT, 16>(__VA_ARGS__); \
        case 32: return FN<GT, 32>(__VA_ARGS__); \
        case 64: return FN<GT, 64>(__VA_ARGS__); \
        default: return FN<GT, 0>(__VA_ARGS__);  \
    }

template <typename GT>
hipError_t step_t(const StepArgs& a, int n_tiles, bool update, hipStream_t s, KernelEvents ev) {
    AGS_K_DISPATCH(step_k, GT, a.K, a, n_tiles, update, s, ev)
}
template <typename GT>
hipError_t update_t(const UpdateArgs& a, hipStream_t s, KernelEvents ev) {
    AGS_K_DISPATCH(update_k, GT, a.K, a, s, ev)
}
template <typename GT>
hipError_t correct_t(const UpdateArgs& a, hipStream_t s, KernelEvents ev) {
    AGS_K_DISPATCH(correct_k, GT, a.K, a, s, ev)
}

}  // namespace

hipError_t launch_step(const StepArgs& a, ags_dtype dt, int n_tiles, bool update, hipStream_t s,
                       KernelEvents ev) {
    return dt == AGS_BF16 ? step_t<uint16_t>(a, n_tiles, update, s, ev)
                          : step_t<float>(a, n_tiles, update, s, ev);
}

hipError_t launch_finalize(const StepArgs& a, int n_chunks, hipStream_t s, KernelEvents ev) {
    return launch(finalize_kernel, dim3(n_chunks), dim3(kBlock), s, a, ev);
}

hipError_t launch_update(const UpdateArgs& a, ags_dtype dt, hipStream_t s, KernelEvents ev) {
    return dt == AGS_BF16 ? update_t<uint16_t>(a, s, ev) : update_t<float>(a, s, ev);
}

hipError_t launch_correct(const UpdateArgs& a, ags_dtype dt, hipStream_t s, KernelEvents ev) {
    return dt == AGS_BF16 ? correct_t<uint16_t>(a, s, ev) : correct_t<float>(a, s, ev);
}

hipError_t launch_set_lr(DevState* state, float lr, hipStream_t s) {
    hipLaunchKernelGGL(set_lr_kernel, dim3(1), dim3(64), 0, s, state, lr);
    return hipGetLastError();
}

}  // namespace ags
