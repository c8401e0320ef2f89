// gfx950 kernels of one AGS step: replica mean + per-tile statistics,
// per-layer finalize (fp64) with the sensitive decision and the gradscale
// refresh, and the fused momentum-SGD update.
//
// All three are HBM-bound streaming kernels (well under 1 flop per byte):
// they use no matrix cores.  Every thread owns groups of 8 consecutive
// elements so that each replica row is read with one 16-byte load (bf16)
// or two (fp32), fully coalesced across the wave.  Reductions are
// atomic-free and in a fixed order (per-thread, wave butterfly, then the
// four waves of the block in index order; per layer in fp64 over tiles),
// so a step is bitwise reproducible.
#include <math.h>

#include "ags_internal.h"

namespace ags {
namespace {

// ---------------------------------------------------------------- loads ---

__device__ __forceinline__ void load8(const float* __restrict__ p, float (&v)[kVec]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// bf16 -> fp32 is exact: a bf16 value is the upper half of an fp32.
__device__ __forceinline__ void load8(const uint16_t* __restrict__ p, float (&v)[kVec]) {
    const uint4 a = *reinterpret_cast<const uint4*>(p);
    v[0] = __uint_as_float(a.x << 16); v[1] = __uint_as_float(a.x & 0xffff0000u);
    v[2] = __uint_as_float(a.y << 16); v[3] = __uint_as_float(a.y & 0xffff0000u);
    v[4] = __uint_as_float(a.z << 16); v[5] = __uint_as_float(a.z & 0xffff0000u);
    v[6] = __uint_as_float(a.w << 16); v[7] = __uint_as_float(a.w & 0xffff0000u);
}

__device__ __forceinline__ float load1(const float* __restrict__ p) { return *p; }
__device__ __forceinline__ float load1(const uint16_t* __restrict__ p) {
    return __uint_as_float(static_cast<uint32_t>(*p) << 16);
}

// Elements [0, n) of a group (n < 8, the ragged end of a layer); the rest
// are 0 and contribute nothing to any sum.
template <typename T>
__device__ __forceinline__ void load_tail(const T* __restrict__ p, int n, float (&v)[kVec]) {
#pragma unroll
    for (int e = 0; e < kVec; ++e) v[e] = (e < n) ? load1(p + e) : 0.0f;
}

__device__ __forceinline__ void store8(float* __restrict__ p, const float (&v)[kVec]) {
    *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

__device__ __forceinline__ void store_tail(float* __restrict__ p, int n, const float (&v)[kVec]) {
#pragma unroll
    for (int e = 0; e < kVec; ++e)
        if (e < n) p[e] = v[e];
}

// ------------------------------------------------------ replica moments ---
//
// Replica mean and spread of one group, with replica 0 as the shift: for
// k >= 1, d_k = g_k - g_0, s1 = sum d_k, s2 = sum d_k^2; then
//   gbar = g_0 + s1 / K   and   sum_k (g_k - gbar)^2 = s2 - s1^2 / K.
// Identical replicas give d_k = 0, hence gbar = g_0 and a spread of exactly
// 0; the spread is formed from differences, never as E[g^2] - E[g]^2.
// The same code produces gbar in the statistics and in the update kernel,
// so both see the same bits.
//
// RMODE selects the small-batch gradient: 0 = replica 0, 1 = mean over
// replicas (no per-replica value needed), 2 = replica r (runtime).

template <typename GT, bool FULL>
__device__ __forceinline__ void load_group(const GT* __restrict__ p, int n, float (&v)[kVec]) {
    if (FULL) load8(p, v);
    else load_tail(p, n, v);
}

// A group of 8 replica values as loaded, before widening to fp32: one
// 16-byte vector for bf16, two for fp32.  Batches of loads are held in this
// form so that a batch costs 64 VGPRs whatever the dtype.
template <typename GT> struct RawGroup;
template <> struct RawGroup<uint16_t> {
    uint4 v;
    __device__ __forceinline__ void load(const uint16_t* __restrict__ p) {
        v = *reinterpret_cast<const uint4*>(p);
    }
    __device__ __forceinline__ void widen(float (&o)[kVec]) const {
        o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
        o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
        o[4] = __uint_as_float(v.z << 16); o[5] = __uint_as_float(v.z & 0xffff0000u);
        o[6] = __uint_as_float(v.w << 16); o[7] = __uint_as_float(v.w & 0xffff0000u);
    }
};
template <> struct RawGroup<float> {
    float4 a, b;
    __device__ __forceinline__ void load(const float* __restrict__ p) {
        a = *reinterpret_cast<const float4*>(p);
        b = *reinterpret_cast<const float4*>(p + 4);
    }
    __device__ __forceinline__ void widen(float (&o)[kVec]) const {
        o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
        o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
    }
};

template <typename GT, int KT, int RMODE, bool FULL>
__device__ __forceinline__ void moments(const GT* __restrict__ g, int64_t stride, int64_t idx,
                                        int n, int K, int r, float invK, float (&gbar)[kVec],
                                        float (&dev)[kVec], float (&gr)[kVec]) {
    float g0[kVec], s1[kVec], s2[kVec];
    load_group<GT, FULL>(g + idx, n, g0);
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        s1[e] = 0.0f;
        s2[e] = 0.0f;
        gr[e] = g0[e];
    }
    auto acc = [&](int k, const float (&x)[kVec]) {
#pragma unroll
        for (int e = 0; e < kVec; ++e) {
            const float d = x[e] - g0[e];
            s1[e] += d;
            s2[e] = fmaf(d, d, s2[e]);
            if (RMODE == 2) gr[e] = (k == r) ? x[e] : gr[e];
        }
    };
    if constexpr (KT > 0 && FULL) {
        // Batches of 64 bytes of replica data per lane (16 bf16 or 8 fp32
        // replicas): every load of a batch is issued before any is used.
        constexpr int KBMAX = 64 / (int)sizeof(RawGroup<GT>);
        constexpr int KB = KT < KBMAX ? KT : KBMAX;
#pragma unroll 1
        for (int kb = 0; kb < KT; kb += KB) {
            RawGroup<GT> x[KB];
#pragma unroll
            for (int j = 0; j < KB; ++j)
                if (kb + j > 0) x[j].load(g + (int64_t)(kb + j) * stride + idx);
#pragma unroll
            for (int j = 0; j < KB; ++j)
                if (kb + j > 0) {
                    float v[kVec];
                    x[j].widen(v);
                    acc(kb + j, v);
                }
        }
    } else {
        // Runtime K, and the ragged end of a layer (rare; unrolling it
        // would raise the register count of the whole kernel).
        int k = 1;
#pragma unroll 1
        for (; k + 3 < K; k += 4) {
            float x[4][kVec];
#pragma unroll
            for (int j = 0; j < 4; ++j) load_group<GT, FULL>(g + (int64_t)(k + j) * stride + idx, n, x[j]);
#pragma unroll
            for (int j = 0; j < 4; ++j) acc(k + j, x[j]);
        }
#pragma unroll 1
        for (; k < K; ++k) {
            float x[kVec];
            load_group<GT, FULL>(g + (int64_t)k * stride + idx, n, x);
            acc(k, x);
        }
    }
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        gbar[e] = fmaf(s1[e], invK, g0[e]);
        const float t = s1[e] * invK;
        dev[e] = fmaxf(fmaf(-t, s1[e], s2[e]), 0.0f);
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

// ------------------------------------------- K1: mean + tile statistics ---

template <typename GT, int KT, int RMODE, bool FULL>
__device__ __forceinline__ void stats_group(const StatsArgs& a, const GT* __restrict__ g,
                                            int64_t idx, int n, int K, float& sw, float& sg,
                                            float& sd, float& ss) {
    float wv[kVec], gb[kVec], dv[kVec], gr[kVec];
    load_group<float, FULL>(a.w + idx, n, wv);
    moments<GT, KT, RMODE, FULL>(g, a.stride, idx, n, K, a.small_replica, a.invK, gb, dv, gr);
    if (a.gbar) {
        if (FULL) store8(a.gbar + idx, gb);
        else store_tail(a.gbar + idx, n, gb);
    }
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        sw = fmaf(wv[e], wv[e], sw);
        sg = fmaf(gb[e], gb[e], sg);
        sd += dv[e];
        // (1/K) sum_k g_k^2 = gbar^2 + (1/K) sum_k (g_k - gbar)^2
        if (RMODE == 1) ss += fmaf(gb[e], gb[e], dv[e] * a.invK);
        else ss = fmaf(gr[e], gr[e], ss);
    }
}

template <typename GT, int KT, int RMODE>
__global__ __launch_bounds__(kBlock) void stats_kernel(StatsArgs a) {
    __shared__ float red[4][kBlock / 64];
    const Tile t = a.tiles[blockIdx.x];
    const GT* __restrict__ g = static_cast<const GT*>(a.grads);
    const int K = KT > 0 ? KT : a.K;
    float sw = 0.0f, sg = 0.0f, sd = 0.0f, ss = 0.0f;
    const int nfull = t.count / kVec;
#pragma unroll 1
    for (int c = threadIdx.x; c < nfull; c += kBlock)
        stats_group<GT, KT, RMODE, true>(a, g, t.begin + (int64_t)c * kVec, kVec, K, sw, sg, sd, ss);
    const int rem = t.count - nfull * kVec;
    if (rem > 0 && (int)threadIdx.x == nfull % kBlock)
        stats_group<GT, KT, RMODE, false>(a, g, t.begin + (int64_t)nfull * kVec, rem, K, sw, sg, sd, ss);

    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    sw = wave_sum(sw);
    sg = wave_sum(sg);
    sd = wave_sum(sd);
    ss = wave_sum(ss);
    if (lane == 0) {
        red[0][wid] = sw;
        red[1][wid] = sg;
        red[2][wid] = sd;
        red[3][wid] = ss;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        Partial p;
        p.w = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
        p.g = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
        p.d = (red[2][0] + red[2][1]) + (red[2][2] + red[2][3]);
        p.s = (red[3][0] + red[3][1]) + (red[3][2] + red[3][3]);
        a.partials[blockIdx.x] = p;
    }
}

// ----------------------------------- K2: per-layer finalize + decision ---
//
// One block.  (A) each wave sums the fp32 tile partials of its layers in
// fp64 (lane-strided, then a butterfly); (B) wave 0 forms G = sum_l G_l,
// Delta = |G - G_prev| / G_prev (inf on a first step, when G_prev <= 0 or
// a value is not finite), sensitive = !(Delta < delta), and commits
// G_prev / step; (C) one thread per layer forms the update coefficients
// and, when due, refreshes gradscale = min(sqrt(S)/(sqrt(G_l)+eps), s_max)
// (1 when a norm is 0) for the steps that follow.

__global__ __launch_bounds__(kFinalizeThreads) void finalize_kernel(FinalizeArgs a) {
    __shared__ int sh_sens;
    __shared__ long long sh_t;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const double invK = 1.0 / (double)a.K;

    for (int l = wid; l < a.n_layers; l += nw) {
        const LayerDev ld = a.layers[l];
        double w = 0.0, g = 0.0, d = 0.0, s = 0.0;
        for (int t = ld.tile_begin + lane; t < ld.tile_end; t += 64) {
            const Partial p = a.partials[t];
            w += (double)p.w;
            g += (double)p.g;
            d += (double)p.d;
            s += (double)p.s;
        }
        w = wave_sum(w);
        g = wave_sum(g);
        d = wave_sum(d);
        s = wave_sum(s);
        if (lane == 0) {
            ags_layer_stats& o = a.lstats[l];
            o.w_sq = w;
            o.g_sq = g;
            o.var = d * invK;
            o.gsmall_sq = s;
        }
    }
    __threadfence_block();
    __syncthreads();

    if (wid == 0) {
        double G = 0.0;
        int nf = 0;
        for (int l = lane; l < a.n_layers; l += 64) {
            const ags_layer_stats& o = a.lstats[l];
            G += o.g_sq;
            nf |= !(isfinite(o.w_sq) && isfinite(o.g_sq) && isfinite(o.var) && isfinite(o.gsmall_sq));
        }
        G = wave_sum(G);
        nf = __any(nf) ? 1 : 0;
        if (lane == 0) {
            const DevState st = *a.state;
            const long long t = st.step + 1;
            const double Gp = st.g_prev;
            double delta;
            if (t == 1 || !(Gp > 0.0) || !isfinite(Gp) || !isfinite(G))
                delta = INFINITY;
            else
                delta = fabs((G - Gp) / Gp);
            const int sens = !(delta < a.delta);
            if (!isfinite(G)) nf = 1;
            ags_global_stats gs;
            gs.step = a.commit ? t : st.step;
            gs.g_sq = G;
            gs.g_sq_prev = (t == 1) ? 0.0 : Gp;
            gs.delta = delta;
            gs.sensitive = sens;
            gs.nonfinite = nf;
            *a.gstats = gs;
            if (a.commit) {
                a.state->g_prev = G;
                a.state->step = t;
            }
            sh_sens = sens;
            sh_t = t;
        }
    }
    __syncthreads();

    const int sens = sh_sens;
    const long long t = sh_t;
    const bool refresh = a.commit && a.mode == AGS_MODE_AGS && a.refresh_every > 0 &&
                         (t % a.refresh_every) == 0;
    const double smax = a.s_max > 0.0 ? a.s_max : sqrt((double)a.K);
    for (int l = threadIdx.x; l < a.n_layers; l += blockDim.x) {
        ags_layer_stats& o = a.lstats[l];
        const uint32_t f = a.layers[l].flags;
        const bool scaled = (f & AGS_LAYER_SCALE) != 0;
        const double lam = (f & AGS_LAYER_DECAY) ? a.weight_decay : 0.0;
        double ca = 1.0, cb = lam;
        if (a.mode == AGS_MODE_AGS) {
            ca = (scaled && !sens) ? a.gradscale[l] : 1.0;
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
        double gsc = a.gradscale[l];
        if (refresh && scaled) {
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
}

// ----------------------------------------------- K3: fused update ---------
//
// d = a_l gbar + b_l w ; m <- mu m + d ; w <- w - eta m, read once, written
// once.  gbar comes from the statistics kernel's buffer or, when re-reading
// the replicas costs no more than that round trip (K * bytes <= 8), is
// recomputed from them by the same code.

template <typename GT, int KT, bool RECOMP, bool FULL>
__device__ __forceinline__ void update_group(const UpdateArgs& a, const GT* __restrict__ g,
                                             int64_t idx, int n, int K, float ca, float cb) {
    float gb[kVec], wv[kVec], mv[kVec];
    load_group<float, FULL>(a.w + idx, n, wv);
    load_group<float, FULL>(a.m + idx, n, mv);
    if (RECOMP) {
        float dv[kVec], gr[kVec];
        moments<GT, KT, 0, FULL>(g, a.stride, idx, n, K, 0, a.invK, gb, dv, gr);
    } else {
        load_group<float, FULL>(a.gbar + idx, n, gb);
    }
#pragma unroll
    for (int e = 0; e < kVec; ++e) {
        const float d = fmaf(ca, gb[e], cb * wv[e]);
        mv[e] = fmaf(a.momentum, mv[e], d);
        wv[e] = fmaf(-a.lr, mv[e], wv[e]);
    }
    if (FULL) {
        store8(a.w + idx, wv);
        store8(a.m + idx, mv);
    } else {
        store_tail(a.w + idx, n, wv);
        store_tail(a.m + idx, n, mv);
    }
}

template <typename GT, int KT, bool RECOMP>
__global__ __launch_bounds__(kBlock) void update_kernel(UpdateArgs a) {
    const Tile t = a.tiles[blockIdx.x];
    const float2 ab = a.coef[t.layer];
    const GT* __restrict__ g = static_cast<const GT*>(a.grads);
    const int K = KT > 0 ? KT : a.K;
    const int nfull = t.count / kVec;
#pragma unroll 1
    for (int c = threadIdx.x; c < nfull; c += kBlock)
        update_group<GT, KT, RECOMP, true>(a, g, t.begin + (int64_t)c * kVec, kVec, K, ab.x, ab.y);
    const int rem = t.count - nfull * kVec;
    if (rem > 0 && (int)threadIdx.x == nfull % kBlock)
        update_group<GT, KT, RECOMP, false>(a, g, t.begin + (int64_t)nfull * kVec, rem, K, ab.x, ab.y);
}

// ----------------------------------------------------------- dispatch ---

template <typename GT, int KT>
hipError_t stats_k(const StatsArgs& a, int n_tiles, hipStream_t s) {
    const dim3 grid(n_tiles), block(kBlock);
    if (a.small_replica == 0)
        hipLaunchKernelGGL((stats_kernel<GT, KT, 0>), grid, block, 0, s, a);
    else if (a.small_replica < 0)
        hipLaunchKernelGGL((stats_kernel<GT, KT, 1>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((stats_kernel<GT, KT, 2>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <typename GT>
hipError_t stats_t(const StatsArgs& a, int n_tiles, hipStream_t s) {
    switch (a.K) {
        case 1: return stats_k<GT, 1>(a, n_tiles, s);
        case 2: return stats_k<GT, 2>(a, n_tiles, s);
        case 4: return stats_k<GT, 4>(a, n_tiles, s);
        case 8: return stats_k<GT, 8>(a, n_tiles, s);
        case 16: return stats_k<GT, 16>(a, n_tiles, s);
        case 32: return stats_k<GT, 32>(a, n_tiles, s);
        case 64: return stats_k<GT, 64>(a, n_tiles, s);
        default: return stats_k<GT, 0>(a, n_tiles, s);
    }
}

template <typename GT, int KT>
hipError_t update_k(const UpdateArgs& a, int n_tiles, hipStream_t s) {
    const dim3 grid(n_tiles), block(kBlock);
    if (a.gbar)
        hipLaunchKernelGGL((update_kernel<GT, KT, false>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((update_kernel<GT, KT, true>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <typename GT>
hipError_t update_t(const UpdateArgs& a, int n_tiles, hipStream_t s) {
    switch (a.K) {
        case 1: return update_k<GT, 1>(a, n_tiles, s);
        case 2: return update_k<GT, 2>(a, n_tiles, s);
        case 4: return update_k<GT, 4>(a, n_tiles, s);
        case 8: return update_k<GT, 8>(a, n_tiles, s);
        case 16: return update_k<GT, 16>(a, n_tiles, s);
        case 32: return update_k<GT, 32>(a, n_tiles, s);
        case 64: return update_k<GT, 64>(a, n_tiles, s);
        default: return update_k<GT, 0>(a, n_tiles, s);
    }
}

}  // namespace

hipError_t launch_stats(const StatsArgs& a, ags_dtype dt, int n_tiles, hipStream_t s) {
    return dt == AGS_BF16 ? stats_t<uint16_t>(a, n_tiles, s) : stats_t<float>(a, n_tiles, s);
}

hipError_t launch_finalize(const FinalizeArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(kFinalizeThreads), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_update(const UpdateArgs& a, ags_dtype dt, int n_tiles, hipStream_t s) {
    return dt == AGS_BF16 ? update_t<uint16_t>(a, n_tiles, s) : update_t<float>(a, n_tiles, s);
}

}  // namespace ags
