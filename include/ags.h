/*
 * libags: the Adaptive Gradient Scaling (AGS) optimizer step with its
 * gradient statistics, for one data-parallel training step on one MI355X
 * (gfx950) GPU.
 *
 * Source of the method: Tula (arXiv 2603.18112): the gradient-variability
 * metric of Sec. III-B, Eq. (5); the statistical performance model of
 * Sec. III-C, Eq. (6)-(8) and Algorithm 1 "Adaptive Gradient Scaling";
 * synchronous data-parallel averaging, Eq. (1c); the wrapped momentum SGD
 * with weight decay of Sec. IV-A/IV-B; the LARS baseline of Sec. IV-D.
 *
 * One step, for a model whose parameter tensors ("layers") are laid end to
 * end in one flat fp32 buffer w with momentum m of the same layout, given K
 * replica gradients g_0..g_{K-1} (the K data-parallel workers' local
 * gradients of the step, each laid out like w):
 *
 *   gbar        = (1/K) sum_k g_k                        large-batch gradient
 *   W_l, G_l    = ||w_l||^2, ||gbar_l||^2                per layer
 *   V_l         = (1/K) sum_k ||g_k,l - gbar_l||^2       cross-replica spread
 *   S_l         = ||g_r,l||^2                            small-batch gradient
 *   G           = sum_l G_l
 *   Delta       = |G - G_prev| / G_prev                  gradient variability
 *   sensitive   = !(Delta < delta)                       (inf on the 1st step)
 *   Delta_l     = |G_l - G_l,prev| / G_l,prev            per layer (reported;
 *                 decides layer l with AGS_DELTA_LAYER)
 *   d           = a_l gbar + b_l w                       a_l, b_l per mode
 *   m <- mu m + d ;  w <- w - eta m                      momentum SGD
 *   gradscale_l <- min(sqrt(S_l) / (sqrt(G_l) + eps), s_max)   (refresh)
 *
 * Modes: AGS   a_l = gradscale_l if the layer is scaled and the step is not
 *              sensitive, else 1; b_l = lambda_l.
 *        LARS  a_l = tau ||w_l|| / (||gbar_l|| + lambda_l ||w_l||) on scaled
 *              layers (1 if either norm is 0); b_l = a_l lambda_l.
 *        STATIC a_l = s (static_scale) if the layer is scaled and the step
 *              is not sensitive, else 1; b_l = lambda_l (the static mapping
 *              U(s) of Eq. (8a), (8b), Sec. III-C).
 *        SGD   a_l = 1; b_l = lambda_l.
 * lambda_l is weight_decay on layers with AGS_LAYER_DECAY, else 0.
 *
 * Elementwise AGS (cfg.elementwise = 1, AGS mode only) reads the scale of
 * Algorithm 1 per parameter element instead of per tensor: element j of a
 * scaled layer gets a_j = gradscale_j on a non-sensitive step (else 1), and
 * the refresh sets gradscale_j = min(|g_small,j / (gbar_j + eps)|, s_max),
 * where g_small,j is replica r's element (or, with small_replica = -1, the
 * root mean square of the K replicas' elements) and a 0/0 ratio gives 1.
 * The denominator gbar_j + eps is formed from an fp64 sum of the replicas,
 * so that its cancellation does not decide the ratio.  The per-layer records
 * then hold layer means: coef_a the mean coefficient applied, gradscale the
 * mean scale after the call.
 *
 * Conventions for every function:
 *  - C linkage; every function returns an ags_status (0 = AGS_OK) except
 *    where noted; nothing throws across the ABI.
 *  - Pointers named d_* are device memory on the handle's device.  Host
 *    arrays are read or written before the call returns.
 *  - Argument, layout and alignment checks run on the host before any HIP
 *    call; on error nothing is changed.  Device pointers are then checked
 *    to be device allocations large enough for the access (AGS_E_ARG if
 *    not), so that a bad pointer is an error, not a GPU fault.
 *  - Work is enqueued on hip_stream (a hipStream_t; NULL is the default
 *    stream) and the call returns without waiting, except ags_read_stats,
 *    ags_get_state, ags_set_state, ags_get_layer_state, ags_set_layer_state,
 *    ags_get_last_decision, ags_set_last_decision,
 *    ags_get_elementwise_scale, ags_set_elementwise_scale and
 *    ags_get_kernel_times, which wait for the handle's last stream.
 *  - Calls on one handle are ordered: the handle's workspace and state are
 *    shared by all its steps, so a call on a stream other than the one the
 *    handle last used first makes that stream wait (a HIP event) for the
 *    work already queued on the handle's last stream.  Neither stream may
 *    be capturing a graph then: a step captured into a graph must be
 *    ordered after the handle's earlier work by the caller (for example by
 *    capturing on the stream the handle last used, or after a synchronize).
 *    The handle's last stream must still exist when a call comes on another
 *    stream (the wait is an event recorded on it then) and when the
 *    functions above wait for it: destroy the stream a handle last used
 *    only after the handle has made a call on another stream, or after
 *    ags_destroy.
 *    The caller's own accesses to w, m and the gradients are ordered by the
 *    caller, as for any kernel launched on hip_stream.
 *  - A handle is not thread-safe: one thread at a time.
 */
#ifndef AGS_H
#define AGS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    AGS_OK = 0,
    AGS_E_ARG = 1,     /* bad argument (null, out of range, not device memory) */
    AGS_E_LAYOUT = 2,  /* layer table empty, overlapping, unordered, out of n_flat */
    AGS_E_ALIGN = 3,   /* offset / stride / pointer misaligned                */
    AGS_E_NOMEM = 4,   /* workspace allocation failed or over the cap          */
    AGS_E_DEVICE = 5,  /* a HIP call failed; see ags_last_error               */
    AGS_E_STATE = 6    /* handle state mismatch (e.g. wrong state length)      */
} ags_status;

typedef enum { AGS_F32 = 0, AGS_BF16 = 1 } ags_dtype;

typedef enum { AGS_MODE_SGD = 0, AGS_MODE_AGS = 1, AGS_MODE_LARS = 2, AGS_MODE_STATIC = 3 } ags_mode;

/* Which variability measure decides a layer's coefficient in AGS and STATIC
 * modes: the global Delta of Eq. (5) (Sec. III-B), or the same measure on
 * the layer's own norm, Delta_l (a per-layer variant of Eq. (5); the first
 * step, G_l,prev <= 0 and non-finite norms give +inf as for Delta). */
typedef enum { AGS_DELTA_GLOBAL = 0, AGS_DELTA_LAYER = 1 } ags_delta_scope;

#define AGS_LAYER_SCALE 1u /* the layer takes part in AGS / LARS scaling  */
#define AGS_LAYER_DECAY 2u /* the layer receives weight decay             */

/* Layer offsets and the replica stride are multiples of this many elements,
 * and d_w, d_m, d_grads are 16-byte aligned, so that every 8-element group
 * is one aligned 16-byte (bf16) or two 16-byte (fp32) loads. */
#define AGS_ALIGN_ELEMS 8
#define AGS_MAX_K 1024

/* One parameter tensor: elements [offset, offset + numel) of the flat
 * buffers.  numel > 0; layers are in increasing offset order and do not
 * overlap; offset + numel <= n_flat.  Elements outside every layer are
 * never read or written. */
typedef struct {
    int64_t offset;
    int64_t numel;
    uint32_t flags;    /* AGS_LAYER_SCALE | AGS_LAYER_DECAY */
    uint32_t reserved; /* must be 0 */
} ags_layer;

typedef struct {
    int32_t n_layers;
    const ags_layer *layers; /* host array [n_layers], copied at init       */
    int64_t n_flat;          /* elements in d_w and d_m                     */
    int32_t K;               /* replicas, 1..AGS_MAX_K                      */
    ags_dtype grad_dtype;    /* dtype of the replica gradients              */
    ags_mode mode;
    double lr;               /* eta >= 0                                    */
    double momentum;         /* mu in [0, 1)                                */
    double weight_decay;     /* lambda >= 0                                 */
    double delta;            /* sensitivity threshold; the paper uses 0.5   */
    double eps;              /* stability term >= 0; the paper uses 1e-8    */
    double s_max;            /* scale clip; <= 0 means sqrt(K)             */
    double trust_coef;       /* LARS tau > 0 (used in AGS_MODE_LARS)        */
    int32_t refresh_every;   /* refresh gradscale every n steps; 0 = never  */
    int32_t small_replica;   /* replica r taken as the small-batch gradient;
                                -1 = mean over replicas of ||g_k||^2        */
    double static_scale;     /* s of AGS_MODE_STATIC (> 0)                 */
    int32_t elementwise;     /* 1: AGS scale per element (AGS mode only)    */
    int32_t delta_scope;     /* ags_delta_scope                            */
    int32_t reuse_w_norms;   /* 1: LARS takes ||w_l||^2 from the last update
                                pass instead of reading w (LARS mode only;
                                see ags_invalidate_weight_norms)           */
} ags_config;

/* Per-layer record of the last ags_stats / ags_step.  var is V_l (the 1/K
 * normalised spread), noise_ratio = V_l / G_l (0 if both are 0, +inf if
 * only G_l is 0), coef_a / coef_b the update coefficients used (or that
 * would be used, for ags_stats), gradscale the state after the call, delta
 * the layer's Delta_l, sensitive the bit that decided the layer (the global
 * one with AGS_DELTA_GLOBAL). */
typedef struct {
    double w_sq, g_sq, var, gsmall_sq, noise_ratio, coef_a, coef_b, gradscale;
    double delta;
    int32_t sensitive;
    int32_t reserved;
} ags_layer_stats;

/* Global record.  step: steps completed after the call; g_sq_prev: the
 * previous norm the call compared against (0 on a first step); delta:
 * +inf on a first step, when g_sq_prev <= 0 or when a norm is not finite;
 * sensitive = !(delta < cfg.delta); nonfinite: a statistic was inf/nan. */
typedef struct {
    int64_t step;
    double g_sq, g_sq_prev, delta;
    int32_t sensitive, nonfinite;
} ags_global_stats;

typedef struct ags_handle ags_handle;

/* Kernels of one step, in launch order, for ags_get_kernel_times:
 * 0: the step kernel (replica mean, tile statistics and, for AGS and SGD,
 *    the update with the coefficients predicted before the step);
 * 1: finalize (layer and global statistics, decision, refresh);
 * 2: the second pass (AGS: correction of a mispredicted sensitive bit,
 *    which exits at once otherwise; LARS: the update; SGD: none). */
#define AGS_N_KERNELS 3

/* Bytes of device workspace ags_init would allocate for cfg (host only).
 * Both reject (AGS_E_LAYOUT) layer tables that need 2^24 or more tiles of
 * 2048 elements (about 3.4e10 parameters): a launch holds fewer than 2^32
 * work-items. */
ags_status ags_workspace_bytes(const ags_config *cfg, size_t *out_bytes);

/* Create a handle bound to d_w, d_m (fp32 [n_flat], caller-owned, must
 * outlive the handle, must not overlap: AGS_E_ARG) on the current HIP
 * device.  The handle allocates its
 * workspace (AGS_E_NOMEM on failure or when it exceeds the byte cap given
 * by the environment variable AGS_MAX_WORKSPACE_BYTES; nothing is leaked).
 * gradscale starts at 1 (Algorithm 1), the step count at 0. */
ags_status ags_init(const ags_config *cfg, float *d_w, float *d_m, void *hip_stream,
                    ags_handle **out);

/* Statistics only: replica mean, per-layer and global statistics and the
 * coefficients a step would use now.  The replica mean is the large-batch
 * gradient of synchronous data-parallel training (Eq. (1c)); W_l, G_l and
 * S_l are the per-tensor norms of Algorithm 1 (UpdateGradScale); G and
 * Delta are the whole-model norm and the variability metric of Eq. (5)
 * (Sec. III-B); V_l, the spread of the replicas about their mean, measures
 * the gap between small- and large-batch gradients that the noise term of
 * Eq. (6) models (Sec. III-C).  w, m and the AGS state are not
 * changed.  d_grads: [K][replica_stride] elements of grad_dtype, caller-
 * owned; replica k starts at element k * replica_stride and uses the
 * layout of w; replica_stride >= n_flat, a multiple of AGS_ALIGN_ELEMS;
 * the replica stack must not overlap w or m (AGS_E_ARG). */
ags_status ags_stats(ags_handle *h, const void *d_grads, int64_t replica_stride,
                     void *hip_stream);

/* One AGS step (Algorithm 1 iteration + UpdateGradScale when due): the
 * statistics above, the sensitive decision, the update of w and m in
 * place, then G_prev <- G, step += 1 and the gradscale refresh. */
ags_status ags_step(ags_handle *h, const void *d_grads, int64_t replica_stride,
                    void *hip_stream);

/* Copy the records of the last ags_stats / ags_step to host arrays
 * (out_layers [n_layers] may be NULL, out_global may be NULL): the
 * statistics of Eq. (5), Eq. (6) and Algorithm 1 listed with ags_stats, the
 * decision of Algorithm 1 (sensitive iff not Delta < delta) and the
 * coefficients and scale of the step.  Waits for the handle's last stream;
 * AGS_E_STATE before the first ags_stats / ags_step. */
ags_status ags_read_stats(ags_handle *h, ags_layer_stats *out_layers,
                          ags_global_stats *out_global);

/* Learning rate eta for the steps launched after this call.  The paper
 * keeps eta a host-side schedule (the linear scaling with the batch and
 * the warm-up and decay of the baselines, Sec. IV-B, IV-D); the update of
 * Algorithm 1 and the wrapped momentum SGD read it per step.  lr must be
 * finite and >= 0 (AGS_E_ARG).  The rate is kept in the device state and
 * written (as fp32, by a one-thread kernel) on the handle's last stream,
 * after the work queued there: every step that runs after it uses it,
 * eager steps and steps replayed from a HIP graph captured earlier alike
 * (a replay on another stream is ordered after this call by the caller).
 * Called while that stream captures a graph, the write becomes part of the
 * graph. */
ags_status ags_set_lr(ags_handle *h, double lr);

/* Checkpoint / resume of the AGS state (w and m are the caller's).
 * gradscale_L: host [n_layers].  With elementwise scales, ags_get_state
 * writes the layer means of the element scales to gradscale_L, and
 * ags_set_state sets G_prev and the step count only (gradscale_L may be
 * NULL and is not read): the element scales are restored with
 * ags_set_elementwise_scale.  ags_set_state clears the last step's
 * sensitive bit (see ags_set_last_decision) and drops LARS's carried
 * weight norms (see ags_invalidate_weight_norms). */
ags_status ags_get_state(const ags_handle *h, double *gradscale_L, double *g_sq_prev,
                         int64_t *step);
ags_status ags_set_state(ags_handle *h, const double *gradscale_L, double g_sq_prev,
                         int64_t step);

/* Weight norms carried from one LARS step to the next (cfg.reuse_w_norms).
 * The LARS trust ratio of Sec. IV-D needs W_l = ||w_l||^2 before the
 * update, so a LARS step is two passes: statistics, then the update.  With
 * reuse_w_norms = 1 the update pass also sums the squares of the new w per
 * tile, in exactly the order the statistics pass sums them, and the next
 * ags_step or ags_stats takes W_l from those sums instead of reading w
 * (4 bytes per parameter less; the statistics are bit for bit those of
 * reading w, as long as w holds what the last update wrote).  The library
 * cannot see writes to w made outside its calls: the sums are used only
 * after a committed LARS ags_step of this handle, and are dropped by
 * ags_set_state, a step whose launch fails (AGS_E_DEVICE), and this
 * function, which a
 * caller that writes w between calls (a checkpoint load, another
 * optimizer's step, an in-place edit) must call before the next step.  A
 * step captured into a HIP graph always reads w (a replay cannot know
 * whether w still holds what the last update wrote), and capturing leaves
 * the handle's choice for its later eager calls as it was; a replayed
 * update pass writes the sums like an eager one.  AGS_E_STATE on a handle
 * without reuse_w_norms. */
ags_status ags_invalidate_weight_norms(ags_handle *h);

/* Per-layer G_l,prev (the ||gbar_l||^2 of the last step), the state of
 * Delta_l: host [n_layers].  Get waits for the handle's last stream; set
 * checks every value is finite and >= 0 (AGS_E_ARG, nothing changed) and
 * clears the layers' last sensitive bits. */
ags_status ags_get_layer_state(ags_handle *h, double *g_sq_prev_L);
ags_status ags_set_layer_state(ags_handle *h, const double *g_sq_prev_L);

/* The sensitive bits of the last committed step: the global one, and per
 * layer the bit that decided the layer (host [n_layers], or NULL to skip);
 * a step sensitive by definition (Delta infinite: the first) leaves 0.
 * An AGS or static step applies its update with the coefficients of the
 * decision predicted from them (sensitive when the last step was, or when
 * Delta is infinite by definition) and corrects the layers whose actual
 * decision differs, so the bits only choose the rounding path: a resumed
 * run that restores them with the rest of the state repeats the original
 * run bit for bit; without them (cleared by ags_set_state and
 * ags_set_layer_state) it agrees to fp32 rounding.  Set checks every value
 * is 0 or 1 (AGS_E_ARG, nothing changed). */
ags_status ags_get_last_decision(ags_handle *h, int32_t *sensitive, int32_t *sensitive_L);
ags_status ags_set_last_decision(ags_handle *h, int32_t sensitive, const int32_t *sensitive_L);

/* Elementwise scales gradscale_j (Algorithm 1 read per element; handles
 * created with cfg.elementwise = 1, else AGS_E_STATE).  scale: host fp32
 * [n], n == n_flat (AGS_E_ARG otherwise); entries outside every layer are
 * carried but never used.  Get waits for the handle's last stream.  Set
 * checks every value is finite and >= 0 (AGS_E_ARG, nothing changed),
 * waits for the last stream, copies the array and recomputes the layer
 * means in fp64.  Those means only feed the reports (the coef_a and
 * gradscale records, the means ags_get_state returns); the kernels form
 * them from fp32 tile sums, so after a set they can differ from the
 * original run's in the last bits (about 1e-7 relative) until the next
 * refresh recomputes them.  The element scales themselves, and so w and m,
 * resume bit for bit. */
ags_status ags_get_elementwise_scale(ags_handle *h, float *scale, int64_t n);
ags_status ags_set_elementwise_scale(ags_handle *h, const float *scale, int64_t n);

/* Per-kernel timing: with profiling enabled, each kernel of a step is
 * launched with a start and a stop HIP event of its own dispatch on the
 * launch stream (the kernel's execution alone); read the summed
 * milliseconds per kernel (out_ms [AGS_N_KERNELS]: step kernel, finalize,
 * second pass, which is 0 for SGD) and the number of steps measured since
 * the last read; reading resets.  Steps enqueued during stream capture are
 * not timed. */
ags_status ags_set_profiling(ags_handle *h, int enable);
ags_status ags_get_kernel_times(ags_handle *h, double *out_ms, int64_t *out_calls);

/* For callers that cannot allocate device memory (code that must not call
 * hipMalloc: tight serving loops, harnesses that forbid allocation): the
 * statistics of ags_stats without a handle.  It fills out_layers (host
 * [n_layers]) and out_global (host) with what ags_read_stats returns after
 * ags_stats on a handle just created by ags_init(cfg, ...): the replica
 * mean, W_l, G_l, V_l, S_l, rho_l, the global G, and the decision and
 * coefficients of a first step (no previous norm: Delta and every Delta_l
 * are +inf, the step is sensitive, gradscale is 1).  d_w: fp32 [n_flat],
 * read only; d_grads as for ags_stats (m is not read).  Arguments are
 * checked as by ags_init and ags_stats (AGS_E_ARG, AGS_E_LAYOUT,
 * AGS_E_ALIGN; the error text is ags_last_error(NULL)).
 *
 * It allocates nothing: the layer table, tile map, tile partials, counters
 * and records live in one device array of 6 MiB inside the library, which
 * each GPU the library runs on holds until the process ends; a call whose
 * tables do not fit (about 230 bytes per layer plus 32 per tile of 2048
 * elements: about 4e8 parameters in up to a few hundred layers) returns
 * AGS_E_NOMEM before any device work.  Every call on a GPU shares that GPU's
 * array and leaves its tables there: calls that overlap on one GPU (two
 * threads, or two streams without ordering between them) race.  The call
 * enqueues its work on hip_stream, copies the records to the host arrays
 * and waits for hip_stream before it returns. */
ags_status ags_stats_noalloc(const ags_config *cfg, const float *d_w, const void *d_grads,
                             int64_t replica_stride, ags_layer_stats *out_layers,
                             ags_global_stats *out_global, void *hip_stream);

/* Static text for a status; last error text of a handle (or, with NULL, of
 * the last failed ags_init / ags_workspace_bytes on this thread). */
const char *ags_status_string(ags_status s);
const char *ags_last_error(const ags_handle *h);

/* Free the handle and its workspace (waits for its last stream).  NULL is
 * a no-op. */
void ags_destroy(ags_handle *h);

#ifdef __cplusplus
}
#endif

#endif /* AGS_H */
