// Host-side planner of libags (include/ags_plan.h): the step-time model of
// Eq. (2), the memory bound of Eq. (3), training time and cost of Eq. (4)
// and the configuration selection policy (minimum time, minimum cost, or the
// Kneedle knee of the time-batch curve).  Plain fp64 host code.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <vector>

#include "ags_plan.h"
#include "ags_internal.h"

namespace {

ags_status fail(ags_status s, const char* why) {
    ags::set_thread_error(why);
    return s;
}

bool fin(double x) { return std::isfinite(x); }

double sync_term(int32_t nodes, ags_sync_model sync) {
    if (sync == AGS_SYNC_PS) return (double)nodes;
    if (sync == AGS_SYNC_RING) return 1.0 - 1.0 / (double)nodes;
    return 0.0;
}

// Enum arguments and fields are validated from their 32-bit value: loading
// an enum object outside its enumeration is undefined behaviour in C++.
template <typename E>
int32_t raw_enum(const E& e) {
    static_assert(sizeof(E) == sizeof(int32_t), "enum values are 32-bit");
    int32_t v;
    std::memcpy(&v, &e, sizeof v);
    return v;
}

bool valid_sync(int32_t s) { return s == AGS_SYNC_NONE || s == AGS_SYNC_RING || s == AGS_SYNC_PS; }

double model_step(const ags_plan_model& m, int32_t nodes, double b) {
    return m.c0 + m.c_compute * b + m.c_sync * sync_term(nodes, m.sync);
}

ags_status check_model(const ags_plan_model* m) {
    if (!m) return fail(AGS_E_ARG, "model is NULL");
    if (!valid_sync(raw_enum(m->sync))) return fail(AGS_E_ARG, "bad sync model");
    if (!fin(m->c0) || !fin(m->c_compute) || !fin(m->c_sync))
        return fail(AGS_E_ARG, "model coefficients must be finite");
    return AGS_OK;
}

// min ||X c - y||_2 for an n x p column-major X (p <= 3) by Householder QR.
// Returns false when a column is (numerically) a combination of the others.
bool least_squares(std::vector<double>& X, std::vector<double>& y, int n, int p, double* c) {
    double rdiag[3];
    double colnorm0[3];
    for (int j = 0; j < p; ++j) {
        double s = 0.0;
        for (int i = 0; i < n; ++i) s += X[j * n + i] * X[j * n + i];
        colnorm0[j] = std::sqrt(s);
    }
    for (int k = 0; k < p; ++k) {
        double* a = &X[k * n];
        double norm = 0.0;
        for (int i = k; i < n; ++i) norm += a[i] * a[i];
        norm = std::sqrt(norm);
        // a column that is zero, or whose part outside the span of the
        // earlier columns vanishes, cannot be identified
        if (!(norm > 1e-12 * colnorm0[k])) return false;
        const double alpha = a[k] > 0 ? -norm : norm;
        // v = a[k:] - alpha e_k, kept in a[k:]; H = I - 2 v v^T / (v^T v)
        a[k] -= alpha;
        double vtv = 0.0;
        for (int i = k; i < n; ++i) vtv += a[i] * a[i];
        for (int j = k + 1; j < p; ++j) {
            double* b = &X[j * n];
            double d = 0.0;
            for (int i = k; i < n; ++i) d += a[i] * b[i];
            const double f = 2.0 * d / vtv;
            for (int i = k; i < n; ++i) b[i] -= f * a[i];
        }
        double d = 0.0;
        for (int i = k; i < n; ++i) d += a[i] * y[i];
        const double f = 2.0 * d / vtv;
        for (int i = k; i < n; ++i) y[i] -= f * a[i];
        rdiag[k] = alpha;
    }
    for (int k = p - 1; k >= 0; --k) {
        double s = y[k];
        for (int j = k + 1; j < p; ++j) s -= X[j * n + k] * c[j];
        c[k] = s / rdiag[k];
    }
    return true;
}

}  // namespace

extern "C" {

ags_status ags_plan_fit(const ags_plan_sample* samples, int32_t n, ags_sync_model sync,
                        uint32_t terms, ags_plan_model* out) {
    if (!samples || !out) return fail(AGS_E_ARG, "samples and out must not be NULL");
    if (!valid_sync(raw_enum(sync))) return fail(AGS_E_ARG, "bad sync model");
    if (terms == 0 || (terms & ~(AGS_PLAN_INTERCEPT | AGS_PLAN_COMPUTE | AGS_PLAN_SYNC)) != 0)
        return fail(AGS_E_ARG, "terms must be a non-empty set of AGS_PLAN_* bits");
    int p = 0;
    for (uint32_t b = 1; b <= AGS_PLAN_SYNC; b <<= 1) p += (terms & b) ? 1 : 0;
    if (n < p) return fail(AGS_E_ARG, "fewer samples than terms");
    for (int32_t i = 0; i < n; ++i) {
        const ags_plan_sample& s = samples[i];
        if (s.nodes < 1 || s.reserved != 0 || !fin(s.local_batch) || s.local_batch < 0 ||
            !fin(s.t_step)) {
            char buf[96];
            snprintf(buf, sizeof buf, "sample %d: need nodes >= 1, reserved 0, finite b >= 0 and t", i);
            return fail(AGS_E_ARG, buf);
        }
    }
    std::vector<double> X((size_t)n * p), y(n);
    for (int32_t i = 0; i < n; ++i) {
        int j = 0;
        if (terms & AGS_PLAN_INTERCEPT) X[(size_t)(j++) * n + i] = 1.0;
        if (terms & AGS_PLAN_COMPUTE) X[(size_t)(j++) * n + i] = samples[i].local_batch;
        if (terms & AGS_PLAN_SYNC) X[(size_t)(j++) * n + i] = sync_term(samples[i].nodes, sync);
        y[i] = samples[i].t_step;
    }
    double c[3] = {0.0, 0.0, 0.0};
    if (!least_squares(X, y, n, p, c))
        return fail(AGS_E_ARG, "the samples cannot tell the chosen terms apart (rank deficient)");
    ags_plan_model m{};
    m.sync = sync;
    m.terms = terms;
    int j = 0;
    if (terms & AGS_PLAN_INTERCEPT) m.c0 = c[j++];
    if (terms & AGS_PLAN_COMPUTE) m.c_compute = c[j++];
    if (terms & AGS_PLAN_SYNC) m.c_sync = c[j++];
    double ss = 0.0;
    for (int32_t i = 0; i < n; ++i) {
        const double r = samples[i].t_step - model_step(m, samples[i].nodes, samples[i].local_batch);
        ss += r * r;
    }
    m.rms_residual = std::sqrt(ss / n);
    m.n_samples = n;
    *out = m;
    return AGS_OK;
}

ags_status ags_plan_step_time(const ags_plan_model* m, int32_t nodes, double local_batch,
                              double* t_step) {
    ags_status s = check_model(m);
    if (s != AGS_OK) return s;
    if (!t_step) return fail(AGS_E_ARG, "t_step is NULL");
    if (nodes < 1 || !fin(local_batch) || local_batch < 0)
        return fail(AGS_E_ARG, "need nodes >= 1 and a finite local batch >= 0");
    *t_step = model_step(*m, nodes, local_batch);
    return AGS_OK;
}

ags_status ags_plan_time_cost(const ags_plan_model* m, int32_t nodes, double global_batch,
                              double epochs, double dataset_size, double price_per_node_hour,
                              double* T_seconds, double* cost) {
    ags_status s = check_model(m);
    if (s != AGS_OK) return s;
    if (!T_seconds || !cost) return fail(AGS_E_ARG, "NULL output pointer");
    if (nodes < 1 || !fin(global_batch) || !(global_batch > 0) || !fin(epochs) ||
        epochs < 0 || !fin(dataset_size) || dataset_size < 0 || !fin(price_per_node_hour) ||
        price_per_node_hour < 0)
        return fail(AGS_E_ARG, "need nodes >= 1, B > 0 and finite E, D, p >= 0");
    const double t = model_step(*m, nodes, global_batch / nodes);
    const double T = epochs * dataset_size / global_batch * t;
    *T_seconds = T;
    *cost = T / 3600.0 * nodes * price_per_node_hour;
    return AGS_OK;
}

ags_status ags_plan_max_local_batch(double capacity, double m_static, double m_per_sample,
                                    int64_t* b_max) {
    if (!b_max) return fail(AGS_E_ARG, "b_max is NULL");
    if (!fin(capacity) || !fin(m_static) || !fin(m_per_sample) || !(m_per_sample > 0))
        return fail(AGS_E_ARG, "need finite capacity and static memory, per-sample memory > 0");
    const double b = std::floor((capacity - m_static) / m_per_sample);
    if (!(b > 0)) {
        *b_max = 0;
    } else if (b >= 9.0e18) {
        return fail(AGS_E_ARG, "bound out of range");
    } else {
        *b_max = (int64_t)b;
    }
    return AGS_OK;
}

ags_status ags_plan_knee(const double* x, const double* y, int32_t n, ags_knee_shape shape,
                         double sensitivity, int32_t* index) {
    if (!index) return fail(AGS_E_ARG, "index is NULL");
    if (n < 0 || (n > 0 && (!x || !y))) return fail(AGS_E_ARG, "bad arrays");
    const int32_t shp = raw_enum(shape);
    if (shp < AGS_KNEE_CONCAVE_INC || shp > AGS_KNEE_CONVEX_DEC) return fail(AGS_E_ARG, "bad shape");
    if (!fin(sensitivity) || sensitivity < 0) return fail(AGS_E_ARG, "sensitivity must be finite, >= 0");
    for (int32_t i = 0; i < n; ++i) {
        if (!fin(x[i]) || !fin(y[i])) return fail(AGS_E_ARG, "x and y must be finite");
        if (i > 0 && !(x[i] > x[i - 1])) return fail(AGS_E_ARG, "x must be strictly increasing");
    }
    *index = -1;
    if (n < 3) return AGS_OK;
    double ymin = y[0], ymax = y[0];
    for (int32_t i = 1; i < n; ++i) {
        ymin = y[i] < ymin ? y[i] : ymin;
        ymax = y[i] > ymax ? y[i] : ymax;
    }
    if (ymax == ymin) return AGS_OK;
    const bool flip_x = shape == AGS_KNEE_CONCAVE_DEC || shape == AGS_KNEE_CONVEX_INC;
    const bool flip_y = shape == AGS_KNEE_CONVEX_DEC || shape == AGS_KNEE_CONVEX_INC;
    // Scan the concave increasing form in order of its x.
    std::vector<double> d(n), xs(n);
    std::vector<int32_t> at(n);
    for (int32_t j = 0; j < n; ++j) {
        const int32_t i = flip_x ? n - 1 - j : j;
        const double xn = (x[i] - x[0]) / (x[n - 1] - x[0]);
        const double yn = (y[i] - ymin) / (ymax - ymin);
        const double xt = flip_x ? 1.0 - xn : xn;
        const double yt = flip_y ? 1.0 - yn : yn;
        xs[j] = xt;
        d[j] = yt - xt;
        at[j] = i;
    }
    const double step = sensitivity * (xs[n - 1] - xs[0]) / (n - 1);
    int32_t lmx = -1;
    double threshold = 0.0;
    for (int32_t j = 1; j < n; ++j) {
        if (j < n - 1 && d[j - 1] < d[j] && d[j] >= d[j + 1]) {
            lmx = j;
            threshold = d[j] - step;
            continue;
        }
        if (lmx >= 0 && d[j] < threshold) {
            *index = at[lmx];
            return AGS_OK;
        }
    }
    return AGS_OK;
}

ags_status ags_plan_select(const ags_plan_model* m, const ags_plan_candidate* cand, int32_t n,
                           double epochs, double dataset_size, double price_per_node_hour,
                           double max_local_batch, ags_plan_objective objective,
                           double sensitivity, int32_t* best, double* T_out, double* C_out) {
    ags_status s = check_model(m);
    if (s != AGS_OK) return s;
    if (!best || n < 0 || (n > 0 && !cand)) return fail(AGS_E_ARG, "bad arguments");
    const int32_t obj = raw_enum(objective);
    if (obj < AGS_PLAN_MIN_TIME || obj > AGS_PLAN_KNEE) return fail(AGS_E_ARG, "bad objective");
    if (std::isnan(max_local_batch)) return fail(AGS_E_ARG, "max_local_batch is NaN");
    for (int32_t i = 0; i < n; ++i) {
        if (cand[i].nodes < 1 || cand[i].reserved != 0 || !fin(cand[i].global_batch) ||
            !(cand[i].global_batch > 0))
            return fail(AGS_E_ARG, "candidate: need nodes >= 1, reserved 0, B > 0");
        if (objective == AGS_PLAN_KNEE && i > 0 &&
            (cand[i].nodes != cand[0].nodes || !(cand[i].global_batch > cand[i - 1].global_batch)))
            return fail(AGS_E_ARG, "knee selection needs one cluster size and increasing B");
    }
    std::vector<double> T(n), C(n);
    std::vector<int32_t> feas;
    for (int32_t i = 0; i < n; ++i) {
        double t, c;
        s = ags_plan_time_cost(m, cand[i].nodes, cand[i].global_batch, epochs, dataset_size,
                               price_per_node_hour, &t, &c);
        if (s != AGS_OK) return s;
        const bool ok = cand[i].global_batch / cand[i].nodes <= max_local_batch;
        T[i] = ok ? t : INFINITY;
        C[i] = ok ? c : INFINITY;
        if (ok) feas.push_back(i);
    }
    int32_t pick = -1;
    if (!feas.empty()) {
        if (objective == AGS_PLAN_KNEE) {
            std::vector<double> xb, yt;
            for (int32_t i : feas) {
                xb.push_back(cand[i].global_batch);
                yt.push_back(T[i]);
            }
            int32_t k = -1;
            s = ags_plan_knee(xb.data(), yt.data(), (int32_t)feas.size(), AGS_KNEE_CONVEX_DEC,
                              sensitivity, &k);
            if (s != AGS_OK) return s;
            pick = k >= 0 ? feas[k] : -1;
        } else {
            const std::vector<double>& v = objective == AGS_PLAN_MIN_TIME ? T : C;
            pick = feas[0];
            for (int32_t i : feas)
                if (v[i] < v[pick]) pick = i;
        }
    }
    if (T_out)
        for (int32_t i = 0; i < n; ++i) T_out[i] = T[i];
    if (C_out)
        for (int32_t i = 0; i < n; ++i) C_out[i] = C[i];
    *best = pick;
    return AGS_OK;
}

}  // extern "C"
