// forge_api.cpp -- the C ABI declared in include/forge.h: argument validation (host only,
// before any HIP call), the per-call scalars of Algorithm 1 computed in fp64, and the
// kernel launches.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "forge.h"
#include "forge_internal.h"

using forge_impl::Args;
using forge_impl::Hyper;

namespace {

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;

struct Range {
    uintptr_t lo, hi;   // [lo, hi)
};

bool overlap(Range a, Range b) { return a.lo < b.hi && b.lo < a.hi; }

Range range_of(const void *p, int64_t bytes)
{
    uintptr_t lo = reinterpret_cast<uintptr_t>(p);
    return Range{lo, lo + static_cast<uintptr_t>(bytes)};
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t moment_bytes(int32_t md) { return md == FORGE_MOMENT_F32 ? 4 : md == FORGE_MOMENT_BF16 ? 2 : 1; }

// Moment dtypes with scale tensors (int8 block scales, fp8 amax rings).
bool is_int8(int32_t md)
{
    return md == FORGE_MOMENT_I8 || md == FORGE_MOMENT_I8_ROW64 || md == FORGE_MOMENT_FP8;
}

// Bytes of one int8 scale tensor of a [d_out, d_in] moment.
int64_t scale_bytes(int32_t md, int64_t d_in, int64_t d_out)
{
    if (md == FORGE_MOMENT_I8_ROW64) return d_out * ((d_in + 63) / 64) * 4;
    if (md == FORGE_MOMENT_FP8) return 4 * forge_impl::AMAX_SLOTS;
    return ((d_out + 255) / 256) * d_in * 4;
}

bool finite(float x) { return std::isfinite(x); }

forge_status check_dtype_moment(int32_t md)
{
    return (md == FORGE_MOMENT_F32 || md == FORGE_MOMENT_BF16 || md == FORGE_MOMENT_I8 ||
            md == FORGE_MOMENT_I8_ROW64 || md == FORGE_MOMENT_FP8)
               ? FORGE_OK : FORGE_ERR_INVALID_DTYPE;
}

forge_status check_dtype_grad(int32_t gd)
{
    return (gd == FORGE_GRAD_BF16 || gd == FORGE_GRAD_F32) ? FORGE_OK : FORGE_ERR_INVALID_DTYPE;
}

// Shape rules; `empty` is set when there is nothing to update.
forge_status check_shape(int64_t T, int64_t d_in, int64_t d_out, bool &empty)
{
    if (T < 0 || d_in < 0 || d_out < 0) return FORGE_ERR_INVALID_SHAPE;
    if (d_in % 8 != 0 || d_out % 8 != 0) return FORGE_ERR_UNSUPPORTED_SHAPE;
    if (T > kMaxElems || d_in > kMaxElems || d_out > kMaxElems) return FORGE_ERR_UNSUPPORTED_SHAPE;
    if (d_in * d_out > kMaxElems || T * d_in > kMaxElems || T * d_out > kMaxElems)
        return FORGE_ERR_UNSUPPORTED_SHAPE;
    empty = (d_in == 0 || d_out == 0);
    return FORGE_OK;
}

forge_status check_hyper(float lr, float b1, float b2, float eps, float wd, int64_t step)
{
    if (step < 1) return FORGE_ERR_INVALID_HYPERPARAM;
    if (!finite(lr) || !finite(b1) || !finite(b2) || !finite(eps) || !finite(wd))
        return FORGE_ERR_INVALID_HYPERPARAM;
    if (!(b1 >= 0.0f && b1 < 1.0f) || !(b2 >= 0.0f && b2 < 1.0f)) return FORGE_ERR_INVALID_HYPERPARAM;
    if (!(eps > 0.0f) || !(lr >= 0.0f)) return FORGE_ERR_INVALID_HYPERPARAM;
    return FORGE_OK;
}

// Per-call scalars in fp64, rounded once to fp32 (Algorithm 1: bias corrections and the
// decoupled decay factor).
Hyper make_hyper(float lr, float b1, float b2, float eps, float wd, int64_t step)
{
    const double t = static_cast<double>(step);
    const double bc1 = 1.0 - std::pow(static_cast<double>(b1), t);
    const double bc2 = 1.0 - std::pow(static_cast<double>(b2), t);
    Hyper h;
    h.b1 = b1;
    h.c1 = static_cast<float>(1.0 - static_cast<double>(b1));
    h.b2 = b2;
    h.c2 = static_cast<float>(1.0 - static_cast<double>(b2));
    h.lr_bc1 = static_cast<float>(static_cast<double>(lr) / bc1);
    h.inv_sqrt_bc2 = static_cast<float>(1.0 / std::sqrt(bc2));
    h.eps = eps;
    h.wdf = static_cast<float>(1.0 - static_cast<double>(lr) * static_cast<double>(wd));
    return h;
}

// The optimizer-state tensors of one step: pointers, alignment and mutual disjointness.
// At most W, m, v, two scale tensors (or amax rings) and the weight's amax ring.
struct StateSet {
    static constexpr int CAP = 8;
    Range r[CAP];
    int n = 0;
    void add(Range x)
    {
        if (n < CAP) r[n++] = x;
    }
};

forge_status check_state(void *W, void *m, void *v, float *ms, float *vs, int64_t d_in,
                         int64_t d_out, int32_t md, StateSet &out)
{
    if (!W || !m || !v) return FORGE_ERR_NULL_POINTER;
    const bool i8 = is_int8(md);
    if (i8 && (!ms || !vs)) return FORGE_ERR_NULL_POINTER;
    if (!aligned16(W) || !aligned16(m) || !aligned16(v)) return FORGE_ERR_MISALIGNED;
    if (i8 && (!aligned16(ms) || !aligned16(vs))) return FORGE_ERR_MISALIGNED;
    const int64_t P = d_in * d_out;
    out.r[0] = range_of(W, 2 * P);
    out.r[1] = range_of(m, moment_bytes(md) * P);
    out.r[2] = range_of(v, moment_bytes(md) * P);
    out.n = 3;
    if (i8) {
        const int64_t nsc = scale_bytes(md, d_in, d_out);
        out.r[3] = range_of(ms, nsc);
        out.r[4] = range_of(vs, nsc);
        out.n = 5;
    }
    for (int i = 0; i < out.n; ++i)
        for (int j = i + 1; j < out.n; ++j)
            if (overlap(out.r[i], out.r[j])) return FORGE_ERR_ALIASING;
    return FORGE_OK;
}

bool disjoint_from(const StateSet &s, Range x)
{
    for (int i = 0; i < s.n; ++i)
        if (overlap(s.r[i], x)) return false;
    return true;
}

forge_status check_inputs(const void *X, const void *dY, int64_t T, int64_t d_in, int64_t d_out)
{
    if (T == 0) return FORGE_OK;
    if (!X || !dY) return FORGE_ERR_NULL_POINTER;
    if (!aligned16(X) || !aligned16(dY)) return FORGE_ERR_MISALIGNED;
    (void)d_in;
    (void)d_out;
    return FORGE_OK;
}

// The current device must be a gfx950; the answer is cached per device ordinal.
forge_status check_device()
{
    static std::mutex mu;
    static int known[64] = {0};   // 0 unknown, 1 ok, 2 not ok
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
        (void)hipGetLastError();
        return FORGE_ERR_NO_DEVICE;
    }
    if (dev >= 64) return FORGE_ERR_NO_DEVICE;
    std::lock_guard<std::mutex> lock(mu);
    if (known[dev] == 0) {
        hipDeviceProp_t prop;
        if (hipGetDeviceProperties(&prop, dev) != hipSuccess) {
            (void)hipGetLastError();
            return FORGE_ERR_NO_DEVICE;
        }
        known[dev] = (std::strncmp(prop.gcnArchName, "gfx950", 6) == 0) ? 1 : 2;
    }
    return known[dev] == 1 ? FORGE_OK : FORGE_ERR_NO_DEVICE;
}

forge_status from_hip(hipError_t e)
{
    if (e == hipSuccess) return FORGE_OK;
    if (e == hipErrorNoDevice || e == hipErrorInvalidDevice) return FORGE_ERR_NO_DEVICE;
    return FORGE_ERR_LAUNCH;
}

Args base_args(const void *X, const void *dY, int64_t T, int64_t d_in, int64_t d_out)
{
    Args a;
    std::memset(&a, 0, sizeof a);
    a.X = static_cast<const uint16_t *>(X);
    a.dY = static_cast<const uint16_t *>(dY);
    a.T = static_cast<int>(T);
    a.d_in = static_cast<int>(d_in);
    a.d_out = static_cast<int>(d_out);
    return a;
}

// The validated launch arguments of a grouped step (empty matrices dropped).
struct GroupPlan {
    StateSet st[FORGE_MAX_GROUP];
    int live[FORGE_MAX_GROUP];
    int nlive = 0;
    Args args[FORGE_MAX_GROUP];
};

// Validation of forge_linear_step_grouped after the dtype, mats and n checks: each matrix,
// then (if any is non-empty) the hyper-parameters and the aliasing rules.
forge_status plan_group(const forge_matrix *mats, int32_t n, int64_t T, int32_t md, float lr,
                        float beta1, float beta2, float eps, float weight_decay, int64_t step,
                        GroupPlan &g)
{
    forge_status s;
    g.nlive = 0;
    for (int i = 0; i < n; ++i) {
        const forge_matrix &x = mats[i];
        bool empty = false;
        if ((s = check_shape(T, x.d_in, x.d_out, empty)) != FORGE_OK) return s;
        if (empty) continue;
        if ((s = check_inputs(x.X, x.dY, T, x.d_in, x.d_out)) != FORGE_OK) return s;
        if ((s = check_state(x.W, x.m, x.v, x.m_scale, x.v_scale, x.d_in, x.d_out, md, g.st[g.nlive])) !=
            FORGE_OK)
            return s;
        g.live[g.nlive++] = i;
    }
    if (g.nlive == 0) return FORGE_OK;
    if ((s = check_hyper(lr, beta1, beta2, eps, weight_decay, step)) != FORGE_OK) return s;
    for (int a = 0; a < g.nlive; ++a) {
        for (int b = 0; b < g.nlive; ++b) {
            const forge_matrix &y = mats[g.live[b]];
            if (T > 0 && (!disjoint_from(g.st[a], range_of(y.X, 2 * T * y.d_in)) ||
                          !disjoint_from(g.st[a], range_of(y.dY, 2 * T * y.d_out))))
                return FORGE_ERR_ALIASING;
            if (b > a)
                for (int k = 0; k < g.st[b].n; ++k)
                    if (!disjoint_from(g.st[a], g.st[b].r[k])) return FORGE_ERR_ALIASING;
        }
    }
    const Hyper h = make_hyper(lr, beta1, beta2, eps, weight_decay, step);
    for (int k = 0; k < g.nlive; ++k) {
        const forge_matrix &x = mats[g.live[k]];
        Args &a = g.args[k];
        a = base_args(x.X, x.dY, T, x.d_in, x.d_out);
        a.W = static_cast<uint16_t *>(x.W);
        a.m = x.m;
        a.v = x.v;
        a.ms = x.m_scale;
        a.vs = x.v_scale;
        a.h = h;
        a.slot = static_cast<int>(step % forge_impl::AMAX_SLOTS);
    }
    return FORGE_OK;
}

// ----------------------------------------------------------------- update rules

struct RuleInfo {
    int epi;        // forge_impl::EpiKind
    int nstate;     // state tensors read and written
    bool uses_w;    // reads and writes W
};

bool rule_info(int32_t opt, RuleInfo &r)
{
    using namespace forge_impl;
    switch (opt) {
    case FORGE_OPT_ADAMW: r = {EPI_ADAMW, 2, true}; return true;
    case FORGE_OPT_SGD: r = {EPI_SGD, 0, true}; return true;
    case FORGE_OPT_SGD_MOMENTUM: r = {EPI_SGDM, 1, true}; return true;
    case FORGE_OPT_ADAGRAD: r = {EPI_ADAGRAD, 1, true}; return true;
    case FORGE_OPT_RMSPROP: r = {EPI_RMSPROP, 1, true}; return true;
    case FORGE_OPT_LION: r = {EPI_LION, 1, true}; return true;
    case FORGE_OPT_NADAM: r = {EPI_NADAM, 2, true}; return true;
    case FORGE_OPT_RADAM: r = {EPI_RADAM, 2, true}; return true;
    case FORGE_OPT_ADAMAX: r = {EPI_ADAMAX, 2, true}; return true;
    case FORGE_OPT_MUON_ACCUMULATE: r = {EPI_MUON, 1, false}; return true;
    default: return false;
    }
}

bool unit_open(float b) { return finite(b) && b >= 0.0f && b < 1.0f; }

// The fields each rule reads must be in range (see forge.h).
forge_status check_rule_hyper(int32_t opt, const forge_hparams &p, int64_t step)
{
    if (step < 1) return FORGE_ERR_INVALID_HYPERPARAM;
    if (!finite(p.lr) || !(p.lr >= 0.0f) || !finite(p.weight_decay)) return FORGE_ERR_INVALID_HYPERPARAM;
    const bool eps_ok = finite(p.eps) && p.eps > 0.0f;
    bool ok = true;
    switch (opt) {
    case FORGE_OPT_ADAMW:
    case FORGE_OPT_RADAM:
    case FORGE_OPT_ADAMAX: ok = unit_open(p.beta1) && unit_open(p.beta2) && eps_ok; break;
    case FORGE_OPT_NADAM:
        ok = unit_open(p.beta1) && unit_open(p.beta2) && eps_ok && finite(p.momentum_decay) &&
             p.momentum_decay >= 0.0f;
        break;
    case FORGE_OPT_SGD: break;
    case FORGE_OPT_SGD_MOMENTUM: ok = unit_open(p.beta1); break;
    case FORGE_OPT_ADAGRAD: ok = eps_ok && finite(p.lr_decay) && p.lr_decay >= 0.0f; break;
    case FORGE_OPT_RMSPROP: ok = unit_open(p.beta2) && eps_ok; break;
    case FORGE_OPT_LION: ok = unit_open(p.beta1) && unit_open(p.beta2); break;
    case FORGE_OPT_MUON_ACCUMULATE: ok = finite(p.beta1) && p.beta1 >= 0.0f && p.beta1 <= 1.0f; break;
    default: ok = false;
    }
    return ok ? FORGE_OK : FORGE_ERR_INVALID_HYPERPARAM;
}

// Per-call scalars of a rule, in fp64, rounded once to fp32 (the formulas of forge.h).
Hyper make_rule_hyper(int32_t opt, const forge_hparams &p, int64_t step)
{
    if (opt == FORGE_OPT_ADAMW) return make_hyper(p.lr, p.beta1, p.beta2, p.eps, p.weight_decay, step);
    const double t = static_cast<double>(step);
    const double lr = p.lr, b1 = p.beta1, b2 = p.beta2, wd = p.weight_decay;
    const double bc1 = 1.0 - std::pow(b1, t), bc2 = 1.0 - std::pow(b2, t);
    Hyper h;
    std::memset(&h, 0, sizeof h);
    h.b1 = p.beta1;
    h.c1 = static_cast<float>(1.0 - b1);
    h.b2 = p.beta2;
    h.c2 = static_cast<float>(1.0 - b2);
    h.eps = p.eps;
    h.lr = p.lr;
    h.wd = p.weight_decay;
    h.wdf = static_cast<float>(1.0 - lr * wd);
    switch (opt) {
    case FORGE_OPT_ADAGRAD: h.lr = static_cast<float>(lr / (1.0 + (t - 1.0) * p.lr_decay)); break;
    case FORGE_OPT_NADAM: {
        const double psi = p.momentum_decay;
        auto mu = [&](double i) { return b1 * (1.0 - 0.5 * std::pow(0.96, i * psi)); };
        double prod = 1.0;
        for (int64_t i = 1; i <= step; ++i) prod *= mu(static_cast<double>(i));
        const double mu_t = mu(t), mu_n = mu(t + 1.0);
        h.inv_sqrt_bc2 = static_cast<float>(1.0 / std::sqrt(bc2));
        h.ka = static_cast<float>(lr * (1.0 - mu_t) / (1.0 - prod));
        h.kb = static_cast<float>(lr * mu_n / (1.0 - prod * mu_n));
        break;
    }
    case FORGE_OPT_RADAM: {
        const double rho_inf = 2.0 / (1.0 - b2) - 1.0;
        const double rho_t = rho_inf - 2.0 * t * std::pow(b2, t) / bc2;
        if (rho_t > 5.0) {
            const double r = std::sqrt((rho_t - 4.0) * (rho_t - 2.0) * rho_inf /
                                       ((rho_inf - 4.0) * (rho_inf - 2.0) * rho_t));
            h.ka = static_cast<float>(lr * r * std::sqrt(bc2) / bc1);
            h.kb = 0.0f;
        } else {
            h.ka = 0.0f;
            h.kb = static_cast<float>(lr / bc1);
        }
        break;
    }
    case FORGE_OPT_ADAMAX: h.lr_bc1 = static_cast<float>(lr / bc1); break;
    default: break;
    }
    return h;
}

}  // namespace

extern "C" {

const char *forge_status_string(int32_t s)
{
    switch (s) {
    case FORGE_OK: return "FORGE_OK: success";
    case FORGE_ERR_NULL_POINTER: return "FORGE_ERR_NULL_POINTER: a required pointer is NULL";
    case FORGE_ERR_INVALID_SHAPE: return "FORGE_ERR_INVALID_SHAPE: a size is negative";
    case FORGE_ERR_UNSUPPORTED_SHAPE:
        return "FORGE_ERR_UNSUPPORTED_SHAPE: d_in and d_out must be multiples of 8 and every tensor below 2^31 elements";
    case FORGE_ERR_INVALID_HYPERPARAM:
        return "FORGE_ERR_INVALID_HYPERPARAM: need step >= 1, 0 <= beta < 1, eps > 0, lr >= 0, all finite";
    case FORGE_ERR_INVALID_DTYPE: return "FORGE_ERR_INVALID_DTYPE: unknown moment or gradient dtype code";
    case FORGE_ERR_MISALIGNED: return "FORGE_ERR_MISALIGNED: tensor pointers must be 16-byte aligned";
    case FORGE_ERR_ALIASING: return "FORGE_ERR_ALIASING: an output tensor overlaps another tensor";
    case FORGE_ERR_NO_DEVICE: return "FORGE_ERR_NO_DEVICE: no gfx950 device is current";
    case FORGE_ERR_LAUNCH: return "FORGE_ERR_LAUNCH: kernel launch failed";
    case FORGE_ERR_INVALID_OPTIMIZER: return "FORGE_ERR_INVALID_OPTIMIZER: unknown optimizer code";
    case FORGE_ERR_SCRATCH_LIMIT:
        return "FORGE_ERR_SCRATCH_LIMIT: the gradient does not fit the library's fixed FORGE_SCRATCH_BYTES buffer";
    default: return "unknown forge_status";
    }
}

forge_status forge_query_tile(int64_t T, int64_t d_in, int64_t d_out, int32_t md, int32_t *rows,
                              int32_t *cols, int32_t *tokens)
{
    if (check_dtype_moment(md) != FORGE_OK) return FORGE_ERR_INVALID_DTYPE;
    if (T < 0 || d_in < 0 || d_out < 0) return FORGE_ERR_INVALID_SHAPE;
    const forge_impl::TileShape t = forge_impl::tile_shape(md);   // one tile per moment kind, any shape
    if (rows) *rows = t.rows;
    if (cols) *cols = t.cols;
    if (tokens) *tokens = t.tokens;
    return FORGE_OK;
}

forge_status forge_linear_step(const void *X, const void *dY, void *W, void *m, void *v,
                               float *m_scale, float *v_scale, int64_t T, int64_t d_in,
                               int64_t d_out, int32_t md, float lr, float beta1, float beta2,
                               float eps, float weight_decay, int64_t step, void *stream)
{
    forge_status s;
    bool empty = false;
    if ((s = check_dtype_moment(md)) != FORGE_OK) return s;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    StateSet st;
    if ((s = check_inputs(X, dY, T, d_in, d_out)) != FORGE_OK) return s;
    if ((s = check_state(W, m, v, m_scale, v_scale, d_in, d_out, md, st)) != FORGE_OK) return s;
    if ((s = check_hyper(lr, beta1, beta2, eps, weight_decay, step)) != FORGE_OK) return s;
    if (T > 0 && (!disjoint_from(st, range_of(X, 2 * T * d_in)) ||
                  !disjoint_from(st, range_of(dY, 2 * T * d_out))))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;

    Args a = base_args(X, dY, T, d_in, d_out);
    a.W = static_cast<uint16_t *>(W);
    a.m = m;
    a.v = v;
    a.ms = m_scale;
    a.vs = v_scale;
    a.h = make_hyper(lr, beta1, beta2, eps, weight_decay, step);
    a.slot = static_cast<int>(step % forge_impl::AMAX_SLOTS);
    return from_hip(forge_impl::launch_fused(a, md, static_cast<hipStream_t>(stream)));
}

static_assert(FORGE_MAX_GROUP == forge_impl::MAX_GROUP, "group bound of the ABI and the kernels");

forge_status forge_linear_step_grouped(const forge_matrix *mats, int32_t n, int64_t T, int32_t md,
                                       float lr, float beta1, float beta2, float eps,
                                       float weight_decay, int64_t step, void *stream)
{
    forge_status s;
    if ((s = check_dtype_moment(md)) != FORGE_OK) return s;
    if (!mats) return FORGE_ERR_NULL_POINTER;
    if (n < 1 || n > FORGE_MAX_GROUP) return FORGE_ERR_INVALID_SHAPE;
    GroupPlan g;
    if ((s = plan_group(mats, n, T, md, lr, beta1, beta2, eps, weight_decay, step, g)) != FORGE_OK) return s;
    if (g.nlive == 0) return FORGE_OK;
    if ((s = check_device()) != FORGE_OK) return s;
    return from_hip(forge_impl::launch_fused_group(g.args, g.nlive, md, static_cast<hipStream_t>(stream)));
}

forge_status forge_linear_step_wfp8(const void *X, const void *dY, void *W, float *w_amax, void *m, void *v,
                                    float *m_amax, float *v_amax, int64_t T, int64_t d_in, int64_t d_out,
                                    int32_t md, float lr, float beta1, float beta2, float eps,
                                    float weight_decay, int64_t step, void *stream)
{
    forge_status s;
    bool empty = false;
    if (md != FORGE_MOMENT_BF16 && md != FORGE_MOMENT_FP8) return FORGE_ERR_INVALID_DTYPE;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    if ((s = check_inputs(X, dY, T, d_in, d_out)) != FORGE_OK) return s;
    const bool f8 = (md == FORGE_MOMENT_FP8);
    if (!W || !w_amax || !m || !v || (f8 && (!m_amax || !v_amax))) return FORGE_ERR_NULL_POINTER;
    if (!aligned16(W) || !aligned16(w_amax) || !aligned16(m) || !aligned16(v) ||
        (f8 && (!aligned16(m_amax) || !aligned16(v_amax))))
        return FORGE_ERR_MISALIGNED;
    const int64_t P = d_in * d_out, ring = 4 * forge_impl::AMAX_SLOTS;
    StateSet st;
    st.add(range_of(W, P));
    st.add(range_of(m, moment_bytes(md) * P));
    st.add(range_of(v, moment_bytes(md) * P));
    if (f8) {
        st.add(range_of(m_amax, ring));
        st.add(range_of(v_amax, ring));
    }
    const Range rw = range_of(w_amax, ring);
    for (int i = 0; i < st.n; ++i) {
        if (overlap(st.r[i], rw)) return FORGE_ERR_ALIASING;
        for (int j = i + 1; j < st.n; ++j)
            if (overlap(st.r[i], st.r[j])) return FORGE_ERR_ALIASING;
    }
    st.add(rw);
    if ((s = check_hyper(lr, beta1, beta2, eps, weight_decay, step)) != FORGE_OK) return s;
    if (T > 0 && (!disjoint_from(st, range_of(X, 2 * T * d_in)) || !disjoint_from(st, range_of(dY, 2 * T * d_out))))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;

    Args a = base_args(X, dY, T, d_in, d_out);
    a.W = static_cast<uint16_t *>(W);          // fp8 codes; the kernel reads it as bytes
    a.wr = w_amax;
    a.m = m;
    a.v = v;
    a.ms = f8 ? m_amax : nullptr;
    a.vs = f8 ? v_amax : nullptr;
    a.h = make_hyper(lr, beta1, beta2, eps, weight_decay, step);
    a.slot = static_cast<int>(step % forge_impl::AMAX_SLOTS);
    return from_hip(forge_impl::launch_fused_wfp8(&a, 1, md, static_cast<hipStream_t>(stream)));
}

forge_status forge_input_grad(const void *dY, const void *W, void *dX, int64_t T, int64_t d_in,
                              int64_t d_out, void *stream)
{
    forge_status s;
    bool empty = false;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (T == 0 || d_in == 0) return FORGE_OK;
    if (!dX) return FORGE_ERR_NULL_POINTER;
    if (d_out > 0 && (!dY || !W)) return FORGE_ERR_NULL_POINTER;
    if (!aligned16(dX)) return FORGE_ERR_MISALIGNED;
    if (d_out > 0 && (!aligned16(dY) || !aligned16(W))) return FORGE_ERR_MISALIGNED;
    const Range rdx = range_of(dX, 2 * T * d_in);
    if (d_out > 0 && (overlap(rdx, range_of(dY, 2 * T * d_out)) || overlap(rdx, range_of(W, 2 * d_in * d_out))))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;
    const forge_impl::DxSeg seg{static_cast<const uint16_t *>(dY), static_cast<const uint16_t *>(W),
                                static_cast<int>(d_out)};
    return from_hip(forge_impl::launch_dx(&seg, d_out > 0 ? 1 : 0, static_cast<uint16_t *>(dX),
                                          static_cast<int>(T), static_cast<int>(d_in),
                                          static_cast<hipStream_t>(stream)));
}

forge_status forge_linear_backward_grouped(const forge_matrix *mats, int32_t n, int64_t T, void *dX,
                                           int32_t md, float lr, float beta1, float beta2, float eps,
                                           float weight_decay, int64_t step, void *stream)
{
    forge_status s;
    if ((s = check_dtype_moment(md)) != FORGE_OK) return s;
    if (!mats) return FORGE_ERR_NULL_POINTER;
    if (n < 1 || n > FORGE_MAX_GROUP) return FORGE_ERR_INVALID_SHAPE;
    const int64_t d_in = mats[0].d_in;
    for (int i = 1; i < n; ++i)
        if (mats[i].d_in != d_in) return FORGE_ERR_INVALID_SHAPE;
    GroupPlan g;
    if ((s = plan_group(mats, n, T, md, lr, beta1, beta2, eps, weight_decay, step, g)) != FORGE_OK) return s;
    const bool has_dx = T > 0 && d_in > 0;
    if (has_dx) {
        if (!dX) return FORGE_ERR_NULL_POINTER;
        if (!aligned16(dX)) return FORGE_ERR_MISALIGNED;
        const Range rdx = range_of(dX, 2 * T * d_in);
        for (int k = 0; k < g.nlive; ++k) {
            const forge_matrix &x = mats[g.live[k]];
            if (!disjoint_from(g.st[k], rdx) || overlap(rdx, range_of(x.X, 2 * T * x.d_in)) ||
                overlap(rdx, range_of(x.dY, 2 * T * x.d_out)))
                return FORGE_ERR_ALIASING;
        }
    }
    if (!has_dx && g.nlive == 0) return FORGE_OK;
    if ((s = check_device()) != FORGE_OK) return s;
    const hipStream_t st = static_cast<hipStream_t>(stream);
    if (has_dx) {
        // dX from the weights as they are before this step (the fused launch below, later in
        // stream order, overwrites them).  Members with d_out == 0 add nothing to the sum.
        forge_impl::DxSeg seg[FORGE_MAX_GROUP];
        for (int k = 0; k < g.nlive; ++k)
            seg[k] = forge_impl::DxSeg{g.args[k].dY, g.args[k].W, g.args[k].d_out};
        if ((s = from_hip(forge_impl::launch_dx(seg, g.nlive, static_cast<uint16_t *>(dX), static_cast<int>(T),
                                                static_cast<int>(d_in), st))) != FORGE_OK)
            return s;
    }
    if (g.nlive == 0) return FORGE_OK;
    return from_hip(forge_impl::launch_fused_group(g.args, g.nlive, md, st));
}

forge_status forge_linear_backward(const void *X, const void *dY, void *W, void *m, void *v,
                                   float *m_scale, float *v_scale, void *dX, int64_t T, int64_t d_in,
                                   int64_t d_out, int32_t md, float lr, float beta1, float beta2,
                                   float eps, float weight_decay, int64_t step, void *stream)
{
    const forge_matrix x{X, dY, W, m, v, m_scale, v_scale, d_in, d_out};
    return forge_linear_backward_grouped(&x, 1, T, dX, md, lr, beta1, beta2, eps, weight_decay, step,
                                         stream);
}

forge_status forge_linear_step_opt(const void *X, const void *dY, void *W, void *s1, void *s2, int64_t T,
                                   int64_t d_in, int64_t d_out, int32_t opt, int32_t md,
                                   const forge_hparams *hp, int64_t step, void *stream)
{
    forge_status s;
    bool empty = false;
    RuleInfo r;
    if (!rule_info(opt, r)) return FORGE_ERR_INVALID_OPTIMIZER;
    if (md != FORGE_MOMENT_F32 && md != FORGE_MOMENT_BF16) return FORGE_ERR_INVALID_DTYPE;
    if (!hp) return FORGE_ERR_NULL_POINTER;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    if ((s = check_inputs(X, dY, T, d_in, d_out)) != FORGE_OK) return s;
    void *t[3] = {r.uses_w ? W : nullptr, r.nstate >= 1 ? s1 : nullptr, r.nstate >= 2 ? s2 : nullptr};
    const bool need[3] = {r.uses_w, r.nstate >= 1, r.nstate >= 2};
    const int64_t P = d_in * d_out;
    const int64_t bytes[3] = {2 * P, moment_bytes(md) * P, moment_bytes(md) * P};
    StateSet st;
    for (int k = 0; k < 3; ++k) {
        if (!need[k]) continue;
        if (!t[k]) return FORGE_ERR_NULL_POINTER;
        if (!aligned16(t[k])) return FORGE_ERR_MISALIGNED;
        st.add(range_of(t[k], bytes[k]));
    }
    for (int i = 0; i < st.n; ++i)
        for (int j = i + 1; j < st.n; ++j)
            if (overlap(st.r[i], st.r[j])) return FORGE_ERR_ALIASING;
    if ((s = check_rule_hyper(opt, *hp, step)) != FORGE_OK) return s;
    if (T > 0 && (!disjoint_from(st, range_of(X, 2 * T * d_in)) || !disjoint_from(st, range_of(dY, 2 * T * d_out))))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;

    Args a = base_args(X, dY, T, d_in, d_out);
    a.W = static_cast<uint16_t *>(t[0]);
    a.m = t[1];
    a.v = t[2];
    a.h = make_rule_hyper(opt, *hp, step);
    return from_hip(forge_impl::launch_fused_rule(&a, 1, r.epi, md, static_cast<hipStream_t>(stream)));
}

forge_status forge_wgrad(const void *X, const void *dY, void *G, int64_t T, int64_t d_in,
                         int64_t d_out, int32_t gd, void *stream)
{
    forge_status s;
    bool empty = false;
    if ((s = check_dtype_grad(gd)) != FORGE_OK) return s;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    if ((s = check_inputs(X, dY, T, d_in, d_out)) != FORGE_OK) return s;
    if (!G) return FORGE_ERR_NULL_POINTER;
    if (!aligned16(G)) return FORGE_ERR_MISALIGNED;
    const Range rg = range_of(G, (gd == FORGE_GRAD_F32 ? 4 : 2) * d_in * d_out);
    if (T > 0 && (overlap(rg, range_of(X, 2 * T * d_in)) || overlap(rg, range_of(dY, 2 * T * d_out))))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;

    Args a = base_args(X, dY, T, d_in, d_out);
    a.G = G;
    return from_hip(forge_impl::launch_wgrad(a, gd == FORGE_GRAD_F32, static_cast<hipStream_t>(stream)));
}

forge_status forge_adamw(const void *G, int32_t gd, void *W, void *m, void *v, float *m_scale,
                         float *v_scale, int64_t d_in, int64_t d_out, int32_t md, float lr,
                         float beta1, float beta2, float eps, float weight_decay, int64_t step,
                         void *stream)
{
    forge_status s;
    bool empty = false;
    if ((s = check_dtype_moment(md)) != FORGE_OK) return s;
    if (md == FORGE_MOMENT_FP8) return FORGE_ERR_INVALID_DTYPE;
    if ((s = check_dtype_grad(gd)) != FORGE_OK) return s;
    if ((s = check_shape(0, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    if (!G) return FORGE_ERR_NULL_POINTER;
    StateSet st;
    if ((s = check_state(W, m, v, m_scale, v_scale, d_in, d_out, md, st)) != FORGE_OK) return s;
    if (!aligned16(G)) return FORGE_ERR_MISALIGNED;
    if ((s = check_hyper(lr, beta1, beta2, eps, weight_decay, step)) != FORGE_OK) return s;
    if (!disjoint_from(st, range_of(G, (gd == FORGE_GRAD_F32 ? 4 : 2) * d_in * d_out)))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;

    Args a = base_args(nullptr, nullptr, 0, d_in, d_out);
    a.G = const_cast<void *>(G);
    a.W = static_cast<uint16_t *>(W);
    a.m = m;
    a.v = v;
    a.ms = m_scale;
    a.vs = v_scale;
    a.h = make_hyper(lr, beta1, beta2, eps, weight_decay, step);
    return from_hip(forge_impl::launch_adamw(a, md, gd == FORGE_GRAD_F32, static_cast<hipStream_t>(stream)));
}

forge_status forge_linear_step_unfused(const void *X, const void *dY, void *W, void *m, void *v,
                                       float *m_scale, float *v_scale, int64_t T, int64_t d_in,
                                       int64_t d_out, int32_t md, float lr, float beta1,
                                       float beta2, float eps, float weight_decay, int64_t step,
                                       void *G_ws, int32_t gd, void *stream)
{
    forge_status s;
    bool empty = false;
    if ((s = check_dtype_moment(md)) != FORGE_OK) return s;
    if (md == FORGE_MOMENT_FP8) return FORGE_ERR_INVALID_DTYPE;
    if ((s = check_dtype_grad(gd)) != FORGE_OK) return s;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    StateSet st;
    if ((s = check_inputs(X, dY, T, d_in, d_out)) != FORGE_OK) return s;
    if ((s = check_state(W, m, v, m_scale, v_scale, d_in, d_out, md, st)) != FORGE_OK) return s;
    if (!G_ws) return FORGE_ERR_NULL_POINTER;
    if (!aligned16(G_ws)) return FORGE_ERR_MISALIGNED;
    if ((s = check_hyper(lr, beta1, beta2, eps, weight_decay, step)) != FORGE_OK) return s;
    const Range rg = range_of(G_ws, (gd == FORGE_GRAD_F32 ? 4 : 2) * d_in * d_out);
    if (!disjoint_from(st, rg)) return FORGE_ERR_ALIASING;
    if (T > 0) {
        const Range rx = range_of(X, 2 * T * d_in), ry = range_of(dY, 2 * T * d_out);
        if (!disjoint_from(st, rx) || !disjoint_from(st, ry) || overlap(rg, rx) || overlap(rg, ry))
            return FORGE_ERR_ALIASING;
    }
    if ((s = forge_wgrad(X, dY, G_ws, T, d_in, d_out, gd, stream)) != FORGE_OK) return s;
    return forge_adamw(G_ws, gd, W, m, v, m_scale, v_scale, d_in, d_out, md, lr, beta1, beta2,
                       eps, weight_decay, step, stream);
}

static_assert(FORGE_SCRATCH_BYTES == forge_impl::SCRATCH_BYTES, "scratch size of the ABI and the library");

forge_status forge_linear_step_unfused_noalloc(const void *X, const void *dY, void *W, void *m, void *v,
                                               float *m_scale, float *v_scale, int64_t T, int64_t d_in,
                                               int64_t d_out, int32_t md, float lr, float beta1, float beta2,
                                               float eps, float weight_decay, int64_t step, int32_t gd,
                                               void *stream)
{
    forge_status s;
    bool empty = false;
    if ((s = check_dtype_moment(md)) != FORGE_OK) return s;
    if (md == FORGE_MOMENT_FP8) return FORGE_ERR_INVALID_DTYPE;
    if ((s = check_dtype_grad(gd)) != FORGE_OK) return s;
    if ((s = check_shape(T, d_in, d_out, empty)) != FORGE_OK) return s;
    if (empty) return FORGE_OK;
    const int64_t g_bytes = (gd == FORGE_GRAD_F32 ? 4 : 2) * d_in * d_out;
    if (g_bytes > FORGE_SCRATCH_BYTES) return FORGE_ERR_SCRATCH_LIMIT;
    StateSet st;
    if ((s = check_inputs(X, dY, T, d_in, d_out)) != FORGE_OK) return s;
    if ((s = check_state(W, m, v, m_scale, v_scale, d_in, d_out, md, st)) != FORGE_OK) return s;
    if ((s = check_hyper(lr, beta1, beta2, eps, weight_decay, step)) != FORGE_OK) return s;
    if (T > 0 && (!disjoint_from(st, range_of(X, 2 * T * d_in)) || !disjoint_from(st, range_of(dY, 2 * T * d_out))))
        return FORGE_ERR_ALIASING;
    if ((s = check_device()) != FORGE_OK) return s;
    void *G = nullptr;
    if (forge_impl::scratch_address(&G) != hipSuccess) {
        (void)hipGetLastError();
        return FORGE_ERR_LAUNCH;
    }
    // The library's buffer is disjoint from every caller tensor; the two calls below
    // validate again (cheaply) and launch the GEMM, then the optimizer, on `stream`.
    if ((s = forge_wgrad(X, dY, G, T, d_in, d_out, gd, stream)) != FORGE_OK) return s;
    return forge_adamw(G, gd, W, m, v, m_scale, v_scale, d_in, d_out, md, lr, beta1, beta2, eps, weight_decay,
                       step, stream);
}

}  // extern "C"
