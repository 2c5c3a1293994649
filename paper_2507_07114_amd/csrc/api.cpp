// C ABI of the lossy step (declared in include/lossy.h): argument checks,
// launch geometry and error reporting around the HIP kernels.
#include "lossy.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>

#include "kernels.h"

using namespace lossy;

static_assert(sizeof(ll_drift) == sizeof(DriftOut), "ll_drift layout");
static_assert(sizeof(DriftPartial) == 32, "partial layout");
static_assert(sizeof(DriftAcc) == 40, "second-level partial layout");
static_assert((size_t)LL_NOALLOC_SCRATCH_BYTES == kNoAllocScratchBytes, "static scratch size");
static_assert(LL_PACE_AUTO == kPaceAuto && LL_PACE_ALWAYS == kPaceAlways &&
                  LL_PACE_NEVER == kPaceNever,
              "pacing modes");

namespace {

thread_local std::string g_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

int ok() {
    g_error.clear();
    return LL_OK;
}

int hip_check(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(LL_EHIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// ceil(p * 2^32): hi32(w) < thr  <=>  hi32(w) / 2^32 < p.
uint64_t threshold(double p) { return (uint64_t)std::ceil(p * 4294967296.0); }

bool prob_ok(double p) { return p >= 0.0 && p <= 1.0; }

// Packets and the largest per-packet grid any element type can need (the
// smallest workgroup, kMinPacketThreads, gives the most chunks per packet);
// drift partials and grid limits are sized for that worst case.
struct Geometry {
    int64_t P = 0;
    int64_t blocks = 0;
};

// Shared checks of (n, d, packet); fills the launch geometry.
int check_shape(int32_t n, int64_t d, int64_t packet, Geometry* g) {
    if (n < 1 || n > kMaxWorkers) return fail(LL_EINVAL, "n=%d outside [1, %d]", n, kMaxWorkers);
    if (d < 0) return fail(LL_EINVAL, "d=%lld is negative", (long long)d);
    if (packet < 1) return fail(LL_EINVAL, "packet=%lld must be at least 1", (long long)packet);
    g->P = (d + packet - 1) / packet;
    const int64_t chunk = (int64_t)kMinPacketThreads * kElems;
    g->blocks = g->P * ((packet + chunk - 1) / chunk);
    if (g->blocks > 0x7FFFFFFFll)
        return fail(LL_EINVAL, "too many workgroups (%lld)", (long long)g->blocks);
    return LL_OK;
}

size_t elem_bytes(int32_t dtype) { return dtype == LL_BF16 ? 2 : 4; }

// Rows [n][ld] of elements of `esize` bytes: every row starts on a 16-byte
// boundary when the base does and ld * esize is a multiple of 16.
int check_rows(const char* name, const void* p, int64_t ld, int64_t d, size_t esize) {
    if (!p) return fail(LL_EINVAL, "%s is NULL", name);
    if (ld < d) return fail(LL_EINVAL, "%s: ld=%lld < d=%lld", name, (long long)ld, (long long)d);
    if (((size_t)ld * esize) % 16 != 0)
        return fail(LL_EALIGN, "%s: ld=%lld elements of %zu bytes is not a multiple of 16 bytes",
                    name, (long long)ld, esize);
    if (!aligned16(p)) return fail(LL_EALIGN, "%s is not 16-byte aligned", name);
    return LL_OK;
}

int check_vec(const char* name, const void* p, bool required) {
    if (!p) return required ? fail(LL_EINVAL, "%s is NULL", name) : LL_OK;
    if (!aligned16(p)) return fail(LL_EALIGN, "%s is not 16-byte aligned", name);
    return LL_OK;
}

int check_dtype(const char* name, int32_t t) {
    if (t != LL_F32 && t != LL_BF16) return fail(LL_EINVAL, "%s: unknown dtype %d", name, t);
    return LL_OK;
}

int check_loss(const char* name, const ll_loss* l) {
    if (!l) return fail(LL_EINVAL, "%s is NULL", name);
    if (l->kind == LL_LOSS_BERNOULLI) {
        if (!prob_ok(l->p)) return fail(LL_EINVAL, "%s: p outside [0, 1]", name);
    } else if (l->kind == LL_LOSS_GILBERT_ELLIOTT) {
        if (!prob_ok(l->p_gb) || !prob_ok(l->p_bg) || !prob_ok(l->loss_good) ||
            !prob_ok(l->loss_bad))
            return fail(LL_EINVAL, "%s: Gilbert-Elliott probability outside [0, 1]", name);
    } else {
        return fail(LL_EINVAL, "%s: unknown loss kind %d", name, l->kind);
    }
    return LL_OK;
}

int make_opt(const ll_opt* opt, uint64_t step, const float* m, const float* v, OptParams* o) {
    if (!opt) return fail(LL_EINVAL, "opt is NULL");
    if (opt->kind != LL_SGD && opt->kind != LL_SGD_MOMENTUM && opt->kind != LL_ADAM)
        return fail(LL_EINVAL, "unknown optimizer kind %d", opt->kind);
    if (opt->kind >= LL_SGD_MOMENTUM) {
        int r = check_vec("m", m, true);
        if (r) return r;
    }
    if (opt->kind == LL_ADAM) {
        int r = check_vec("v", v, true);
        if (r) return r;
    }
    o->kind = opt->kind;
    o->lr = opt->lr;
    o->momentum = opt->momentum;
    o->beta1 = opt->beta1;
    o->beta2 = opt->beta2;
    o->eps = opt->eps;
    const double t1 = (double)step + 1.0;
    o->bc1 = (float)(1.0 - std::pow((double)opt->beta1, t1));
    o->bc2 = (float)(1.0 - std::pow((double)opt->beta2, t1));
    if (opt->kind == LL_ADAM && (!(o->bc1 > 0.0f) || !(o->bc2 > 0.0f)))
        return fail(LL_EINVAL, "Adam betas must lie in [0, 1)");
    return LL_OK;
}

GeParams make_ge(const ll_loss* l) {
    GeParams g;
    g.seed = l->seed;
    g.thr_gb = threshold(l->p_gb);
    g.thr_bg = threshold(l->p_bg);
    g.thr_loss_good = threshold(l->loss_good);
    g.thr_loss_bad = threshold(l->loss_bad);
    return g;
}

size_t round256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace layout: [drift partials][gradient masks][broadcast masks]
// [Gilbert-Elliott scratch for two directions], each region 256-byte aligned.
struct GeScratch {
    int64_t S = 0;  // segments per chain
    size_t tmaps = 0, comps = 0, state = 0, per_dir = 0;
};

GeScratch ge_scratch(int32_t n, int64_t P) {
    GeScratch g;
    g.S = (P + kGeSeg - 1) / kGeSeg;
    g.tmaps = round256((size_t)n * (size_t)g.S * kThreads);
    g.comps = round256((size_t)n * (size_t)g.S);
    g.state = round256((size_t)n);
    g.per_dir = g.tmaps + g.comps + g.state;
    return g;
}

// The partials region holds one partial per workgroup followed by the
// kReduceGroups second-level partials.
struct WsLayout {
    size_t partials = 0, groups_off = 0, masks = 0, ge = 0, total = 0;
    GeScratch gs;
};

WsLayout ws_layout(int32_t n, const Geometry& g) {
    WsLayout w;
    w.groups_off = round256((size_t)g.blocks * sizeof(DriftPartial));
    w.partials = w.groups_off + round256(kReduceBytes);
    w.masks = round256((size_t)n * (size_t)g.P);
    w.gs = ge_scratch(n, g.P);
    w.ge = 2 * w.gs.per_dir;
    w.total = w.partials + 2 * w.masks + w.ge;
    return w;
}

// Variants of the step (ll_ext), validated; defaults when ext is NULL.
struct ExtView {
    int est = LL_EST_ARRIVED_MEAN;
    int owner = -1;
    const uint8_t* reliable = nullptr;
    void* g_prev = nullptr;
    uint16_t* ages = nullptr;
    double q = 0.0;
    int parity = 0;  // packets per parity group, 0 = no parity packets
};

int read_ext(const ll_ext* e, int32_t n, ExtView* v) {
    if (!e) return LL_OK;
    if (e->estimator != LL_EST_ARRIVED_MEAN && e->estimator != LL_EST_HORVITZ_THOMPSON &&
        e->estimator != LL_EST_STALE_FILL)
        return fail(LL_EINVAL, "unknown estimator %d", e->estimator);
    if (e->owner < -1 || e->owner >= n) return fail(LL_EINVAL, "owner=%d outside [-1, n)", e->owner);
    if (!(e->arrival_prob >= 0.0 && e->arrival_prob <= 1.0))
        return fail(LL_EINVAL, "arrival_prob outside [0, 1]");
    if (e->parity_group < 0 || e->parity_group > kMaxParityGroup)
        return fail(LL_EINVAL, "parity_group=%d outside [0, %d]", e->parity_group, kMaxParityGroup);
    v->est = e->estimator;
    v->owner = e->owner;
    v->reliable = e->reliable;
    v->g_prev = e->g_prev;
    v->ages = e->ages;
    v->q = e->arrival_prob;
    v->parity = e->parity_group;
    return LL_OK;
}

// Parity-packet mask launch for up to two Bernoulli directions.
int make_parity(const ExtView& x, int32_t n, int64_t P, uint64_t step, ParityLaunch* L) {
    L->ndir = 0;
    L->n = n;
    L->G = x.parity;
    L->span = x.parity * (kThreads / x.parity);
    L->P = P;
    L->spans = (P + L->span - 1) / L->span;
    L->step = step;
    if (2 * (int64_t)n * L->spans > 0x7FFFFFFFll) return fail(LL_EINVAL, "too many workgroups");
    return LL_OK;
}

void add_parity_job(ParityLaunch* L, const ll_loss* l, int dir, const ExtView& x,
                    uint8_t* arrived) {
    MaskJob& j = L->job[L->ndir++];
    j.dir = (uint64_t)dir;
    j.seed = l->seed;
    j.thr = threshold(l->p);
    j.owner = x.owner;
    j.reliable = x.reliable;
    j.arrived = arrived;
}

// Aggregation variant for the kernels; q is the Horvitz-Thompson arrival
// probability already resolved by the caller.
int make_variant(const ExtView& x, double q, const void* g_prev_checked, AggVariant* v) {
    v->kind = x.est;
    v->owner = x.owner;
    v->reliable = x.reliable;
    v->g_prev = const_cast<void*>(g_prev_checked);
    v->invq = 1.0f;
    v->parity_group = 0;
    v->q = q;
    v->ge_derived = 0;
    v->p_gb = v->p_bg = v->loss_good = v->loss_bad = 0.0;
    if (x.est == LL_EST_HORVITZ_THOMPSON) {
        if (!(q > 0.0 && q <= 1.0))
            return fail(LL_EINVAL, "Horvitz-Thompson needs an arrival probability in (0, 1]");
        v->invq = (float)(1.0 / q);
    }
    return LL_OK;
}

// Aggregation variant of the fused step.  An explicit Horvitz-Thompson
// arrival_prob is used as given; 0 asks for each packet's exact arrival
// probability under the gradient loss, derived in the kernel: 1 - p for
// Bernoulli loss, turned per packet into q + (1 - q) q^(g - r) under parity
// packets (a packet also arrives when it alone was lost in its group and the
// parity packet came through), and the chain's marginal at the packet under
// Gilbert-Elliott loss (positive only if neither state loses everything).
int fused_variant(const ExtView& x, const ll_loss* loss_g, AggVariant* var) {
    const bool derive = x.est == LL_EST_HORVITZ_THOMPSON && x.q == 0.0;
    const bool ge = loss_g->kind == LL_LOSS_GILBERT_ELLIOTT;
    double q = x.q;
    if (derive && ge) {
        if (!(loss_g->loss_good < 1.0 && loss_g->loss_bad < 1.0))
            return fail(LL_EINVAL, "Horvitz-Thompson under Gilbert-Elliott loss with a state "
                                   "that loses every packet needs arrival_prob");
        q = 1.0;  // replaced per packet
    } else if (derive) {
        q = 1.0 - loss_g->p;
    }
    int r = make_variant(x, q, x.g_prev, var);
    if (r) return r;
    if (derive && ge) {
        var->ge_derived = 1;
        var->p_gb = loss_g->p_gb;
        var->p_bg = loss_g->p_bg;
        var->loss_good = loss_g->loss_good;
        var->loss_bad = loss_g->loss_bad;
    }
    if (derive && x.parity) var->parity_group = x.parity;
    return LL_OK;
}

// Fill one direction's Gilbert-Elliott job with its scratch carved from `base`.
GeJob make_ge_job(const ll_loss* l, int dir, uint8_t* state, uint8_t* arrived,
                  const GeScratch& gs, uint8_t* base) {
    GeJob j;
    j.ge = make_ge(l);
    j.dir = (uint64_t)dir;
    j.state = state;
    j.arrived = arrived;
    j.tmaps = base;
    j.comps = base + gs.tmaps;
    j.state_in = base + gs.tmaps + gs.comps;
    j.owner = -1;
    j.reliable = nullptr;
    return j;
}

// Long-run fraction of transfers that arrive under a loss process (with
// parity recovery over groups of g packets when g > 0); only used to lay out
// the pacing schedule.
double expected_arrival(const ll_loss* l, int g) {
    double q;
    if (l->kind == LL_LOSS_BERNOULLI) {
        q = 1.0 - l->p;
    } else {
        const double s = l->p_gb + l->p_bg;
        const double bad = s > 0.0 ? l->p_gb / s : 0.0;
        q = 1.0 - (bad * l->loss_bad + (1.0 - bad) * l->loss_good);
    }
    if (g > 0) q = q + (1.0 - q) * std::pow(q, (double)g);
    return q;
}

}  // namespace

extern "C" {

int ll_set_pacing(const ll_pacing* cfg) {
    if (!cfg) return fail(LL_EINVAL, "cfg is NULL");
    if (cfg->mode != LL_PACE_AUTO && cfg->mode != LL_PACE_ALWAYS && cfg->mode != LL_PACE_NEVER)
        return fail(LL_EINVAL, "unknown pacing mode %d", cfg->mode);
    if (!(cfg->bytes_per_s > 0.0 && cfg->bytes_per_s < 1e15))
        return fail(LL_EINVAL, "bytes_per_s must lie in (0, 1e15)");
    if (!(cfg->bytes_per_s_f32 > 0.0 && cfg->bytes_per_s_f32 < 1e15))
        return fail(LL_EINVAL, "bytes_per_s_f32 must lie in (0, 1e15)");
    if (!(cfg->gap_us >= 0.0 && cfg->gap_us <= 1e4))
        return fail(LL_EINVAL, "gap_us must lie in [0, 1e4]");
    if (!(cfg->lead_us >= 0.0 && cfg->lead_us <= 1e4))
        return fail(LL_EINVAL, "lead_us must lie in [0, 1e4]");
    if (cfg->overlap != 1 && cfg->overlap != 2)
        return fail(LL_EINVAL, "overlap=%d must be 1 or 2", cfg->overlap);
    if (cfg->resident < cfg->overlap || cfg->resident > 4)
        return fail(LL_EINVAL, "resident=%d must lie in [overlap, 4]", cfg->resident);
    if (!(cfg->headroom > 0.0 && cfg->headroom <= 1.0))
        return fail(LL_EINVAL, "headroom must lie in (0, 1]");
    if (!(cfg->tail_us >= 0.0 && cfg->tail_us <= 1e4))
        return fail(LL_EINVAL, "tail_us must lie in [0, 1e4]");
    if (cfg->persistent != 0 && cfg->persistent != 1)
        return fail(LL_EINVAL, "persistent=%d must be 0 or 1", cfg->persistent);
    if (cfg->persistent && (cfg->overlap != 1 || cfg->resident != 1))
        return fail(LL_EINVAL, "persistent pacing needs overlap=1 and resident=1");
    set_pace_setting(PaceSetting{cfg->mode, cfg->bytes_per_s, cfg->gap_us, cfg->lead_us,
                                 cfg->overlap, cfg->resident, cfg->headroom, cfg->tail_us,
                                 cfg->persistent, cfg->bytes_per_s_f32});
    return ok();
}

int ll_get_pacing(ll_pacing* out) {
    if (!out) return fail(LL_EINVAL, "out is NULL");
    const PaceSetting st = get_pace_setting();
    out->mode = st.mode;
    out->bytes_per_s = st.bytes_per_s;
    out->gap_us = st.gap_us;
    out->lead_us = st.lead_us;
    out->overlap = st.overlap;
    out->resident = st.resident;
    out->headroom = st.headroom;
    out->tail_us = st.tail_us;
    out->persistent = st.persistent;
    out->bytes_per_s_f32 = st.bytes_per_s_f32;
    return ok();
}

const char* ll_last_error(void) { return g_error.c_str(); }

size_t ll_workspace_bytes(int32_t n, int64_t d, int64_t packet) {
    Geometry g;
    if (check_shape(n, d, packet, &g) != LL_OK) return 0;
    return ws_layout(n, g).total;
}

size_t ll_masks_workspace_bytes(int32_t n, int64_t num_packets) {
    if (n < 1 || n > kMaxWorkers || num_packets < 0) return 0;
    return ge_scratch(n, num_packets).per_dir;
}

int ll_masks(int32_t n, int64_t num_packets, uint64_t step, int32_t dir, const ll_loss* loss,
             uint8_t* ge_state, uint8_t* arrived, void* workspace, size_t ws_bytes,
             const ll_ext* ext, void* stream) {
    if (n < 1 || n > kMaxWorkers) return fail(LL_EINVAL, "n=%d outside [1, %d]", n, kMaxWorkers);
    if (num_packets < 0) return fail(LL_EINVAL, "num_packets is negative");
    if (dir != LL_DIR_GRAD && dir != LL_DIR_BCAST) return fail(LL_EINVAL, "unknown direction %d", dir);
    int r = check_loss("loss", loss);
    if (r) return r;
    ExtView x;
    if ((r = read_ext(ext, n, &x))) return r;
    if (!arrived) return fail(LL_EINVAL, "arrived is NULL");
    const bool ge = loss->kind == LL_LOSS_GILBERT_ELLIOTT;
    if (ge && x.parity) return fail(LL_EINVAL, "parity packets need Bernoulli loss");
    if (ge && !ge_state) return fail(LL_EINVAL, "ge_state is NULL for a Gilbert-Elliott process");
    const GeScratch gs = ge_scratch(n, num_packets);
    if (ge && (!workspace || ws_bytes < gs.per_dir))
        return fail(LL_EINVAL, "workspace of %zu bytes is smaller than %zu", ws_bytes, gs.per_dir);
    if (num_packets == 0) return ok();
    if ((int64_t)n * gs.S > 0x7FFFFFFFll) return fail(LL_EINVAL, "too many workgroups");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (x.parity) {
        ParityLaunch PL;
        if ((r = make_parity(x, n, num_packets, step, &PL))) return r;
        add_parity_job(&PL, loss, dir, x, arrived);
        return hip_check(launch_masks_parity(PL, s), "ll_masks");
    }
    if (!ge)
        return hip_check(launch_masks_bernoulli(n, num_packets, step, dir, loss->seed,
                                                threshold(loss->p), x.owner, x.reliable, arrived,
                                                s),
                         "ll_masks");
    GeLaunch L;
    L.n = n;
    L.P = num_packets;
    L.S = gs.S;
    L.step = step;
    L.job[0] = make_ge_job(loss, dir, ge_state, arrived, gs, reinterpret_cast<uint8_t*>(workspace));
    L.job[0].owner = x.owner;
    L.job[0].reliable = x.reliable;
    L.job[1] = L.job[0];
    return hip_check(launch_masks_ge(L, 1, s), "ll_masks");
}

int lossy_aggregate(int32_t n, int64_t d, int64_t packet, int32_t gdtype, const void* grads,
                    int64_t ld_g, const uint8_t* arrived, float fallback_lambda,
                    const float* theta, float* g_hat, int32_t* counts, const ll_ext* ext,
                    void* stream) {
    Geometry g;
    int r = check_shape(n, d, packet, &g);
    if (r) return r;
    if ((r = check_dtype("gdtype", gdtype))) return r;
    if (d == 0) return ok();
    if ((r = check_rows("grads", grads, ld_g, d, elem_bytes(gdtype)))) return r;
    if (!arrived) return fail(LL_EINVAL, "arrived is NULL");
    if ((r = check_vec("g_hat", g_hat, true))) return r;
    if ((r = check_vec("theta", theta, fallback_lambda != 0.0f))) return r;
    ExtView x;
    if ((r = read_ext(ext, n, &x))) return r;
    if (x.est == LL_EST_STALE_FILL && (r = check_rows("g_prev", x.g_prev, ld_g, d, elem_bytes(gdtype)))) return r;
    AggParams p;
    if ((r = make_variant(x, x.q, x.g_prev, &p.var))) return r;
    p.n = n;
    p.d = d;
    p.L = packet;
    p.P = g.P;
    p.cpp = 0;
    p.grads = grads;
    p.ld = ld_g;
    p.arrived = arrived;
    p.lam = fallback_lambda;
    p.theta = theta;
    p.g_hat = g_hat;
    p.counts = counts;
    return hip_check(launch_aggregate(gdtype, p, reinterpret_cast<hipStream_t>(stream)),
                     "lossy_aggregate");
}

int ll_ages_update(int32_t n, int64_t num_packets, const uint8_t* arrived_bc, uint16_t* ages,
                   void* stream) {
    if (n < 1 || n > kMaxWorkers) return fail(LL_EINVAL, "n=%d outside [1, %d]", n, kMaxWorkers);
    if (num_packets < 0) return fail(LL_EINVAL, "num_packets is negative");
    if (num_packets == 0) return ok();
    if (!arrived_bc) return fail(LL_EINVAL, "arrived_bc is NULL");
    if (!ages) return fail(LL_EINVAL, "ages is NULL");
    return hip_check(launch_ages_update((int64_t)n * num_packets, arrived_bc, ages,
                                        reinterpret_cast<hipStream_t>(stream)),
                     "ll_ages_update");
}

int shard_step(const ll_opt* opt, int64_t d, uint64_t step, float* theta, float* m, float* v,
               const float* g_hat, void* stream) {
    if (d < 0) return fail(LL_EINVAL, "d is negative");
    if (d == 0) return ok();
    OptParams o;
    int r = make_opt(opt, step, m, v, &o);
    if (r) return r;
    if ((r = check_vec("theta", theta, true))) return r;
    if ((r = check_vec("g_hat", g_hat, true))) return r;
    if ((d + kThreads * kElems - 1) / (kThreads * kElems) > 0x7FFFFFFFll)
        return fail(LL_EINVAL, "d too large");
    return hip_check(launch_shard_step(d, o, theta, m, v, g_hat,
                                       reinterpret_cast<hipStream_t>(stream)),
                     "shard_step");
}

int lossy_broadcast(int32_t n, int64_t d, int64_t packet, const float* theta, int32_t rdtype,
                    void* replicas, int64_t ld_r, const uint8_t* arrived_bc, void* stream) {
    Geometry g;
    int r = check_shape(n, d, packet, &g);
    if (r) return r;
    if ((r = check_dtype("rdtype", rdtype))) return r;
    if (d == 0) return ok();
    if ((r = check_vec("theta", theta, true))) return r;
    if ((r = check_rows("replicas", replicas, ld_r, d, elem_bytes(rdtype)))) return r;
    if (!arrived_bc) return fail(LL_EINVAL, "arrived_bc is NULL");
    BcastParams p;
    p.n = n;
    p.d = d;
    p.L = packet;
    p.P = g.P;
    p.cpp = 0;
    p.theta = theta;
    p.replicas = replicas;
    p.ld = ld_r;
    p.arrived = arrived_bc;
    return hip_check(launch_broadcast(rdtype, p, reinterpret_cast<hipStream_t>(stream)),
                     "lossy_broadcast");
}

int drift_stats(int32_t n, int64_t d, int64_t packet, int32_t rdtype, const void* replicas,
                int64_t ld_r, const float* theta, const uint8_t* arrived_bc, void* workspace,
                size_t ws_bytes, ll_drift* out, void* stream) {
    Geometry g;
    int r = check_shape(n, d, packet, &g);
    if (r) return r;
    if ((r = check_dtype("rdtype", rdtype))) return r;
    if (!out) return fail(LL_EINVAL, "out is NULL");
    if ((r = check_vec("out", out, true))) return r;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (d == 0) return hip_check(launch_drift_zero(reinterpret_cast<DriftOut*>(out), s), "drift_stats");
    if ((r = check_rows("replicas", replicas, ld_r, d, elem_bytes(rdtype)))) return r;
    if ((r = check_vec("theta", theta, false))) return r;
    const WsLayout w = ws_layout(n, g);
    if (!workspace || ws_bytes < w.total)
        return fail(LL_EINVAL, "workspace of %zu bytes is smaller than %zu", ws_bytes, w.total);
    if ((r = check_vec("workspace", workspace, true))) return r;
    DriftParams p;
    p.n = n;
    p.d = d;
    p.L = packet;
    p.P = g.P;
    p.cpp = 0;
    p.replicas = replicas;
    p.ld = ld_r;
    p.theta = theta;
    p.arrived = arrived_bc;
    p.partials = reinterpret_cast<DriftPartial*>(workspace);
    p.groups = reinterpret_cast<DriftAcc*>(reinterpret_cast<uint8_t*>(workspace) + w.groups_off);
    return hip_check(launch_drift(rdtype, p, n, d, theta != nullptr,
                                  reinterpret_cast<DriftOut*>(out), s),
                     "drift_stats");
}

}  // extern "C"

namespace {

// The fused step behind lossy_step_fused and lossy_step_fused_noalloc; `fn`
// names the entry point in error messages.
int step_fused(const char* fn, int32_t n, int64_t d, int64_t packet, uint64_t step,
               const ll_loss* loss_g, const ll_loss* loss_b, uint8_t* ge_state_g,
               uint8_t* ge_state_b, int32_t gdtype, const void* grads, int64_t ld_g,
               const ll_opt* opt, float* theta, float* m, float* v, int32_t rdtype,
               void* replicas, int64_t ld_r, uint8_t* arrived_g, uint8_t* arrived_b,
               int32_t* counts, void* workspace, size_t ws_bytes, ll_drift* drift,
               const ll_ext* ext, void* stream) {
    Geometry g;
    int r = check_shape(n, d, packet, &g);
    if (r) return r;
    if ((r = check_loss("loss_g", loss_g))) return r;
    if ((r = check_loss("loss_b", loss_b))) return r;
    if ((r = check_dtype("gdtype", gdtype))) return r;
    if ((r = check_dtype("rdtype", rdtype))) return r;
    ExtView x;
    if ((r = read_ext(ext, n, &x))) return r;
    const bool ge_g = loss_g->kind == LL_LOSS_GILBERT_ELLIOTT;
    const bool ge_b = loss_b->kind == LL_LOSS_GILBERT_ELLIOTT;
    if (ge_g && !ge_state_g) return fail(LL_EINVAL, "ge_state_g is NULL for a Gilbert-Elliott process");
    if (ge_b && !ge_state_b) return fail(LL_EINVAL, "ge_state_b is NULL for a Gilbert-Elliott process");
    if (x.parity && (ge_g || ge_b)) return fail(LL_EINVAL, "parity packets need Bernoulli loss");
    if (drift && (r = check_vec("drift", drift, true))) return r;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (d == 0) {
        if (drift) return hip_check(launch_drift_zero(reinterpret_cast<DriftOut*>(drift), s), fn);
        return ok();
    }
    if ((r = check_rows("grads", grads, ld_g, d, elem_bytes(gdtype)))) return r;
    if ((r = check_rows("replicas", replicas, ld_r, d, elem_bytes(rdtype)))) return r;
    if ((r = check_vec("theta", theta, true))) return r;
    OptParams o;
    if ((r = make_opt(opt, step, m, v, &o))) return r;
    if (x.est == LL_EST_STALE_FILL && (r = check_rows("g_prev", x.g_prev, ld_g, d, elem_bytes(gdtype)))) return r;
    AggVariant var;
    if ((r = fused_variant(x, loss_g, &var))) return r;
    const WsLayout w = ws_layout(n, g);
    const bool need_ws = drift || ge_g || ge_b || x.parity;
    if (need_ws) {
        if (!workspace || ws_bytes < w.total)
            return fail(LL_EINVAL, "workspace of %zu bytes is smaller than %zu", ws_bytes, w.total);
        if ((r = check_vec("workspace", workspace, true))) return r;
    }
    uint8_t* ws = reinterpret_cast<uint8_t*>(workspace);

    FusedParams p;
    p.n = n;
    p.d = d;
    p.L = packet;
    p.P = g.P;
    p.cpp = 0;
    p.step = step;
    p.out_g = arrived_g;
    p.out_b = arrived_b;
    p.counts = counts;
    p.grads = grads;
    p.ld_g = ld_g;
    p.opt = o;
    p.lam = opt->fallback_lambda;
    p.theta = theta;
    p.m = m;
    p.v = v;
    p.replicas = replicas;
    p.ld_r = ld_r;
    p.partials = drift ? reinterpret_cast<DriftPartial*>(ws) : nullptr;
    p.groups = drift ? reinterpret_cast<DriftAcc*>(ws + w.groups_off) : nullptr;
    p.var = var;
    p.ages = x.ages;
    const bool have_ws = workspace && ws_bytes >= w.total && aligned16(workspace);
    for (int dir = 0; dir < 2; ++dir) {
        uint8_t* out = dir == 0 ? arrived_g : arrived_b;
        p.pre[dir] = out ? out : (have_ws ? ws + w.partials + dir * w.masks : nullptr);
    }

    const ll_loss* losses[2] = {loss_g, loss_b};
    uint8_t* states[2] = {ge_state_g, ge_state_b};
    uint8_t* outs[2] = {arrived_g, arrived_b};
    GeLaunch L;
    L.n = n;
    L.P = g.P;
    L.S = w.gs.S;
    L.step = step;
    int nge = 0;
    for (int dir = 0; dir < 2; ++dir) {
        const ll_loss* l = losses[dir];
        if (l->kind == LL_LOSS_BERNOULLI) {
            p.src[dir] = MaskSource{true, l->seed, threshold(l->p), nullptr, x.owner, x.reliable};
        } else {
            // Sequential chain: the scan writes the masks, the step reads them.
            uint8_t* dst = outs[dir] ? outs[dir] : ws + w.partials + dir * w.masks;
            L.job[nge] = make_ge_job(l, dir, states[dir], dst, w.gs,
                                     ws + w.partials + 2 * w.masks + dir * w.gs.per_dir);
            L.job[nge].owner = x.owner;
            L.job[nge].reliable = x.reliable;
            ++nge;
            p.src[dir] = MaskSource{false, 0, 0, dst, -1, nullptr};
            if (dir == 0) p.out_g = nullptr;  // already written by the scan
            else p.out_b = nullptr;
        }
    }
    if (x.parity) {
        // Recovery needs a whole group's arrivals: masks go through memory.
        ParityLaunch PL;
        if ((r = make_parity(x, n, g.P, step, &PL))) return r;
        for (int dir = 0; dir < 2; ++dir) {
            uint8_t* dst = outs[dir] ? outs[dir] : ws + w.partials + dir * w.masks;
            add_parity_job(&PL, losses[dir], dir, x, dst);
            p.src[dir] = MaskSource{false, 0, 0, dst, -1, nullptr};
        }
        p.out_g = p.out_b = nullptr;
        r = hip_check(launch_masks_parity(PL, s), fn);
        if (r) return r;
    }
    if (nge) {
        if ((int64_t)nge * n * w.gs.S > 0x7FFFFFFFll) return fail(LL_EINVAL, "too many workgroups");
        if (nge == 1) L.job[1] = L.job[0];
        r = hip_check(launch_masks_ge(L, nge, s), fn);
        if (r) return r;
    }
    const PaceHint hint{expected_arrival(loss_g, x.parity), expected_arrival(loss_b, x.parity)};
    return hip_check(launch_fused(gdtype, rdtype, p, reinterpret_cast<DriftOut*>(drift), hint, s),
                     fn);
}

}  // namespace

extern "C" {

int lossy_step_fused(int32_t n, int64_t d, int64_t packet, uint64_t step, const ll_loss* loss_g,
                     const ll_loss* loss_b, uint8_t* ge_state_g, uint8_t* ge_state_b,
                     int32_t gdtype, const void* grads, int64_t ld_g, const ll_opt* opt,
                     float* theta, float* m, float* v, int32_t rdtype, void* replicas,
                     int64_t ld_r, uint8_t* arrived_g, uint8_t* arrived_b, int32_t* counts,
                     void* workspace, size_t ws_bytes, ll_drift* drift, const ll_ext* ext,
                     void* stream) {
    return step_fused("lossy_step_fused", n, d, packet, step, loss_g, loss_b, ge_state_g,
                      ge_state_b, gdtype, grads, ld_g, opt, theta, m, v, rdtype, replicas, ld_r,
                      arrived_g, arrived_b, counts, workspace, ws_bytes, drift, ext, stream);
}

int lossy_step_fused_noalloc(int32_t n, int64_t d, int64_t packet, uint64_t step,
                             const ll_loss* loss_g, const ll_loss* loss_b, uint8_t* ge_state_g,
                             uint8_t* ge_state_b, int32_t gdtype, const void* grads,
                             int64_t ld_g, const ll_opt* opt, float* theta, float* m, float* v,
                             int32_t rdtype, void* replicas, int64_t ld_r, uint8_t* arrived_g,
                             uint8_t* arrived_b, int32_t* counts, ll_drift* drift,
                             const ll_ext* ext, void* stream) {
    static const char* fn = "lossy_step_fused_noalloc";
    Geometry g;
    int r = check_shape(n, d, packet, &g);
    if (r) return r;
    const size_t need = ws_layout(n, g).total;
    if (need > kNoAllocScratchBytes)
        return fail(LL_EINVAL,
                    "%s: n=%d, d=%lld, packet=%lld need %zu bytes of scratch, more than the "
                    "%zu bytes of its static scratch; use lossy_step_fused with a workspace",
                    fn, n, (long long)d, (long long)packet, need, kNoAllocScratchBytes);
    void* ws = nullptr;
    if ((r = hip_check(noalloc_scratch(&ws), fn))) return r;
    return step_fused(fn, n, d, packet, step, loss_g, loss_b, ge_state_g, ge_state_b, gdtype,
                      grads, ld_g, opt, theta, m, v, rdtype, replicas, ld_r, arrived_g,
                      arrived_b, counts, ws, kNoAllocScratchBytes, drift, ext, stream);
}

}  // extern "C"
