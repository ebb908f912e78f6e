// Exploration sampler, Droplet Search and the combined approach (Sections 2.1-2.3).
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <functional>
#include <limits>
#include <unordered_map>
#include <unordered_set>

#include "ds_internal.h"

namespace ds {
const Space &space_of(const ds_space *s);
}

using namespace ds;

namespace {

// SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): state advances by the golden
// gamma, output is the two-multiply finaliser of the state.
struct SplitMix64 {
    uint64_t state;
    explicit SplitMix64(uint64_t seed) : state(seed) {}
    uint64_t next() {
        state += 0x9E3779B97F4A7C15ull;
        uint64_t z = state;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    // Uniform on [0, n): reject the top partial block of 2^64 mod n values.
    uint32_t below(uint32_t n) {
        const uint64_t lim = (n & (n - 1)) == 0 ? 0 : (~uint64_t(0) / n) * n;
        for (;;) {
            const uint64_t z = next();
            if (lim == 0 || z < lim) return uint32_t(z % n);
        }
    }
};

double now_s() {
    using clk = std::chrono::steady_clock;
    return std::chrono::duration<double>(clk::now().time_since_epoch()).count();
}

Meas to_meas(const ds_measurement &m, int rc) {
    Meas r;
    r.full = m;
    r.status = rc != DS_OK ? rc : m.status;
    if (r.status != DS_OK) {
        r.median = std::numeric_limits<double>::infinity();
        r.full.median_ms = r.median;
        return r;
    }
    const int n = std::max(0, std::min<int>(m.n_repeats, DS_MAX_REPEATS));
    r.repeats.assign(m.repeats_ms, m.repeats_ms + n);
    r.median = m.median_ms;
    if (!(r.median == r.median)) r.median = std::numeric_limits<double>::infinity();
    return r;
}

void trace_push(ds_trace *tr, int stage, const Meas &m, uint64_t key) {
    if (!tr) return;
    if (tr->n < tr->cap && tr->entries) {
        ds_trace_entry &e = tr->entries[tr->n];
        e.stage = stage;
        e.status = m.status;
        e.key = key;
        e.median_ms = m.median;
    }
    tr->n++;
}

using MeasureFn = std::function<Meas(const int32_t *idx, double best_so_far)>;

// The draw sequence of the exploration sampler.
std::vector<std::vector<int32_t>> draw_points(const Space &sp, uint64_t seed, int n_explore) {
    std::vector<std::vector<int32_t>> out;
    if (n_explore <= 0) return out;
    SplitMix64 rng(seed);
    std::unordered_set<uint64_t> seen;
    int64_t draws = 0;
    const int64_t max_draws = 100 * int64_t(n_explore);
    std::vector<int32_t> idx(sp.nknobs);
    while (int(out.size()) < n_explore && draws < max_draws) {
        ++draws;
        for (int a = 0; a < sp.nknobs; ++a) idx[a] = int32_t(rng.below(uint32_t(sp.values[a].size())));
        const uint64_t k = sp.key(idx.data());
        if (seen.count(k) || !sp.geometry(idx.data()).valid) continue;
        seen.insert(k);
        out.push_back(idx);
    }
    return out;
}

struct DropletOut {
    std::vector<int32_t> best;
    Meas meas;
    int measured = 0;
    int moves = 0;
    int failed = 0;
    int status = DS_OK;
};

// Droplet Search from `start` over the cached measurements `cache`.
DropletOut droplet(const Space &sp, const int32_t *start, int budget, double alpha,
                   uint32_t frozen, std::unordered_map<uint64_t, Meas> &cache,
                   const MeasureFn &measure, double &best_so_far, ds_trace *trace) {
    DropletOut out;
    std::vector<int32_t> cur(start, start + sp.nknobs);
    uint64_t kcur = sp.key(cur.data());
    if (!cache.count(kcur)) {
        Meas m = measure(cur.data(), best_so_far);
        if (m.status != DS_OK) out.failed++;
        else best_so_far = best_so_far > 0 ? std::min(best_so_far, m.median) : m.median;
        cache[kcur] = m;
        out.measured++;
        trace_push(trace, 1, m, kcur);
    }
    int nb_measured = 0;
    std::vector<std::vector<int32_t>> nbs;
    std::vector<int32_t> nb(sp.nknobs);
    for (;;) {
        nbs.clear();
        for (int a = 0; a < sp.nknobs; ++a) {
            if (frozen & (1u << a)) continue;
            for (int d = -1; d <= 1; d += 2) {
                const int j = cur[a] + d;
                if (j < 0 || j >= int(sp.values[a].size())) continue;
                nb = cur;
                nb[a] = j;
                if (sp.geometry(nb.data()).valid) nbs.push_back(nb);
            }
        }
        bool stop = false;
        for (const auto &p : nbs) {
            const uint64_t k = sp.key(p.data());
            if (cache.count(k)) continue;
            if (nb_measured >= budget) {
                out.status = DS_EBUDGET;
                stop = true;
                break;
            }
            Meas m = measure(p.data(), best_so_far);
            if (m.status != DS_OK) out.failed++;
            else best_so_far = best_so_far > 0 ? std::min(best_so_far, m.median) : m.median;
            cache[k] = m;
            nb_measured++;
            out.measured++;
            trace_push(trace, 2, m, k);
        }
        if (stop || nbs.empty()) break;
        size_t b = 0;
        for (size_t i = 1; i < nbs.size(); ++i)
            if (cache[sp.key(nbs[i].data())].median < cache[sp.key(nbs[b].data())].median) b = i;
        const Meas &mb = cache[sp.key(nbs[b].data())];
        if (better(mb, cache[kcur], alpha)) {
            cur = nbs[b];
            kcur = sp.key(cur.data());
            out.moves++;
        } else {
            break;
        }
    }
    out.best = cur;
    out.meas = cache[kcur];
    return out;
}

MeasureFn make_measure(const Space &sp, const ds_tune_cfg *cfg, const ds_tune_io *io,
                       const float *ref, ds_measure_fn fn, void *ctx) {
    if (fn) {
        return [&sp, fn, ctx](const int32_t *idx, double) {
            ds_measurement m;
            std::memset(&m, 0, sizeof m);
            const ds_sched s = make_sched(sp, idx);
            const int rc = fn(ctx, &s, &m);
            return to_meas(m, rc);
        };
    }
    ds_tune_io local = *io;
    local.ref = ref;
    ds_measure_cfg mc = cfg->measure;
    return [&sp, local, mc](const int32_t *idx, double best) {
        ds_measurement m;
        std::memset(&m, 0, sizeof m);
        const ds_sched s = make_sched(sp, idx);
        const int rc = ds_measure(&s, &local, &mc, best, &m);
        return to_meas(m, rc);
    };
}

void fill_result(ds_tune_result *res, const Space &sp, const DropletOut &d) {
    res->best = make_sched(sp, d.best.data());
    res->best_ms = d.meas.median;
    res->best_meas = d.meas.full;
    res->status = d.status;
    res->n_moves = d.moves;
}

// Prepares the measurement context: GPU mode needs buffers and a reference.
int prepare(const Space &sp, const ds_tune_cfg *cfg, const ds_tune_io *io, ds_measure_fn fn,
            float **owned_ref) {
    *owned_ref = nullptr;
    if (fn) return DS_OK;
    if (sp.op == 0) {
        set_error("a generic lattice needs a measurement callback");
        return DS_EINVAL;
    }
    if (!io || !io->x || !io->w || !io->y) {
        set_error("GPU measurement needs io with x, w and y");
        return DS_EINVAL;
    }
    if (cfg->measure.check && !io->ref) return reference_output(sp, io, owned_ref);
    return DS_OK;
}

}  // namespace

namespace ds {

double ranksum_p_less(const std::vector<double> &a, const std::vector<double> &b) {
    const size_t n1 = a.size(), n2 = b.size();
    if (n1 == 0 || n2 == 0) return 1.0;
    std::vector<std::pair<double, int>> pooled;
    pooled.reserve(n1 + n2);
    for (double v : a) pooled.emplace_back(v, 0);
    for (double v : b) pooled.emplace_back(v, 1);
    std::sort(pooled.begin(), pooled.end());
    const size_t n = pooled.size();
    double r1 = 0.0, ties = 0.0;
    for (size_t i = 0; i < n;) {
        size_t j = i;
        while (j + 1 < n && pooled[j + 1].first == pooled[i].first) ++j;
        const double rank = 0.5 * double(i + j) + 1.0;
        for (size_t t = i; t <= j; ++t)
            if (pooled[t].second == 0) r1 += rank;
        const double g = double(j - i + 1);
        ties += g * g * g - g;
        i = j + 1;
    }
    const double u1 = r1 - double(n1) * double(n1 + 1) / 2.0;
    const double mu = double(n1) * double(n2) / 2.0;
    const double var = double(n1) * double(n2) / 12.0 *
                       (double(n + 1) - ties / (double(n) * double(n - 1)));
    if (!(var > 0.0)) return 1.0;
    const double z = (u1 - mu + 0.5) / std::sqrt(var);
    return 0.5 * std::erfc(-z / std::sqrt(2.0));
}

bool better(const Meas &a, const Meas &b, double alpha) {
    if (a.status != DS_OK || !std::isfinite(a.median)) return false;
    if (b.status != DS_OK || !std::isfinite(b.median)) return true;
    if (!(a.median < b.median)) return false;
    if (alpha >= 1.0) return true;
    return ranksum_p_less(a.repeats, b.repeats) < alpha;
}

}  // namespace ds

extern "C" {

void ds_measure_cfg_default(ds_measure_cfg *cfg) {
    if (!cfg) return;
    cfg->warmup = 3;
    cfg->repeat = 11;
    cfg->min_repeat_ms = 0.5;
    cfg->max_number = 200;
    cfg->slow_cut = 4.0;
    cfg->tol = 1e-4;
    cfg->check = 1;
    cfg->graph = 1;
}

void ds_tune_cfg_default(ds_tune_cfg *cfg) {
    if (!cfg) return;
    cfg->n_explore = 300;
    cfg->budget = 100;
    cfg->alpha = 0.05;
    cfg->seed = 240620037ull;
    cfg->frozen_mask = 0;
    ds_measure_cfg_default(&cfg->measure);
}

int ansor_draw(const ds_space *space, uint64_t seed, int n_explore, ds_sched *out, int *n_out) {
    if (!space || !n_out || n_explore < 0 || (n_explore > 0 && !out)) {
        set_error("bad ansor_draw arguments");
        return DS_EINVAL;
    }
    const Space &sp = space_of(space);
    const auto pts = draw_points(sp, seed, n_explore);
    for (size_t i = 0; i < pts.size(); ++i) out[i] = make_sched(sp, pts[i].data());
    *n_out = int(pts.size());
    return pts.empty() && n_explore > 0 ? DS_EEXHAUSTED : DS_OK;
}

int ansor_sample(const ds_space *space, uint64_t seed, int n_explore, const ds_tune_io *io,
                 const ds_measure_cfg *mcfg, ds_sched *best, double *best_ms, ds_trace *trace) {
    if (!space || !best || !best_ms || n_explore < 0) {
        set_error("bad ansor_sample arguments");
        return DS_EINVAL;
    }
    const Space &sp = space_of(space);
    ds_tune_cfg cfg;
    ds_tune_cfg_default(&cfg);
    if (mcfg) cfg.measure = *mcfg;
    if (trace) trace->n = 0;
    float *owned = nullptr;
    int rc = prepare(sp, &cfg, io, nullptr, &owned);
    if (rc != DS_OK) return rc;
    const MeasureFn measure = make_measure(sp, &cfg, io, owned ? owned : io->ref, nullptr, nullptr);
    const auto pts = draw_points(sp, seed, n_explore);
    double best_so_far = 0.0;
    int ib = -1;
    double tb = std::numeric_limits<double>::infinity();
    for (size_t i = 0; i < pts.size(); ++i) {
        Meas m = measure(pts[i].data(), best_so_far);
        trace_push(trace, 0, m, sp.key(pts[i].data()));
        if (m.status == DS_OK)
            best_so_far = best_so_far > 0 ? std::min(best_so_far, m.median) : m.median;
        if (ib < 0 || m.median < tb) {
            ib = int(i);
            tb = m.median;
        }
    }
    free_device(owned);
    if (ib < 0) {
        set_error("no valid point to sample");
        return DS_EEXHAUSTED;
    }
    *best = make_sched(sp, pts[ib].data());
    *best_ms = tb;
    return DS_OK;
}

int droplet_tune_ex(const ds_space *space, const ds_sched *start, int budget,
                    const ds_tune_cfg *cfg_in, const ds_tune_io *io, ds_measure_fn fn, void *ctx,
                    ds_tune_result *res, ds_trace *trace) {
    if (!space || !res || budget < 0) {
        set_error("bad droplet_tune_ex arguments");
        return DS_EINVAL;
    }
    std::memset(res, 0, sizeof *res);
    const Space &sp = space_of(space);
    ds_tune_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_tune_cfg_default(&cfg);
    if (trace) trace->n = 0;
    int32_t st[DS_MAX_KNOBS] = {0};
    if (start) {
        if (!sched_matches(sp, start) || !sp.in_range(start->idx)) {
            set_error("start point does not belong to the space");
            return DS_EINVAL;
        }
        if (!sp.valid(start->idx)) {
            set_error("start point is not a valid schedule");
            return DS_EINVALID_SCHED;
        }
        std::memcpy(st, start->idx, sizeof(int32_t) * sp.nknobs);
    } else {
        ds_sched o;
        const int rc = sched_origin(space, &o);
        if (rc != DS_OK) return rc;
        std::memcpy(st, o.idx, sizeof(int32_t) * sp.nknobs);
    }
    float *owned = nullptr;
    int rc = prepare(sp, &cfg, io, fn, &owned);
    if (rc != DS_OK) return rc;
    const MeasureFn measure = make_measure(sp, &cfg, io, owned ? owned : (io ? io->ref : nullptr),
                                           fn, ctx);
    const double t0 = now_s();
    std::unordered_map<uint64_t, Meas> cache;
    double best_so_far = 0.0;
    const DropletOut d = droplet(sp, st, budget, cfg.alpha, cfg.frozen_mask, cache, measure,
                                 best_so_far, trace);
    free_device(owned);
    fill_result(res, sp, d);
    res->seed_point = make_sched(sp, st);
    res->seed_ms = cache[sp.key(st)].median;
    res->n_droplet_measured = d.measured;
    res->n_failed = d.failed;
    res->droplet_s = res->wall_s = now_s() - t0;
    return DS_OK;
}

int ds_tune(const ds_space *space, const ds_tune_cfg *cfg_in, const ds_tune_io *io,
            ds_measure_fn fn, void *ctx, ds_tune_result *res, ds_trace *trace) {
    if (!space || !res) {
        set_error("bad ds_tune arguments");
        return DS_EINVAL;
    }
    std::memset(res, 0, sizeof *res);
    const Space &sp = space_of(space);
    ds_tune_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_tune_cfg_default(&cfg);
    if (cfg.n_explore < 0 || cfg.budget < 0) {
        set_error("negative n_explore or budget");
        return DS_EINVAL;
    }
    if (trace) trace->n = 0;
    float *owned = nullptr;
    int rc = prepare(sp, &cfg, io, fn, &owned);
    if (rc != DS_OK) return rc;
    const MeasureFn measure = make_measure(sp, &cfg, io, owned ? owned : (io ? io->ref : nullptr),
                                           fn, ctx);
    const double t0 = now_s();
    const auto pts = draw_points(sp, cfg.seed, cfg.n_explore);
    if (pts.empty()) {
        free_device(owned);
        set_error("no valid point to sample");
        return DS_EEXHAUSTED;
    }
    std::unordered_map<uint64_t, Meas> cache;
    double best_so_far = 0.0;
    int ib = -1, failed = 0;
    double tb = std::numeric_limits<double>::infinity();
    for (size_t i = 0; i < pts.size(); ++i) {
        Meas m = measure(pts[i].data(), best_so_far);
        const uint64_t k = sp.key(pts[i].data());
        trace_push(trace, 0, m, k);
        if (m.status != DS_OK) failed++;
        else best_so_far = best_so_far > 0 ? std::min(best_so_far, m.median) : m.median;
        if (ib < 0 || m.median < tb) {
            ib = int(i);
            tb = m.median;
        }
        cache[k] = m;
    }
    const double t1 = now_s();
    const DropletOut d = droplet(sp, pts[ib].data(), cfg.budget, cfg.alpha, cfg.frozen_mask,
                                 cache, measure, best_so_far, trace);
    const double t2 = now_s();
    free_device(owned);
    fill_result(res, sp, d);
    res->seed_point = make_sched(sp, pts[ib].data());
    res->seed_ms = tb;
    res->n_explore_measured = int(pts.size());
    res->n_droplet_measured = d.measured;
    res->n_failed = failed + d.failed;
    res->explore_s = t1 - t0;
    res->droplet_s = t2 - t1;
    res->wall_s = t2 - t0;
    return DS_OK;
}

int ds_gen_uniform(uint64_t seed, int64_t n, float *out) {
    if (n < 0 || (n > 0 && !out)) {
        set_error("bad ds_gen_uniform arguments");
        return DS_EINVAL;
    }
    SplitMix64 rng(seed);
    for (int64_t i = 0; i < n; ++i) {
        const double u = double(rng.next() >> 40) * (1.0 / 16777216.0);
        out[i] = float(2.0 * u - 1.0);
    }
    return DS_OK;
}

}  // extern "C"
