// Exploration sampler, Droplet Search and the combined approach (Sections 2.1-2.3),
// the exploitation strategies it is compared with (Section 3, RQ4) and the
// whole-network trial split (Section 2.1, Termination in Ansor).
#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstring>
#include <functional>
#include <limits>
#include <memory>
#include <new>
#include <unordered_map>
#include <unordered_set>

#include "ds_internal.h"

namespace ds {
const Space &space_of(const ds_space *s);
}

using namespace ds;

// Measurements of one space, keyed by lattice key; remembers the space's axes
// so that a cache cannot be used with another space.
struct ds_cache {
    int op = 0;
    int64_t shape[9] = {0};
    std::vector<std::vector<int32_t>> values;
    std::unordered_map<uint64_t, Meas> map;
};

namespace {

bool cache_fits(const ds_cache *c, const Space &sp) {
    return c && c->op == sp.op && c->values == sp.values &&
           std::equal(c->shape, c->shape + 9, sp.shape);
}

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
    // Uniform double in [0, 1) from the top 53 bits.
    double uniform01() { return double(next() >> 11) * (1.0 / 9007199254740992.0); }
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

// The draw sequence of the exploration sampler (Section 2.1, sketch
// annotation; Section 2.3, step 1).  The kernel family -- the mfma knob of
// the conv and matmul spaces -- stands for the sketch: each draw first picks
// a family uniformly among those that still have an undrawn valid point,
// then one of that family's undrawn valid points uniformly (in key order,
// removed once drawn).  A generic lattice is a single family.  Sampling stops
// at n_explore points or when every valid point has been drawn.
int sketch_axis(const Space &sp) {
    if (sp.op == DS_OP_CONV2D_NCHW) return 7;
    if (sp.op == DS_OP_MATMUL_RM) return 5;
    return -1;
}

struct ExploreSampler {
    const Space &sp;
    SplitMix64 rng;
    std::vector<std::vector<uint64_t>> pool;   // undrawn valid keys per family, key order
    std::vector<int> live;
    ExploreSampler(const Space &s, uint64_t seed) : sp(s), rng(seed) {
        const int sa = sketch_axis(sp);
        pool.resize(sa < 0 ? 1 : sp.values[sa].size());
        std::vector<int32_t> idx(sp.nknobs);
        for (uint64_t k = 0; k < sp.size; ++k) {
            sp.from_key(k, idx.data());
            if (sp.geometry(idx.data()).valid) pool[sa < 0 ? 0 : idx[sa]].push_back(k);
        }
    }
    // The next point, or false once every valid point has been drawn.
    bool next(int32_t *idx) {
        live.clear();
        for (size_t f = 0; f < pool.size(); ++f)
            if (!pool[f].empty()) live.push_back(int(f));
        if (live.empty()) return false;
        std::vector<uint64_t> &p = pool[live[rng.below(uint32_t(live.size()))]];
        const uint32_t j = rng.below(uint32_t(p.size()));
        sp.from_key(p[j], idx);
        p.erase(p.begin() + j);
        return true;
    }
};

std::vector<std::vector<int32_t>> draw_points(const Space &sp, uint64_t seed, int n_explore) {
    std::vector<std::vector<int32_t>> out;
    if (n_explore <= 0) return out;
    ExploreSampler smp(sp, seed);
    std::vector<int32_t> idx(sp.nknobs);
    while (int(out.size()) < n_explore && smp.next(idx.data())) out.push_back(idx);
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

// Droplet Search from `start` over the cached measurements `cache`.  With
// `line`, every move along one axis is followed by steps further along that
// axis in the same direction, one charged trial each, while a step is valid and
// better; the neighbourhood scan then resumes from where the steps stopped.
DropletOut droplet(const Space &sp, const int32_t *start, int budget, double alpha,
                   uint32_t frozen, std::unordered_map<uint64_t, Meas> &cache,
                   const MeasureFn &measure, double &best_so_far, ds_trace *trace,
                   bool line = false) {
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
        // The fastest measured neighbour (ties: first in neighbour order).  When
        // the budget ran out part-way through the neighbourhood, the neighbours
        // measured before it did still compete: they were paid for.
        int b = -1;
        for (size_t i = 0; i < nbs.size(); ++i) {
            auto it = cache.find(sp.key(nbs[i].data()));
            if (it == cache.end()) continue;
            if (b < 0 || it->second.median < cache[sp.key(nbs[size_t(b)].data())].median) b = int(i);
        }
        if (b < 0) break;
        const Meas &mb = cache[sp.key(nbs[size_t(b)].data())];
        if (!better(mb, cache[kcur], alpha)) break;
        int axis = 0;
        while (nbs[size_t(b)][axis] == cur[axis]) ++axis;
        const int dir = nbs[size_t(b)][axis] - cur[axis];
        cur = nbs[size_t(b)];
        kcur = sp.key(cur.data());
        out.moves++;
        while (line) {
            const int j = cur[axis] + dir;
            if (j < 0 || j >= int(sp.values[axis].size())) break;
            nb = cur;
            nb[axis] = j;
            if (!sp.geometry(nb.data()).valid) break;
            const uint64_t k = sp.key(nb.data());
            if (!cache.count(k)) {
                if (nb_measured >= budget) {
                    out.status = DS_EBUDGET;
                    stop = true;
                    break;
                }
                Meas m = measure(nb.data(), best_so_far);
                if (m.status != DS_OK) out.failed++;
                else best_so_far = best_so_far > 0 ? std::min(best_so_far, m.median) : m.median;
                cache[k] = m;
                nb_measured++;
                out.measured++;
                trace_push(trace, 2, m, k);
            }
            if (!better(cache[k], cache[kcur], alpha)) break;
            cur = nb;
            kcur = k;
            out.moves++;
        }
        if (stop) break;
    }
    out.best = cur;
    out.meas = cache[kcur];
    return out;
}

using Cache = std::unordered_map<uint64_t, Meas>;

void note_best(double &best_so_far, const Meas &m) {
    if (m.status == DS_OK) best_so_far = best_so_far > 0 ? std::min(best_so_far, m.median) : m.median;
}

struct ExploreOut {
    int ib = -1;           // fastest drawn point (ties: first drawn)
    double tb = std::numeric_limits<double>::infinity();
    int measured = 0;
    int failed = 0;
};

// Measures the drawn points into cache (cached points keep their measurement).
ExploreOut explore(const Space &sp, const std::vector<std::vector<int32_t>> &pts, Cache &cache,
                   const MeasureFn &measure, double &best_so_far, ds_trace *trace) {
    ExploreOut out;
    for (size_t i = 0; i < pts.size(); ++i) {
        const uint64_t k = sp.key(pts[i].data());
        auto it = cache.find(k);
        if (it == cache.end()) {
            Meas m = measure(pts[i].data(), best_so_far);
            trace_push(trace, 0, m, k);
            if (m.status != DS_OK) out.failed++;
            note_best(best_so_far, m);
            it = cache.emplace(k, std::move(m)).first;
            out.measured++;
        }
        if (out.ib < 0 || it->second.median < out.tb) {
            out.ib = int(i);
            out.tb = it->second.median;
        }
    }
    return out;
}

// Charging rules shared by Random, Grid and GA: cached candidates are skipped
// without charge; an invalid candidate is a failed trial (or skipped when
// valid_only); every other candidate is measured.
struct ExploitRun {
    const Space &sp;
    Cache &cache;
    const MeasureFn &measure;
    int budget;
    bool valid_only;
    double &best_so_far;
    ds_trace *trace;
    int charged = 0;
    int failed = 0;
    std::vector<uint64_t> order;

    bool exhausted() const { return charged >= budget; }

    bool try_point(const int32_t *idx) {
        const uint64_t k = sp.key(idx);
        if (cache.count(k)) return false;
        Meas m;
        if (!sp.valid(idx)) {
            if (valid_only) return false;
            m.status = DS_EINVALID_SCHED;
            m.median = std::numeric_limits<double>::infinity();
            m.full.status = DS_EINVALID_SCHED;
            m.full.median_ms = m.median;
        } else {
            m = measure(idx, best_so_far);
            note_best(best_so_far, m);
        }
        if (m.status != DS_OK) failed++;
        trace_push(trace, 2, m, k);
        cache.emplace(k, std::move(m));
        charged++;
        order.push_back(k);
        return true;
    }
};

// Independent uniform draws of every axis index; ends after max_draws draws.
struct RandomStream {
    SplitMix64 &rng;
    int64_t max_draws;
    int64_t draws = 0;

    bool next(const Space &sp, std::vector<int32_t> &out) {
        if (draws >= max_draws) return false;
        ++draws;
        out.resize(sp.nknobs);
        for (int a = 0; a < sp.nknobs; ++a) out[a] = int32_t(rng.below(uint32_t(sp.values[a].size())));
        return true;
    }
};

int roulette(SplitMix64 &rng, const std::vector<double> &w) {
    double total = 0.0;
    for (double v : w) total += v;
    if (!(total > 0.0)) return int(rng.below(uint32_t(w.size())));
    const double r = rng.uniform01() * total;
    double cum = 0.0;
    for (size_t i = 0; i < w.size(); ++i) {
        cum += w[i];
        if (cum > r) return int(i);
    }
    return int(w.size()) - 1;
}

double fitness(const Meas &m) {
    if (m.status != DS_OK || !std::isfinite(m.median) || !(m.median > 0.0)) return 0.0;
    return 1.0 / m.median;
}

// Genetic algorithm: generation zero is the start plus pop-1 Random draws; each
// next generation keeps the `elite` fastest points seen so far and adds
// children (roulette-selected parents, one-point crossover, per-gene mutation;
// 50 attempts at a new point, then a Random draw).
void run_ga(const Space &sp, ExploitRun &run, const std::vector<int32_t> &start, uint64_t seed,
            int pop, int elite, double mutation) {
    SplitMix64 rng(seed);
    RandomStream rs{rng, 100 * int64_t(run.budget)};
    const int d = sp.nknobs;
    std::vector<uint64_t> seen{sp.key(start.data())};     // GA members in measurement order
    std::vector<int32_t> tmp(d);
    auto from_stream = [&](std::vector<int32_t> &out) {
        while (rs.next(sp, tmp)) {
            if (run.exhausted()) return false;
            if (run.try_point(tmp.data())) {
                seen.push_back(sp.key(tmp.data()));
                out = tmp;
                return true;
            }
        }
        return false;
    };
    std::vector<std::vector<int32_t>> gen{start};
    while (int(gen.size()) < pop && !run.exhausted()) {
        std::vector<int32_t> p;
        if (!from_stream(p)) break;
        gen.push_back(p);
    }
    std::vector<int> rank;
    std::vector<double> weights;
    std::vector<int32_t> cand(d), p(d);
    while (!run.exhausted() && !gen.empty()) {
        rank.resize(seen.size());
        for (size_t i = 0; i < seen.size(); ++i) rank[i] = int(i);
        std::sort(rank.begin(), rank.end(), [&](int a, int b) {
            const double ma = run.cache.at(seen[a]).median, mb = run.cache.at(seen[b]).median;
            if (ma < mb) return true;
            if (mb < ma) return false;
            return a < b;
        });
        std::vector<std::vector<int32_t>> nxt;
        for (int i = 0; i < elite && i < int(rank.size()); ++i) {
            sp.from_key(seen[rank[i]], p.data());
            nxt.push_back(p);
        }
        weights.resize(gen.size());
        for (size_t i = 0; i < gen.size(); ++i)
            weights[i] = fitness(run.cache.at(sp.key(gen[i].data())));
        bool ended = false;
        while (int(nxt.size()) < pop && !run.exhausted()) {
            bool found = false;
            for (int attempt = 0; attempt < 50; ++attempt) {
                const int i = roulette(rng, weights);
                const int j = roulette(rng, weights);
                const int c = int(rng.below(uint32_t(d)));
                for (int a = 0; a < d; ++a) cand[a] = a < c ? gen[i][a] : gen[j][a];
                for (int a = 0; a < d; ++a)
                    if (rng.uniform01() < mutation)
                        cand[a] = int32_t(rng.below(uint32_t(sp.values[a].size())));
                if (run.cache.count(sp.key(cand.data()))) continue;
                if (run.valid_only && !sp.valid(cand.data())) continue;
                found = true;
                break;
            }
            if (found) {
                run.try_point(cand.data());
                seen.push_back(sp.key(cand.data()));
                nxt.push_back(cand);
            } else {
                if (!from_stream(p)) {
                    ended = true;
                    break;
                }
                nxt.push_back(p);
            }
        }
        gen.swap(nxt);
        if (ended) break;
    }
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
    Cache cache;
    double best_so_far = 0.0;
    const ExploreOut e = explore(sp, pts, cache, measure, best_so_far, trace);
    const double t1 = now_s();
    const DropletOut d = droplet(sp, pts[e.ib].data(), cfg.budget, cfg.alpha, cfg.frozen_mask,
                                 cache, measure, best_so_far, trace);
    const double t2 = now_s();
    free_device(owned);
    fill_result(res, sp, d);
    res->seed_point = make_sched(sp, pts[e.ib].data());
    res->seed_ms = e.tb;
    res->n_explore_measured = e.measured;
    res->n_droplet_measured = d.measured;
    res->n_failed = e.failed + d.failed;
    res->explore_s = t1 - t0;
    res->droplet_s = t2 - t1;
    res->wall_s = t2 - t0;
    return DS_OK;
}

int ds_cache_create(const ds_space *space, ds_cache **out) {
    if (!space || !out) {
        set_error("bad ds_cache_create arguments");
        return DS_EINVAL;
    }
    const Space &sp = space_of(space);
    ds_cache *c = new (std::nothrow) ds_cache;
    if (!c) return DS_ENOMEM;
    c->op = sp.op;
    std::copy(sp.shape, sp.shape + 9, c->shape);
    c->values = sp.values;
    *out = c;
    return DS_OK;
}

void ds_cache_destroy(ds_cache *cache) { delete cache; }

int ds_cache_clone(const ds_cache *cache, ds_cache **out) {
    if (!cache || !out) {
        set_error("bad ds_cache_clone arguments");
        return DS_EINVAL;
    }
    ds_cache *c = new (std::nothrow) ds_cache(*cache);
    if (!c) return DS_ENOMEM;
    *out = c;
    return DS_OK;
}

int ds_cache_size(const ds_cache *cache) {
    if (!cache) {
        set_error("null cache");
        return DS_EINVAL;
    }
    return int(cache->map.size());
}

int ds_cache_get(const ds_cache *cache, const ds_sched *s, ds_measurement *out) {
    if (!cache || !s || !out || s->nknobs != int(cache->values.size())) {
        set_error("bad ds_cache_get arguments");
        return DS_EINVAL;
    }
    uint64_t key = 0, radix = 1;
    for (size_t a = 0; a < cache->values.size(); ++a) {
        const int n = int(cache->values[a].size());
        if (s->idx[a] < 0 || s->idx[a] >= n) {
            set_error("schedule index out of range");
            return DS_EINVAL;
        }
        key += uint64_t(s->idx[a]) * radix;
        radix *= uint64_t(n);
    }
    auto it = cache->map.find(key);
    if (it == cache->map.end()) return 0;
    *out = it->second.full;
    out->status = it->second.status;
    out->median_ms = it->second.median;
    return 1;
}

int ds_explore(const ds_space *space, const ds_tune_cfg *cfg_in, const ds_tune_io *io,
               ds_measure_fn fn, void *ctx, ds_cache *cache, ds_tune_result *res,
               ds_trace *trace) {
    if (!space || !res || !cache) {
        set_error("bad ds_explore arguments");
        return DS_EINVAL;
    }
    std::memset(res, 0, sizeof *res);
    const Space &sp = space_of(space);
    if (!cache_fits(cache, sp)) {
        set_error("cache belongs to another space");
        return DS_EINVAL;
    }
    ds_tune_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_tune_cfg_default(&cfg);
    if (cfg.n_explore < 0) {
        set_error("negative n_explore");
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
    double best_so_far = 0.0;
    const ExploreOut e = explore(sp, pts, cache->map, measure, best_so_far, trace);
    free_device(owned);
    const Meas &mb = cache->map.at(sp.key(pts[e.ib].data()));
    res->seed_point = res->best = make_sched(sp, pts[e.ib].data());
    res->seed_ms = res->best_ms = e.tb;
    res->best_meas = mb.full;
    res->n_explore_measured = e.measured;
    res->n_failed = e.failed;
    res->explore_s = res->wall_s = now_s() - t0;
    return DS_OK;
}

void ds_exploit_cfg_default(ds_exploit_cfg *cfg) {
    if (!cfg) return;
    cfg->kind = DS_EXPLOIT_DROPLET;
    cfg->budget = 100;
    cfg->seed = 240620037ull;
    cfg->valid_only = 0;
    cfg->pop = 20;
    cfg->elite = 3;
    cfg->mutation = 0.1;
}

int ds_exploit(const ds_space *space, const ds_sched *start, const ds_exploit_cfg *cfg_in,
               const ds_tune_cfg *tcfg_in, const ds_tune_io *io, ds_measure_fn fn, void *ctx,
               ds_cache *cache, ds_tune_result *res, ds_trace *trace) {
    if (!space || !start || !res) {
        set_error("bad ds_exploit arguments");
        return DS_EINVAL;
    }
    std::memset(res, 0, sizeof *res);
    const Space &sp = space_of(space);
    ds_exploit_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_exploit_cfg_default(&cfg);
    ds_tune_cfg tcfg;
    if (tcfg_in) tcfg = *tcfg_in;
    else ds_tune_cfg_default(&tcfg);
    if (cfg.kind < DS_EXPLOIT_DROPLET || cfg.kind > DS_EXPLOIT_DROPLET_LINE || cfg.budget < 0 ||
        (cfg.kind == DS_EXPLOIT_GA &&
         (cfg.pop < 2 || cfg.elite < 0 || cfg.elite >= cfg.pop || !(cfg.mutation >= 0.0)))) {
        set_error("bad exploitation settings");
        return DS_EINVAL;
    }
    if (cache && !cache_fits(cache, sp)) {
        set_error("cache belongs to another space");
        return DS_EINVAL;
    }
    if (!sched_matches(sp, start) || !sp.in_range(start->idx)) {
        set_error("start point does not belong to the space");
        return DS_EINVAL;
    }
    if (!sp.valid(start->idx)) {
        set_error("start point is not a valid schedule");
        return DS_EINVALID_SCHED;
    }
    if (trace) trace->n = 0;
    float *owned = nullptr;
    int rc = prepare(sp, &tcfg, io, fn, &owned);
    if (rc != DS_OK) return rc;
    const MeasureFn measure = make_measure(sp, &tcfg, io, owned ? owned : (io ? io->ref : nullptr),
                                           fn, ctx);
    Cache local;
    Cache &c = cache ? cache->map : local;
    const std::vector<int32_t> st(start->idx, start->idx + sp.nknobs);
    const uint64_t k0 = sp.key(st.data());
    double best_so_far = 0.0;
    for (const auto &kv : c) note_best(best_so_far, kv.second);
    const double t0 = now_s();
    if (cfg.kind == DS_EXPLOIT_DROPLET || cfg.kind == DS_EXPLOIT_DROPLET_LINE) {
        const DropletOut d = droplet(sp, st.data(), cfg.budget, tcfg.alpha, tcfg.frozen_mask, c,
                                     measure, best_so_far, trace,
                                     cfg.kind == DS_EXPLOIT_DROPLET_LINE);
        fill_result(res, sp, d);
        res->n_droplet_measured = d.measured;
        res->n_failed = d.failed;
    } else {
        int start_measured = 0, start_failed = 0;
        if (!c.count(k0)) {
            Meas m = measure(st.data(), best_so_far);
            trace_push(trace, 1, m, k0);
            note_best(best_so_far, m);
            start_failed = m.status != DS_OK;
            c.emplace(k0, std::move(m));
            start_measured = 1;
        }
        ExploitRun run{sp, c, measure, cfg.budget, cfg.valid_only != 0, best_so_far, trace, 0, 0, {}};
        if (cfg.kind == DS_EXPLOIT_RANDOM) {
            SplitMix64 rng(cfg.seed);
            RandomStream rs{rng, 100 * int64_t(cfg.budget)};
            std::vector<int32_t> p;
            while (!run.exhausted() && rs.next(sp, p)) run.try_point(p.data());
        } else if (cfg.kind == DS_EXPLOIT_GRID) {
            std::vector<int32_t> p(sp.nknobs);
            for (uint64_t i = 1; i < sp.size && !run.exhausted(); ++i) {
                sp.from_key((k0 + i) % sp.size, p.data());
                run.try_point(p.data());
            }
        } else {
            run_ga(sp, run, st, cfg.seed, cfg.pop, cfg.elite, cfg.mutation);
        }
        uint64_t kb = k0;
        for (uint64_t k : run.order)
            if (c.at(k).median < c.at(kb).median) kb = k;
        std::vector<int32_t> b(sp.nknobs);
        sp.from_key(kb, b.data());
        res->best = make_sched(sp, b.data());
        res->best_ms = c.at(kb).median;
        res->best_meas = c.at(kb).full;
        res->status = DS_OK;
        res->n_droplet_measured = start_measured + run.charged;
        res->n_failed = start_failed + run.failed;
    }
    free_device(owned);
    res->seed_point = *start;
    res->seed_ms = c.at(k0).median;
    res->droplet_s = res->wall_s = now_s() - t0;
    return DS_OK;
}

int ds_tune_tasks(const ds_task *tasks, int n_tasks, int total_trials, const ds_tune_cfg *cfg_in,
                  ds_tune_result *results, ds_round *rounds, int rounds_cap, int *n_rounds,
                  double *network_ms) {
    if (!tasks || n_tasks <= 0 || total_trials < 0 || !results || (rounds_cap > 0 && !rounds) ||
        rounds_cap < 0) {
        set_error("bad ds_tune_tasks arguments");
        return DS_EINVAL;
    }
    for (int t = 0; t < n_tasks; ++t)
        if (!tasks[t].space || !(tasks[t].weight >= 0.0)) {
            set_error("task %d has no space or a negative weight", t);
            return DS_EINVAL;
        }
    ds_tune_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_tune_cfg_default(&cfg);
    if (cfg.budget < 0) {
        set_error("negative budget");
        return DS_EINVAL;
    }
    const int q = std::max(1, std::min(total_trials / n_tasks, 64));
    struct TaskState {
        const Space *sp = nullptr;
        float *owned = nullptr;
        MeasureFn measure;
        std::unique_ptr<ExploreSampler> smp;
        int taken = 0;
        bool ended = false;
        Cache cache;
        std::vector<int32_t> best;
        double best_t = std::numeric_limits<double>::infinity();
        double best_so_far = 0.0;
        int failed = 0;
        double explore_s = 0.0;
    };
    std::vector<TaskState> st(n_tasks);
    int rc = DS_OK;
    for (int t = 0; t < n_tasks && rc == DS_OK; ++t) {
        TaskState &T = st[t];
        T.sp = &space_of(tasks[t].space);
        rc = prepare(*T.sp, &cfg, &tasks[t].io, tasks[t].fn, &T.owned);
        if (rc != DS_OK) break;
        T.measure = make_measure(*T.sp, &cfg, &tasks[t].io,
                                 T.owned ? T.owned : tasks[t].io.ref, tasks[t].fn, tasks[t].ctx);
        T.smp.reset(new ExploreSampler(*T.sp, tasks[t].seed));
    }
    auto release = [&]() {
        for (auto &T : st) free_device(T.owned);
    };
    if (rc != DS_OK) {
        release();
        return rc;
    }
    for (int t = 0; t < n_tasks; ++t) std::memset(&results[t], 0, sizeof results[t]);
    int nr = 0;
    int64_t spent = 0;
    // Next n points of task t's sampler stream (the prefix rule of ansor_draw).
    auto run_round = [&](int t, int n) {
        TaskState &T = st[t];
        const Space &sp = *T.sp;
        const double t0 = now_s();
        const int target = T.taken + n;
        std::vector<int32_t> idx(sp.nknobs);
        int got = 0;
        while (T.taken < target && T.smp->next(idx.data())) {
            const uint64_t k = sp.key(idx.data());
            T.taken++;
            got++;
            Meas m = T.measure(idx.data(), T.best_so_far);
            if (m.status != DS_OK) T.failed++;
            note_best(T.best_so_far, m);
            if (T.best.empty() || m.median < T.best_t) {
                T.best = idx;
                T.best_t = m.median;
            }
            T.cache.emplace(k, std::move(m));
        }
        if (T.taken < target) T.ended = true;
        spent += got;
        if (nr < rounds_cap) rounds[nr] = ds_round{t, got};
        nr++;
        T.explore_s += now_s() - t0;
    };
    for (int t = 0; t < n_tasks; ++t) run_round(t, q);
    while (spent < total_trials) {
        int pick = -1;
        for (int t = 0; t < n_tasks; ++t) {
            if (st[t].ended || st[t].best.empty()) continue;
            if (pick < 0 || tasks[t].weight * st[t].best_t > tasks[pick].weight * st[pick].best_t)
                pick = t;
        }
        if (pick < 0) break;
        run_round(pick, int(std::min<int64_t>(q, total_trials - spent)));
    }
    double net = 0.0;
    for (int t = 0; t < n_tasks; ++t) {
        TaskState &T = st[t];
        ds_tune_result &r = results[t];
        r.n_explore_measured = T.taken;
        r.explore_s = T.explore_s;
        if (T.best.empty()) {
            r.status = DS_EEXHAUSTED;
            r.best_ms = r.seed_ms = std::numeric_limits<double>::infinity();
            continue;
        }
        const double t0 = now_s();
        const DropletOut d = droplet(*T.sp, T.best.data(), cfg.budget, cfg.alpha, cfg.frozen_mask,
                                     T.cache, T.measure, T.best_so_far, nullptr);
        fill_result(&r, *T.sp, d);
        r.seed_point = make_sched(*T.sp, T.best.data());
        r.seed_ms = T.best_t;
        r.n_droplet_measured = d.measured;
        r.n_failed = T.failed + d.failed;
        r.droplet_s = now_s() - t0;
        r.wall_s = r.explore_s + r.droplet_s;
        net += tasks[t].weight * r.best_ms;
    }
    release();
    if (n_rounds) *n_rounds = nr;
    if (network_ms) *network_ms = net;
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
