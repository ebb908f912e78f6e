/*
 * droplet.h -- C ABI of the MI355X (gfx950) schedule-tuning library.
 *
 * The library implements the measurement-driven core of the combined
 * explore/exploit kernel scheduler of "Explore as a Storm, Exploit as a
 * Raindrop" (Canesche, Verma, Pereira): a schedule-parameterised fp32 kernel family (NCHW conv2d and
 * row-major matmul) written in HIP for gfx950, a hipEvent measurement harness,
 * a seeded exploration sampler and Droplet Search coordinate descent.
 *
 * Conventions for every entry point:
 *   - The return value is a status: DS_OK (0) or a negative DS_E* code.  No
 *     C++ exception crosses the ABI.  ds_last_error() gives a thread-local
 *     message for the last failing call on the calling thread.
 *   - Device pointers are plain HIP device addresses owned by the caller
 *     (allocated through PyTorch or hipMalloc), contiguous, 16-byte aligned.
 *   - Streams are the caller's; work is enqueued asynchronously unless the
 *     entry point says it synchronises.
 *   - ds_sched is a plain value type owned by the caller; ds_space is opaque
 *     and owned by the library until sched_space_destroy().
 */
#ifndef DROPLET_H
#define DROPLET_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
enum {
    DS_OK = 0,
    DS_EINVAL = -1,          /* bad argument (null pointer, bad shape, bad index) */
    DS_EUNSUPPORTED = -2,    /* unknown op, or no device of the supported kind */
    DS_EINVALID_SCHED = -3,  /* schedule outside the valid search space: nothing launched */
    DS_EHIP = -4,            /* a HIP runtime call failed; see ds_last_error() */
    DS_EPARITY = -5,         /* output failed the parity check against the reference */
    DS_EBUDGET = -6,         /* Droplet stopped because its trial budget ran out (informational) */
    DS_EEXHAUSTED = -7,      /* the lattice has no (more) valid point to draw */
    DS_ENOMEM = -8           /* host or device allocation failed */
};

/* ---- operations -------------------------------------------------------- */
enum {
    DS_OP_CONV2D_NCHW = 1,   /* shape = {N,C,H,W,K,R,S,stride,pad}             */
    DS_OP_MATMUL_RM = 2      /* shape = {M,N,K}                                */
};

#define DS_MAX_KNOBS 12
#define DS_MAX_REPEATS 64

/*
 * A schedule: one point of the search space of a kernel family at a shape
 * (Definition 1: an annotation of a sketch; Section 2.2: its coordinates).
 * idx[a] is the position on axis a's ordered value list.  Entries of shape
 * and idx beyond the op's length are ignored and should be zero.
 */
typedef struct {
    int32_t op;
    int32_t nknobs;
    int64_t shape[9];
    int32_t idx[DS_MAX_KNOBS];
} ds_sched;

typedef struct ds_space ds_space;

/*
 * sched_space_create -- the kernel search space of one kernel family at one
 * shape (Definition 1).  conv2d axes, in order: tk, th, tw, tc (powers of two
 * 1..64 kept if <= K, P, Q, C; th and tw also keep the smallest power of two
 * >= P, Q), unroll {0,16,64,512}, lds {0,1}, ks {1,2,4,...,32} (kept if
 * <= C), mfma {0,1,2,3}, vec {1,4} (floats per lane of the global -> LDS
 * copies).
 * conv mfma: 0 VALU FMA; 1 fp32 MFMA over 16-step groups of the (c, r, s)
 * reduction (a per-chunk offset table locates each tap); 2 fp32 MFMA over
 * (tap, channel quad) steps, LDS staging only, where ks first splits every
 * chunk's quads between up to four wave groups of one workgroup (summed in
 * LDS) and the rest across workgroups; 3 the same over band tiles: th * tw
 * consecutive pixels of the output flattened over (image, row, column).  Only
 * band tiles may reach past the output's height or width.  matmul axes: bm,
 * bn {16,...,256} (kept if <= M, N), bk {4,...,64} (kept if <= K), unroll,
 * dbuf {0,1}, mfma {0,1}, ks {1,2,4,8} (kept if <= K), vec {1,4} (floats per
 * lane of the operand loads).  The
 * smallest value of a clipped axis is always kept.  A point is valid when its
 * kernel fits the hardware (threads, LDS, workgroups) and the register budget
 * of its compiled instance (no spill), and, for vec 4, an operand can move 16
 * bytes per lane.  Accepted shapes: conv N >= 0 (0 is the empty
 * batch), C,H,W,K,R,S,stride >= 1, pad >= 0, at least one output position;
 * matmul M >= 0, N,K >= 1.  *out receives a new space (free it with
 * sched_space_destroy).  Errors: DS_EINVAL, DS_EUNSUPPORTED, DS_ENOMEM.
 */
int sched_space_create(int op, const int64_t *shape, int shape_len, ds_space **out);

/*
 * sched_space_create_lattice -- a generic lattice for exercising the search
 * drivers with a caller-supplied cost (Section 2.2, Example 3 is such a
 * lattice).  nvalues[a] values per axis, taken consecutively from values[].
 * Every point is valid unless invalid_keys (nullable, n_invalid entries)
 * lists its key.  The space has op 0 and cannot be launched.
 */
int sched_space_create_lattice(int nknobs, const int32_t *nvalues, const int32_t *values,
                               const uint64_t *invalid_keys, int n_invalid, ds_space **out);

void sched_space_destroy(ds_space *space);

/* op, number of axes and number of lattice points (valid or not). */
int sched_space_info(const ds_space *space, int *op, int *nknobs, uint64_t *size);

/* Axis a: name (static string), number of values and the value list (owned
 * by the space). */
int sched_space_axis(const ds_space *space, int axis, const char **name, int *nvalues,
                     const int32_t **values);

/* 1 if s is a valid point of the space, 0 if not, < 0 on a bad argument.  The
 * search space of a sketch is the set of its valid annotations (Definition 1);
 * Section 3 (RQ4) notes that some annotations give kernels that cannot run,
 * which is what this predicate excludes. */
int sched_valid(const ds_space *space, const ds_sched *s);

/* Mixed-radix key of a point of the lattice whose coordinates are the knob
 * indices (Section 2.2, Example 3): sum over axes of idx[a] * prod_{b<a}
 * nvalues[b]. */
int sched_key(const ds_space *space, const ds_sched *s, uint64_t *key);
int sched_from_key(const ds_space *space, uint64_t key, ds_sched *out);

/*
 * sched_neighbors -- the neighbourhood of Section 2.2: points one index step
 * away on one axis, axis order ascending, the -1 step before the +1 step;
 * out-of-range and invalid points are left out.  Writes min(n, cap) points,
 * *n_out = n (at most 2 * nknobs).
 */
int sched_neighbors(const ds_space *space, const ds_sched *s, ds_sched *out, int cap,
                    int *n_out);

/* The point that applies no optimisation (Section 2.2, step 1): index 0 on
 * every axis, or the first valid point in key order.  DS_EEXHAUSTED if none. */
int sched_origin(const ds_space *space, ds_sched *out);

/* Launch geometry and derived template parameters of a point (valid or not). */
typedef struct {
    int32_t valid;
    int32_t threads;      /* workgroup size */
    int64_t grid;         /* number of workgroups (1-D) */
    int32_t lds_bytes;    /* dynamic LDS per workgroup */
    int32_t acc;          /* fp32 accumulators per lane */
    int32_t unroll_eff;   /* unroll factor of the reduction loop (conv MFMA: the
                             number of 16-step groups read ahead, 1..3) */
    int32_t t0, t1;       /* conv VALU: channels, pixels per thread; conv MFMA:
                             16-channel blocks, 16-pixel blocks per wave;
                             matmul VALU: rows, cols per thread; matmul MFMA:
                             wave tile rows, cols */
    int32_t red;          /* conv: reduction length per chunk; matmul: k per MFMA/FMA step */
    int64_t chunks;       /* conv: reduction chunks; matmul: K-steps */
} ds_geometry;
int sched_geometry(const ds_space *space, const ds_sched *s, ds_geometry *out);

/*
 * ansor_draw -- the exploration sampler's draw sequence without measuring
 * (Section 2.3, step 1; Section 2.1 annotation initialisation read as uniform
 * draws): per draw, one index per axis from SplitMix64(seed), unbiased by
 * rejection; invalid and repeated points are rejected; stops after n_explore
 * distinct valid points or 100 * n_explore draws.  Writes *n_out points to out
 * (capacity n_explore).
 */
int ansor_draw(const ds_space *space, uint64_t seed, int n_explore, ds_sched *out, int *n_out);

/* 1 if a compiled kernel instance implements valid schedule s, 0 if not
 * (host only, launches nothing). */
int sched_has_kernel(const ds_space *space, const ds_sched *s);

/* Kernel families (the sketches whose annotations the spaces enumerate). */
enum {
    DS_KERNEL_CONV_VALU = 1,  /* conv_valu<KPT, PPT, UF, LDS> */
    DS_KERNEL_CONV_MFMA = 2,  /* conv_mfma<TKB, NPB, D, LDS> (conv mfma = 1) */
    DS_KERNEL_MM_VALU = 3,    /* mm_valu<RM, RN, BK, UF, DB> */
    DS_KERNEL_MM_MFMA = 4,    /* mm_mfma<WM, WN, BK, UF, DB, KG> */
    DS_KERNEL_CONV_MFMA2 = 5  /* conv_mfma2<TKB, NPB, U, KG> (conv mfma = 2 and 3) */
};

/* The compiled program a valid schedule selects (Definition 1: an annotated
 * sketch is a concrete program): its template instance, its launch geometry
 * and a hash of its kernel-argument block (buffer pointers left null), so two
 * schedules launch identical work iff instance and args_hash agree.  With
 * with_attrs = 1 the instance's compiled attributes are read with
 * hipFuncGetAttributes (needs a device); with 0 no HIP call is made. */
typedef struct {
    int32_t family;                /* DS_KERNEL_* */
    int32_t nparams;
    int32_t params[6];             /* template parameters in declaration order */
    int32_t instance;              /* family * 4096 + slot in the family's table */
    int32_t threads;               /* workgroup size */
    int64_t grid;                  /* workgroups */
    int32_t lds_bytes;             /* dynamic LDS per workgroup */
    int32_t splits;                /* reduction splits across workgroups (> 1: reduce launch) */
    uint64_t args_hash;
    int32_t num_regs;              /* with_attrs: registers per lane */
    int32_t max_threads_per_block; /* with_attrs: the instance's launch bound */
    int64_t local_bytes;           /* with_attrs: scratch per lane (register spills) */
    int64_t static_lds_bytes;      /* with_attrs: statically declared LDS */
} ds_kernel_info;

/* Errors: DS_EINVAL, DS_EINVALID_SCHED (s not valid), DS_EUNSUPPORTED (no
 * compiled instance), DS_EHIP (attribute query failed). */
int sched_kernel_info(const ds_space *space, const ds_sched *s, int with_attrs,
                      ds_kernel_info *out);

/* Every valid point of a kernel space in key order with the program it
 * selects: keys[i], instances[i] and args_hashes[i] as sched_kernel_info
 * reports them (host only, no HIP call).  Writes min(n, cap) entries; *n_out
 * = n, the number of valid points.  For tests and tools. */
int sched_space_programs(const ds_space *space, uint64_t *keys, int32_t *instances,
                         uint64_t *args_hashes, int64_t cap, int64_t *n_out);

/* ---- kernels ------------------------------------------------------------ */

/*
 * kernel_run -- launch the kernel that schedule s selects (Definition 1: an
 * annotated sketch is a concrete program).  conv: x = input [N,C,H,W], w =
 * weight [K,C,R,S], y = output [N,K,P,Q] with P = (H+2pad-R)/stride+1 and
 * Q likewise; y[n,k,p,q] = sum_{c,r,s} x[n,c,p*stride-pad+r,q*stride-pad+s] *
 * w[k,c,r,s], out-of-range inputs read as 0.  matmul: x = A [M,K], w = B
 * [K,N], y = C [M,N] = A*B, row-major.  fp32 in, out and accumulate.
 * Asynchronous on stream; y is overwritten.  An empty output launches nothing.
 * A split reduction (ks > 1) writes its partial outputs to a workspace the
 * library keeps per (device, stream): split launches on different streams do
 * not share partials.  When a stream's workspace is too small it is replaced
 * by a larger one (hipMalloc; the old one is kept until ds_shutdown, since a
 * graph captured earlier may still use it, and the stream is synchronised
 * first).  Under stream capture nothing may be allocated: a split schedule
 * whose workspace does not exist yet on that stream returns DS_EUNSUPPORTED
 * (run it once on the stream before capturing, or use kernel_run_noalloc).
 * Errors: DS_EINVAL, DS_EINVALID_SCHED (nothing launched), DS_EHIP,
 * DS_ENOMEM, DS_EUNSUPPORTED.
 */
int kernel_run(int op, const ds_sched *s, const float *x, const float *w, float *y,
               hipStream_t stream);

/*
 * kernel_run_noalloc -- kernel_run for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  It launches the same kernels as kernel_run, but the
 * partial outputs of a split reduction (ks > 1) go to a fixed array in device
 * memory (one per device, DS_NOALLOC_MAX_FLOATS floats = 32 MiB, held by the
 * library until the process ends) instead of a library-allocated workspace.
 * It calls no hipMalloc or hipFree.  A split schedule whose partials (ks *
 * output elements) exceed DS_NOALLOC_MAX_FLOATS floats is rejected with
 * DS_EINVAL and launches nothing.  Every call on one device shares that device's array:
 * calls that overlap in time on one device (different streams, or different
 * host threads) race on it and give wrong outputs; order them on one stream.
 * The array is fully rewritten by each split launch before it is read, so it
 * needs no clearing.  Arguments, layout and other errors as kernel_run.
 */
#define DS_NOALLOC_MAX_FLOATS 8388608
int kernel_run_noalloc(int op, const ds_sched *s, const float *x, const float *w, float *y,
                       hipStream_t stream);

/* The library's plain one-thread-per-output kernel for the same operation
 * (used as the in-tuning reference when the caller supplies none). */
int kernel_run_reference(int op, const int64_t *shape, const float *x, const float *w, float *y,
                         hipStream_t stream);

/* ---- measurement -------------------------------------------------------- */

typedef struct {
    int32_t warmup;        /* untimed launches before timing (default 3) */
    int32_t repeat;        /* timed repeats (default 11, at most DS_MAX_REPEATS) */
    double min_repeat_ms;  /* launches per repeat chosen so a repeat lasts this long (0.5) */
    int32_t max_number;    /* cap on launches per repeat (200) */
    double slow_cut;       /* a candidate whose first launch is slower than
                              slow_cut * best_so_far is timed once only (4.0; 0 = never) */
    double tol;            /* parity: max|y-ref| <= tol * max|ref| (1e-4) */
    int32_t check;         /* 1: parity-check the first launch against ref */
    int32_t graph;         /* 1: time each repeat as one replay of a HIP graph holding
                              `number` launches, on a library-owned stream (after
                              synchronising io->stream); the output of the last
                              replay is parity-checked again.  0: launch from the host
                              on io->stream (default 1) */
} ds_measure_cfg;

/* Fills cfg with the defaults above. */
void ds_measure_cfg_default(ds_measure_cfg *cfg);

typedef struct {
    int32_t status;        /* DS_OK, DS_EPARITY, DS_EHIP, DS_EINVALID_SCHED */
    int32_t n_repeats;
    int32_t number;        /* launches per repeat */
    int32_t cut;           /* 1 if timed once because of slow_cut */
    double median_ms;      /* median over repeats of (repeat time / number); +inf on failure */
    double mean_ms;
    double min_ms;
    double first_ms;       /* time of the parity launch */
    double max_err;        /* parity: max |y - ref| */
    double max_ref;        /* parity: max |ref| */
    int64_t nonfinite;     /* parity: count of non-finite outputs */
    double repeats_ms[DS_MAX_REPEATS];
} ds_measurement;

/* Buffers a measurement runs on.  ref (nullable) is the fp32 reference output
 * used by the parity check. */
typedef struct {
    const float *x;
    const float *w;
    float *y;
    const float *ref;
    hipStream_t stream;
} ds_tune_io;

/*
 * ds_measure -- one trial, the observed execution of a concrete schedule
 * (Section 2.1, "Termination in Ansor"; each search step of Section 2.2 is
 * such a measurement): parity-check the first launch (y is
 * pre-filled with NaN; the check fails on NaN/Inf or max|y-ref| > tol*max|ref|),
 * warm up, then time cfg->repeat repeats of `number` launches between two
 * hipEvents on io->stream.  Synchronises the stream.  best_so_far_ms (0 = none)
 * drives slow_cut.  out->status is the trial's status; the return value is
 * DS_OK unless an argument is bad.
 */
int ds_measure(const ds_sched *s, const ds_tune_io *io, const ds_measure_cfg *cfg,
               double best_so_far_ms, ds_measurement *out);

/* Per-launch time of an empty kernel in the same harness (the dispatch floor),
 * host launches or graph replays as cfg->graph says. */
int ds_empty_kernel_floor(hipStream_t stream, const ds_measure_cfg *cfg, ds_measurement *out);

/* Floats the sink of ds_mfma_ceiling must hold: one per thread of its grid
 * (1024 workgroups of 256 threads). */
#define DS_MFMA_CEILING_SINK 262144

/* ds_mfma_ceiling -- the fp32 MFMA rate this device sustains with no memory
 * traffic: every wave (four on each SIMD) issues back-to-back 16x16x4 fp32
 * MFMAs into 16 independent accumulator blocks, iters rounds of 16.  A
 * calibration of the measurement, like the empty-kernel floor (the paper
 * defines no such operation): the rate the tuned MFMA kernels can approach on
 * this device, next to the published peak, which assumes the nominal clock.
 * sink: device buffer of at least
 * DS_MFMA_CEILING_SINK floats, owned by the caller, overwritten.  Launches
 * one timed kernel per repeat (cfg->warmup untimed first); *flop receives
 * the flop of one launch, out->median_ms its time.  Errors: DS_EINVAL (null
 * pointer, iters < 1, sink too small), DS_EHIP. */
int ds_mfma_ceiling(hipStream_t stream, float *sink, int64_t sink_elems, int iters,
                    const ds_measure_cfg *cfg, ds_measurement *out, double *flop);

/* ---- tuning --------------------------------------------------------------- */

/* A measurement callback: fills *out for schedule s, returns DS_OK or an error
 * (an error is a failed trial with infinite time). */
typedef int (*ds_measure_fn)(void *ctx, const ds_sched *s, ds_measurement *out);

typedef struct {
    int32_t n_explore;     /* exploration samples (300, Section 3 RQ1) */
    int32_t budget;        /* Droplet trial cap (100, Section 3 RQ2) */
    double alpha;          /* significance of "faster" (0.05; >= 1: plain median <) */
    uint64_t seed;         /* sampler seed */
    uint32_t frozen_mask;  /* bit a set: axis a is held at the start's value */
    ds_measure_cfg measure;
} ds_tune_cfg;

void ds_tune_cfg_default(ds_tune_cfg *cfg);

typedef struct {
    ds_sched best;
    double best_ms;
    ds_sched seed_point;          /* best exploration sample (the Droplet start) */
    double seed_ms;
    int32_t status;               /* DS_OK, DS_EBUDGET (informational), DS_EEXHAUSTED, ... */
    int32_t n_explore_measured;
    int32_t n_droplet_measured;   /* new measurements made by Droplet (start included) */
    int32_t n_failed;             /* failed trials (parity, launch) */
    int32_t n_moves;              /* accepted Droplet moves */
    double wall_s, explore_s, droplet_s;
    ds_measurement best_meas;
} ds_tune_result;

typedef struct {
    int32_t stage;                /* 0 explore, 1 droplet start, 2 droplet neighbour */
    int32_t status;
    uint64_t key;
    double median_ms;
} ds_trace_entry;

typedef struct {
    ds_trace_entry *entries;      /* caller-owned array of cap entries */
    int32_t cap;
    int32_t n;                    /* entries written (the library sets it) */
} ds_trace;

/*
 * ansor_sample -- the exploration of the combined approach (Sections 2.1 and
 * 2.3): draw n_explore points (as ansor_draw) and measure each on the GPU; *best is the fastest (ties: first drawn).  If io->ref is NULL
 * the library computes a reference with kernel_run_reference.
 */
int ansor_sample(const ds_space *space, uint64_t seed, int n_explore, const ds_tune_io *io,
                 const ds_measure_cfg *cfg, ds_sched *best, double *best_ms, ds_trace *trace);

/*
 * droplet_tune_ex -- Droplet Search (Section 2.2) from start (NULL = the
 * no-optimisation origin): measure the uncached valid neighbours of the
 * current point, move to the fastest if it is faster (median lower and, for
 * alpha < 1, one-sided rank-sum p < alpha, the 95% criterion of Section 3
 * RQ4/RQ5), else stop.  At most `budget` neighbour measurements; the start is
 * measured once more if needed.  fn NULL measures on the GPU with io (ref as in
 * ansor_sample); otherwise fn(ctx, ...) supplies every measurement.
 */
int droplet_tune_ex(const ds_space *space, const ds_sched *start, int budget,
                    const ds_tune_cfg *cfg, const ds_tune_io *io, ds_measure_fn fn, void *ctx,
                    ds_tune_result *res, ds_trace *trace);

/*
 * ds_tune -- the combined approach (Section 2.3): explore cfg->n_explore
 * samples, give the best to Droplet Search with cfg->budget, run it to
 * convergence.  Samples are cached, so Droplet never re-measures them.
 */
int ds_tune(const ds_space *space, const ds_tune_cfg *cfg, const ds_tune_io *io,
            ds_measure_fn fn, void *ctx, ds_tune_result *res, ds_trace *trace);

/* ---- measurement cache, exploration, exploitation strategies --------------- */

/*
 * ds_cache -- the measurements of one space, keyed by lattice key (opaque,
 * library-owned until ds_cache_destroy).  Exploration fills it; every
 * exploitation strategy skips points it holds and adds what it measures, so
 * several strategies can start from one exploration (Section 3, RQ4: each
 * technique exploits the same best exploration sample).  A cache is bound to
 * the space it was created for (same op, shape and axes).
 */
typedef struct ds_cache ds_cache;

int ds_cache_create(const ds_space *space, ds_cache **out);
void ds_cache_destroy(ds_cache *cache);
/* Deep copy (so each strategy starts from the same exploration state). */
int ds_cache_clone(const ds_cache *cache, ds_cache **out);
/* Number of cached points (>= 0) or a negative status. */
int ds_cache_size(const ds_cache *cache);
/* 1 and *out filled if s is cached, 0 if not, < 0 on error. */
int ds_cache_get(const ds_cache *cache, const ds_sched *s, ds_measurement *out);

/*
 * ds_explore -- the exploration alone (Section 2.3, first step): draw
 * cfg->n_explore points (as ansor_draw with cfg->seed) and measure each into
 * cache; a point already cached keeps its measurement and is not measured
 * again.  res->seed_point / seed_ms (and
 * best / best_ms) are the fastest drawn point (ties: first drawn);
 * n_explore_measured counts new measurements; n_failed and explore_s are
 * filled.  DS_EEXHAUSTED if nothing can be drawn.
 */
int ds_explore(const ds_space *space, const ds_tune_cfg *cfg, const ds_tune_io *io,
               ds_measure_fn fn, void *ctx, ds_cache *cache, ds_tune_result *res,
               ds_trace *trace);

/* Exploitation strategies compared in Section 3, RQ4. */
enum {
    DS_EXPLOIT_DROPLET = 0,  /* Droplet Search (Section 2.2): converges, at most budget trials */
    DS_EXPLOIT_RANDOM = 1,   /* independent uniform draws of each axis index */
    DS_EXPLOIT_GRID = 2,     /* mixed-radix walk key(start)+1, +2, ... (first axis fastest) */
    DS_EXPLOIT_GA = 3,       /* genetic algorithm: elitism, roulette selection by 1/time,
                                one-point crossover, per-gene mutation */
    DS_EXPLOIT_DROPLET_LINE = 4  /* Droplet Search with line steps: after each move along
                                    one axis, keep stepping that way (one charged trial per
                                    step) while the step is valid and better, then scan the
                                    neighbourhood again (the paper calls Droplet a line search
                                    and presents it without its speculative steps, Section
                                    2.2; this is one reading of those steps) */
};

typedef struct {
    int32_t kind;          /* DS_EXPLOIT_* */
    int32_t budget;        /* charged trials (100, Section 3 RQ4) */
    uint64_t seed;         /* SplitMix64 stream of Random and GA */
    int32_t valid_only;    /* 0: an invalid candidate is a failed trial that costs one
                              trial, as in the paper's host framework (default);
                              1: invalid candidates are skipped without charge.
                              Droplet visits valid neighbours only, either way. */
    int32_t pop;           /* GA population (20; >= 2) */
    int32_t elite;         /* GA elites kept per generation (3; 0 <= elite < pop) */
    double mutation;       /* GA per-gene mutation probability (0.1) */
} ds_exploit_cfg;

void ds_exploit_cfg_default(ds_exploit_cfg *cfg);

/*
 * ds_exploit -- run one strategy from start (must be a valid point).  The start
 * is measured (not charged) unless cached.  Random, Grid and GA skip cached
 * candidates without charge, stop after cfg->budget charged trials or when
 * their candidate stream ends (Random: 100*budget draws; Grid: back at the
 * start; GA: neither crossover nor the Random stream yields a new point), and
 * return the fastest of the start and their trials (ties: earliest).  Droplet
 * and Droplet with line steps run as droplet_tune_ex with cfg->budget (they
 * visit valid points only, so valid_only has no effect on them).
 * tcfg supplies alpha, frozen_mask (Droplet) and the measurement settings.
 * cache may be NULL (a private one is used).  res->n_droplet_measured counts
 * the strategy's measurements (start included when measured), res->n_failed
 * its failed trials, res->droplet_s its wall-clock.  Trace stages: 1 start,
 * 2 trial.
 */
int ds_exploit(const ds_space *space, const ds_sched *start, const ds_exploit_cfg *cfg,
               const ds_tune_cfg *tcfg, const ds_tune_io *io, ds_measure_fn fn, void *ctx,
               ds_cache *cache, ds_tune_result *res, ds_trace *trace);

/* One kernel (task) of a network for ds_tune_tasks. */
typedef struct {
    const ds_space *space;
    ds_tune_io io;         /* GPU buffers of this task (used when fn is NULL) */
    ds_measure_fn fn;      /* NULL: measure on the GPU; else fn(ctx, ...) */
    void *ctx;
    double weight;         /* occurrences of the kernel in the network */
    uint64_t seed;         /* this task's exploration stream */
} ds_task;

typedef struct {
    int32_t task;
    int32_t trials;
} ds_round;

/*
 * ds_tune_tasks -- one exploration budget for a whole network (Section 2.1,
 * Termination in Ansor; Section 3 setup): each task first receives
 * q = max(1, min(total_trials / n_tasks, 64)) trials in task order; while fewer
 * than total_trials were spent, the live task with the largest weight *
 * best time (ties: lowest index) receives min(q, total_trials - spent) more; a
 * task whose stream ends leaves the worklist.  A task's trials are the next
 * points of its sampler stream (the first n of ansor_draw(seed, n)).  Then
 * Droplet Search runs per task from its best sample with cfg->budget and
 * cfg->alpha.  results[t] holds task t's outcome; rounds (nullable, cap
 * rounds_cap) the allocation order; *n_rounds the number of rounds;
 * *network_ms = sum(weight * best_ms).
 */
int ds_tune_tasks(const ds_task *tasks, int n_tasks, int total_trials, const ds_tune_cfg *cfg,
                  ds_tune_result *results, ds_round *rounds, int rounds_cap, int *n_rounds,
                  double *network_ms);

/*
 * droplet_tune -- the four-argument form: builds the space, allocates seeded
 * U[-1,1) inputs on the current device (SplitMix64 streams 240620037 for x / A
 * and 240620038 for w, 240620039 for B), runs Droplet Search from start
 * (NULL = origin) with `budget` on
 * the default stream, frees everything, returns the best point and its median
 * time in ms.
 */
int droplet_tune(int op, const int64_t *shape, const ds_sched *start, int budget, ds_sched *best,
                 double *best_ms);

/* ---- misc ------------------------------------------------------------------ */

const char *ds_last_error(void);

/* Host-side U[-1,1) SplitMix64 stream (the same definition the tests' input
 * generator uses), for inputs the library creates itself. */
int ds_gen_uniform(uint64_t seed, int64_t n, float *out);

/* Current device: compute units, peak engine clock (kHz), arch name. */
int ds_device_info(int *cus, int *clock_khz, char *arch, int arch_len);

/* Number of compiled kernel instances (all families). */
int ds_num_instances(void);

/* Release library-owned device buffers of every device. */
void ds_shutdown(void);

#ifdef __cplusplus
}
#endif

#endif /* DROPLET_H */
