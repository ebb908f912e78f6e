// Internal declarations shared by the library's translation units.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

#include "droplet.h"

namespace ds {

// ---- errors ---------------------------------------------------------------
void set_error(const char *fmt, ...);
const char *last_error();

// ---- lattice ----------------------------------------------------------------
constexpr int kLdsLimit = 163840;     // bytes of LDS per workgroup on gfx950
constexpr int kThreadsLimit = 1024;
constexpr int64_t kGridLimit = 2147483647;

// LDS stages of a matmul K-tile: one without dbuf; with dbuf three when they
// fit in LDS (two tiles in flight while one is consumed), else two.
constexpr int mm_stages(int bm, int bn, int bk, int dbuf) {
    return !dbuf ? 1 : (int64_t(3) * (bm * bk + bk * bn) * 4 <= kLdsLimit ? 3 : 2);
}

// Wave groups splitting each K-tile of the MFMA matmul inside a workgroup:
// two for a reduction split (ks >= 2) when the K-tile has at least 8 steps.
constexpr int mm_wave_groups(int mfma, int ks, int bk) { return mfma && ks >= 2 && bk >= 8 ? 2 : 1; }

struct Geometry {
    bool valid = false;
    int threads = 0;
    int64_t grid = 0;
    int lds_bytes = 0;
    int acc = 0;
    int unroll_eff = 1;
    int t0 = 0, t1 = 0;
    int red = 0;
    int64_t chunks = 0;
};

struct Space {
    int op = 0;                       // 0: generic lattice (no kernel)
    int nknobs = 0;
    int64_t shape[9] = {0};
    std::vector<std::vector<int32_t>> values;
    std::vector<const char *> names;
    std::vector<uint64_t> invalid_keys;   // generic lattices only (sorted)
    uint64_t size = 1;

    bool in_range(const int32_t *idx) const;
    uint64_t key(const int32_t *idx) const;
    void from_key(uint64_t key, int32_t *idx) const;
    Geometry geometry(const int32_t *idx) const;
    bool valid(const int32_t *idx) const;
    int value(const int32_t *idx, int axis) const { return values[axis][idx[axis]]; }
};

// Builds the space of a kernel family at a shape; returns DS_OK or an error.
int build_space(int op, const int64_t *shape, int shape_len, Space &out);

// Conv output extent.
inline int64_t conv_out_dim(int64_t in, int64_t f, int64_t st, int64_t pd) {
    return (in + 2 * pd - f) / st + 1;
}

ds_sched make_sched(const Space &sp, const int32_t *idx);
bool sched_matches(const Space &sp, const ds_sched *s);

// ---- launch plans -------------------------------------------------------------
// Division by a run-time invariant d in [1, 2^31) for dividends n in [0, 2^31)
// (Granlund & Montgomery, "Division by invariant integers using
// multiplication", PLDI 1994): q = (umulhi(n, m) + n) >> s with
// s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1.
struct FastDiv {
    uint32_t m;
    int s;
};

inline FastDiv make_fastdiv(int d) {
    int s = 0;
    while ((int64_t(1) << s) < d) ++s;
    const uint64_t m = ((uint64_t(1) << 32) * ((uint64_t(1) << s) - uint64_t(d))) / uint64_t(d) + 1;
    return FastDiv{uint32_t(m), s};
}

// Arguments of the conv kernels (passed by value).
struct ConvArgs {
    const float *x;
    const float *w;
    float *y;
    int N, C, H, W, K, R, S, st, pd, P, Q;
    int tk, th, tw, tc;
    int tiles_k, tiles_p, tiles_q, ks;
    int chunks, cps;      // reduction chunks, chunks per split
    int red, wrow;        // reduction length per chunk, LDS weight row stride
    int hs, ws;           // halo tile extent
    int npx, npl;         // pixels per tile, lanes covering pixels (VALU)
    int ltw;              // log2(tw)
    int nbuf, buf;        // LDS buffers (1 or 2) and floats per buffer (16-byte multiple)
    float *part;          // ks > 1: split z writes its partial output at part + z * N*K*P*Q
    int w4;               // bit 0: weight rows staged with 16-byte copies (C*R*S, tc*R*S,
                          //    wrow multiples of 4 and w 16-byte aligned); bit 1: halo
                          //    rows too (aligned layout, tk*wrow a multiple of 4, x
                          //    16-byte aligned); bit 2: aligned halo layout (W a
                          //    multiple of 4 and tw*st >= 16: rows start at the
                          //    16-byte boundary at or before the tile's first column)
    FastDiv f_hw, f_ws, f_red, f_rs, f_s, f_wrow;   // divisions by hs*ws, ws, red, R*S, S, wrow
};

struct MatmulArgs {
    const float *A;
    const float *B;
    float *C;
    int M, N, K;
    int tiles_m, tiles_n, ks;
    int nkt, kps;         // K-tiles, K-tiles per split
    int vecA, vecB;       // 1: 16-byte loads along K of A / along N of B are legal
    int direct;           // 1: every tile is full and aligned: K-tiles go straight to LDS
    float *part;          // ks > 1: split z writes its partial C at part + z * M*N
    int gm;               // tile rows per group of the XCD tile order (mm_group_rows)
};

// Tile rows per group of the matmul tile order: the power of two (at most
// tiles_m) that minimises the A rows plus B columns, in elements, touched by
// the contiguous tile range of one XCD (ties: the smaller), so that range is
// square in elements whatever the tile's aspect.
inline int mm_group_rows(int tiles_m, int tiles_n, int ks, int bm, int bn) {
    const int64_t tiles = int64_t(tiles_m) * tiles_n * ks;
    const int64_t per_xcd = tiles > 8 ? (tiles + 7) / 8 : 1;
    int best = 1;
    int64_t cost = INT64_MAX;
    for (int gm = 1; gm <= tiles_m && gm > 0; gm *= 2) {
        const int64_t rows = gm < per_xcd ? gm : per_xcd;
        int64_t cols = (per_xcd + gm - 1) / gm;
        if (cols > tiles_n) cols = tiles_n;
        const int64_t c = rows * bm + cols * bn;
        if (c < cost) {
            cost = c;
            best = gm;
        }
    }
    return best;
}

struct Plan {
    const void *func = nullptr;
    int family = 0;           // DS_KERNEL_* of the selected instance
    int nparams = 0;
    int params[6] = {0, 0, 0, 0, 0, 0};   // its template parameters
    int slot = -1;            // its slot in the family's instance table
    int threads = 0;
    int64_t grid = 0;
    int lds = 0;
    int splits = 1;           // non-empty reduction splits; > 1: partials reduced into y
    int64_t y_elems = 0;
    int op = 0;
    ConvArgs conv{};
    MatmulArgs mm{};
};

// Builds the plan of schedule s for buffers (x, w, y); DS_EINVALID_SCHED if s is
// not a valid point.
int make_plan(const ds_sched *s, const float *x, const float *w, float *y, Plan &plan);
int attach_workspace(Plan &plan, hipStream_t stream);   // split reductions: per-stream partials
int launch_plan(const Plan &plan, hipStream_t stream);

// Kernel instance lookup (compiled template instances).
const void *conv_valu_instance(int kpt, int ppt, int uf, int lds);
const void *conv_mfma_instance(int tkb, int npb, int d, int lds);
const void *mm_valu_instance(int rm, int rn, int bk, int uf, int dbuf);
const void *mm_mfma_instance(int wm, int wn, int bk, int uf, int dbuf, int kg);
int count_instances();

// ---- measurement -----------------------------------------------------------------
struct Meas {
    int status = DS_OK;
    double median = 0;
    std::vector<double> repeats;
    ds_measurement full{};
};

// Rank-sum test: one-sided p-value that a is stochastically smaller than b.
double ranksum_p_less(const std::vector<double> &a, const std::vector<double> &b);
bool better(const Meas &a, const Meas &b, double alpha);

// Device helpers (harness).
int fill_async(float *p, int64_t n, float v, hipStream_t stream);
int reference_output(const Space &sp, const ds_tune_io *io, float **ref_out);
void free_device(void *p);

}  // namespace ds
