// Internal declarations shared by the library's translation units.
#pragma once

#include <algorithm>
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

// Arguments of the channel-quad MFMA conv (conv_mfma2, mfma = 2).  A
// workgroup stages, per reduction chunk of tc channels, the weights of its tk
// output channels ([kl][c_l*R*S + r*S + s], rows wrow floats apart) and the
// input halo of its tile ([c_l][hy][hx], channels cs floats apart) in LDS; one
// MFMA k-step takes four consecutive channels (a "quad") at one tap (r, s), so
// both operands are read at a uniform offset from a per-lane base.
struct Conv2Args {
    const float *x;
    const float *w;
    float *y;
    float *part;          // ksw > 1: split z writes its partial output at part + z * N*K*P*Q
    int N, C, H, W, K, R, S, st, pd, P, Q;
    int tk, th, tw, tc;   // tc: real channels of a full chunk (C when C < 4)
    int tiles_k, tiles_p, tiles_q, ksw;   // ksw: reduction splits across workgroups
                          //    (band tiles: tiles_p = 1, tiles_q = bands, no image axis)
    int band;             // band tiles (tw >= Q): a tile is th * tw consecutive pixels of
                          //    the flattened (image, row, column) output space
    int hp;               // band tiles: padded rows per image, (P - 1) * st + R; image n's
                          //    output row p reads padded rows n * hp + p * st + r
    int F;                // band tiles: N * P * Q
    int st4;              // output stores of 4 consecutive pixels are 16-byte aligned (y and
                          //    partials 16-byte aligned; P*Q, and for rectangles Q and tw,
                          //    multiples of 4)
    int chunks, cps;      // reduction chunks, chunks per split
    int t4;               // channel quads per chunk (channel slots / 4)
    int hs, ws, cs;       // halo rows, halo row stride, halo channel stride (floats)
    int wrow;             // weight row stride (floats; 4 * odd for 16-byte weight copies,
                          //    else 2 * odd)
    int npx, ltw, wpx, lwpx;   // tile pixels, log2(tw), pixel waves and log2
    int bufw, buf;        // floats of the weight part of a buffer, of a whole buffer
    int nbuf;             // LDS buffers (2 when a workgroup walks more than one chunk)
    int hal;              // aligned halo layout: rows start at the 16-byte boundary at
                          //    or before the tile's first column (W % 4 == 0, tw*st >= 16)
    int vw, vh;           // 16-byte copies of weight / halo units (else 4-byte)
    int nw4, nh4;         // copy units of a chunk (weights, halo)
    int ncopy;            // copy units per thread per kind
    int rc;               // copy units per thread the instance holds in registers (RC)
    int regs;             // ncopy <= rc: a full chunk's sources stay in registers
    int wr_u, hc_u, hr_u; // copy units per weight row, halo channel, halo row
    int w_dk, w_dc;       // blockDim in (weight row, unit) mixed radix
    int h_dc, h_dr;       // blockDim in (halo channel, unit) mixed radix
    FastDiv f_wru, f_hcu, f_hru, f_rs, f_s, f_tk, f_tq, f_tp, f_ksw;
    FastDiv f_q, f_p, f_hp, f_pq;   // band tiles: Q, P, hp, P*Q
};

// Launch shape of a conv_mfma2 point.
struct Conv2Shape {
    bool valid = false;
    int tkb = 0, npb = 0, u = 1, kg = 1;   // template parameters
    int threads = 0;
    int64_t grid = 0;
    int64_t lds = 0;
    int red = 0;                          // channel slots x taps of one chunk
};

constexpr int kConv2MaxCopies = 12;       // copy units per thread of a valid point

// Copy units per thread a conv_mfma2 instance keeps in registers across
// chunks (its RC template parameter): 4 when a point needs no more, or when
// its workgroups walk a single chunk (the registers that frees buy many
// instances more waves per SIMD), else 12.
constexpr int kConv2FewCopies = 4;

// Register budget of the compiled conv_mfma2 instances (no spill; launch bound
// 256 * KG): TKB x NPB blocks per wave and TKB + NPB operand floats per quad.
constexpr bool conv2_regs_ok(int tkb, int npb, int kg) {
    return tkb * npb <= (kg == 4 ? 4 : kg == 2 ? 16 : 32) &&
           tkb + npb <= (kg == 4 ? 8 : kg == 2 ? 12 : 20);
}

// Copy units of conv_mfma2 for its copy widths (vw, vh) and thread count.
inline void conv2_units(Conv2Args &a, int threads) {
    const int tc4 = 4 * a.t4;
    a.nw4 = a.vw ? a.bufw / 4 : a.bufw;
    a.nh4 = int(a.vh ? int64_t(tc4) * a.cs / 4 : std::min<int64_t>(int64_t(tc4) * a.cs, INT32_MAX));
    a.ncopy = std::max((a.nw4 + threads - 1) / threads, (a.nh4 + threads - 1) / threads);
    // (a workgroup that walks one chunk never reuses its sources: the 4-unit
    // instance, whatever the count)
    a.rc = a.ncopy <= kConv2FewCopies || a.cps <= 1 ? kConv2FewCopies : kConv2MaxCopies;
    a.regs = a.ncopy <= a.rc;
    a.wr_u = a.vw ? a.wrow / 4 : a.wrow;
    a.hc_u = a.vh ? a.cs / 4 : a.cs;
    a.hr_u = a.vh ? a.ws / 4 : a.ws;
    a.w_dk = threads / a.wr_u; a.w_dc = threads % a.wr_u;
    a.h_dc = threads / a.hc_u; a.h_dr = threads % a.hc_u;
    a.f_wru = make_fastdiv(a.wr_u); a.f_hcu = make_fastdiv(a.hc_u); a.f_hru = make_fastdiv(a.hr_u);
}

// Halo rows of a band of npx consecutive output pixels (flattened over
// image, row, column): it spans at most D output rows, and consecutive rows
// are st padded rows apart inside an image and R across an image boundary
// (image n's rows start at n * hp, hp = (P - 1) * st + R), so the padded
// rows it reads number at most (D - 1) * st + X * max(0, R - st) + R with X
// the image boundaries among its D rows.
inline int64_t conv2_band_rows(int64_t N, int64_t P, int64_t Q, int64_t R, int64_t st, int64_t npx) {
    const int64_t d = std::max<int64_t>(1, std::min(N * P, 1 + (npx - 1 + Q - 1) / Q));
    const int64_t x = std::min(N - 1, (d - 1 + P - 1) / P);
    return (d - 1) * st + std::max<int64_t>(0, x) * std::max<int64_t>(0, R - st) + R;
}

// Set-up of conv_mfma2 for shape sh and knob values (depth D = 1..3 from the
// unroll knob; the k-steps unrolled per loop step are U = 2^(D-1) quads).
// The in-workgroup reduction split KG is the largest of 4, 2, 1 not above ks
// that divides the quads of a chunk into whole U-blocks and fits 1024
// threads; the rest of ks splits across workgroups.  Rectangular tiles
// (band false) are th x tw pixels of one image, within its P x Q; band tiles
// are th * tw consecutive pixels of the output flattened over (image, row,
// column), across row and image boundaries, whose halo is a range of padded
// rows.  Fills a (buffers aside) and returns the shape with its
// validity: a tile of at least one 16x16 block, chunks of whole channel quads
// (tc >= 4, or for fewer than four image channels tc = 1 standing for all of
// them), the register budget of the compiled instances (no spill), the copy
// units a thread holds, LDS, and copy offsets within 31 bits.
inline Conv2Shape conv2_setup(const int64_t *sh, int tk, int th, int tw, int tc, int depth, int ks,
                              int vec, bool band, Conv2Args &a) {
    Conv2Shape g;
    a = Conv2Args();
    a.N = int(sh[0]); a.C = int(sh[1]); a.H = int(sh[2]); a.W = int(sh[3]); a.K = int(sh[4]);
    a.R = int(sh[5]); a.S = int(sh[6]); a.st = int(sh[7]); a.pd = int(sh[8]);
    a.P = int(conv_out_dim(sh[2], sh[5], sh[7], sh[8]));
    a.Q = int(conv_out_dim(sh[3], sh[6], sh[7], sh[8]));
    a.tk = tk; a.th = th; a.tw = tw;
    const int RS = a.R * a.S;
    bool ok = tk >= 16 && th * tw >= 16 && (tc >= 4 || (a.C < 4 && tc == 1));
    a.band = band;
    ok = ok && (band || (th <= a.P && tw <= a.Q));
    a.tc = a.C < 4 ? a.C : tc;
    const int tc4 = (a.tc + 3) / 4 * 4;
    a.t4 = tc4 / 4;
    a.npx = th * tw;
    a.wpx = std::min(4, std::max(1, a.npx / 16));
    a.lwpx = a.wpx >= 4 ? 2 : a.wpx - 1;
    int l = 0;
    while ((1 << l) < tw) ++l;
    a.ltw = l;
    g.tkb = std::max(1, tk / 16);
    g.npb = std::max(1, a.npx / (16 * a.wpx));
    g.u = 1 << (depth - 1);
    int kg = std::min(ks, 4);
    while (kg > 1 && (a.t4 % (kg * g.u) != 0 || 64 * a.wpx * kg > 1024)) kg /= 2;
    g.kg = kg;
    a.ksw = ks / kg;
    const int body = g.tkb * g.npb;
    ok = ok && 4 * body <= 128 && a.t4 % (kg * g.u) == 0 && conv2_regs_ok(g.tkb, g.npb, kg);
    a.chunks = int((a.C + a.tc - 1) / a.tc);
    a.cps = (a.chunks + a.ksw - 1) / a.ksw;
    ok = ok && a.ksw <= a.chunks;
    const int64_t span_w = a.band ? a.Q : tw;         // output columns a halo row covers
    int64_t hs = int64_t(th - 1) * a.st + a.R;
    if (a.band) {
        hs = conv2_band_rows(a.N, a.P, a.Q, a.R, a.st, a.npx);
        a.hp = (a.P - 1) * a.st + a.R;
    }
    a.hs = int(std::min<int64_t>(hs, INT32_MAX));
    const bool halo16 = vec == 4 && a.W % 4 == 0 && span_w * a.st >= 16;
    a.ws = int(halo16 ? ((span_w - 1) * a.st + a.S + 3 + 3) / 4 * 4 : (span_w - 1) * a.st + a.S);
    int64_t cs = hs * a.ws;
    cs += ((16 - cs % 32) + 32) % 32;                 // cs = 16 mod 32: the four lane groups'
    a.cs = int(std::min<int64_t>(cs, INT32_MAX));     // channels fall on disjoint banks
    a.vw = vec == 4 && (int64_t(a.C) * RS) % 4 == 0 && (int64_t(a.tc) * RS) % 4 == 0;
    // Weight rows: the 16 rows of a block are read together, one float each,
    // by lanes of the same channel, 32 lanes at a time.  4 * odd floats apart
    // (16-byte copies need rows of whole 16-byte groups) puts them on 8 banks
    // of each 4-bank group; 2 * odd puts them on 16 distinct banks.
    const int64_t unit = a.vw ? 4 : 2;
    int64_t odd = (int64_t(tc4) * RS + unit - 1) / unit;
    if (odd % 2 == 0) ++odd;
    a.wrow = int(std::min<int64_t>(unit * odd, INT32_MAX));
    a.hal = halo16;
    a.vh = halo16;
    ok = ok && (vec == 1 || a.vw || a.vh);
    a.bufw = int(std::min<int64_t>(int64_t(tk) * a.wrow, INT32_MAX));
    const int64_t buf = int64_t(tk) * a.wrow + int64_t(tc4) * a.cs;
    a.buf = int(std::min<int64_t>(buf, INT32_MAX));
    a.nbuf = a.cps > 1 ? 2 : 1;
    g.threads = 64 * a.wpx * kg;
    conv2_units(a, g.threads);
    // a full chunk's copy units are held in registers (chunks with channel
    // slots past C, C < 4, compute theirs as they go)
    ok = ok && (a.C < 4 || a.ncopy <= kConv2MaxCopies);
    a.tiles_k = int((a.K + tk - 1) / tk);
    int64_t grid;
    if (a.band) {
        const int64_t F = int64_t(a.N) * a.P * a.Q;
        a.F = int(std::min<int64_t>(F, INT32_MAX));
        a.tiles_p = 1;
        a.tiles_q = int((F + a.npx - 1) / a.npx);
        grid = int64_t(a.ksw) * a.tiles_k * a.tiles_q;
        // copy offsets from the band's first image: at most `imgs` images
        const int64_t imgs = std::min<int64_t>(a.N, 1 + (a.npx - 1 + int64_t(a.P) * a.Q - 1) /
                                                          (int64_t(a.P) * a.Q));
        ok = ok && (imgs * a.C + tc4) * int64_t(a.H) * a.W < (int64_t(1) << 29);
    } else {
        a.tiles_p = int((a.P + th - 1) / th);
        a.tiles_q = int((a.Q + tw - 1) / tw);
        grid = int64_t(a.N) * a.ksw * a.tiles_k * a.tiles_p * a.tiles_q;
        ok = ok && int64_t(tc4) * a.H * a.W < (int64_t(1) << 29);
    }
    ok = ok && int64_t(tk) * a.C * RS < (int64_t(1) << 29);
    a.f_rs = make_fastdiv(RS); a.f_s = make_fastdiv(a.S);
    a.f_tk = make_fastdiv(a.tiles_k); a.f_tq = make_fastdiv(std::max(1, a.tiles_q));
    a.f_tp = make_fastdiv(a.tiles_p); a.f_ksw = make_fastdiv(a.ksw);
    a.f_q = make_fastdiv(a.Q); a.f_p = make_fastdiv(a.P); a.f_hp = make_fastdiv(std::max(1, a.hp));
    a.f_pq = make_fastdiv(std::max(1, a.P * a.Q));
    a.st4 = band ? (int64_t(a.P) * a.Q) % 4 == 0 : a.Q % 4 == 0 && tw % 4 == 0;
    // buffers; the wave groups' partial tiles; the output staging rows (16
    // rows of 68 floats per pixel wave)
    g.lds = std::max<int64_t>({4 * int64_t(a.nbuf) * buf,
                               int64_t(16) * (kg - 1) * a.wpx * 64 * body,
                               int64_t(4) * 16 * 68 * a.wpx});
    g.grid = grid;
    g.red = tc4 * RS;
    g.valid = ok && g.lds <= kLdsLimit && g.threads <= kThreadsLimit && g.grid <= kGridLimit;
    return g;
}

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
    Conv2Args conv2{};        // family DS_KERNEL_CONV_MFMA2
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
const void *conv_mfma2_instance(int tkb, int npb, int u, int kg, int rc);
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
