// Schedule lattices of the two kernel families (Definition 1: the search space
// of a sketch is every valid annotation; Section 2.2: one coordinate axis per
// varying parameter, neighbours one step away on one axis).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "ds_internal.h"

namespace ds {

namespace {

thread_local std::string g_error;

const int32_t kPow2to64[] = {1, 2, 4, 8, 16, 32, 64};
const int32_t kUnroll[] = {0, 16, 64, 512};
const int32_t kSplit[] = {1, 2, 4, 8};
// conv splits reach 32: a batch-1 layer with few output pixels fills the
// chip only through its reduction
const int32_t kConvSplit[] = {1, 2, 4, 8, 16, 32};
const int32_t kMmTile[] = {16, 32, 64, 128, 256};
const int32_t kMmBk[] = {4, 8, 16, 32, 64};
const int32_t kOnOff[] = {0, 1};
const int32_t kConvMfma[] = {0, 1, 2, 3};
const int32_t kVec[] = {1, 4};

const char *kConvNames[] = {"tk", "th", "tw", "tc", "unroll", "lds", "ks", "mfma", "vec"};
const char *kMmNames[] = {"bm", "bn", "bk", "unroll", "dbuf", "mfma", "ks", "vec"};
const char *kGenericNames[] = {"p0", "p1", "p2", "p3", "p4", "p5",
                               "p6", "p7", "p8", "p9", "p10", "p11"};

// Values of `list` that do not exceed `extent`; the smallest value if none does.
template <size_t L>
std::vector<int32_t> clipped(const int32_t (&list)[L], int64_t extent) {
    std::vector<int32_t> out;
    for (int32_t v : list)
        if (v <= extent) out.push_back(v);
    if (out.empty()) out.push_back(*std::min_element(list, list + L));
    return out;
}

// The clipped list plus the smallest value that covers `extent`, if the list
// has one above it: a tile may span a whole output row or column.
template <size_t L>
std::vector<int32_t> covering(const int32_t (&list)[L], int64_t extent) {
    std::vector<int32_t> out = clipped(list, extent);
    for (int32_t v : list)
        if (v >= extent) {
            if (v > out.back()) out.push_back(v);
            break;
        }
    return out;
}

// Largest value of the clipped list.
template <size_t L>
int64_t clipped_max(const int32_t (&list)[L], int64_t extent) {
    int64_t best = -1;
    for (int32_t v : list)
        if (v <= extent && v > best) best = v;
    return best >= 0 ? best : *std::min_element(list, list + L);
}

template <size_t L>
std::vector<int32_t> all_of(const int32_t (&list)[L]) {
    return std::vector<int32_t>(list, list + L);
}

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

int pow2_floor(int64_t v) {
    int p = 1;
    while (int64_t(p) * 2 <= v) p *= 2;
    return p;
}

Geometry conv_geometry(const int64_t *sh, const int32_t *v) {
    const int64_t N = sh[0], C = sh[1], H = sh[2], W = sh[3], K = sh[4], R = sh[5], S = sh[6],
                  st = sh[7], pd = sh[8];
    const int64_t P = conv_out_dim(H, R, st, pd), Q = conv_out_dim(W, S, st, pd);
    const int tk = v[0], th = v[1], tw = v[2], tc = v[3], unroll = v[4], lds = v[5], ks = v[6],
              mfma = v[7], vec = v[8];
    Geometry g;
    const int npx = th * tw;
    const int outs = tk * npx;
    if (mfma >= 2) {
        // channel-quad MFMA family (mfma 2: rectangular tiles, mfma 3: band
        // tiles): LDS staging only; its unroll depth is taken like the other
        // MFMA family's (3 from 16 unrolled steps, 2 from 4), over its 16x16
        // blocks
        const int body2 = std::max(1, tk / 16) * std::max(1, npx / (16 * std::min(4, std::max(1, npx / 16))));
        const int ue = unroll == 0 ? 1 : std::min(16, pow2_floor(std::max(1, unroll / body2)));
        const int depth = ue >= 16 ? 3 : (ue >= 4 ? 2 : 1);
        Conv2Args a;
        const Conv2Shape c = conv2_setup(sh, tk, th, tw, tc, depth, ks, vec, mfma == 3, a);
        g.threads = c.threads;
        g.grid = c.grid;
        g.lds_bytes = int(std::min<int64_t>(c.lds, INT32_MAX));
        g.acc = 4 * c.tkb * c.npb;
        g.unroll_eff = depth;
        g.t0 = c.tkb;
        g.t1 = c.npb;
        g.red = c.red;
        g.chunks = a.chunks;
        g.valid = c.valid && lds == 1;
        return g;
    }
    // tiles past the output's height or width exist only as band tiles
    if (th > P || tw > Q) return g;
    bool ok;
    int body, wrow;
    if (!mfma) {
        // Lanes take pixels first, then groups of channels; one wave at least,
        // or the largest tile a smaller shape allows.
        const int64_t biggest =
            clipped_max(kPow2to64, K) * clipped_max(kPow2to64, P) * clipped_max(kPow2to64, Q);
        ok = outs >= std::min<int64_t>(64, biggest);
        int kpt, ppt;
        if (npx >= 256) {
            g.threads = 256;
            ppt = npx / 256;
            kpt = tk;
        } else {
            g.threads = std::min(256, outs);
            const int groups = std::max(1, g.threads / npx);
            kpt = std::max(1, tk / groups);
            ppt = 1;
        }
        g.acc = kpt * ppt;
        body = g.acc;
        ok = ok && g.acc <= 64;
        g.red = int(tc * R * S);
        wrow = g.red;
        g.t0 = kpt;
        g.t1 = ppt;
    } else {
        // Up to four waves split the pixels (one per 16-pixel block for tiles
        // under 64 pixels); 16x16 output blocks per wave.
        const int waves = std::min(4, std::max(1, npx / 16));
        g.threads = 64 * waves;
        ok = tk >= 16 && npx >= 16;
        const int tkb = std::max(1, tk / 16), npb = std::max(1, npx / (16 * waves));
        g.acc = 4 * tkb * npb;
        body = tkb * npb;
        ok = ok && g.acc <= 128;
        g.red = int(cdiv(tc * R * S, 16) * 16);
        wrow = g.red + 4;
        g.t0 = tkb;
        g.t1 = npb;
    }
    // aligned halo layout (16-byte copies, image rows of whole 16-byte groups,
    // tiles of at least 16 input columns): rows start at the 16-byte boundary
    // at or before the tile's first column, up to 3 more columns, rounded to 4
    const bool halo16 = vec == 4 && W % 4 == 0 && int64_t(tw) * st >= 16;
    const int64_t hs = int64_t(th - 1) * st + R;
    const int64_t ws = halo16 ? cdiv(int64_t(tw - 1) * st + S + 3, 4) * 4 : int64_t(tw - 1) * st + S;
    g.chunks = std::max<int64_t>(1, cdiv(C, tc));
    int64_t lds_bytes;
    if (lds) {
        // Two buffers (weights + halo + a zero float, 16-byte rounded) when a
        // workgroup walks more than one chunk, then the offset table.
        const int64_t nbuf = cdiv(g.chunks, ks) > 1 ? 2 : 1;
        const int64_t buf = cdiv(int64_t(tk) * wrow + tc * hs * ws + 1, 4) * 4;
        // + the reduction table and the staging source tables
        lds_bytes = 4 * (nbuf * buf + int64_t(g.red) + int64_t(tk) * wrow + int64_t(tc) * hs * ws);
    } else {
        lds_bytes = 8 * int64_t(g.red);
    }
    g.lds_bytes = int(std::min<int64_t>(lds_bytes, INT32_MAX));
    g.grid = N * ks * cdiv(K, tk) * cdiv(P, th) * cdiv(Q, tw);
    g.unroll_eff = unroll == 0 ? 1 : std::min(16, pow2_floor(std::max(1, unroll / body)));
    if (mfma) {
        // The MFMA family unrolls its group loop by its read-ahead depth D
        // (1..3); its D+1 operand sets hold 4*(tkb + npb) floats each.  Register
        // budget of the compiled instances (no spill): at most 96 such floats,
        // or 192 with D = 1.
        g.unroll_eff = g.unroll_eff >= 16 ? 3 : (g.unroll_eff >= 4 ? 2 : 1);
        const int ring = (g.unroll_eff + 1) * 4 * (g.t0 + g.t1);
        ok = ok && (ring <= 96 || (g.unroll_eff == 1 && ring <= 192));
    } else {
        // register budget: 64 accumulators on the global path fit only a
        // loop unrolled less than 8 times
        ok = ok && !(lds == 0 && g.acc == 64 && g.unroll_eff >= 8);
    }
    // vec = 4 (16-byte global -> LDS copies) needs LDS staging by whole waves
    // and at least one operand whose staged rows are whole 16-byte groups
    if (vec == 4) {
        const bool w16 = (C * R * S) % 4 == 0 && (int64_t(tc) * R * S) % 4 == 0 && wrow % 4 == 0;
        const bool h16 = halo16 && (int64_t(tk) * wrow) % 4 == 0;
        ok = ok && lds && g.threads % 64 == 0 && (w16 || h16);
    }
    g.valid = ok && lds_bytes <= kLdsLimit && g.threads <= kThreadsLimit && ks <= g.chunks &&
              g.grid <= kGridLimit;
    return g;
}

Geometry mm_geometry(const int64_t *sh, const int32_t *v) {
    const int64_t M = sh[0], N = sh[1], K = sh[2];
    const int bm = v[0], bn = v[1], bk = v[2], unroll = v[3], dbuf = v[4], mfma = v[5], ks = v[6],
              vec = v[7];
    Geometry g;
    bool ok;
    int body, kstep;
    if (!mfma) {
        const int rm = bm / 16, rn = bn / 16;
        g.acc = rm * rn;
        body = g.acc;
        kstep = 1;
        ok = g.acc <= 128;
        g.t0 = rm;
        g.t1 = rn;
    } else {
        ok = bm >= 32 && bn >= 32;
        const int wm = bm / 2, wn = bn / 2;
        int blocks;
        if (wm >= 32 && wn >= 32) {
            kstep = 2;
            blocks = (wm / 32) * (wn / 32);
            g.acc = 16 * blocks;
        } else {
            kstep = 4;
            blocks = std::max(1, wm / 16) * std::max(1, wn / 16);
            g.acc = 4 * blocks;
        }
        body = blocks;
        ok = ok && g.acc <= 256;
        g.t0 = wm;
        g.t1 = wn;
    }
    const int trip = std::max(1, bk / kstep);
    if (unroll == 0)
        g.unroll_eff = 1;
    else if (trip * body <= unroll)
        g.unroll_eff = trip;
    else
        g.unroll_eff = std::min(trip, pow2_floor(std::max(1, unroll / body)));
    // a reduction split first splits each K-tile between wave groups of one
    // workgroup, then the K-tiles between workgroups (partials + reduce)
    const int kg = mm_wave_groups(mfma, ks, bk);
    const int wgs = ks / kg;
    // Register budget of the compiled instances (no spill): two wave groups
    // (512 threads) leave half the registers per lane, so at most 64
    // accumulators; a 128x128 wave tile with a 16-deep K-tile unrolled 8
    // times and one LDS stage does not fit; a VALU tile whose next K-tile is
    // staged through registers (dbuf) fits (rm + rn) * unroll <= 512.
    if (mfma)
        ok = ok && (kg == 1 || g.acc <= 64) &&
             !(g.acc == 256 && !dbuf && bk == 16 && g.unroll_eff == 8);
    else
        ok = ok && (!dbuf || (g.t0 + g.t1) * g.unroll_eff <= 512);
    const int64_t lds = std::max<int64_t>(int64_t(mm_stages(bm, bn, bk, dbuf)) * (bm * bk + bk * bn),
                                          kg > 1 ? int64_t(bm) * bn : 0) * 4;
    g.lds_bytes = int(std::min<int64_t>(lds, INT32_MAX));
    g.red = kstep;
    g.chunks = cdiv(K, bk);
    g.grid = cdiv(M, bm) * cdiv(N, bn) * wgs;
    g.threads = 256 * kg;
    // vec = 4 (16-byte operand loads) needs rows of A (K) or of B (N) in whole
    // 16-byte groups
    ok = ok && (vec == 1 || K % 4 == 0 || N % 4 == 0);
    g.valid = ok && lds <= kLdsLimit && g.threads <= kThreadsLimit && wgs <= g.chunks &&
              g.grid <= kGridLimit;
    return g;
}

}  // namespace

void set_error(const char *fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
}

const char *last_error() { return g_error.c_str(); }

bool Space::in_range(const int32_t *idx) const {
    for (int a = 0; a < nknobs; ++a)
        if (idx[a] < 0 || idx[a] >= int32_t(values[a].size())) return false;
    return true;
}

uint64_t Space::key(const int32_t *idx) const {
    uint64_t k = 0, radix = 1;
    for (int a = 0; a < nknobs; ++a) {
        k += uint64_t(idx[a]) * radix;
        radix *= values[a].size();
    }
    return k;
}

void Space::from_key(uint64_t k, int32_t *idx) const {
    for (int a = 0; a < nknobs; ++a) {
        const uint64_t n = values[a].size();
        idx[a] = int32_t(k % n);
        k /= n;
    }
}

Geometry Space::geometry(const int32_t *idx) const {
    int32_t v[DS_MAX_KNOBS];
    for (int a = 0; a < nknobs; ++a) v[a] = values[a][idx[a]];
    if (op == DS_OP_CONV2D_NCHW) return conv_geometry(shape, v);
    if (op == DS_OP_MATMUL_RM) return mm_geometry(shape, v);
    Geometry g;
    g.valid = !std::binary_search(invalid_keys.begin(), invalid_keys.end(), key(idx));
    return g;
}

bool Space::valid(const int32_t *idx) const { return in_range(idx) && geometry(idx).valid; }

int build_space(int op, const int64_t *sh, int shape_len, Space &sp) {
    if (!sh) {
        set_error("shape is null");
        return DS_EINVAL;
    }
    sp = Space();
    sp.op = op;
    if (op == DS_OP_CONV2D_NCHW) {
        if (shape_len != 9) {
            set_error("conv2d shape has 9 entries, got %d", shape_len);
            return DS_EINVAL;
        }
        const int64_t N = sh[0], C = sh[1], H = sh[2], W = sh[3], K = sh[4], R = sh[5],
                      S = sh[6], st = sh[7], pd = sh[8];
        if (N < 0 || C < 1 || H < 1 || W < 1 || K < 1 || R < 1 || S < 1 || st < 1 || pd < 0) {
            set_error("bad conv2d shape");
            return DS_EINVAL;
        }
        if (H + 2 * pd < R || W + 2 * pd < S) {
            set_error("conv2d shape has no output position");
            return DS_EINVAL;
        }
        const int64_t P = conv_out_dim(H, R, st, pd), Q = conv_out_dim(W, S, st, pd);
        if (N * C * H * W > INT32_MAX || K * C * R * S > INT32_MAX || N * K * P * Q > INT32_MAX ||
            R > 255 || S > 255 || st > 64 || pd > 64 || H > 65535 || W > 65535) {
            set_error("conv2d shape exceeds the 32-bit index range of the kernels");
            return DS_EUNSUPPORTED;
        }
        for (int i = 0; i < 9; ++i) sp.shape[i] = sh[i];
        sp.values = {clipped(kPow2to64, K), covering(kPow2to64, P), covering(kPow2to64, Q),
                     clipped(kPow2to64, C), all_of(kUnroll), all_of(kOnOff),
                     clipped(kConvSplit, C), all_of(kConvMfma), all_of(kVec)};
        sp.names.assign(kConvNames, kConvNames + 9);
    } else if (op == DS_OP_MATMUL_RM) {
        if (shape_len != 3) {
            set_error("matmul shape has 3 entries, got %d", shape_len);
            return DS_EINVAL;
        }
        const int64_t M = sh[0], N = sh[1], K = sh[2];
        if (M < 0 || N < 1 || K < 1) {
            set_error("bad matmul shape");
            return DS_EINVAL;
        }
        if (M * K > INT32_MAX || K * N > INT32_MAX || M * N > INT32_MAX) {
            set_error("matmul shape exceeds the 32-bit extent range of the kernels");
            return DS_EUNSUPPORTED;
        }
        for (int i = 0; i < 3; ++i) sp.shape[i] = sh[i];
        sp.values = {clipped(kMmTile, M), clipped(kMmTile, N), clipped(kMmBk, K),
                     all_of(kUnroll),     all_of(kOnOff),      all_of(kOnOff),
                     clipped(kSplit, K),  all_of(kVec)};
        sp.names.assign(kMmNames, kMmNames + 8);
    } else {
        set_error("unknown op %d", op);
        return DS_EUNSUPPORTED;
    }
    sp.nknobs = int(sp.values.size());
    sp.size = 1;
    for (auto &v : sp.values) sp.size *= v.size();
    return DS_OK;
}

ds_sched make_sched(const Space &sp, const int32_t *idx) {
    ds_sched s;
    std::memset(&s, 0, sizeof s);
    s.op = sp.op;
    s.nknobs = sp.nknobs;
    for (int i = 0; i < 9; ++i) s.shape[i] = sp.shape[i];
    for (int a = 0; a < sp.nknobs; ++a) s.idx[a] = idx[a];
    return s;
}

bool sched_matches(const Space &sp, const ds_sched *s) {
    if (s->op != sp.op || s->nknobs != sp.nknobs) return false;
    const int n = sp.op == DS_OP_CONV2D_NCHW ? 9 : (sp.op == DS_OP_MATMUL_RM ? 3 : 0);
    for (int i = 0; i < n; ++i)
        if (s->shape[i] != sp.shape[i]) return false;
    return true;
}

}  // namespace ds

using namespace ds;

struct ds_space {
    Space sp;
};

extern "C" {

const char *ds_last_error(void) { return ds::last_error(); }

int sched_space_create(int op, const int64_t *shape, int shape_len, ds_space **out) {
    if (!out) {
        set_error("out is null");
        return DS_EINVAL;
    }
    *out = nullptr;
    ds_space *s = new (std::nothrow) ds_space;
    if (!s) {
        set_error("out of host memory");
        return DS_ENOMEM;
    }
    const int rc = build_space(op, shape, shape_len, s->sp);
    if (rc != DS_OK) {
        delete s;
        return rc;
    }
    *out = s;
    return DS_OK;
}

int sched_space_create_lattice(int nknobs, const int32_t *nvalues, const int32_t *values,
                               const uint64_t *invalid_keys, int n_invalid, ds_space **out) {
    if (!out || !nvalues || !values || nknobs < 1 || nknobs > DS_MAX_KNOBS || n_invalid < 0 ||
        (n_invalid > 0 && !invalid_keys)) {
        set_error("bad lattice description");
        return DS_EINVAL;
    }
    *out = nullptr;
    ds_space *s = new (std::nothrow) ds_space;
    if (!s) {
        set_error("out of host memory");
        return DS_ENOMEM;
    }
    Space &sp = s->sp;
    sp.op = 0;
    sp.nknobs = nknobs;
    int off = 0;
    for (int a = 0; a < nknobs; ++a) {
        if (nvalues[a] < 1) {
            delete s;
            set_error("axis %d has no value", a);
            return DS_EINVAL;
        }
        sp.values.emplace_back(values + off, values + off + nvalues[a]);
        off += nvalues[a];
        sp.names.push_back(kGenericNames[a]);
        sp.size *= uint64_t(nvalues[a]);
    }
    sp.invalid_keys.assign(invalid_keys, invalid_keys + n_invalid);
    std::sort(sp.invalid_keys.begin(), sp.invalid_keys.end());
    *out = s;
    return DS_OK;
}

void sched_space_destroy(ds_space *space) { delete space; }

int sched_space_info(const ds_space *space, int *op, int *nknobs, uint64_t *size) {
    if (!space) {
        set_error("space is null");
        return DS_EINVAL;
    }
    if (op) *op = space->sp.op;
    if (nknobs) *nknobs = space->sp.nknobs;
    if (size) *size = space->sp.size;
    return DS_OK;
}

int sched_space_axis(const ds_space *space, int axis, const char **name, int *nvalues,
                     const int32_t **values) {
    if (!space || axis < 0 || axis >= space->sp.nknobs) {
        set_error("bad space or axis");
        return DS_EINVAL;
    }
    if (name) *name = space->sp.names[axis];
    if (nvalues) *nvalues = int(space->sp.values[axis].size());
    if (values) *values = space->sp.values[axis].data();
    return DS_OK;
}

static int check_point(const ds_space *space, const ds_sched *s) {
    if (!space || !s) {
        set_error("null argument");
        return DS_EINVAL;
    }
    if (!sched_matches(space->sp, s)) {
        set_error("schedule does not belong to this space (op, shape or knob count differ)");
        return DS_EINVAL;
    }
    return DS_OK;
}

int sched_valid(const ds_space *space, const ds_sched *s) {
    const int rc = check_point(space, s);
    if (rc != DS_OK) return rc;
    return space->sp.valid(s->idx) ? 1 : 0;
}

int sched_key(const ds_space *space, const ds_sched *s, uint64_t *key) {
    int rc = check_point(space, s);
    if (rc != DS_OK) return rc;
    if (!key || !space->sp.in_range(s->idx)) {
        set_error("index out of range");
        return DS_EINVAL;
    }
    *key = space->sp.key(s->idx);
    return DS_OK;
}

int sched_from_key(const ds_space *space, uint64_t key, ds_sched *out) {
    if (!space || !out || key >= space->sp.size) {
        set_error("bad key");
        return DS_EINVAL;
    }
    int32_t idx[DS_MAX_KNOBS] = {0};
    space->sp.from_key(key, idx);
    *out = make_sched(space->sp, idx);
    return DS_OK;
}

int sched_neighbors(const ds_space *space, const ds_sched *s, ds_sched *out, int cap,
                    int *n_out) {
    int rc = check_point(space, s);
    if (rc != DS_OK) return rc;
    if (!n_out || cap < 0 || (cap > 0 && !out) || !space->sp.in_range(s->idx)) {
        set_error("bad neighbour query");
        return DS_EINVAL;
    }
    const Space &sp = space->sp;
    int n = 0;
    int32_t idx[DS_MAX_KNOBS];
    for (int a = 0; a < sp.nknobs; ++a) {
        for (int d = -1; d <= 1; d += 2) {
            const int j = s->idx[a] + d;
            if (j < 0 || j >= int(sp.values[a].size())) continue;
            std::memcpy(idx, s->idx, sizeof(int32_t) * sp.nknobs);
            idx[a] = j;
            if (!sp.geometry(idx).valid) continue;
            if (n < cap) out[n] = make_sched(sp, idx);
            ++n;
        }
    }
    *n_out = n;
    return DS_OK;
}

int sched_origin(const ds_space *space, ds_sched *out) {
    if (!space || !out) {
        set_error("null argument");
        return DS_EINVAL;
    }
    const Space &sp = space->sp;
    int32_t idx[DS_MAX_KNOBS] = {0};
    if (sp.valid(idx)) {
        *out = make_sched(sp, idx);
        return DS_OK;
    }
    for (uint64_t k = 0; k < sp.size; ++k) {
        sp.from_key(k, idx);
        if (sp.geometry(idx).valid) {
            *out = make_sched(sp, idx);
            return DS_OK;
        }
    }
    set_error("the space has no valid point");
    return DS_EEXHAUSTED;
}

int sched_geometry(const ds_space *space, const ds_sched *s, ds_geometry *out) {
    int rc = check_point(space, s);
    if (rc != DS_OK) return rc;
    if (!out || !space->sp.in_range(s->idx)) {
        set_error("index out of range");
        return DS_EINVAL;
    }
    const Geometry g = space->sp.geometry(s->idx);
    out->valid = g.valid;
    out->threads = g.threads;
    out->grid = g.grid;
    out->lds_bytes = g.lds_bytes;
    out->acc = g.acc;
    out->unroll_eff = g.unroll_eff;
    out->t0 = g.t0;
    out->t1 = g.t1;
    out->red = g.red;
    out->chunks = g.chunks;
    return DS_OK;
}

}  // extern "C"

// Accessor for the other translation units.
namespace ds {
const Space &space_of(const ds_space *s) { return s->sp; }
}  // namespace ds
