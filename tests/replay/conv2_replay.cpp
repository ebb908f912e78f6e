// CPU replay of the channel-quad conv kernel's index arithmetic (conv mfma 2
// and 3, kern_conv.hip: conv_mfma2), for tests only.
//
// For one schedule it walks every workgroup, thread and lane the kernel
// would run, with the launch geometry of conv2_setup (the library's own
// set-up), and checks what the GPU cannot report: every global read lies in
// its tensor, every global->LDS copy lands inside the workgroup's LDS size
// (the geometry's lds bytes) and, for 16-byte copies, on 16-byte boundaries;
// every LDS read of an operand stays in its buffer and never reads a word
// that was not written (unless only discarded outputs depend on it); every
// output is written exactly once (per split); each output tile counts one
// arrival per non-empty split; and the fp64 result of the replayed
// multiply-adds equals a direct convolution.  The replay mirrors the
// kernel's arithmetic by hand: a change to one needs the same change here.
//
// stdin, one schedule per line:
//   N C H W K R S stride pad  tk th tw tc depth ks vec misaligned band
// stdout: "ok ..." or "FAIL ..." per line; exit status 1 on the first failure.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>

#include "ds_internal.h"

namespace ds {
void set_error(const char *, ...) {}
}
using namespace ds;

namespace {

int fdv(int n, FastDiv f) {
    const unsigned hi = unsigned((uint64_t(unsigned(n)) * uint64_t(f.m)) >> 32);
    return int((hi + unsigned(n)) >> f.s);
}

// xcd_tile of kern_common.h
int xcd_tile(int b, int nwg) {
    const int q = nwg >> 3, r = nwg & 7;
    const int x = b & 7, j = b >> 3;
    return x * q + (x < r ? x : r) + j;
}

struct Cursor {
    int kl, wc, hc, hu;
    void start(const Conv2Args &a, int t) {
        kl = fdv(t, a.f_wru);
        wc = t - kl * a.wr_u;
        hc = fdv(t, a.f_hcu);
        hu = t - hc * a.hc_u;
    }
    void next(const Conv2Args &a) {
        wc += a.w_dc;
        const bool cw = wc >= a.wr_u;
        wc -= cw ? a.wr_u : 0;
        kl += a.w_dk + (cw ? 1 : 0);
        hu += a.h_dr;
        const bool ch = hu >= a.hc_u;
        hu -= ch ? a.hc_u : 0;
        hc += a.h_dc + (ch ? 1 : 0);
    }
};

long g_errors = 0;
#define CHECK(c, ...)                                         \
    do {                                                      \
        if (!(c) && g_errors++ < 8) {                         \
            fprintf(stderr, __VA_ARGS__);                     \
            fprintf(stderr, "\n");                            \
        }                                                     \
    } while (0)

bool replay(const int64_t *sh, int tk, int th, int tw, int tc, int depth, int ks, int vec, bool mis,
            bool band, char *summary, size_t nsum) {
    Conv2Args a;
    const Conv2Shape c = conv2_setup(sh, tk, th, tw, tc, depth, ks, vec, band, a);
    if (!c.valid) {
        snprintf(summary, nsum, "invalid point");
        return false;
    }
    if (mis) {   // operands 4 bytes off a 16-byte boundary: 4-byte copies, same layout
        a.vw = 0;
        a.vh = 0;
        a.st4 = 0;
        conv2_units(a, c.threads);
    }
    const int TKB = c.tkb, NPB = c.npb, U = c.u, KG = c.kg;
    const int N = a.N, C = a.C, H = a.H, W = a.W, K = a.K, R = a.R, S = a.S;
    const int RS = R * S, PQ = a.P * a.Q;
    const size_t nx = size_t(N) * C * H * W, nw = size_t(K) * C * RS, ny = size_t(N) * K * PQ;
    std::mt19937 rng(20240620);
    std::uniform_real_distribution<double> ud(-1, 1);
    std::vector<double> x(nx), w(nw);
    for (auto &v : x) v = ud(rng);
    for (auto &v : w) v = ud(rng);
    std::vector<double> part(size_t(a.ksw) * ny, NAN);
    std::vector<int> written(size_t(a.ksw) * ny, 0);
    const int nthr = c.threads, nwave = nthr / 64;
    const int64_t grid = c.grid;
    const int lds_f = int(c.lds / 4);
    CHECK(nthr == 64 * a.wpx * KG, "threads %d", nthr);
    CHECK(grid % a.ksw == 0, "grid %% ksw");
    std::vector<int> arrivals(grid / a.ksw, 0);
    std::vector<char> seen(grid, 0);
    const int nsplit = (a.chunks + a.cps - 1) / a.cps;
    const int tc4 = 4 * a.t4;

    for (int64_t b = 0; b < grid; ++b) {
        const int t0 = xcd_tile(int(b), int(grid));
        CHECK(t0 >= 0 && t0 < grid && !seen[t0], "workgroup order is not a permutation at %ld", (long)b);
        if (t0 < 0 || t0 >= grid) continue;
        seen[t0] = 1;
        const int t1 = fdv(t0, a.f_tk), kt = t0 - t1 * a.tiles_k;
        const int t2 = fdv(t1, a.f_tq), qt = t1 - t2 * a.tiles_q;
        const int t3 = fdv(t2, a.f_tp), pt = t2 - t3 * a.tiles_p;
        const int n = fdv(t3, a.f_ksw), z = t3 - n * a.ksw;
        const int ci0 = z * a.cps, ci1 = std::min(ci0 + a.cps, a.chunks);
        if (ci0 >= ci1) continue;
        {
            const int64_t tile = ((int64_t(n) * a.tiles_p + pt) * a.tiles_q + qt) * a.tiles_k + kt;
            CHECK(tile < int64_t(arrivals.size()), "tile %ld", (long)tile);
            if (tile < int64_t(arrivals.size())) arrivals[tile]++;
        }
        int n0 = n, g0 = 0, rows = a.hs;
        if (a.band) {
            const int f0 = qt * a.npx, fl = std::min(f0 + a.npx, a.F) - 1;
            const int r0 = fdv(f0, a.f_q), rl = fdv(fl, a.f_q);
            n0 = fdv(r0, a.f_p);
            const int nl = fdv(rl, a.f_p);
            g0 = (r0 - n0 * a.P) * a.st;
            rows = (nl - n0) * a.hp + (rl - nl * a.P) * a.st + a.R - g0;
            CHECK(rows > 0 && rows <= a.hs, "band rows %d of %d", rows, a.hs);
        }
        const int hy0 = pt * a.th * a.st - a.pd;
        const int col0 = (a.band ? 0 : qt * a.tw * a.st) - a.pd;
        const int hx0 = a.hal ? col0 & ~3 : col0;
        const int kvalid = a.K - kt * a.tk;
        const size_t wk = size_t(kt) * a.tk * C * RS, xn = size_t(n0) * C * H * W;
        auto creal_of = [&](int ci) { return std::min(a.tc, a.C - ci * a.tc); };
        auto halo_src = [&](int hc, int hy, int hx) {
            int gy, img = 0;
            if (a.band) {
                const int gr = g0 + hy;
                img = fdv(gr, a.f_hp);
                gy = gr - img * a.hp - a.pd;
            } else {
                gy = hy0 + hy;
            }
            const int gx = hx0 + hx;
            const bool in = hy < rows && gy >= 0 && gy < H && gx >= 0 && gx < W;
            return in ? ((img * C + hc) * H + gy) * W + gx : -1;
        };
        std::vector<double> lds(std::max(lds_f, 1), NAN);
        // one lane's global->LDS copy of `floats` floats (bytes offset from base)
        auto copy = [&](const std::vector<double> &src, size_t base, int off, int floats, int dst) {
            CHECK(off >= 0 && off % 4 == 0, "copy offset %d", off);
            const size_t e = base + size_t(off) / 4;
            CHECK(e + floats <= src.size(), "global read past the tensor (%zu of %zu)", e, src.size());
            CHECK(dst >= 0 && dst + floats <= lds_f, "LDS write at %d past %d floats", dst, lds_f);
            if (floats == 4) CHECK(e % 4 == 0 && dst % 4 == 0, "16-byte copy not 16-byte aligned");
            for (int i = 0; i < floats; ++i)
                if (e + i < src.size() && dst + i >= 0 && dst + i < lds_f) lds[dst + i] = src[e + i];
        };
        const bool reuse = a.regs && ci1 - ci0 > 1;
        std::vector<int> sw(size_t(nthr) * kConv2MaxCopies, -1), shv(size_t(nthr) * kConv2MaxCopies, -1);
        if (reuse) {
            for (int tid = 0; tid < nthr; ++tid) {
                Cursor cur;
                cur.start(a, tid);
                const int gw = a.vw ? 4 : 1, gh = a.vh ? 4 : 1;
                for (int u = 0; u < a.ncopy; ++u) {
                    const int kl = std::min(cur.kl, kvalid - 1);
                    const int col = std::min(gw * cur.wc, a.tc * RS - gw);
                    sw[tid * kConv2MaxCopies + u] = cur.kl < a.tk ? 4 * (kl * C * RS + col) : -1;
                    const int hy = fdv(cur.hu, a.f_hru);
                    const int hx = gh * (cur.hu - hy * a.hr_u);
                    const int o = halo_src(cur.hc, hy, hx);
                    shv[tid * kConv2MaxCopies + u] = cur.hc >= tc4 ? -1 : hy >= a.hs ? 0 : o >= 0 ? 4 * o : -1;
                    cur.next(a);
                }
            }
        }
        auto issue = [&](int ci, int bi) {
            const int wt = bi * a.buf, xs = wt + a.bufw;
            const size_t wb = wk + size_t(ci) * a.tc * RS, xb = xn + size_t(ci) * a.tc * H * W;
            const int creal = creal_of(ci);
            if (creal < tc4)   // channel slots past C: the buffer is zeroed first
                for (int e = 0; e < a.buf; ++e) lds[wt + e] = 0;
            for (int tid = 0; tid < nthr; ++tid) {
                const int lane_base = (tid >> 6) * 64, lane = tid & 63;
                if (creal >= tc4 && reuse) {
                    for (int u = 0; u < a.ncopy; ++u) {
                        const int d = u * nthr + lane_base + lane;
                        const int ow = sw[tid * kConv2MaxCopies + u], oh = shv[tid * kConv2MaxCopies + u];
                        if (ow >= 0) copy(w, wb, ow, a.vw ? 4 : 1, a.vw ? wt + 4 * d : wt + d);
                        if (oh >= 0) copy(x, xb, oh, a.vh ? 4 : 1, a.vh ? xs + 4 * d : xs + d);
                    }
                    continue;
                }
                const int gw = a.vw ? 4 : 1, gh = a.vh ? 4 : 1;
                Cursor cur;
                cur.start(a, tid);
                for (int u = 0; u < a.ncopy; ++u, cur.next(a)) {
                    const int d = u * nthr + lane_base + lane;
                    const int col = gw * cur.wc;
                    if (cur.kl < a.tk && cur.kl < kvalid && col < creal * RS)
                        copy(w, wb, 4 * (cur.kl * C * RS + col), gw, a.vw ? wt + 4 * d : wt + d);
                    const int hy = fdv(cur.hu, a.f_hru);
                    const int hx = gh * (cur.hu - hy * a.hr_u);
                    const int o = halo_src(cur.hc, hy, hx);
                    if (cur.hc < creal && hy < a.hs && o >= 0) copy(x, xb, 4 * o, gh, a.vh ? xs + 4 * d : xs + d);
                }
            }
        };
        const bool border = a.band ? a.pd > 0 : hy0 < 0 || hy0 + a.hs > H || hx0 < 0 || hx0 + a.ws > W;
        if (border)
            for (int bi = 0; bi < a.nbuf; ++bi)
                for (int e = a.bufw; e < a.buf; ++e) lds[bi * a.buf + e] = 0;

        // lane bases
        std::vector<int> bbase(size_t(nwave) * NPB * 64), ooff(bbase.size());
        std::vector<char> pvalid(bbase.size());
        const int shift = a.hal ? col0 & 3 : 0;
        for (int wu = 0; wu < nwave; ++wu) {
            const int wp = wu & (a.wpx - 1);
            for (int lane = 0; lane < 64; ++lane) {
                const int li = lane & 15, lg = lane >> 4;
                for (int bk = 0; bk < NPB; ++bk) {
                    const int pix = (wp * NPB + bk) * 16 + li;
                    const size_t id = (size_t(wu) * NPB + bk) * 64 + lane;
                    if (a.band) {
                        const int f = qt * a.npx + pix, fc = std::min(f, a.F - 1);
                        const int r = fdv(fc, a.f_q), q = fc - r * a.Q;
                        const int img = fdv(r, a.f_p), p = r - img * a.P;
                        pvalid[id] = f < a.F;
                        bbase[id] = a.bufw + lg * a.cs + ((img - n0) * a.hp + p * a.st - g0) * a.ws + q * a.st + shift;
                    } else {
                        const int py = pix >> a.ltw, px = pix & (a.tw - 1);
                        const int p = pt * a.th + py, q = qt * a.tw + px;
                        pvalid[id] = pix < a.npx && p < a.P && q < a.Q;
                        bbase[id] = a.bufw + lg * a.cs + py * a.st * a.ws + px * a.st + shift;
                    }
                }
            }
        }
        // chunk loop: every wave's k-steps over the chunk in its buffer
        std::vector<double> acc(size_t(nwave) * TKB * NPB * 256, 0.0);
        const int sa = 4 * KG * RS, sb = 4 * KG * a.cs;
        const int tg = (a.t4 / (KG * U)) * RS;
        issue(ci0, 0);
        for (int ci = ci0; ci < ci1; ++ci) {
            const int bo = ((ci - ci0) & 1) * a.buf;
            for (int wu = 0; wu < nwave; ++wu) {
                const int g = wu >> a.lwpx;
                for (int t = 0; t < tg; ++t) {
                    const int cq = fdv(t, a.f_rs), rs = t - cq * RS;
                    const int r = fdv(rs, a.f_s), s = rs - r * S;
                    const int q = 4 * (cq * U * KG + g);
                    const int oa = q * RS + rs, ob = q * a.cs + r * a.ws + s;
                    for (int u = 0; u < U; ++u)
                        for (int i = 0; i < TKB; ++i)
                            for (int bk = 0; bk < NPB; ++bk)
                                for (int m = 0; m < 16; ++m)
                                    for (int col = 0; col < 16; ++col) {
                                        double sum = 0;
                                        for (int k4 = 0; k4 < 4; ++k4) {
                                            const int ia = bo + m * a.wrow + k4 * RS + i * 16 * a.wrow + oa + u * sa;
                                            const size_t id = (size_t(wu) * NPB + bk) * 64 + k4 * 16 + col;
                                            const int ib = bo + bbase[id] + ob + u * sb;
                                            CHECK(ia >= bo && ia < bo + a.bufw, "weight read at %d outside [%d, %d)", ia, bo, bo + a.bufw);
                                            CHECK(ib >= bo + a.bufw && ib < bo + a.buf, "halo read at %d outside [%d, %d)", ib, bo + a.bufw, bo + a.buf);
                                            const double av = ia >= 0 && ia < lds_f ? lds[ia] : NAN;
                                            const double bv = ib >= 0 && ib < lds_f ? lds[ib] : NAN;
                                            if (kt * a.tk + i * 16 + m < K && pvalid[id])
                                                CHECK(!std::isnan(av) && !std::isnan(bv), "unwritten LDS word read for a kept output");
                                            sum += av * bv;
                                        }
                                        acc[((size_t(wu) * TKB + i) * NPB + bk) * 256 + m * 16 + col] += sum;
                                    }
                }
            }
            if (ci + 1 < ci1) issue(ci + 1, ((ci - ci0) & 1) ^ 1);
        }
        // wave groups meet in group 0; its waves store 16 channels x up to 64
        // pixels per pass, 4 consecutive pixels per lane
        const int BG = NPB < 4 ? NPB : 4, ROW = 16 * BG + 4, LPR = 4 * BG;
        for (int wu = 0; wu < nwave; ++wu) {
            const int g = wu >> a.lwpx, wp = wu & (a.wpx - 1);
            if (g > 0) continue;
            for (int h = 1; h < KG; ++h) {
                const int wv = (h << a.lwpx) | wp;
                for (size_t e = 0; e < size_t(TKB) * NPB * 256; ++e)
                    acc[size_t(wu) * TKB * NPB * 256 + e] += acc[size_t(wv) * TKB * NPB * 256 + e];
            }
            CHECK(wp * 16 * 68 + 16 * 68 <= lds_f, "output staging past the LDS size");
            const size_t nkpq = ny, yoff = size_t(n) * K * PQ;
            auto emit = [&](size_t o, double v) {
                const size_t idx = size_t(z) * nkpq + yoff + o;
                CHECK(yoff + o < ny, "output write past the end");
                if (yoff + o >= ny) return;
                part[idx] = v;
                written[idx]++;
            };
            auto each4 = [&](int k, int pix, const double *val) {
                if (k >= K) return;
                if (a.band) {
                    const int f0 = qt * a.npx + pix;
                    if (a.st4 && f0 + 3 < a.F) {
                        const int img = fdv(f0, a.f_pq);
                        const size_t o = size_t(img) * K * PQ + size_t(k) * PQ + (f0 - img * PQ);
                        CHECK(o % 4 == 0, "16-byte output store not aligned");
                        for (int e = 0; e < 4; ++e) emit(o + e, val[e]);
                        return;
                    }
                    for (int e = 0; e < 4; ++e) {
                        const int fe = f0 + e;
                        if (fe >= a.F) break;
                        const int img = fdv(fe, a.f_pq);
                        emit(size_t(img) * K * PQ + size_t(k) * PQ + (fe - img * PQ), val[e]);
                    }
                } else {
                    const int py = pix >> a.ltw, px = pix & (a.tw - 1);
                    const int p = pt * a.th + py, q = qt * a.tw + px;
                    if (a.st4 && p < a.P && q + 3 < a.Q) {
                        const size_t o = size_t(k) * PQ + size_t(p) * a.Q + q;
                        CHECK(o % 4 == 0, "16-byte output store not aligned");
                        for (int e = 0; e < 4; ++e) emit(o + e, val[e]);
                        return;
                    }
                    for (int e = 0; e < 4; ++e) {
                        const int pe = pt * a.th + ((pix + e) >> a.ltw), qe = qt * a.tw + ((pix + e) & (a.tw - 1));
                        if (pe < a.P && qe < a.Q) emit(size_t(k) * PQ + size_t(pe) * a.Q + qe, val[e]);
                    }
                }
            };
            std::vector<double> stage(16 * ROW);
            for (int i = 0; i < TKB; ++i)
                for (int b0 = 0; b0 < NPB; b0 += BG) {
                    for (int lane = 0; lane < 64; ++lane) {
                        const int li = lane & 15, lg = lane >> 4;
                        for (int bb = 0; bb < BG; ++bb)
                            for (int v = 0; v < 4; ++v)
                                stage[(4 * lg + v) * ROW + bb * 16 + li] =
                                    acc[((size_t(wu) * TKB + i) * NPB + b0 + bb) * 256 + (4 * lg + v) * 16 + li];
                    }
                    for (int r0 = 0; r0 < 16; r0 += 64 / LPR)
                        for (int lane = 0; lane < 64; ++lane) {
                            const int row = r0 + lane / LPR, c4 = lane % LPR;
                            each4(kt * a.tk + i * 16 + row, (wp * NPB + b0) * 16 + 4 * c4, &stage[row * ROW + 4 * c4]);
                        }
                }
        }
    }
    for (int64_t t = 0; t < grid; ++t) CHECK(seen[t], "tile %ld never visited", (long)t);
    for (size_t t = 0; t < arrivals.size(); ++t)
        CHECK(arrivals[t] == nsplit, "tile %zu: %d arrivals, %d splits", t, arrivals[t], nsplit);
    // partials summed in split order (the reduce launch); direct convolution
    double maxerr = 0, maxref = 0;
    for (size_t e = 0; e < ny; ++e) {
        double s = 0;
        for (int zz = 0; zz < nsplit; ++zz) {
            CHECK(written[zz * ny + e] == 1, "output %zu of split %d written %d times", e, zz, written[zz * ny + e]);
            s += part[zz * ny + e];
        }
        const int q = int(e % a.Q), p = int(e / a.Q % a.P), k = int(e / PQ % K), nn = int(e / (size_t(PQ) * K));
        double ref = 0;
        for (int ch = 0; ch < C; ++ch)
            for (int r = 0; r < R; ++r)
                for (int s2 = 0; s2 < S; ++s2) {
                    const int iy = p * a.st - a.pd + r, ix = q * a.st - a.pd + s2;
                    if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                    ref += x[((size_t(nn) * C + ch) * H + iy) * W + ix] * w[((size_t(k) * C + ch) * R + r) * S + s2];
                }
        maxerr = std::max(maxerr, std::isnan(s) ? INFINITY : std::fabs(s - ref));
        maxref = std::max(maxref, std::fabs(ref));
    }
    CHECK(maxerr <= 1e-9 * std::max(1.0, maxref), "max error %g (max |ref| %g)", maxerr, maxref);
    snprintf(summary, nsum, "band=%d tkb=%d npb=%d u=%d kg=%d ksw=%d grid=%ld lds=%d err=%.2g", a.band, TKB,
             NPB, U, KG, a.ksw, (long)grid, int(c.lds), maxerr);
    return g_errors == 0;
}

}  // namespace

int main() {
    int64_t sh[9];
    int tk, th, tw, tc, depth, ks, vec, mis, band;
    while (scanf("%ld %ld %ld %ld %ld %ld %ld %ld %ld %d %d %d %d %d %d %d %d %d", &sh[0], &sh[1], &sh[2],
                 &sh[3], &sh[4], &sh[5], &sh[6], &sh[7], &sh[8], &tk, &th, &tw, &tc, &depth, &ks, &vec,
                 &mis, &band) == 18) {
        char summary[256];
        const bool ok = replay(sh, tk, th, tw, tc, depth, ks, vec, mis != 0, band != 0, summary, sizeof summary);
        printf("%s %s\n", ok ? "ok" : "FAIL", summary);
        fflush(stdout);
        if (!ok) return 1;
    }
    return 0;
}
