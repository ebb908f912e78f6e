// NCHW fp32 conv2d kernel family for gfx950.
//
// y[n,k,p,q] = sum_{c,r,s} x[n,c,p*st-pd+r,q*st-pd+s] * w[k,c,r,s]
//
// One workgroup computes a tk x th x tw output tile (channels x rows x cols)
// of one image, over the input-channel chunks of its reduction split.  The
// reduction inside a chunk runs over kr = c_l*R*S + r*S + s; an offset table
// in LDS turns kr into the position of the tap, so the loop has no division.
//
//   conv_valu: VALU FMA.  Lanes take pixels first, then groups of KPT output
//              channels; each lane accumulates KPT x PPT outputs.
//   conv_mfma: implicit GEMM on v_mfma_f32_16x16x4f32 (M = channels, N =
//              pixels, K = kr).  Up to four waves split the pixels of the tile
//              (one per 16-pixel block below 64 pixels); a wave holds TKB x
//              NPB 16x16 blocks.  Lane group g (lanes
//              16g..16g+15) feeds reduction steps kr = 16*j + 4*g + v, v < 4,
//              for both operands, so a 16-byte LDS read gives four steps of A.
//              The operands of the D next 16-step groups are read while the
//              MFMAs of the current one run (D, 1 to 3, is the unroll knob's
//              read-ahead depth: D+1 operand sets, loop unrolled by D+1).
//
// LDS layout (lds=1): [weights tk x wrow][input halo tc x hs x ws][zero] per buffer,
//                    then [table red][weight sources tk x wrow][halo sources tc x hs x ws]
//             (lds=0): [table red x {offset, info}]
// A split (ks > 1) stores its partial output tile; a reduce kernel sums the
// splits into y in split order.
#include <utility>

#include "kern_common.h"

namespace ds {

namespace {

__device__ __forceinline__ int fdiv(int n, FastDiv f) {
    return int((__umulhi(unsigned(n), f.m) + unsigned(n)) >> f.s);
}

// A zero in device memory: loads of positions that read zero are pointed here.
__device__ const float kZero[1] = {0.f};

// Global-memory pointers (a select between two generic pointers would make
// the load a flat load, whose wait counts are conservative).
typedef const __attribute__((address_space(1))) float gfloat;
__device__ __forceinline__ gfloat *gptr(const float *p) { return (gfloat *)(p); }

__device__ __forceinline__ void conv_tile_coords(const ConvArgs &a, int &n, int &z, int &kt,
                                                 int &pt, int &qt) {
    int t = xcd_tile(blockIdx.x, gridDim.x);
    kt = t % a.tiles_k;
    t /= a.tiles_k;
    qt = t % a.tiles_q;
    t /= a.tiles_q;
    pt = t % a.tiles_p;
    t /= a.tiles_p;
    z = t % a.ks;
    n = t / a.ks;
}

// Offset table for one chunk (identical for every chunk).  real = tc*R*S taps;
// entries real..red-1 are padding: their weights are zero, and in LDS mode they
// point at the first halo element (a finite value inside the halo for every
// pixel offset); in global mode their valid bit is clear and they read zero.
// LDS mode stores byte offsets, so a read address is one add to a lane base.
__device__ __forceinline__ void build_table(const ConvArgs &a, int *tab, bool lds) {
    const int RS = a.R * a.S;
    const int real = a.tc * RS;
    for (int e = threadIdx.x; e < a.red; e += blockDim.x) {
        const int c_l = fdiv(e, a.f_rs), rs = e - c_l * RS;
        const int r = fdiv(rs, a.f_s), s = rs - r * a.S;
        if (lds) {
            tab[e] = 4 * (e < real ? c_l * a.hs * a.ws + r * a.ws + s : 0);   // bytes
        } else {
            tab[2 * e] = e < real ? c_l * a.H * a.W + r * a.W + s : 0;
            tab[2 * e + 1] = e < real ? int(0x80000000u | unsigned(c_l << 16) | unsigned(r << 8) |
                                            unsigned(s))
                                      : 0;
        }
    }
}

// Offset (within one output channel's weights) of staged reduction index kr of
// the chunk starting at channel c0; false if kr reads zero.
__device__ __forceinline__ bool weight_src(const ConvArgs &a, int kr, int c0, int real, int crs,
                                           int &gofs) {
    const int RS = a.R * a.S;
    gofs = c0 * RS + kr;
    return kr < real && gofs < crs;
}

// Stage the input halo of chunk c0 and the weights of the tile into LDS.  Each
// thread issues kBatch independent loads before writing any of them, so the
// global-load latency is paid once per batch rather than once per element.
constexpr int kBatch = 8;

// Image column of LDS halo column 0: the tile's first input column, or, with
// the aligned halo layout (w4 bit 2), the 16-byte boundary at or before it (so
// halo rows can travel 16 bytes per lane).
__device__ __forceinline__ int halo_x0(const ConvArgs &a, int qt) {
    const int x0 = qt * a.tw * a.st - a.pd;
    return a.w4 & 4 ? x0 - (x0 & 3) : x0;
}
// Column of the tile's first input column inside a halo row.
__device__ __forceinline__ int halo_shift(const ConvArgs &a, int qt) {
    return a.w4 & 4 ? (qt * a.tw * a.st - a.pd) & 3 : 0;
}

__device__ __forceinline__ void stage_chunk(const ConvArgs &a, int n, int kt, int pt, int qt,
                                            int c0, float *wt, float *xs) {
    const int RS = a.R * a.S;
    const int real = a.tc * RS;
    const int hw = a.hs * a.ws;
    const int nh = a.tc * hw;
    const int hy0 = pt * a.th * a.st - a.pd, hx0 = halo_x0(a, qt);
    const float *xn = a.x + (size_t)n * a.C * a.H * a.W;
    const int nt = blockDim.x;
    for (int e0 = threadIdx.x; e0 < nh; e0 += kBatch * nt) {
        float v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int e = e0 + u * nt;
            // unconditional load (element 0 where the position reads zero),
            // select after: a guarded load would drain the loads in flight
            const int c_l = fdiv(e, a.f_hw), rem = e - c_l * hw;
            const int hy = fdiv(rem, a.f_ws), hx = rem - hy * a.ws;
            const int c = c0 + c_l, gy = hy0 + hy, gx = hx0 + hx;
            const bool ok = e < nh && c < a.C && gy >= 0 && gy < a.H && gx >= 0 && gx < a.W;
            const float t = xn[ok ? ((size_t)c * a.H + gy) * a.W + gx : 0];
            v[u] = ok ? t : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int e = e0 + u * nt;
            if (e < nh) xs[e] = v[u];
        }
    }
    if (threadIdx.x == 0) xs[nh] = 0.f;
    const int nw = a.tk * a.red;
    const int crs = a.C * RS;
    for (int e0 = threadIdx.x; e0 < nw; e0 += kBatch * nt) {
        float v[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int e = e0 + u * nt;
            const int kl = fdiv(e, a.f_red), kr = e - kl * a.red;
            const int k = kt * a.tk + kl;
            int gofs;
            const bool ok = e < nw && weight_src(a, kr, c0, real, crs, gofs) && k < a.K;
            const float t = a.w[ok ? (size_t)k * crs + gofs : 0];
            v[u] = ok ? t : 0.f;
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int e = e0 + u * nt;
            if (e < nw) {
                const int kl = fdiv(e, a.f_red), kr = e - kl * a.red;
                wt[kl * a.wrow + kr] = v[u];
            }
        }
    }
}

#define DS_GLOBAL(p) ((const __attribute__((address_space(1))) void *)(p))
#define DS_LOCAL(p) ((__attribute__((address_space(3))) void *)(p))

// The same staging as stage_chunk, issued as asynchronous global -> LDS copies
// (4 bytes per lane; a wave's instruction fills 64 consecutive LDS floats);
// positions that read zero (padding, channels past C, reduction padding) are
// written with ordinary LDS stores.  Needs a whole number of waves.
__device__ __forceinline__ void dma_chunk(const ConvArgs &a, int n, int kt, int pt, int qt, int c0,
                                          float *wt, float *xs) {
    const int RS = a.R * a.S;
    const int real = a.tc * RS;
    const int crs = a.C * RS;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nwv = blockDim.x >> 6;
    const int npw = a.tk * a.wrow;
    for (int base = wid * 64; base < npw; base += nwv * 64) {
        const int p = base + lane;
        if (p < npw) {
            const int kl = fdiv(p, a.f_wrow), kr = p - kl * a.wrow;
            const int k = kt * a.tk + kl;
            int gofs;
            if (kr < a.red && weight_src(a, kr, c0, real, crs, gofs) && k < a.K)
                __builtin_amdgcn_global_load_lds(DS_GLOBAL(a.w + (size_t)k * crs + gofs),
                                                 DS_LOCAL(wt + base), 4, 0, 0);
            else if (kr < a.red)
                wt[p] = 0.f;
        }
    }
    const int hw = a.hs * a.ws;
    const int nh = a.tc * hw;
    const int hy0 = pt * a.th * a.st - a.pd, hx0 = halo_x0(a, qt);
    const float *xn = a.x + (size_t)n * a.C * a.H * a.W;
    for (int base = wid * 64; base < nh; base += nwv * 64) {
        const int p = base + lane;
        if (p < nh) {
            const int c_l = fdiv(p, a.f_hw), rem = p - c_l * hw;
            const int hy = fdiv(rem, a.f_ws), hx = rem - hy * a.ws;
            const int c = c0 + c_l, gy = hy0 + hy, gx = hx0 + hx;
            if (c < a.C && gy >= 0 && gy < a.H && gx >= 0 && gx < a.W)
                __builtin_amdgcn_global_load_lds(
                    DS_GLOBAL(xn + ((size_t)c * a.H + gy) * a.W + gx), DS_LOCAL(xs + base), 4, 0, 0);
            else
                xs[p] = 0.f;
        }
    }
    if (threadIdx.x == 0) xs[nh] = 0.f;
}

// Waits for this wave's outstanding copies and LDS operations, then barriers
// the workgroup (no memory fence: the waits make every wave's LDS writes
// complete before any wave passes).
__device__ __forceinline__ void chunk_barrier() {
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Stages chunk ci of this workgroup into LDS buffer b.
// Source offsets of every LDS position of one chunk, relative to the chunk's
// base (weights: row kt*tk, column c0*R*S; halo: image n, channel c0), -1
// where the position reads zero.  Identical for every chunk that ends at or
// before channel C, so they are built once per workgroup.
__device__ __forceinline__ void build_stage_tables(const ConvArgs &a, int kt, int pt, int qt,
                                                   int *wsrc, int *xsrc) {
    const int RS = a.R * a.S;
    const int real = a.tc * RS;
    const int crs = a.C * RS;
    const int npw = a.tk * a.wrow;
    if (a.w4 & 1) {
        // 16-byte groups: a group of four positions is valid or not as a whole
        for (int q = threadIdx.x; q < (npw >> 2); q += blockDim.x) {
            const int p = q << 2;
            const int kl = fdiv(p, a.f_wrow), kr = p - kl * a.wrow;
            wsrc[q] = kr < real && kt * a.tk + kl < a.K ? kl * crs + kr : -1;
        }
    } else {
        for (int p = threadIdx.x; p < npw; p += blockDim.x) {
            const int kl = fdiv(p, a.f_wrow), kr = p - kl * a.wrow;
            wsrc[p] = kr < real && kt * a.tk + kl < a.K ? kl * crs + kr : -1;
        }
    }
    const int hw = a.hs * a.ws;
    const int nh = a.tc * hw;
    const int hy0 = pt * a.th * a.st - a.pd, hx0 = halo_x0(a, qt);
    // 16-byte groups when image rows allow (W % 4 == 0: a group starting at a
    // multiple of 4 is inside a row or outside it as a whole)
    const int gsz = a.w4 & 2 ? 4 : 1;
    for (int q = threadIdx.x; q < nh / gsz; q += blockDim.x) {
        const int p = q * gsz;
        const int c_l = fdiv(p, a.f_hw), rem = p - c_l * hw;
        const int hy = fdiv(rem, a.f_ws), hx = rem - hy * a.ws;
        const int gy = hy0 + hy, gx = hx0 + hx;
        xsrc[q] = gy >= 0 && gy < a.H && gx >= 0 && gx < a.W ? (c_l * a.H + gy) * a.W + gx : -1;
    }
}

// dma_chunk driven by the tables: one table read and one copy per position;
// positions that read zero are never written (both buffers are zeroed once).
// A wave takes its positions kCopyBatch instructions at a time: the batch's
// table reads are all issued before its first copy, so one LDS latency is
// paid per batch rather than per copy.
constexpr int kCopyBatch = 8;

template <int BYTES>
__device__ __forceinline__ void copy_from_table(const float *src, const int *tabv, int n,
                                                float *dst) {
    constexpr int W = BYTES / 4;   // floats per lane
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nwv = blockDim.x >> 6;
    const int step = nwv * 64;
    for (int base = wid * 64; base < n; base += kCopyBatch * step) {
        int e[kCopyBatch];
#pragma unroll
        for (int u = 0; u < kCopyBatch; ++u) {
            const int q = base + u * step + lane;
            const int t = tabv[q < n ? q : 0];
            e[u] = q < n ? t : -1;
        }
#pragma unroll
        for (int u = 0; u < kCopyBatch; ++u) {
            if (e[u] < 0) continue;
            if constexpr (BYTES == 16)
                __builtin_amdgcn_global_load_lds(DS_GLOBAL(src + e[u]),
                                                 DS_LOCAL(dst + W * (base + u * step)), 16, 0, 0);
            else
                __builtin_amdgcn_global_load_lds(DS_GLOBAL(src + e[u]),
                                                 DS_LOCAL(dst + W * (base + u * step)), 4, 0, 0);
        }
    }
}

__device__ __forceinline__ void dma_chunk_tab(const ConvArgs &a, int n, int kt, int c0,
                                              const int *wsrc, const int *xsrc, float *wt,
                                              float *xs) {
    const int RS = a.R * a.S;
    const float *wb = a.w + (size_t)kt * a.tk * a.C * RS + (size_t)c0 * RS;
    const float *xb = a.x + ((size_t)n * a.C + c0) * a.H * a.W;
    const int npw = a.tk * a.wrow;
    // weights: 16 bytes per lane (one instruction fills 256 floats) when rows allow
    if (a.w4 & 1) copy_from_table<16>(wb, wsrc, npw >> 2, wt);
    else copy_from_table<4>(wb, wsrc, npw, wt);
    if (a.w4 & 2) copy_from_table<16>(xb, xsrc, (a.tc * a.hs * a.ws) >> 2, xs);
    else copy_from_table<4>(xb, xsrc, a.tc * a.hs * a.ws, xs);
}

// LDS staging set-up of a workgroup: the offset tables and zeroed buffers for
// the table-driven copies (whole waves only), then a barrier.
__device__ __forceinline__ void stage_init(const ConvArgs &a, float *smem, int kt, int pt, int qt,
                                           int *wsrc, int *xsrc) {
    if ((blockDim.x & 63) == 0) {
        build_stage_tables(a, kt, pt, qt, wsrc, xsrc);
        floatx4 *z4 = reinterpret_cast<floatx4 *>(smem);
        for (int e = threadIdx.x; e < (a.nbuf * a.buf) >> 2; e += blockDim.x)
            z4[e] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();
}

// WHOLE: the workgroup is whole waves (always for conv_mfma).  Only then are
// the asynchronous copies used; the register-staged fallback is left out of
// such kernels, because its loads into registers, merged into the chunk loop,
// make the compiler wait for every copy in flight before the next LDS read.
template <bool WHOLE>
__device__ __forceinline__ void stage_to(const ConvArgs &a, float *smem, int b, int n, int kt, int pt,
                                         int qt, int ci, const int *wsrc, const int *xsrc) {
    float *wt = smem + b * a.buf;
    float *xs = wt + a.tk * a.wrow;
    const int c0 = ci * a.tc;
    if (WHOLE || (blockDim.x & 63) == 0) {
        if (c0 + a.tc <= a.C) dma_chunk_tab(a, n, kt, c0, wsrc, xsrc, wt, xs);
        else dma_chunk(a, n, kt, pt, qt, c0, wt, xs);      // channel tail
    } else {
        stage_chunk(a, n, kt, pt, qt, c0, wt, xs);
    }
}

// Chunk staging with the copy sources held in registers: the tables are the
// same for every chunk, so when a thread's share of a kind (weights, halo)
// fits in kRegCopies entries it reads them once, after stage_init, and each
// chunk's copies of that kind need no LDS read (a table read before every copy
// left the copies waiting on LDS latency).  Thread t's u-th copy of a kind
// fills position u*blockDim + t (wave-uniform destination per u).  A kind
// that does not fit is copied from its LDS table; the channel tail and
// workgroups of partial waves go through stage_to.
constexpr int kRegCopies = 8;

struct RegStage {
    int w[kRegCopies], h[kRegCopies];
    bool onw, onh;

    __device__ __forceinline__ void init(const ConvArgs &a, const int *wsrc, const int *xsrc) {
        const int nt = blockDim.x;
        const int nw = a.w4 & 1 ? (a.tk * a.wrow) >> 2 : a.tk * a.wrow;
        const int nh = a.w4 & 2 ? (a.tc * a.hs * a.ws) >> 2 : a.tc * a.hs * a.ws;
        onw = (nt & 63) == 0 && nw <= kRegCopies * nt;
        onh = (nt & 63) == 0 && nh <= kRegCopies * nt;
#pragma unroll
        for (int u = 0; u < kRegCopies; ++u) {
            const int q = u * nt + threadIdx.x;
            w[u] = onw && q < nw ? wsrc[q] : -1;
            h[u] = onh && q < nh ? xsrc[q] : -1;
        }
    }

    // One copy of a kind; lanes without a position (-1) are masked off.  The
    // empty asm makes the compiler compare the offset at every copy instead of
    // computing the lane masks once per workgroup: held in scalar registers
    // those masks were spilled, and each copy read its mask back with two lane
    // reads.  One compare per copy measured 1-2% faster on the small layers.
    template <int BYTES>
    __device__ __forceinline__ static void copy(const float *base, int off, float *dst) {
        __asm__ volatile("" : "+v"(off));
        if (off < 0) return;
        if constexpr (BYTES == 16)
            __builtin_amdgcn_global_load_lds(DS_GLOBAL(base + off), DS_LOCAL(dst), 16, 0, 0);
        else
            __builtin_amdgcn_global_load_lds(DS_GLOBAL(base + off), DS_LOCAL(dst), 4, 0, 0);
    }

    template <bool WHOLE>
    __device__ __forceinline__ void to(const ConvArgs &a, float *smem, int b, int n, int kt, int pt,
                                       int qt, int ci, const int *wsrc, const int *xsrc) const {
        const int c0 = ci * a.tc;
        if (!(onw || onh) || c0 + a.tc > a.C) {
            stage_to<WHOLE>(a, smem, b, n, kt, pt, qt, ci, wsrc, xsrc);
            return;
        }
        float *wt = smem + b * a.buf;
        float *xs = wt + a.tk * a.wrow;
        const int RS = a.R * a.S;
        const float *wb = a.w + (size_t)kt * a.tk * a.C * RS + (size_t)c0 * RS;
        const float *xb = a.x + ((size_t)n * a.C + c0) * a.H * a.W;
        const int slot = threadIdx.x & ~63, nt = blockDim.x;
        const int npw = a.tk * a.wrow;
        if (!onw) {
            if (a.w4 & 1) copy_from_table<16>(wb, wsrc, npw >> 2, wt);
            else copy_from_table<4>(wb, wsrc, npw, wt);
        } else if (a.w4 & 1) {
#pragma unroll
            for (int u = 0; u < kRegCopies; ++u) copy<16>(wb, w[u], wt + 4 * (u * nt + slot));
        } else {
#pragma unroll
            for (int u = 0; u < kRegCopies; ++u) copy<4>(wb, w[u], wt + u * nt + slot);
        }
        const int nh = a.tc * a.hs * a.ws;
        if (!onh) {
            if (a.w4 & 2) copy_from_table<16>(xb, xsrc, nh >> 2, xs);
            else copy_from_table<4>(xb, xsrc, nh, xs);
        } else if (a.w4 & 2) {
#pragma unroll
            for (int u = 0; u < kRegCopies; ++u) copy<16>(xb, h[u], xs + 4 * (u * nt + slot));
        } else {
#pragma unroll
            for (int u = 0; u < kRegCopies; ++u) copy<4>(xb, h[u], xs + u * nt + slot);
        }
    }
};

// Software pipeline over the 16-step groups of a chunk with D groups read
// ahead: operand set r%(D+1) holds group r; the reads of group g+D are issued
// before the MFMAs of group g, so those MFMAs need not wait for them.  The
// loop is unrolled by D+1, so every set index is a compile-time constant and
// the body has no branch (its wait counts stay exact).  Reads past the last
// group re-read the last group into a set that is never consumed.
template <int D, class Ops, class Load, class Mma>
__device__ __forceinline__ void group_ring(int ngroups, Load &&load, Mma &&mma) {
    constexpr int RG = D + 1;
    Ops o[RG];
#pragma unroll
    for (int r = 0; r < D; ++r) load(min(r, ngroups - 1), o[r]);
    int kg = 0;
    for (; kg + RG <= ngroups; kg += RG) {
#pragma unroll
        for (int r = 0; r < RG; ++r) {
            load(min(kg + r + D, ngroups - 1), o[(r + D) % RG]);
            mma(o[r]);
        }
    }
    // fewer than RG groups remain; groups kg .. kg+D-1 are loaded
#pragma unroll
    for (int r = 0; r < RG - 1; ++r) {
        if (kg + r < ngroups) {
            if (kg + r + D < ngroups) load(kg + r + D, o[(r + D) % RG]);
            mma(o[r]);
        }
    }
}

template <int KPT, int PPT, int UF, int LDS>
__global__ __launch_bounds__(256) void conv_valu(ConvArgs a) {
    extern __shared__ float smem[];
    int n, z, kt, pt, qt;
    conv_tile_coords(a, n, z, kt, pt, qt);
    const int ci0 = z * a.cps, ci1 = min(ci0 + a.cps, a.chunks);
    if (ci0 >= ci1) return;

    const int tid = threadIdx.x;
    const int pl = tid % a.npl, g = tid / a.npl;
    const int k0 = kt * a.tk + g * KPT;
    const int PQ = a.P * a.Q;

    int poff[PPT], iy0[PPT], ix0[PPT], oq[PPT];
    bool pv[PPT];
#pragma unroll
    for (int j = 0; j < PPT; ++j) {
        const int pix = pl + a.npl * j;
        const int py = pix >> a.ltw, px = pix & (a.tw - 1);
        const int p = pt * a.th + py, q = qt * a.tw + px;
        pv[j] = pix < a.npx && p < a.P && q < a.Q;
        poff[j] = py * a.st * a.ws + px * a.st + halo_shift(a, qt);
        iy0[j] = p * a.st - a.pd;
        ix0[j] = q * a.st - a.pd;
        oq[j] = p * a.Q + q;
    }

    float acc[KPT][PPT];
#pragma unroll
    for (int i = 0; i < KPT; ++i)
#pragma unroll
        for (int j = 0; j < PPT; ++j) acc[i][j] = 0.f;

    int *tab = LDS ? reinterpret_cast<int *>(smem + a.nbuf * a.buf) : reinterpret_cast<int *>(smem);
    int *wsrc = tab + a.red, *xsrc = wsrc + a.tk * a.wrow;     // LDS staging tables
    // the set-up and the first copies also run at raised priority
    __builtin_amdgcn_s_setprio(3);
    build_table(a, tab, LDS);
    RegStage rs;
    if (LDS) {
        stage_init(a, smem, kt, pt, qt, wsrc, xsrc);
        rs.init(a, wsrc, xsrc);
        rs.template to<false>(a, smem, 0, n, kt, pt, qt, ci0, wsrc, xsrc);
    }
    __builtin_amdgcn_s_setprio(0);

    const int RS = a.R * a.S;
    const int crs = a.C * RS;
    for (int ci = ci0; ci < ci1; ++ci) {
        const int c0 = ci * a.tc;
        if (LDS) {
            const int bi = (ci - ci0) & 1;
            chunk_barrier();
            if (ci + 1 < ci1) {
                // the copies are issued at raised wave priority: next to waves
                // that issue MFMAs back to back their vector instructions
                // otherwise wait for issue slots
                __builtin_amdgcn_s_setprio(3);
                rs.template to<false>(a, smem, bi ^ 1, n, kt, pt, qt, ci + 1, wsrc, xsrc);
                __builtin_amdgcn_s_setprio(0);
            }
            const float *wt = smem + bi * a.buf;
            const float *xs = wt + a.tk * a.wrow;
            const float *wg = wt + g * KPT * a.wrow;
            const char *xp[PPT];
#pragma unroll
            for (int j = 0; j < PPT; ++j) xp[j] = reinterpret_cast<const char *>(xs + poff[j]);
#pragma unroll UF
            for (int kr = 0; kr < a.red; ++kr) {
                const int off = tab[kr];
                float xv[PPT];
#pragma unroll
                for (int j = 0; j < PPT; ++j) xv[j] = *reinterpret_cast<const float *>(xp[j] + off);
#pragma unroll
                for (int i = 0; i < KPT; ++i) {
                    const float wv = wg[i * a.wrow + kr];
#pragma unroll
                    for (int j = 0; j < PPT; ++j) acc[i][j] = fmaf(wv, xv[j], acc[i][j]);
                }
            }
        } else {
            if (ci == ci0) __syncthreads();
            const float *xc = a.x + ((size_t)n * a.C + c0) * a.H * a.W;
#pragma unroll UF
            for (int kr = 0; kr < a.red; ++kr) {
                const int goff = tab[2 * kr];
                const unsigned info = unsigned(tab[2 * kr + 1]);
                const int c_l = int((info >> 16) & 0x7fffu);
                const int r = int((info >> 8) & 0xffu), s = int(info & 0xffu);
                const bool cok = (info & 0x80000000u) && c0 + c_l < a.C;
                float xv[PPT];
#pragma unroll
                for (int j = 0; j < PPT; ++j) {
                    const int iy = iy0[j] + r, ix = ix0[j] + s;
                    const bool ok = cok && pv[j] && iy >= 0 && iy < a.H && ix >= 0 && ix < a.W;
                    const float t = xc[ok ? goff + iy0[j] * a.W + ix0[j] : 0];
                    xv[j] = ok ? t : 0.f;
                }
#pragma unroll
                for (int i = 0; i < KPT; ++i) {
                    const int k = k0 + i;
                    const bool wok = cok && k < a.K;
                    const float t = a.w[wok ? (size_t)k * crs + c0 * RS + kr : 0];
                    const float wv = wok ? t : 0.f;
#pragma unroll
                    for (int j = 0; j < PPT; ++j) acc[i][j] = fmaf(wv, xv[j], acc[i][j]);
                }
            }
        }
    }

    float *yn = (a.ks > 1 ? a.part + (size_t)z * a.N * a.K * PQ : a.y) + (size_t)n * a.K * PQ;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
        const int k = k0 + i;
        if (k >= a.K) continue;
#pragma unroll
        for (int j = 0; j < PPT; ++j)
            if (pv[j]) yn[(size_t)k * PQ + oq[j]] = acc[i][j];
    }
}

template <int TKB, int NPB, int D, int LDS>
__global__ __launch_bounds__(256) void conv_mfma(ConvArgs a) {
    extern __shared__ float smem[];
    int n, z, kt, pt, qt;
    conv_tile_coords(a, n, z, kt, pt, qt);
    const int ci0 = z * a.cps, ci1 = min(ci0 + a.cps, a.chunks);
    if (ci0 >= ci1) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wid = tid >> 6;
    const int li = lane & 15, lg = lane >> 4;
    const int PQ = a.P * a.Q;

    int poff[NPB], iy0[NPB], ix0[NPB], oq[NPB];
    bool pv[NPB];
#pragma unroll
    for (int b = 0; b < NPB; ++b) {
        const int pix = (wid * NPB + b) * 16 + li;
        const int py = pix >> a.ltw, px = pix & (a.tw - 1);
        const int p = pt * a.th + py, q = qt * a.tw + px;
        pv[b] = pix < a.npx && p < a.P && q < a.Q;
        poff[b] = py * a.st * a.ws + px * a.st + halo_shift(a, qt);
        iy0[b] = p * a.st - a.pd;
        ix0[b] = q * a.st - a.pd;
        oq[b] = p * a.Q + q;
    }

    floatx4 acc[TKB][NPB];
#pragma unroll
    for (int i = 0; i < TKB; ++i)
#pragma unroll
        for (int b = 0; b < NPB; ++b) acc[i][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    int *tab = LDS ? reinterpret_cast<int *>(smem + a.nbuf * a.buf) : reinterpret_cast<int *>(smem);
    int *wsrc = tab + a.red, *xsrc = wsrc + a.tk * a.wrow;     // LDS staging tables
    // the set-up and the first copies also run at raised priority
    __builtin_amdgcn_s_setprio(3);
    build_table(a, tab, LDS);
    RegStage rs;
    if (LDS) {
        stage_init(a, smem, kt, pt, qt, wsrc, xsrc);
        rs.init(a, wsrc, xsrc);
        rs.template to<true>(a, smem, 0, n, kt, pt, qt, ci0, wsrc, xsrc);
    }
    __builtin_amdgcn_s_setprio(0);

    const int RS = a.R * a.S;
    const int crs = a.C * RS;
    const int ngroups = a.red / 16;
    for (int ci = ci0; ci < ci1; ++ci) {
        const int c0 = ci * a.tc;
        if (LDS) {
            const int bi = (ci - ci0) & 1;
            chunk_barrier();
            if (ci + 1 < ci1) {
                // the next chunk's copies go to the other buffer, issued at
                // raised wave priority: next to waves that issue MFMAs back to
                // back their vector instructions otherwise wait for issue slots
                __builtin_amdgcn_s_setprio(3);
                rs.template to<true>(a, smem, bi ^ 1, n, kt, pt, qt, ci + 1, wsrc, xsrc);
                __builtin_amdgcn_s_setprio(0);
            }
            const float *wt = smem + bi * a.buf;
            const float *xs = wt + a.tk * a.wrow;
            {
                // lane bases: pixel b of the halo, row i*16+li of the weights
                const char *bp[NPB];
#pragma unroll
                for (int b = 0; b < NPB; ++b) bp[b] = reinterpret_cast<const char *>(xs + poff[b]);
                const float *ap[TKB];
#pragma unroll
                for (int i = 0; i < TKB; ++i) ap[i] = wt + (i * 16 + li) * a.wrow + 4 * lg;
                struct Ops {
                    floatx4 a[TKB];
                    float b[4][NPB];
                };
                auto load = [&](int kg, Ops &o) {
                    const int kb = kg * 16 + 4 * lg;
                    // the offsets are read as float-typed data: an int-typed
                    // LDS read makes the compiler wait for every copy in flight
                    // (the buffers this loop reads are already complete: the
                    // chunk barrier waited for their copies)
                    const floatx4 offf =
                        *reinterpret_cast<const floatx4 *>(reinterpret_cast<const float *>(tab) + kb);
                    const int offv[4] = {__float_as_int(offf[0]), __float_as_int(offf[1]),
                                         __float_as_int(offf[2]), __float_as_int(offf[3])};
#pragma unroll
                    for (int i = 0; i < TKB; ++i)
                        o.a[i] = *reinterpret_cast<const floatx4 *>(ap[i] + kg * 16);
#pragma unroll
                    for (int v = 0; v < 4; ++v)
#pragma unroll
                        for (int b = 0; b < NPB; ++b)
                            o.b[v][b] = *reinterpret_cast<const float *>(bp[b] + offv[v]);
                };
                auto mma = [&](const Ops &o) {
#pragma unroll
                    for (int v = 0; v < 4; ++v)
#pragma unroll
                        for (int i = 0; i < TKB; ++i)
#pragma unroll
                            for (int b = 0; b < NPB; ++b)
                                acc[i][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                    o.a[i][v], o.b[v][b], acc[i][b], 0, 0, 0);
                };
                group_ring<D, Ops>(ngroups, load, mma);
            }
        } else {
            if (ci == ci0) __syncthreads();
            const float *xc = a.x + ((size_t)n * a.C + c0) * a.H * a.W;
            // Software pipeline: the operands of the D next 16-step groups are
            // loaded while the MFMAs of the current one run.  Positions that
            // read zero load the zero in device memory, so no select waits on
            // a load.
            struct Ops {
                float A[4][TKB];
                float B[4][NPB];
            };
            auto gload = [&](int kg, Ops &o) {
                const int kb = kg * 16 + 4 * lg;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int kr = kb + v;
                    const int goff = tab[2 * kr];
                    const unsigned info = unsigned(tab[2 * kr + 1]);
                    const int c_l = int((info >> 16) & 0x7fffu);
                    const int r = int((info >> 8) & 0xffu), s = int(info & 0xffu);
                    const bool cok = (info & 0x80000000u) && c0 + c_l < a.C;
#pragma unroll
                    for (int i = 0; i < TKB; ++i) {
                        const int k = kt * a.tk + i * 16 + li;
                        const bool wok = cok && k < a.K;
                        o.A[v][i] = *(wok ? gptr(a.w + (size_t)k * crs + c0 * RS + kr) : gptr(kZero));
                    }
#pragma unroll
                    for (int b = 0; b < NPB; ++b) {
                        const int iy = iy0[b] + r, ix = ix0[b] + s;
                        const bool ok = cok && pv[b] && iy >= 0 && iy < a.H && ix >= 0 && ix < a.W;
                        o.B[v][b] = *(ok ? gptr(xc + goff + iy0[b] * a.W + ix0[b]) : gptr(kZero));
                    }
                }
            };
            auto gmma = [&](const Ops &o) {
#pragma unroll
                for (int v = 0; v < 4; ++v)
#pragma unroll
                    for (int i = 0; i < TKB; ++i)
#pragma unroll
                        for (int b = 0; b < NPB; ++b)
                            acc[i][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.A[v][i], o.B[v][b],
                                                                            acc[i][b], 0, 0, 0);
            };
            group_ring<D, Ops>(ngroups, gload, gmma);
        }
    }

    // 16x16 block: lane holds rows 4*lg + v (channels), column li (pixel).
    float *yn = (a.ks > 1 ? a.part + (size_t)z * a.N * a.K * PQ : a.y) + (size_t)n * a.K * PQ;
#pragma unroll
    for (int i = 0; i < TKB; ++i)
#pragma unroll
        for (int b = 0; b < NPB; ++b) {
            if (!pv[b]) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int k = kt * a.tk + i * 16 + 4 * lg + v;
                if (k < a.K) yn[(size_t)k * PQ + oq[b]] = acc[i][b][v];
            }
        }
}

// ---- channel-quad MFMA conv (mfma = 2) -----------------------------------------
//
// Implicit GEMM on v_mfma_f32_16x16x4f32 with the reduction ordered by tap:
// a k-step multiplies one channel quad (lane group g holds channel 4q + g) at
// one tap (r, s).  Both operands then sit at a uniform offset from a per-lane
// base -- weight row 16i + li, column (4q + g)*R*S + r*S + s; halo channel
// 4q + g, row py*st + r, column px*st + s -- so the loop reads them with plain
// 4-byte LDS reads and needs no offset table.  A step takes U quads at once;
// the operands of the next step are read while the current one multiplies.
// KG wave groups split the quads of every chunk (group g takes quads g,
// g+KG, ...) and meet in LDS at the end, so a reduction split needs no second
// launch.  Copy sources of a full chunk are the same for every chunk and are
// computed once per thread; the next chunk's copies are issued right after
// the chunk barrier, into the other buffer.

namespace q4 {

__device__ __forceinline__ int fdv(int n, FastDiv f) {
    return int((__umulhi(unsigned(n), f.m) + unsigned(n)) >> f.s);
}

// Copy unit u * blockDim + tid of a chunk as (weight row, unit in row) and
// (halo channel, unit in channel), advanced by blockDim units at a time.
struct Cursor {
    int kl, wc, hc, hu;
    __device__ __forceinline__ void start(const Conv2Args &a, int t) {
        kl = fdv(t, a.f_wru);
        wc = t - kl * a.wr_u;
        hc = fdv(t, a.f_hcu);
        hu = t - hc * a.hc_u;
    }
    __device__ __forceinline__ void next(const Conv2Args &a) {
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

template <int BYTES>
__device__ __forceinline__ void copy(const char *base, unsigned off, float *dst) {
    if constexpr (BYTES == 16)
        __builtin_amdgcn_global_load_lds(DS_GLOBAL(base + off), DS_LOCAL(dst), 16, 0, 0);
    else
        __builtin_amdgcn_global_load_lds(DS_GLOBAL(base + off), DS_LOCAL(dst), 4, 0, 0);
}

}  // namespace q4

// Waves per SIMD each conv_mfma2 instance is compiled to allow: the most of
// 4, 3 and 2 (instances that hold 12 copy units per thread in registers) or
// of 6, 5, 4, 3 and 2 (those that hold 4) for which its registers fit without
// spilling, found by compiling every instance under each bound; others keep
// the compiler's choice.  On its own the compiler keeps the
// accumulators in AGPRs beside the VGPRs and ends at fewer waves:
// conv_mfma2<4, 4, 1, 1, 12>, for one, takes 164 VGPRs + 64 AGPRs (2 waves)
// unbounded and 152 VGPRs (3 waves) bounded; with 4 copy units, 119 VGPRs (4
// waves).  An instance is keyed TKB·10000 + NPB·100 + U·10 + KG.
constexpr int kConv2Waves4[] = {
    10111, 10112, 10114, 10121, 10122, 10124, 10141, 10142, 10144, 10211, 10212, 10214,
    10221, 10222, 10224, 10241, 10242, 10244, 10411, 10412, 10414, 10421, 10422, 10424,
    10441, 10442, 10444, 10811, 10812, 20111, 20112, 20114, 20121, 20122, 20124, 20141,
    20142, 20144, 20211, 20212, 20214, 20221, 20222, 20224, 20241, 20242, 20244, 20411,
    20412, 40111, 40112, 40114, 40121, 40122, 40124, 40141, 40142, 40144, 40211, 40212,
    40221, 40222};
constexpr int kConv2Waves3[] = {
    10821, 10822, 10841, 10842, 20421, 20422, 20441, 20442, 20811, 20812, 40241, 40242,
    40411, 40412};
constexpr int kConv2Waves2[] = {
    11621, 20821, 20841, 40441, 40811};
constexpr int kConv2FewWaves6[] = {
    10111, 10112, 10114, 10121, 10122, 10124, 10141, 10142, 10144, 10211, 10212, 10214,
    10221, 10222, 10224, 10241, 10242, 10244, 10411, 10412, 10414, 10421, 10422, 10424,
    20111, 20112, 20114, 20121, 20122, 20124, 20141, 20142, 20144, 20211, 20212, 20214,
    20221, 20222, 20224, 20241, 20242, 20244, 40111, 40112, 40114, 40121, 40122, 40124,
    40141, 40142, 40144, 40211, 40212};
constexpr int kConv2FewWaves5[] = {
    10441, 10442, 10444, 10811, 10812, 20411, 20412};
constexpr int kConv2FewWaves4[] = {
    40221, 40222, 40411, 40412};
constexpr int kConv2FewWaves3[] = {
    10821, 10822, 10841, 10842, 11611, 20421, 20422, 20441, 20442, 20811, 20812, 40241,
    40242};
constexpr int kConv2FewWaves2[] = {
    11621, 11641, 20821, 20822, 20841, 20842, 21611, 40421, 40422, 40441, 40442, 40811};
constexpr int conv2_waves(int tkb, int npb, int u, int kg, int rc) {
    const int key = tkb * 10000 + npb * 100 + u * 10 + kg;
    if (rc == kConv2FewCopies) {
        for (int k : kConv2FewWaves6)
            if (k == key) return 6;
        for (int k : kConv2FewWaves5)
            if (k == key) return 5;
        for (int k : kConv2FewWaves4)
            if (k == key) return 4;
        for (int k : kConv2FewWaves3)
            if (k == key) return 3;
        for (int k : kConv2FewWaves2)
            if (k == key) return 2;
        return 1;
    }
    for (int k : kConv2Waves4)
        if (k == key) return 4;
    for (int k : kConv2Waves3)
        if (k == key) return 3;
    for (int k : kConv2Waves2)
        if (k == key) return 2;
    return 1;
}

template <int TKB, int NPB, int U, int KG, int RC>
__global__ __launch_bounds__(256 * KG, conv2_waves(TKB, NPB, U, KG, RC)) void conv_mfma2(Conv2Args a) {
    extern __shared__ float smem[];
    using q4::fdv;
    // tile of this workgroup (tile order: k, q, p, split, image)
    const int t0 = xcd_tile(blockIdx.x, gridDim.x);
    const int t1 = fdv(t0, a.f_tk);
    const int kt = t0 - t1 * a.tiles_k;
    const int t2 = fdv(t1, a.f_tq);
    const int qt = t1 - t2 * a.tiles_q;
    const int t3 = fdv(t2, a.f_tp);
    const int pt = t2 - t3 * a.tiles_p;
    const int n = fdv(t3, a.f_ksw);
    const int z = t3 - n * a.ksw;
    const int ci0 = z * a.cps, ci1 = min(ci0 + a.cps, a.chunks);
    if (ci0 >= ci1) return;

    const int tid = threadIdx.x, nthr = blockDim.x;
    const int lane = tid & 63;
    const int wu = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = wu >> a.lwpx, wp = wu & (a.wpx - 1);
    const int li = lane & 15, lg = lane >> 4;
    const int RS = a.R * a.S;
    const int PQ = a.P * a.Q;
    const int slot = wu * 64;
    const int tc4 = 4 * a.t4;
    // A band tile starts at pixel qt * npx of the flattened output: image n0,
    // padded row g0 of that image; its halo is the `rows` padded rows from
    // there (image boundaries included), each one whole output row wide.
    int n0 = n, g0 = 0, rows = a.hs;
    if (a.band) {
        const int f0 = qt * a.npx, fl = min(f0 + a.npx, a.F) - 1;
        const int r0 = fdv(f0, a.f_q), rl = fdv(fl, a.f_q);
        n0 = fdv(r0, a.f_p);
        const int nl = fdv(rl, a.f_p);
        g0 = (r0 - n0 * a.P) * a.st;
        rows = (nl - n0) * a.hp + (rl - nl * a.P) * a.st + a.R - g0;
    }
    const int hy0 = pt * a.th * a.st - a.pd;
    const int col0 = (a.band ? 0 : qt * a.tw * a.st) - a.pd;
    const int hx0 = a.hal ? col0 & ~3 : col0;
    const int kvalid = a.K - kt * a.tk;
    const float *wk = a.w + (size_t)kt * a.tk * a.C * RS;
    const float *xn = a.x + (size_t)n0 * a.C * a.H * a.W;
    auto creal_of = [&](int ci) { return min(a.tc, a.C - ci * a.tc); };
    // Float offset of halo position (channel hc, row hy, column hx) from the
    // chunk's first channel of image n0, or -1 outside the image (left zero).
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
        const bool in = hy < rows && gy >= 0 && gy < a.H && gx >= 0 && gx < a.W;
        return in ? ((img * a.C + hc) * a.H + gy) * a.W + gx : -1;
    };

    // Copy sources of a full chunk (byte offsets from its weight / image
    // base, the same for every full chunk): thread t's u-th unit of a kind is
    // unit u * blockDim + t.  Weight rows past K and the row padding re-read a
    // valid float (their LDS positions feed only discarded outputs, or are
    // never read); halo rows of the channel padding read any valid float
    // (never read); -1: nothing to copy (past the buffer, or outside the
    // image: left zero).
    // (held only when the workgroup walks more than one chunk: a single
    // chunk's units are computed as they are issued, so the first copies leave
    // sooner)
    const bool reuse = a.regs && ci1 - ci0 > 1;
    int sw[RC], sh[RC];
    if (reuse) {
        q4::Cursor cur;
        cur.start(a, tid);
        const int gw = a.vw ? 4 : 1, gh = a.vh ? 4 : 1;
#pragma unroll
        for (int u = 0; u < RC; ++u) {
            sw[u] = sh[u] = -1;
            if (u < a.ncopy) {
                const int kl = min(cur.kl, kvalid - 1);
                const int col = min(gw * cur.wc, a.tc * RS - gw);
                sw[u] = cur.kl < a.tk ? 4 * (kl * a.C * RS + col) : -1;
                const int hy = fdv(cur.hu, a.f_hru);
                const int hx = gh * (cur.hu - hy * a.hr_u);
                const int o = halo_src(cur.hc, hy, hx);
                sh[u] = cur.hc >= tc4 ? -1 : hy >= a.hs ? 0 : o >= 0 ? 4 * o : -1;
                cur.next(a);
            }
        }
    }
    auto issue_full = [&](int ci, int b) {
        const char *wb = reinterpret_cast<const char *>(wk + (size_t)ci * a.tc * RS);
        const char *xb = reinterpret_cast<const char *>(xn + (size_t)ci * a.tc * a.H * a.W);
        float *wt = smem + b * a.buf;
        float *xs = wt + a.bufw;
#pragma unroll
        for (int u = 0; u < RC; ++u) {
            if (u >= a.ncopy) break;
            const int d = u * nthr + slot;
            if (sw[u] >= 0) {
                if (a.vw) q4::copy<16>(wb, unsigned(sw[u]), wt + 4 * d);
                else q4::copy<4>(wb, unsigned(sw[u]), wt + d);
            }
            if (sh[u] >= 0) {
                if (a.vh) q4::copy<16>(xb, unsigned(sh[u]), xs + 4 * d);
                else q4::copy<4>(xb, unsigned(sh[u]), xs + d);
            }
        }
    };
    // Units computed as they are issued: a chunk with channel slots past C
    // (its buffer zeroed first), a workgroup's only chunk, or every chunk when
    // a thread's units do not fit the registers the instance holds them in
    // (more than RC units: 4-byte copies of misaligned operands).
    auto issue_units = [&](int ci, int b, bool zero) {
        float *wt = smem + b * a.buf;
        float *xs = wt + a.bufw;
        if (zero) {
            for (int e = tid; e < a.buf / 4; e += nthr)
                reinterpret_cast<floatx4 *>(wt)[e] = floatx4{0.f, 0.f, 0.f, 0.f};
            __syncthreads();
        }
        const int creal = creal_of(ci);
        const char *wb = reinterpret_cast<const char *>(wk + (size_t)ci * a.tc * RS);
        const char *xb = reinterpret_cast<const char *>(xn + (size_t)ci * a.tc * a.H * a.W);
        const int gw = a.vw ? 4 : 1, gh = a.vh ? 4 : 1;
        q4::Cursor cur;
        cur.start(a, tid);
        for (int u = 0; u < a.ncopy; ++u, cur.next(a)) {
            const int d = u * nthr + slot;
            const int col = gw * cur.wc;
            if (cur.kl < a.tk && cur.kl < kvalid && col < creal * RS) {
                if (a.vw) q4::copy<16>(wb, unsigned(4 * (cur.kl * a.C * RS + col)), wt + 4 * d);
                else q4::copy<4>(wb, unsigned(4 * (cur.kl * a.C * RS + col)), wt + d);
            }
            const int hy = fdv(cur.hu, a.f_hru);
            const int hx = gh * (cur.hu - hy * a.hr_u);
            const int o = halo_src(cur.hc, hy, hx);
            if (cur.hc < creal && hy < a.hs && o >= 0) {
                if (a.vh) q4::copy<16>(xb, unsigned(4 * o), xs + 4 * d);
                else q4::copy<4>(xb, unsigned(4 * o), xs + d);
            }
        }
    };

    // Halo positions outside the image are never copied: zero the halo part
    // of every buffer once when the tile's halo reaches past the image (a
    // band's does wherever there is zero padding).
    const bool border = a.band ? a.pd > 0
                               : hy0 < 0 || hy0 + a.hs > a.H || hx0 < 0 || hx0 + a.ws > a.W;
    if (border) {
        const int per = (a.buf - a.bufw) / 4;
        for (int e = tid; e < a.nbuf * per; e += nthr) {
            const int b = e >= per ? 1 : 0;
            reinterpret_cast<floatx4 *>(smem + b * a.buf + a.bufw)[e - b * per] =
                floatx4{0.f, 0.f, 0.f, 0.f};
        }
        __syncthreads();
    }
    auto issue = [&](int ci, int b) {
        if (creal_of(ci) < tc4) issue_units(ci, b, true);
        else if (reuse) issue_full(ci, b);
        else issue_units(ci, b, false);
    };
    issue(ci0, 0);

    // lane bases (floats) inside a buffer
    int bb[NPB];
    const int shift = a.hal ? col0 & 3 : 0;
#pragma unroll
    for (int b = 0; b < NPB; ++b) {
        const int pix = (wp * NPB + b) * 16 + li;
        if (a.band) {
            // pixels past the output read the last one's operands (discarded)
            const int f = qt * a.npx + pix;
            const int fc = min(f, a.F - 1);
            const int r = fdv(fc, a.f_q), q = fc - r * a.Q;
            const int img = fdv(r, a.f_p), p = r - img * a.P;
            bb[b] = a.bufw + lg * a.cs + ((img - n0) * a.hp + p * a.st - g0) * a.ws + q * a.st + shift;
        } else {
            // pixels past the output read in-buffer operands (discarded)
            const int py = pix >> a.ltw, px = pix & (a.tw - 1);
            bb[b] = a.bufw + lg * a.cs + py * a.st * a.ws + px * a.st + shift;
        }
    }
    const int ab = li * a.wrow + lg * RS;
    const int sa = 4 * KG * RS, sb = 4 * KG * a.cs;   // quad strides of one group

    floatx4 acc[TKB][NPB];
#pragma unroll
    for (int i = 0; i < TKB; ++i)
#pragma unroll
        for (int b = 0; b < NPB; ++b) acc[i][b] = floatx4{0.f, 0.f, 0.f, 0.f};

    // Step t of a group in a chunk: quad block cq = t / RS (quads
    // (cq*U + u)*KG + g, u < U) at tap rs = t % RS.
    const int tg = (a.t4 / (KG * U)) * RS;
    auto offs = [&](int t, int &oa, int &ob) {
        t = min(t, tg - 1);   // past the last step: re-read it (never multiplied)
        const int cq = fdv(t, a.f_rs), rs = t - cq * RS;
        const int r = fdv(rs, a.f_s), s = rs - r * a.S;
        const int q = 4 * (cq * U * KG + g);
        oa = q * RS + rs;
        ob = q * a.cs + r * a.ws + s;
    };
    struct Ops {
        float A[U][TKB];
        float B[U][NPB];
    };
    for (int ci = ci0; ci < ci1; ++ci) {
        const int bi = (ci - ci0) & 1;
        chunk_barrier();
        if (ci + 1 < ci1) issue(ci + 1, bi ^ 1);
        const float *buf = smem + bi * a.buf;
        auto load = [&](int t, Ops &o) {
            int oa, ob;
            offs(t, oa, ob);
#pragma unroll
            for (int u = 0; u < U; ++u) {
#pragma unroll
                for (int i = 0; i < TKB; ++i) o.A[u][i] = buf[ab + i * 16 * a.wrow + oa + u * sa];
#pragma unroll
                for (int b = 0; b < NPB; ++b) o.B[u][b] = buf[bb[b] + ob + u * sb];
            }
        };
        auto mma = [&](const Ops &o) {
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int i = 0; i < TKB; ++i)
#pragma unroll
                    for (int b = 0; b < NPB; ++b) {
                        acc[i][b] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.A[u][i], o.B[u][b],
                                                                        acc[i][b], 0, 0, 0);
                        // one LDS read between consecutive MFMAs
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
        };
        Ops o[2];
        load(0, o[0]);
        int j = 0;
        for (; j + 2 <= tg; j += 2) {
            load(j + 1, o[1]);
            mma(o[0]);
            load(j + 2, o[0]);
            mma(o[1]);
        }
        if (j < tg) mma(o[0]);
    }

    // wave groups 1..KG-1 hand their partial tiles to group 0 through LDS
    if constexpr (KG > 1) {
        __syncthreads();
        floatx4 *red = reinterpret_cast<floatx4 *>(smem);
        constexpr int per_wave = 64 * TKB * NPB;
        if (g > 0) {
            floatx4 *dst = red + ((g - 1) * a.wpx + wp) * per_wave;
#pragma unroll
            for (int i = 0; i < TKB; ++i)
#pragma unroll
                for (int b = 0; b < NPB; ++b) dst[(i * NPB + b) * 64 + lane] = acc[i][b];
        }
        __syncthreads();
        if (g == 0) {
#pragma unroll
            for (int h = 1; h < KG; ++h) {
                const floatx4 *src = red + ((h - 1) * a.wpx + wp) * per_wave;
#pragma unroll
                for (int i = 0; i < TKB; ++i)
#pragma unroll
                    for (int b = 0; b < NPB; ++b) acc[i][b] += src[(i * NPB + b) * 64 + lane];
            }
        }
    }
    // Stores go through LDS: a 16x16 block leaves a lane one pixel of four
    // channels, so each wave of group 0 writes 16 channels x up to 64 pixels
    // at a time to its own LDS rows and reads them back as 4 consecutive
    // pixels of one channel per lane -- 16-byte stores, runs of up to 256
    // bytes per channel row.  The LDS is free once every wave is past its
    // last operand (or reduction) read.
    __syncthreads();
    if (g > 0) return;
    constexpr int BG = NPB < 4 ? NPB : 4;              // blocks per pass
    constexpr int ROW = 16 * BG + 4;                    // staging row stride (floats)
    constexpr int LPR = 4 * BG;                         // lanes per channel row
    float *stage = smem + wp * (16 * 68);
    float *yn = (a.ksw > 1 ? a.part + (size_t)z * a.N * a.K * PQ : a.y) + (size_t)n * a.K * PQ;
    auto put = [&](int k, int pix, floatx4 val) {
        if (k >= a.K) return;
        if (a.band) {
            const int f = qt * a.npx + pix;
            if (a.st4 && f + 3 < a.F) {
                const int img = fdv(f, a.f_pq);
                *reinterpret_cast<floatx4 *>(yn + (size_t)img * a.K * PQ + (size_t)k * PQ +
                                             (f - img * PQ)) = val;
                return;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int fe = f + e;
                if (fe >= a.F) break;
                const int img = fdv(fe, a.f_pq);
                yn[(size_t)img * a.K * PQ + (size_t)k * PQ + (fe - img * PQ)] = val[e];
            }
        } else {
            const int py = pix >> a.ltw, px = pix & (a.tw - 1);
            const int p = pt * a.th + py, q = qt * a.tw + px;
            if (a.st4 && p < a.P && q + 3 < a.Q) {
                *reinterpret_cast<floatx4 *>(yn + (size_t)k * PQ + p * a.Q + q) = val;
                return;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int pe = pt * a.th + ((pix + e) >> a.ltw), qe = qt * a.tw + ((pix + e) & (a.tw - 1));
                if (pe < a.P && qe < a.Q) yn[(size_t)k * PQ + pe * a.Q + qe] = val[e];
            }
        }
    };
#pragma unroll
    for (int i = 0; i < TKB; ++i)
#pragma unroll
        for (int b0 = 0; b0 < NPB; b0 += BG) {
#pragma unroll
            for (int bb = 0; bb < BG; ++bb)
#pragma unroll
                for (int v = 0; v < 4; ++v) stage[(4 * lg + v) * ROW + bb * 16 + li] = acc[i][b0 + bb][v];
#pragma unroll
            for (int r0 = 0; r0 < 16; r0 += 64 / LPR) {
                const int row = r0 + lane / LPR, c4 = lane % LPR;
                const floatx4 val = *reinterpret_cast<const floatx4 *>(stage + row * ROW + 4 * c4);
                put(kt * a.tk + i * 16 + row, (wp * NPB + b0) * 16 + 4 * c4, val);
            }
        }
}

// ---- instance registry --------------------------------------------------------
// conv_valu slots: ((log2 KPT * 5 + log2 PPT) * 5 + log2 UF) * 2 + LDS
// conv_mfma slots: ((log2 TKB * 7 + log2 NPB) * 3 + D - 1) * 2 + LDS
// conv_mfma2 slots: (((log2 TKB * 6 + log2 NPB) * 3 + log2 U) * 3 + log2 KG) * 2 + (RC == 4)
constexpr int kValuSlots = kConvValuSlots;
constexpr int kMfmaSlots = kConvMfmaSlots;

}  // namespace

extern const void *g_conv_valu[kConvValuSlots];
extern const void *g_conv_mfma[kConvMfmaSlots];
extern const void *g_conv_mfma2[kConvMfma2Slots];

#ifndef DS_SLICE
#define DS_SLICE 0
#define DS_NSLICES 1
#endif

namespace {

template <int I>
void reg_valu() {
    constexpr int lds = I % 2, iuf = (I / 2) % 5, ippt = (I / 10) % 5, ikpt = I / 50;
    constexpr int KPT = 1 << ikpt, PPT = 1 << ippt, UF = 1 << iuf;
    if constexpr (KPT * PPT <= 64 && conv_uf_reachable(KPT * PPT, UF) && I % DS_NSLICES == DS_SLICE)
        g_conv_valu[I] = reinterpret_cast<const void *>(&conv_valu<KPT, PPT, UF, lds>);
}

template <int I>
void reg_mfma() {
    constexpr int lds = I % 2, D = (I / 2) % 3 + 1, inpb = (I / 6) % 7, itkb = I / 42;
    constexpr int TKB = 1 << itkb, NPB = 1 << inpb;
    if constexpr (TKB * NPB <= 32 && conv_mfma_depth_ok(TKB, NPB, D) &&
                  I % DS_NSLICES == DS_SLICE)
        g_conv_mfma[I] = reinterpret_cast<const void *>(&conv_mfma<TKB, NPB, D, lds>);
}

template <int I>
void reg_mfma2() {
    constexpr int few = I % 2, J = I / 2;
    constexpr int ikg = J % 3, iu = (J / 3) % 3, inpb = (J / 9) % 6, itkb = J / 54;
    constexpr int TKB = 1 << itkb, NPB = 1 << inpb, U = 1 << iu, KG = 1 << ikg;
    constexpr int RC = few ? kConv2FewCopies : kConv2MaxCopies;
    if constexpr (conv2_regs_ok(TKB, NPB, KG) && I % DS_NSLICES == DS_SLICE)
        g_conv_mfma2[I] = reinterpret_cast<const void *>(&conv_mfma2<TKB, NPB, U, KG, RC>);
}

template <size_t... I>
void reg_all_mfma2(std::index_sequence<I...>) {
    (reg_mfma2<int(I)>(), ...);
}

template <size_t... I>
void reg_all(std::index_sequence<I...>) {
    (reg_valu<int(I)>(), ...);
}
template <size_t... I>
void reg_all_mfma(std::index_sequence<I...>) {
    (reg_mfma<int(I)>(), ...);
}

struct Registrar {
    Registrar() {
        reg_all(std::make_index_sequence<kValuSlots>{});
        reg_all_mfma(std::make_index_sequence<kMfmaSlots>{});
        reg_all_mfma2(std::make_index_sequence<kConvMfma2Slots>{});
    }
};
const Registrar registrar;

}  // namespace

}  // namespace ds
