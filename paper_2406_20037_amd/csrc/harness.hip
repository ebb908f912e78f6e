// Launch plans, kernel_run, reference kernels and the hipEvent measurement
// harness (the "trial" of Section 2.1: observing one schedule's execution).
#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <limits>
#include <map>
#include <mutex>
#include <set>
#include <utility>
#include <vector>

#include "kern_common.h"
#include "kern_reduce.h"

namespace ds {

const Space &space_of(const ds_space *s);

const void *g_conv_valu[kConvValuSlots];
const void *g_conv_mfma[kConvMfmaSlots];
const void *g_conv_mfma2[kConvMfma2Slots];
const void *g_mm_valu[kMmValuSlots];
const void *g_mm_mfma[kMmMfmaSlots];

namespace {

int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }

int log2_exact(int v) {
    if (v < 1 || (v & (v - 1))) return -1;
    int l = 0;
    while ((1 << l) < v) ++l;
    return l;
}

bool hip_ok(hipError_t e, const char *what) {
    if (e == hipSuccess) return true;
    set_error("%s: %s", what, hipGetErrorString(e));
    return false;
}

// ---- small kernels ------------------------------------------------------------

// Fills n floats with v: 16-byte stores over the aligned body, scalar head and tail.
__global__ void fill_kernel(float *p, int64_t n, float v) {
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    const int64_t tid = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t head = int64_t((16 - (reinterpret_cast<uintptr_t>(p) & 15)) & 15) / 4;
    const int64_t h = head < n ? head : n;
    const int64_t body = (n - h) / 4;
    floatx4 *q = reinterpret_cast<floatx4 *>(p + h);
    const floatx4 v4 = {v, v, v, v};
    for (int64_t i = tid; i < body; i += stride) q[i] = v4;
    if (tid < h) p[tid] = v;
    const int64_t t0 = h + 4 * body;
    if (tid < n - t0) p[t0 + tid] = v;
}

constexpr int kCeilBlocks = 16;                // accumulator blocks per wave

__global__ void fill_u32_kernel(unsigned *p, int n) {
    if (int(threadIdx.x) < n) p[threadIdx.x] = 0u;
}

// max |y - ref| and max |ref| (as order-preserving bit patterns of
// non-negative floats) and the count of non-finite y.
__global__ __launch_bounds__(256) void parity_kernel(const float *y, const float *ref, int64_t n,
                                                     unsigned *out) {
    float me = 0.f, mr = 0.f;
    unsigned bad = 0;
    const int64_t stride = int64_t(gridDim.x) * blockDim.x;
    for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) {
        const float a = y[i], b = ref[i];
        if (!isfinite(a)) bad++;
        else me = fmaxf(me, fabsf(a - b));
        mr = fmaxf(mr, fabsf(b));
    }
    for (int off = 32; off > 0; off >>= 1) {
        me = fmaxf(me, __shfl_xor(me, off));
        mr = fmaxf(mr, __shfl_xor(mr, off));
        bad += __shfl_xor(bad, off);
    }
    if ((threadIdx.x & 63) == 0) {
        atomicMax(out + 0, __float_as_uint(me));
        atomicMax(out + 1, __float_as_uint(mr));
        atomicAdd(out + 2, bad);
    }
}

__global__ void empty_kernel() {}

// The fp32 MFMA pipe under a pure MFMA load: every wave issues back-to-back
// 16x16x4 MFMAs into 16 independent accumulator blocks from register
// operands, with no memory access in the loop; one float per thread leaves
// through sink so the work is kept.
__global__ __launch_bounds__(256) void mfma_ceiling_kernel(float *sink, int iters) {
    const int lane = threadIdx.x & 63;
    const float a = 1.0f + 1e-3f * lane, b = 1.0f - 1e-3f * lane;
    floatx4 acc[kCeilBlocks];
#pragma unroll
    for (int i = 0; i < kCeilBlocks; ++i) acc[i] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int i = 0; i < kCeilBlocks; ++i)
            acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[i], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kCeilBlocks; ++i) s += acc[i][0] + acc[i][1] + acc[i][2] + acc[i][3];
    sink[int64_t(blockIdx.x) * blockDim.x + threadIdx.x] = s;
}

// One thread per output, reduction in the definition's order (c, r, s / k).
__global__ __launch_bounds__(256) void conv_ref_kernel(ConvArgs a) {
    const int64_t total = int64_t(a.N) * a.K * a.P * a.Q;
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= total) return;
    int64_t f = i;
    const int q = int(f % a.Q);
    f /= a.Q;
    const int p = int(f % a.P);
    f /= a.P;
    const int k = int(f % a.K);
    const int n = int(f / a.K);
    float acc = 0.f;
    for (int c = 0; c < a.C; ++c)
        for (int r = 0; r < a.R; ++r) {
            const int iy = p * a.st - a.pd + r;
            if (iy < 0 || iy >= a.H) continue;
            for (int s = 0; s < a.S; ++s) {
                const int ix = q * a.st - a.pd + s;
                if (ix < 0 || ix >= a.W) continue;
                acc = fmaf(a.x[((size_t(n) * a.C + c) * a.H + iy) * a.W + ix],
                           a.w[((size_t(k) * a.C + c) * a.R + r) * a.S + s], acc);
            }
        }
    a.y[i] = acc;
}

__global__ __launch_bounds__(256) void mm_ref_kernel(MatmulArgs a) {
    const int64_t total = int64_t(a.M) * a.N;
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int m = int(i / a.N), nn = int(i % a.N);
    float acc = 0.f;
    for (int k = 0; k < a.K; ++k)
        acc = fmaf(a.A[size_t(m) * a.K + k], a.B[size_t(k) * a.N + nn], acc);
    a.C[i] = acc;
}

// ---- per-device state ------------------------------------------------------------

constexpr int kMaxDevices = 64;
std::mutex g_mu;
unsigned *g_parity_buf[kMaxDevices];     // 4 words per device, library-owned
hipStream_t g_graph_stream[kMaxDevices];  // capture / replay stream per device
// Partial outputs of split reductions: one buffer per (device, stream), so
// split launches on different streams never share partials.  A buffer that
// grows is retired, not freed: a graph the caller captured earlier may still
// hold its address.  Retired and live buffers are freed by ds_shutdown.
struct SplitWs {
    float *p = nullptr;
    int64_t elems = 0;
};
std::map<std::pair<int, hipStream_t>, SplitWs> g_split_ws;
std::vector<std::pair<int, void *>> g_split_retired;
std::set<std::pair<int, const void *>> g_lds_attr;

// Split-reduction partials of kernel_run_noalloc: a fixed array in device
// memory (one copy per device, held until the process ends), so that entry
// point never allocates.  Host code never passes the array's name to a kernel:
// g_scratch[dev] holds the address the runtime reports for this device.
constexpr int64_t kScratchFloats = DS_NOALLOC_MAX_FLOATS;   // 32 MiB
static __device__ __align__(256) float scratch[kScratchFloats];
float *g_scratch[kMaxDevices];

int current_device(int &dev) {
    if (!hip_ok(hipGetDevice(&dev), "hipGetDevice")) return DS_EHIP;
    if (dev < 0 || dev >= kMaxDevices) {
        set_error("device index %d out of range", dev);
        return DS_EUNSUPPORTED;
    }
    return DS_OK;
}

int parity_buffer(unsigned **out) {
    int dev;
    int rc = current_device(dev);
    if (rc != DS_OK) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_parity_buf[dev]) {
        void *p = nullptr;
        if (!hip_ok(hipMalloc(&p, 16), "hipMalloc(parity)")) return DS_ENOMEM;
        g_parity_buf[dev] = static_cast<unsigned *>(p);
    }
    *out = g_parity_buf[dev];
    return DS_OK;
}

int graph_stream(hipStream_t *out) {
    int dev;
    int rc = current_device(dev);
    if (rc != DS_OK) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_graph_stream[dev]) {
        hipStream_t st;
        if (!hip_ok(hipStreamCreateWithFlags(&st, hipStreamNonBlocking), "hipStreamCreate"))
            return DS_EHIP;
        g_graph_stream[dev] = st;
    }
    *out = g_graph_stream[dev];
    return DS_OK;
}

// The split-reduction workspace of `stream` on the current device, grown to at
// least `elems` floats.  Growing allocates a new buffer (at least twice the
// old size) and retires the old one after the stream's queued work is done;
// while the stream is being captured nothing may be allocated, so a capture
// needs the buffer to exist already (one uncaptured call of the same schedule
// on that stream creates it).
int split_workspace(int64_t elems, hipStream_t stream, float **out) {
    int dev;
    int rc = current_device(dev);
    if (rc != DS_OK) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    SplitWs &ws = g_split_ws[{dev, stream}];
    if (ws.elems < elems) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (!hip_ok(hipStreamIsCapturing(stream, &cap), "hipStreamIsCapturing")) return DS_EHIP;
        if (cap != hipStreamCaptureStatusNone) {
            set_error("split reduction needs %lld workspace floats on a stream under capture; run "
                      "the schedule once on that stream outside capture first, or use "
                      "kernel_run_noalloc",
                      (long long)elems);
            return DS_EUNSUPPORTED;
        }
        const int64_t grow = std::max<int64_t>(elems, 2 * ws.elems);
        void *p = nullptr;
        if (!hip_ok(hipMalloc(&p, size_t(grow) * sizeof(float)), "hipMalloc(split workspace)"))
            return DS_ENOMEM;
        if (ws.p) {
            if (!hip_ok(hipStreamSynchronize(stream), "hipStreamSynchronize")) {
                (void)hipFree(p);
                return DS_EHIP;
            }
            g_split_retired.emplace_back(dev, ws.p);
        }
        ws.p = static_cast<float *>(p);
        ws.elems = grow;
    }
    *out = ws.p;
    return DS_OK;
}

// This device's address of `scratch`, looked up on the first call on the
// device (with that device current) and kept.
int scratch_ptr(float **out) {
    int dev;
    int rc = current_device(dev);
    if (rc != DS_OK) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        if (!hip_ok(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)"))
            return DS_EHIP;
        if (!p) {
            set_error("hipGetSymbolAddress(scratch) returned a null address");
            return DS_EHIP;
        }
        g_scratch[dev] = static_cast<float *>(p);
    }
    *out = g_scratch[dev];
    return DS_OK;
}

int ensure_lds_attr(const void *func, int lds) {
    if (lds <= 65536) return DS_OK;
    int dev;
    int rc = current_device(dev);
    if (rc != DS_OK) return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_lds_attr.count({dev, func})) return DS_OK;
    if (!hip_ok(hipFuncSetAttribute(func, hipFuncAttributeMaxDynamicSharedMemorySize, lds),
                "hipFuncSetAttribute(MaxDynamicSharedMemorySize)"))
        return DS_EHIP;
    g_lds_attr.insert({dev, func});
    return DS_OK;
}

void fill_conv_args(const Space &sp, const float *x, const float *w, float *y, ConvArgs &a) {
    std::memset(&a, 0, sizeof a);
    a.x = x;
    a.w = w;
    a.y = y;
    a.N = int(sp.shape[0]);
    a.C = int(sp.shape[1]);
    a.H = int(sp.shape[2]);
    a.W = int(sp.shape[3]);
    a.K = int(sp.shape[4]);
    a.R = int(sp.shape[5]);
    a.S = int(sp.shape[6]);
    a.st = int(sp.shape[7]);
    a.pd = int(sp.shape[8]);
    a.P = int(conv_out_dim(a.H, a.R, a.st, a.pd));
    a.Q = int(conv_out_dim(a.W, a.S, a.st, a.pd));
}

void fill_mm_args(const Space &sp, const float *A, const float *B, float *C, MatmulArgs &a) {
    std::memset(&a, 0, sizeof a);
    a.A = A;
    a.B = B;
    a.C = C;
    a.M = int(sp.shape[0]);
    a.N = int(sp.shape[1]);
    a.K = int(sp.shape[2]);
    a.gm = 1;
}

double elapsed_ms(hipEvent_t a, hipEvent_t b) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return std::numeric_limits<double>::quiet_NaN();
    return double(ms);
}

struct Events {
    std::vector<hipEvent_t> ev;
    ~Events() {
        for (auto e : ev) (void)hipEventDestroy(e);
    }
    bool make(int n) {
        for (int i = 0; i < n; ++i) {
            hipEvent_t e;
            if (!hip_ok(hipEventCreate(&e), "hipEventCreate")) return false;
            ev.push_back(e);
        }
        return true;
    }
};

// Times `repeat` repeats of `number` launches of fn on stream.
template <class F>
int time_repeats(F &&fn, hipStream_t stream, int number, int repeat, double *rep) {
    Events E;
    if (!E.make(repeat + 1)) return DS_EHIP;
    if (!hip_ok(hipEventRecord(E.ev[0], stream), "hipEventRecord")) return DS_EHIP;
    for (int r = 0; r < repeat; ++r) {
        for (int i = 0; i < number; ++i) {
            const int rc = fn();
            if (rc != DS_OK) return rc;
        }
        if (!hip_ok(hipEventRecord(E.ev[r + 1], stream), "hipEventRecord")) return DS_EHIP;
    }
    if (!hip_ok(hipEventSynchronize(E.ev[repeat]), "hipEventSynchronize")) return DS_EHIP;
    for (int r = 0; r < repeat; ++r) rep[r] = elapsed_ms(E.ev[r], E.ev[r + 1]) / number;
    return DS_OK;
}

// Times `repeat` replays of a graph holding `number` launches of fn(stream).
template <class F>
int time_graph(F &&fn, hipStream_t caller, int number, int repeat, double *rep) {
    hipStream_t st;
    int rc = graph_stream(&st);
    if (rc != DS_OK) return rc;
    if (!hip_ok(hipStreamSynchronize(caller), "hipStreamSynchronize")) return DS_EHIP;
    hipGraph_t graph = nullptr;
    hipGraphExec_t exec = nullptr;
    if (!hip_ok(hipStreamBeginCapture(st, hipStreamCaptureModeRelaxed), "hipStreamBeginCapture"))
        return DS_EHIP;
    for (int i = 0; i < number && rc == DS_OK; ++i) rc = fn(st);
    const hipError_t ec = hipStreamEndCapture(st, &graph);
    if (rc != DS_OK || !hip_ok(ec, "hipStreamEndCapture")) {
        if (graph) (void)hipGraphDestroy(graph);
        return rc != DS_OK ? rc : DS_EHIP;
    }
    rc = DS_OK;
    if (!hip_ok(hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0), "hipGraphInstantiate"))
        rc = DS_EHIP;
    Events E;
    if (rc == DS_OK && !E.make(repeat + 1)) rc = DS_EHIP;
    if (rc == DS_OK && (!hip_ok(hipGraphLaunch(exec, st), "hipGraphLaunch") ||
                        !hip_ok(hipEventRecord(E.ev[0], st), "hipEventRecord")))
        rc = DS_EHIP;
    for (int r = 0; r < repeat && rc == DS_OK; ++r)
        if (!hip_ok(hipGraphLaunch(exec, st), "hipGraphLaunch") ||
            !hip_ok(hipEventRecord(E.ev[r + 1], st), "hipEventRecord"))
            rc = DS_EHIP;
    if (rc == DS_OK && !hip_ok(hipStreamSynchronize(st), "hipStreamSynchronize")) rc = DS_EHIP;
    if (rc == DS_OK)
        for (int r = 0; r < repeat; ++r) rep[r] = elapsed_ms(E.ev[r], E.ev[r + 1]) / number;
    if (exec) (void)hipGraphExecDestroy(exec);
    (void)hipGraphDestroy(graph);
    return rc;
}

void summarise(ds_measurement *out, int n) {
    std::vector<double> v(out->repeats_ms, out->repeats_ms + n);
    std::sort(v.begin(), v.end());
    out->n_repeats = n;
    out->median_ms = n % 2 ? v[n / 2] : 0.5 * (v[n / 2 - 1] + v[n / 2]);
    out->min_ms = v.front();
    double s = 0;
    for (double t : v) s += t;
    out->mean_ms = s / n;
}

}  // namespace

// ---- instance lookup ---------------------------------------------------------------

const void *conv_valu_instance(int kpt, int ppt, int uf, int lds) {
    const int a = log2_exact(kpt), b = log2_exact(ppt), c = log2_exact(uf);
    if (a < 0 || a > 6 || b < 0 || b > 4 || c < 0 || c > 4 || (lds & ~1)) return nullptr;
    return g_conv_valu[((a * 5 + b) * 5 + c) * 2 + lds];
}

const void *conv_mfma_instance(int tkb, int npb, int d, int lds) {
    const int a = log2_exact(tkb), b = log2_exact(npb);
    if (a < 0 || a > 2 || b < 0 || b > 6 || d < 1 || d > 3 || (lds & ~1)) return nullptr;
    return g_conv_mfma[((a * 7 + b) * 3 + d - 1) * 2 + lds];
}

const void *conv_mfma2_instance(int tkb, int npb, int u, int kg, int rc) {
    const int a = log2_exact(tkb), b = log2_exact(npb), c = log2_exact(u), d = log2_exact(kg);
    if (a < 0 || a > 2 || b < 0 || b > 5 || c < 0 || c > 2 || d < 0 || d > 2) return nullptr;
    if (rc != kConv2FewCopies && rc != kConv2MaxCopies) return nullptr;
    return g_conv_mfma2[(((a * 6 + b) * 3 + c) * 3 + d) * 2 + (rc == kConv2FewCopies)];
}

const void *mm_valu_instance(int rm, int rn, int bk, int uf, int dbuf) {
    const int a = log2_exact(rm), b = log2_exact(rn), k = log2_exact(bk) - 2, c = log2_exact(uf);
    if (a < 0 || a > 4 || b < 0 || b > 4 || k < 0 || k > 4 || c < 0 || c > 6 || (dbuf & ~1))
        return nullptr;
    return g_mm_valu[(((a * 5 + b) * 5 + k) * 7 + c) * 2 + dbuf];
}

const void *mm_mfma_instance(int wm, int wn, int bk, int uf, int dbuf, int kg) {
    const int a = log2_exact(wm) - 4, b = log2_exact(wn) - 4, k = log2_exact(bk) - 2,
              c = log2_exact(uf);
    if (a < 0 || a > 3 || b < 0 || b > 3 || k < 0 || k > 4 || c < 0 || c > 6 || (dbuf & ~1) ||
        kg < 1 || kg > 2)
        return nullptr;
    return g_mm_mfma[((((a * 4 + b) * 5 + k) * 7 + c) * 2 + dbuf) * 2 + (kg - 1)];
}

int count_instances() {
    int n = 0;
    for (auto p : g_conv_valu) n += p != nullptr;
    for (auto p : g_conv_mfma) n += p != nullptr;
    for (auto p : g_conv_mfma2) n += p != nullptr;
    for (auto p : g_mm_valu) n += p != nullptr;
    for (auto p : g_mm_mfma) n += p != nullptr;
    return n;
}

// ---- plans -------------------------------------------------------------------------

int make_plan(const ds_sched *s, const float *x, const float *w, float *y, Plan &plan) {
    if (!s) {
        set_error("schedule is null");
        return DS_EINVAL;
    }
    Space sp;
    const int len = s->op == DS_OP_CONV2D_NCHW ? 9 : 3;
    int rc = build_space(s->op, s->shape, len, sp);
    if (rc != DS_OK) return rc;
    if (s->nknobs != sp.nknobs || !sp.in_range(s->idx)) {
        set_error("schedule index vector does not fit the space");
        return DS_EINVAL;
    }
    const Geometry g = sp.geometry(s->idx);
    if (!g.valid) {
        set_error("schedule is not a valid point of its search space");
        return DS_EINVALID_SCHED;
    }
    plan = Plan();
    plan.op = s->op;
    plan.threads = g.threads;
    plan.grid = g.grid;
    plan.lds = g.lds_bytes;
    if (s->op == DS_OP_CONV2D_NCHW && sp.value(s->idx, 7) >= 2) {
        Conv2Args &a = plan.conv2;
        const Conv2Shape c = conv2_setup(sp.shape, sp.value(s->idx, 0), sp.value(s->idx, 1),
                                         sp.value(s->idx, 2), sp.value(s->idx, 3), g.unroll_eff,
                                         sp.value(s->idx, 6), sp.value(s->idx, 8),
                                         sp.value(s->idx, 7) == 3, a);
        a.x = x;
        a.w = w;
        a.y = y;
        // 16-byte copies only from 16-byte aligned operands (else 4-byte
        // copies into the same layout)
        const int vw0 = a.vw, vh0 = a.vh;
        if (reinterpret_cast<uintptr_t>(w) % 16 != 0) a.vw = 0;
        if (reinterpret_cast<uintptr_t>(x) % 16 != 0) a.vh = 0;
        if (a.vw != vw0 || a.vh != vh0) conv2_units(a, c.threads);
        // 16-byte output stores only into a 16-byte aligned output (and
        // partials: the workspace is)
        if (reinterpret_cast<uintptr_t>(y) % 16 != 0) a.st4 = 0;
        plan.func = conv_mfma2_instance(c.tkb, c.npb, c.u, c.kg, a.rc);
        plan.family = DS_KERNEL_CONV_MFMA2;
        plan.nparams = 5;
        const int pr[5] = {c.tkb, c.npb, c.u, c.kg, a.rc};
        std::memcpy(plan.params, pr, sizeof pr);
        plan.slot = (((log2_exact(c.tkb) * 6 + log2_exact(c.npb)) * 3 + log2_exact(c.u)) * 3 +
                     log2_exact(c.kg)) * 2 + (a.rc == kConv2FewCopies);
        plan.splits = a.ksw > 1 ? int(cdiv64(a.chunks, a.cps)) : 1;
        plan.y_elems = int64_t(a.N) * a.K * a.P * a.Q;
    } else if (s->op == DS_OP_CONV2D_NCHW) {
        ConvArgs &a = plan.conv;
        fill_conv_args(sp, x, w, y, a);
        a.tk = sp.value(s->idx, 0);
        a.th = sp.value(s->idx, 1);
        a.tw = sp.value(s->idx, 2);
        a.tc = sp.value(s->idx, 3);
        const int lds = sp.value(s->idx, 5);
        a.ks = sp.value(s->idx, 6);
        const int mfma = sp.value(s->idx, 7);
        a.tiles_k = int(cdiv64(a.K, a.tk));
        a.tiles_p = int(cdiv64(a.P, a.th));
        a.tiles_q = int(cdiv64(a.Q, a.tw));
        a.chunks = int(g.chunks);
        a.cps = int(cdiv64(a.chunks, a.ks));
        a.red = g.red;
        a.wrow = mfma ? g.red + 4 : g.red;
        a.hs = (a.th - 1) * a.st + a.R;
        // aligned halo layout when image rows are whole 16-byte groups and the
        // tile is at least 16 columns wide: rows start at the 16-byte boundary
        // at or before the tile's first column (up to 3 more columns, rounded
        // to 4); otherwise rows hold exactly the tile's input columns
        // (only with 16-byte copies, vec = 4)
        const int vec = sp.value(s->idx, 8);
        const bool halo16 = vec == 4 && a.W % 4 == 0 && a.tw * a.st >= 16;
        a.ws = halo16 ? int(cdiv64(int64_t(a.tw - 1) * a.st + a.S + 3, 4) * 4)
                      : (a.tw - 1) * a.st + a.S;
        a.npx = a.th * a.tw;
        a.npl = std::min(a.npx, 256);
        a.ltw = log2_exact(a.tw);
        a.f_hw = make_fastdiv(a.hs * a.ws);
        a.f_ws = make_fastdiv(a.ws);
        a.f_red = make_fastdiv(a.red);
        a.f_rs = make_fastdiv(a.R * a.S);
        a.f_s = make_fastdiv(a.S);
        a.f_wrow = make_fastdiv(a.wrow);
        // bit 0: weight rows staged 16 bytes per lane; bit 1: halo rows too;
        // bit 2: aligned halo layout (16-byte copies only with vec = 4, and
        // only from 16-byte aligned operands)
        a.w4 = (vec == 4 && (a.C * a.R * a.S) % 4 == 0 && (a.tc * a.R * a.S) % 4 == 0 &&
                        a.wrow % 4 == 0 && reinterpret_cast<uintptr_t>(w) % 16 == 0
                    ? 1
                    : 0) |
               (halo16 && (int64_t(a.tk) * a.wrow) % 4 == 0 &&
                        reinterpret_cast<uintptr_t>(x) % 16 == 0
                    ? 2
                    : 0) |
               (halo16 ? 4 : 0);
        a.nbuf = cdiv64(a.chunks, a.ks) > 1 ? 2 : 1;
        a.buf = int(cdiv64(int64_t(a.tk) * a.wrow + int64_t(a.tc) * a.hs * a.ws + 1, 4) * 4);
        plan.func = mfma ? conv_mfma_instance(g.t0, g.t1, g.unroll_eff, lds)
                         : conv_valu_instance(g.t0, g.t1, g.unroll_eff, lds);
        plan.family = mfma ? DS_KERNEL_CONV_MFMA : DS_KERNEL_CONV_VALU;
        plan.nparams = 4;
        const int pr[4] = {g.t0, g.t1, g.unroll_eff, lds};
        std::memcpy(plan.params, pr, sizeof pr);
        plan.slot = mfma ? ((log2_exact(g.t0) * 7 + log2_exact(g.t1)) * 3 + g.unroll_eff - 1) * 2 + lds
                         : ((log2_exact(g.t0) * 5 + log2_exact(g.t1)) * 5 + log2_exact(g.unroll_eff)) *
                                   2 + lds;
        plan.splits = a.ks > 1 ? int(cdiv64(a.chunks, a.cps)) : 1;
        plan.y_elems = int64_t(a.N) * a.K * a.P * a.Q;
    } else {
        MatmulArgs &a = plan.mm;
        fill_mm_args(sp, x, w, y, a);
        const int bm = sp.value(s->idx, 0), bn = sp.value(s->idx, 1), bk = sp.value(s->idx, 2);
        const int dbuf = sp.value(s->idx, 4), mfma = sp.value(s->idx, 5);
        const int kg = mm_wave_groups(mfma, sp.value(s->idx, 6), bk);
        a.ks = sp.value(s->idx, 6) / kg;
        a.tiles_m = int(cdiv64(a.M, bm));
        a.tiles_n = int(cdiv64(a.N, bn));
        a.nkt = int(g.chunks);
        a.kps = int(cdiv64(a.nkt, a.ks));
        // 16-byte operand loads only with vec = 4 (and aligned operands)
        const int vec = sp.value(s->idx, 7);
        a.vecA = vec == 4 && (a.K % 4 == 0) && (reinterpret_cast<uintptr_t>(x) % 16 == 0);
        a.vecB = vec == 4 && (a.N % 4 == 0) && (reinterpret_cast<uintptr_t>(w) % 16 == 0);
        a.direct = a.vecA && a.vecB && a.M % bm == 0 && a.N % bn == 0 && a.K % bk == 0;
        a.gm = mm_group_rows(a.tiles_m, a.tiles_n, a.ks, bm, bn);
        plan.func = mfma ? mm_mfma_instance(g.t0, g.t1, bk, g.unroll_eff, dbuf, kg)
                         : mm_valu_instance(g.t0, g.t1, bk, g.unroll_eff, dbuf);
        plan.family = mfma ? DS_KERNEL_MM_MFMA : DS_KERNEL_MM_VALU;
        plan.nparams = mfma ? 6 : 5;
        const int pr[6] = {g.t0, g.t1, bk, g.unroll_eff, dbuf, kg};
        std::memcpy(plan.params, pr, sizeof pr);
        const int lb = log2_exact(bk) - 2, lu = log2_exact(g.unroll_eff);
        plan.slot = mfma ? ((((log2_exact(g.t0) - 4) * 4 + (log2_exact(g.t1) - 4)) * 5 + lb) * 7 + lu) *
                                   4 + dbuf * 2 + (kg - 1)
                         : (((log2_exact(g.t0) * 5 + log2_exact(g.t1)) * 5 + lb) * 7 + lu) * 2 + dbuf;
        plan.splits = a.ks > 1 ? int(cdiv64(a.nkt, a.kps)) : 1;
        plan.y_elems = int64_t(a.M) * a.N;
    }
    if (!plan.func) {
        set_error("no compiled kernel instance for this schedule");
        return DS_EUNSUPPORTED;
    }
    return DS_OK;
}

int64_t workspace_elems(const Plan &plan) {
    if (plan.splits <= 1 || plan.y_elems == 0 || plan.grid == 0) return 0;
    // Splits that own no reduction step exit early; the reduce kernel sums only
    // the first plan.splits partial slices.
    const int ks = plan.family == DS_KERNEL_CONV_MFMA2 ? plan.conv2.ksw
                   : plan.op == DS_OP_CONV2D_NCHW      ? plan.conv.ks
                                                       : plan.mm.ks;
    return int64_t(ks) * plan.y_elems;
}

void set_workspace(Plan &plan, float *part) {
    if (plan.family == DS_KERNEL_CONV_MFMA2) plan.conv2.part = part;
    else if (plan.op == DS_OP_CONV2D_NCHW) plan.conv.part = part;
    else plan.mm.part = part;
}

int attach_workspace(Plan &plan, hipStream_t stream) {
    const int64_t elems = workspace_elems(plan);
    if (elems == 0) return DS_OK;
    float *part = nullptr;
    const int rc = split_workspace(elems, stream, &part);
    if (rc != DS_OK) return rc;
    set_workspace(plan, part);
    return DS_OK;
}

int fill_async(float *p, int64_t n, float v, hipStream_t stream) {
    if (n <= 0) return DS_OK;
    const int64_t blocks = std::min<int64_t>(cdiv64(cdiv64(n, 4), 256), 2048);
    hipLaunchKernelGGL(fill_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, p, n, v);
    return hip_ok(hipGetLastError(), "fill launch") ? DS_OK : DS_EHIP;
}

int launch_plan(const Plan &plan, hipStream_t stream) {
    if (plan.grid == 0 || plan.y_elems == 0) return DS_OK;
    if (plan.splits > kMaxSplits) {      // the lattice's split axes stop at 32
        set_error("more than %d reduction splits", kMaxSplits);
        return DS_EUNSUPPORTED;
    }
    int rc = ensure_lds_attr(plan.func, plan.lds);
    if (rc != DS_OK) return rc;
    void *args[1];
    if (plan.family == DS_KERNEL_CONV_MFMA2) args[0] = const_cast<Conv2Args *>(&plan.conv2);
    else if (plan.op == DS_OP_CONV2D_NCHW) args[0] = const_cast<ConvArgs *>(&plan.conv);
    else args[0] = const_cast<MatmulArgs *>(&plan.mm);
    if (!hip_ok(hipLaunchKernel(plan.func, dim3(unsigned(plan.grid)), dim3(plan.threads), args,
                                size_t(plan.lds), stream),
                "hipLaunchKernel"))
        return DS_EHIP;
    if (plan.splits > 1) {
        const bool c2 = plan.family == DS_KERNEL_CONV_MFMA2;
        float *y = c2 ? plan.conv2.y : plan.op == DS_OP_CONV2D_NCHW ? plan.conv.y : plan.mm.C;
        const float *part = c2 ? plan.conv2.part
                               : plan.op == DS_OP_CONV2D_NCHW ? plan.conv.part : plan.mm.part;
        const int64_t n4 = cdiv64(plan.y_elems, 4);
        const int64_t blocks = std::min<int64_t>(cdiv64(n4, 256), 4096);
        int64_t n = plan.y_elems;
        void *rargs[] = {const_cast<float **>(&part), &y, &n};
        if (!hip_ok(hipLaunchKernel(split_reduce_kernel_for(plan.splits), dim3(unsigned(blocks)),
                                    dim3(256), rargs, 0, stream),
                    "split reduce launch"))
            return DS_EHIP;
        if (!hip_ok(hipGetLastError(), "split reduce launch")) return DS_EHIP;
    }
    return DS_OK;
}

int reference_output(const Space &sp, const ds_tune_io *io, float **ref_out) {
    *ref_out = nullptr;
    int64_t n;
    if (sp.op == DS_OP_CONV2D_NCHW) {
        const int64_t P = conv_out_dim(sp.shape[2], sp.shape[5], sp.shape[7], sp.shape[8]);
        const int64_t Q = conv_out_dim(sp.shape[3], sp.shape[6], sp.shape[7], sp.shape[8]);
        n = sp.shape[0] * sp.shape[4] * P * Q;
    } else {
        n = sp.shape[0] * sp.shape[1];
    }
    if (n == 0) return DS_OK;
    void *p = nullptr;
    if (!hip_ok(hipMalloc(&p, size_t(n) * sizeof(float)), "hipMalloc(reference)")) return DS_ENOMEM;
    const int rc = kernel_run_reference(sp.op, sp.shape, io->x, io->w, static_cast<float *>(p),
                                        io->stream);
    if (rc != DS_OK || !hip_ok(hipStreamSynchronize(io->stream), "reference kernel")) {
        (void)hipFree(p);
        return rc != DS_OK ? rc : DS_EHIP;
    }
    *ref_out = static_cast<float *>(p);
    return DS_OK;
}

void free_device(void *p) {
    if (p) (void)hipFree(p);
}

}  // namespace ds

using namespace ds;

extern "C" {

int kernel_run(int op, const ds_sched *s, const float *x, const float *w, float *y,
               hipStream_t stream) {
    if (!s || s->op != op) {
        set_error("schedule missing or for another op");
        return DS_EINVAL;
    }
    Plan plan;
    int rc = make_plan(s, x, w, y, plan);
    if (rc != DS_OK) return rc;
    if (plan.y_elems > 0 && plan.grid > 0 && (!x || !w || !y)) {
        set_error("null buffer");
        return DS_EINVAL;
    }
    rc = attach_workspace(plan, stream);
    if (rc != DS_OK) return rc;
    return launch_plan(plan, stream);
}

int kernel_run_noalloc(int op, const ds_sched *s, const float *x, const float *w, float *y,
                       hipStream_t stream) {
    if (!s || s->op != op) {
        set_error("schedule missing or for another op");
        return DS_EINVAL;
    }
    Plan plan;
    int rc = make_plan(s, x, w, y, plan);
    if (rc != DS_OK) return rc;
    if (plan.y_elems > 0 && plan.grid > 0 && (!x || !w || !y)) {
        set_error("null buffer");
        return DS_EINVAL;
    }
    const int64_t elems = workspace_elems(plan);
    if (elems > kScratchFloats) {
        set_error("kernel_run_noalloc: the split reduction needs %lld partial floats, more than the "
                  "%lld of its fixed scratch; use a schedule with fewer splits or kernel_run",
                  (long long)elems, (long long)kScratchFloats);
        return DS_EINVAL;
    }
    if (elems > 0) {
        float *p = nullptr;
        rc = scratch_ptr(&p);
        if (rc != DS_OK) return rc;
        set_workspace(plan, p);
    }
    return launch_plan(plan, stream);
}

int kernel_run_reference(int op, const int64_t *shape, const float *x, const float *w, float *y,
                         hipStream_t stream) {
    Space sp;
    int rc = build_space(op, shape, op == DS_OP_CONV2D_NCHW ? 9 : 3, sp);
    if (rc != DS_OK) return rc;
    int64_t total;
    if (op == DS_OP_CONV2D_NCHW) {
        ConvArgs a;
        fill_conv_args(sp, x, w, y, a);
        total = int64_t(a.N) * a.K * a.P * a.Q;
        if (total == 0) return DS_OK;
        if (!x || !w || !y) {
            set_error("null buffer");
            return DS_EINVAL;
        }
        hipLaunchKernelGGL(conv_ref_kernel, dim3(unsigned(cdiv64(total, 256))), dim3(256), 0,
                           stream, a);
    } else {
        MatmulArgs a;
        fill_mm_args(sp, x, w, y, a);
        total = int64_t(a.M) * a.N;
        if (total == 0) return DS_OK;
        if (!x || !w || !y) {
            set_error("null buffer");
            return DS_EINVAL;
        }
        hipLaunchKernelGGL(mm_ref_kernel, dim3(unsigned(cdiv64(total, 256))), dim3(256), 0,
                           stream, a);
    }
    return hip_ok(hipGetLastError(), "reference launch") ? DS_OK : DS_EHIP;
}

}  // extern "C"

namespace {

// Parity of y against ref (NaN/Inf count, max |y - ref|, max |ref|); synchronises.
int parity_check(const float *y, const float *ref, int64_t n, double tol, hipStream_t stream,
                 ds_measurement *out) {
    unsigned *buf = nullptr;
    int rc = parity_buffer(&buf);
    if (rc != DS_OK) return rc;
    hipLaunchKernelGGL(fill_u32_kernel, dim3(1), dim3(64), 0, stream, buf, 4);
    const int64_t blocks = std::min<int64_t>(cdiv64(n, 256), 1024);
    hipLaunchKernelGGL(parity_kernel, dim3(unsigned(blocks)), dim3(256), 0, stream, y, ref, n, buf);
    unsigned host[4] = {0, 0, 0, 0};
    if (!hip_ok(hipGetLastError(), "parity launch") ||
        !hip_ok(hipMemcpyAsync(host, buf, 16, hipMemcpyDeviceToHost, stream), "parity copy") ||
        !hip_ok(hipStreamSynchronize(stream), "parity sync"))
        return DS_EHIP;
    float fe, fr;
    std::memcpy(&fe, &host[0], 4);
    std::memcpy(&fr, &host[1], 4);
    out->max_err = std::max(out->max_err, double(fe));
    out->max_ref = std::max(out->max_ref, double(fr));
    out->nonfinite += host[2];
    if (host[2] != 0 || !(double(fe) <= tol * double(fr))) {
        set_error("parity failed: max_err %.3g, max_ref %.3g, non-finite %u", double(fe), double(fr),
                  host[2]);
        return DS_EPARITY;
    }
    return DS_OK;
}

}  // namespace

extern "C" {

int ds_measure(const ds_sched *s, const ds_tune_io *io, const ds_measure_cfg *cfg_in,
               double best_so_far_ms, ds_measurement *out) {
    if (!s || !io || !out) {
        set_error("null argument");
        return DS_EINVAL;
    }
    std::memset(out, 0, sizeof *out);
    out->median_ms = out->mean_ms = out->min_ms = std::numeric_limits<double>::infinity();
    ds_measure_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_measure_cfg_default(&cfg);
    cfg.repeat = std::max(1, std::min(cfg.repeat, DS_MAX_REPEATS));
    cfg.max_number = std::max(1, cfg.max_number);
    cfg.warmup = std::max(0, cfg.warmup);

    Plan plan;
    int rc = make_plan(s, io->x, io->w, io->y, plan);
    if (rc != DS_OK) {
        out->status = rc;
        return rc == DS_EINVALID_SCHED ? DS_OK : rc;
    }
    if (plan.y_elems > 0 && (!io->x || !io->w || !io->y)) {
        set_error("null buffer");
        return DS_EINVAL;
    }
    rc = attach_workspace(plan, io->stream);
    if (rc != DS_OK) {
        out->status = rc;
        return DS_OK;
    }
    const hipStream_t stream = io->stream;
    const bool check = cfg.check && io->ref && plan.y_elems > 0;
    auto launch = [&]() { return launch_plan(plan, stream); };
    auto launch_on = [&](hipStream_t st) { return launch_plan(plan, st); };
    auto fail = [&](int code) {
        out->status = code;
        out->median_ms = out->mean_ms = out->min_ms = std::numeric_limits<double>::infinity();
        return DS_OK;
    };

    // Parity launch on a NaN-filled output.
    if (check) {
        rc = fill_async(io->y, plan.y_elems, std::numeric_limits<float>::quiet_NaN(), stream);
        if (rc != DS_OK) return fail(rc);
    }
    double first[1];
    rc = time_repeats(launch, stream, 1, 1, first);
    if (rc != DS_OK) return fail(rc);
    out->first_ms = first[0];
    if (check) {
        rc = parity_check(io->y, io->ref, plan.y_elems, cfg.tol, stream, out);
        if (rc != DS_OK) return fail(rc);
    }
    if (cfg.slow_cut > 0 && best_so_far_ms > 0 && out->first_ms > cfg.slow_cut * best_so_far_ms) {
        out->cut = 1;
        out->number = 1;
        out->repeats_ms[0] = out->first_ms;
        summarise(out, 1);
        return DS_OK;
    }
    // Warm-up, which also calibrates the number of launches per repeat.
    double warm = out->first_ms;
    if (cfg.warmup > 0) {
        double w[1];
        rc = time_repeats(launch, stream, cfg.warmup, 1, w);
        if (rc != DS_OK) return fail(rc);
        warm = w[0];
    }
    const double per = std::max(warm, 1e-4);
    const int number = int(std::max(1.0, std::min(double(cfg.max_number),
                                                  std::ceil(cfg.min_repeat_ms / per))));
    if (cfg.graph) {
        if (check) {
            rc = fill_async(io->y, plan.y_elems, std::numeric_limits<float>::quiet_NaN(), stream);
            if (rc != DS_OK) return fail(rc);
        }
        rc = time_graph(launch_on, stream, number, cfg.repeat, out->repeats_ms);
        if (rc != DS_OK) return fail(rc);
        if (check) {
            rc = parity_check(io->y, io->ref, plan.y_elems, cfg.tol, stream, out);
            if (rc != DS_OK) return fail(rc);
        }
    } else {
        rc = time_repeats(launch, stream, number, cfg.repeat, out->repeats_ms);
        if (rc != DS_OK) return fail(rc);
    }
    out->number = number;
    summarise(out, cfg.repeat);
    return DS_OK;
}

int ds_empty_kernel_floor(hipStream_t stream, const ds_measure_cfg *cfg_in, ds_measurement *out) {
    if (!out) {
        set_error("null argument");
        return DS_EINVAL;
    }
    std::memset(out, 0, sizeof *out);
    ds_measure_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_measure_cfg_default(&cfg);
    cfg.repeat = std::max(1, std::min(cfg.repeat, DS_MAX_REPEATS));
    auto launch_on = [&](hipStream_t st) {
        hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, st);
        return hip_ok(hipGetLastError(), "empty launch") ? DS_OK : DS_EHIP;
    };
    auto launch = [&]() { return launch_on(stream); };
    double w[1];
    int rc = time_repeats(launch, stream, std::max(1, cfg.warmup), 1, w);
    if (rc != DS_OK) return rc;
    const int number = std::max(1, std::min(cfg.max_number,
                                            int(std::ceil(cfg.min_repeat_ms / std::max(w[0], 1e-4)))));
    if (cfg.graph) rc = time_graph(launch_on, stream, number, cfg.repeat, out->repeats_ms);
    else rc = time_repeats(launch, stream, number, cfg.repeat, out->repeats_ms);
    if (rc != DS_OK) return rc;
    out->number = number;
    summarise(out, cfg.repeat);
    return DS_OK;
}

int ds_mfma_ceiling(hipStream_t stream, float *sink, int64_t sink_elems, int iters,
                    const ds_measure_cfg *cfg_in, ds_measurement *out, double *flop) {
    if (!sink || !out || !flop || iters < 1) {
        set_error("bad ds_mfma_ceiling arguments");
        return DS_EINVAL;
    }
    if (sink_elems < DS_MFMA_CEILING_SINK) {
        set_error("ds_mfma_ceiling needs a sink of %lld floats, got %lld",
                  (long long)DS_MFMA_CEILING_SINK, (long long)sink_elems);
        return DS_EINVAL;
    }
    std::memset(out, 0, sizeof *out);
    ds_measure_cfg cfg;
    if (cfg_in) cfg = *cfg_in;
    else ds_measure_cfg_default(&cfg);
    cfg.repeat = std::max(1, std::min(cfg.repeat, DS_MAX_REPEATS));
    // four waves on each of the 1024 SIMDs of a 256-CU part
    const int blocks = int(DS_MFMA_CEILING_SINK / 256);
    *flop = double(blocks) * 4 * iters * kCeilBlocks * 2048.0;
    auto launch_on = [&](hipStream_t st) {
        hipLaunchKernelGGL(mfma_ceiling_kernel, dim3(blocks), dim3(256), 0, st, sink, iters);
        return hip_ok(hipGetLastError(), "mfma ceiling launch") ? DS_OK : DS_EHIP;
    };
    auto launch = [&]() { return launch_on(stream); };
    double w[1];
    int rc = time_repeats(launch, stream, std::max(1, cfg.warmup), 1, w);
    if (rc != DS_OK) return rc;
    rc = time_repeats(launch, stream, 1, cfg.repeat, out->repeats_ms);
    if (rc != DS_OK) return rc;
    out->number = 1;
    summarise(out, cfg.repeat);
    return DS_OK;
}

int droplet_tune(int op, const int64_t *shape, const ds_sched *start, int budget, ds_sched *best,
                 double *best_ms) {
    if (!shape || !best || !best_ms || budget < 0) {
        set_error("bad droplet_tune arguments");
        return DS_EINVAL;
    }
    ds_space *space = nullptr;
    int rc = sched_space_create(op, shape, op == DS_OP_CONV2D_NCHW ? 9 : 3, &space);
    if (rc != DS_OK) return rc;
    Space sp;
    build_space(op, shape, op == DS_OP_CONV2D_NCHW ? 9 : 3, sp);
    int64_t nx, nw, ny;
    if (op == DS_OP_CONV2D_NCHW) {
        const int64_t P = conv_out_dim(sp.shape[2], sp.shape[5], sp.shape[7], sp.shape[8]);
        const int64_t Q = conv_out_dim(sp.shape[3], sp.shape[6], sp.shape[7], sp.shape[8]);
        nx = sp.shape[0] * sp.shape[1] * sp.shape[2] * sp.shape[3];
        nw = sp.shape[4] * sp.shape[1] * sp.shape[5] * sp.shape[6];
        ny = sp.shape[0] * sp.shape[4] * P * Q;
    } else {
        nx = sp.shape[0] * sp.shape[2];
        nw = sp.shape[2] * sp.shape[1];
        ny = sp.shape[0] * sp.shape[1];
    }
    const uint64_t base = 240620037ull;
    std::vector<float> hx(size_t(std::max<int64_t>(nx, 1))), hw(size_t(std::max<int64_t>(nw, 1)));
    ds_gen_uniform(base, nx, hx.data());
    ds_gen_uniform(op == DS_OP_CONV2D_NCHW ? base + 1 : base + 2, nw, hw.data());
    void *dx = nullptr, *dw = nullptr, *dy = nullptr;
    rc = DS_OK;
    if (!hip_ok(hipMalloc(&dx, size_t(std::max<int64_t>(nx, 1)) * 4), "hipMalloc(x)") ||
        !hip_ok(hipMalloc(&dw, size_t(std::max<int64_t>(nw, 1)) * 4), "hipMalloc(w)") ||
        !hip_ok(hipMalloc(&dy, size_t(std::max<int64_t>(ny, 1)) * 4), "hipMalloc(y)"))
        rc = DS_ENOMEM;
    if (rc == DS_OK &&
        (!hip_ok(hipMemcpy(dx, hx.data(), size_t(nx) * 4, hipMemcpyHostToDevice), "copy x") ||
         !hip_ok(hipMemcpy(dw, hw.data(), size_t(nw) * 4, hipMemcpyHostToDevice), "copy w")))
        rc = DS_EHIP;
    if (rc == DS_OK) {
        ds_tune_cfg cfg;
        ds_tune_cfg_default(&cfg);
        ds_tune_io io = {static_cast<float *>(dx), static_cast<float *>(dw),
                         static_cast<float *>(dy), nullptr, nullptr};
        ds_tune_result res;
        rc = droplet_tune_ex(space, start, budget, &cfg, &io, nullptr, nullptr, &res, nullptr);
        if (rc == DS_OK) {
            *best = res.best;
            *best_ms = res.best_ms;
        }
    }
    free_device(dx);
    free_device(dw);
    free_device(dy);
    sched_space_destroy(space);
    return rc;
}

int ds_device_info(int *cus, int *clock_khz, char *arch, int arch_len) {
    int dev;
    int rc = current_device(dev);
    if (rc != DS_OK) return rc;
    hipDeviceProp_t prop;
    if (!hip_ok(hipGetDeviceProperties(&prop, dev), "hipGetDeviceProperties")) return DS_EHIP;
    if (cus) *cus = prop.multiProcessorCount;
    if (clock_khz) *clock_khz = prop.clockRate;
    if (arch && arch_len > 0) {
        std::strncpy(arch, prop.gcnArchName, size_t(arch_len) - 1);
        arch[arch_len - 1] = 0;
    }
    return DS_OK;
}

int ds_num_instances(void) { return count_instances(); }

int sched_has_kernel(const ds_space *space, const ds_sched *s) {
    const int v = sched_valid(space, s);
    if (v <= 0) return v;
    Plan plan;
    const int rc = make_plan(s, nullptr, nullptr, nullptr, plan);
    if (rc == DS_OK) return 1;
    return rc == DS_EUNSUPPORTED ? 0 : rc;
}

int sched_kernel_info(const ds_space *space, const ds_sched *s, int with_attrs,
                      ds_kernel_info *out) {
    if (!out) {
        set_error("out is null");
        return DS_EINVAL;
    }
    std::memset(out, 0, sizeof *out);
    const int v = sched_valid(space, s);
    if (v < 0) return v;
    if (v == 0) {
        set_error("schedule is not a valid point of its search space");
        return DS_EINVALID_SCHED;
    }
    Plan plan;
    int rc = make_plan(s, nullptr, nullptr, nullptr, plan);
    if (rc != DS_OK) return rc;
    out->family = plan.family;
    out->nparams = plan.nparams;
    for (int i = 0; i < 6; ++i) out->params[i] = plan.params[i];
    out->instance = plan.family * 4096 + plan.slot;
    out->threads = plan.threads;
    out->grid = plan.grid;
    out->lds_bytes = plan.lds;
    out->splits = plan.splits;
    // FNV-1a over the kernel's argument block (buffer pointers are null here)
    const unsigned char *b = plan.family == DS_KERNEL_CONV_MFMA2
                                 ? reinterpret_cast<const unsigned char *>(&plan.conv2)
                             : plan.op == DS_OP_CONV2D_NCHW
                                 ? reinterpret_cast<const unsigned char *>(&plan.conv)
                                 : reinterpret_cast<const unsigned char *>(&plan.mm);
    const size_t nb = plan.family == DS_KERNEL_CONV_MFMA2 ? sizeof plan.conv2
                      : plan.op == DS_OP_CONV2D_NCHW     ? sizeof plan.conv
                                                         : sizeof plan.mm;
    uint64_t h = 1469598103934665603ull;
    for (size_t i = 0; i < nb; ++i) h = (h ^ b[i]) * 1099511628211ull;
    out->args_hash = h;
    if (with_attrs) {
        hipFuncAttributes fa;
        if (!hip_ok(hipFuncGetAttributes(&fa, plan.func), "hipFuncGetAttributes")) return DS_EHIP;
        out->num_regs = fa.numRegs;
        out->max_threads_per_block = fa.maxThreadsPerBlock;
        out->local_bytes = int64_t(fa.localSizeBytes);
        out->static_lds_bytes = int64_t(fa.sharedSizeBytes);
    }
    return DS_OK;
}

int sched_space_programs(const ds_space *space, uint64_t *keys, int32_t *instances,
                         uint64_t *args_hashes, int64_t cap, int64_t *n_out) {
    if (!space || !n_out || cap < 0 || (cap > 0 && (!keys || !instances || !args_hashes))) {
        set_error("bad arguments");
        return DS_EINVAL;
    }
    const Space &sp = space_of(space);
    if (sp.op != DS_OP_CONV2D_NCHW && sp.op != DS_OP_MATMUL_RM) {
        set_error("a generic lattice has no kernel");
        return DS_EINVAL;
    }
    int64_t n = 0;
    int32_t idx[DS_MAX_KNOBS] = {0};
    for (uint64_t k = 0; k < sp.size; ++k) {
        sp.from_key(k, idx);
        if (!sp.geometry(idx).valid) continue;
        if (n < cap) {
            const ds_sched s = make_sched(sp, idx);
            ds_kernel_info info;
            const int rc = sched_kernel_info(space, &s, 0, &info);
            if (rc != DS_OK) return rc;
            keys[n] = k;
            instances[n] = info.instance;
            args_hashes[n] = info.args_hash;
        }
        ++n;
    }
    *n_out = n;
    return DS_OK;
}

void ds_shutdown(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return;
    for (int d = 0; d < kMaxDevices; ++d) {
        bool ws = false;
        for (auto &e : g_split_ws) ws = ws || e.first.first == d;
        for (auto &e : g_split_retired) ws = ws || e.first == d;
        if (!g_parity_buf[d] && !g_graph_stream[d] && !ws) continue;
        if (hipSetDevice(d) == hipSuccess) {
            (void)hipDeviceSynchronize();
            if (g_parity_buf[d]) (void)hipFree(g_parity_buf[d]);
            if (g_graph_stream[d]) (void)hipStreamDestroy(g_graph_stream[d]);
            for (auto &e : g_split_ws)
                if (e.first.first == d && e.second.p) (void)hipFree(e.second.p);
            for (auto &e : g_split_retired)
                if (e.first == d) (void)hipFree(e.second);
        }
        g_parity_buf[d] = nullptr;
        g_graph_stream[d] = nullptr;
    }
    g_split_ws.clear();
    g_split_retired.clear();
    (void)hipSetDevice(cur);
    g_lds_attr.clear();
}

}  // extern "C"
