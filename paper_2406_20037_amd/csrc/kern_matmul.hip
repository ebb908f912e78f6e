// Row-major fp32 matmul kernel family for gfx950: C[M,N] = A[M,K] * B[K,N].
//
// A workgroup of 256 threads computes a BM x BN tile of C over the K-tiles of
// its split.  Each K-tile (BK deep) is staged through LDS:
//   As[BM][BK]  k contiguous in 16-byte slots; slot j of row r is stored at
//               j ^ swz(r), so the 16-byte reads of eight consecutive rows at
//               one k land on distinct banks without padding,
//   Bs[BK][BN]  n contiguous.
// When every tile is full and the operands are 16-byte aligned (a.direct), the
// K-tiles travel straight from global memory into LDS (global_load_lds, no
// register staging); with dbuf the next ST-1 K-tiles are in flight while the
// current one is consumed (ST = 3 stages when they fit in LDS, else 2).
// Otherwise tiles are staged through registers with bounds checks (zero
// outside A and B) and, with dbuf, written to the other LDS stage after the
// current one is consumed.
//
//   mm_valu: VALU FMA; thread (ty, tx) of a 16x16 grid owns RM rows x RN
//            columns (contiguous).
//   mm_mfma: KG groups of 2x2 waves; each wave a WM x WN tile of fp32 MFMA
//            blocks (v_mfma_f32_32x32x2f32 when WM, WN >= 32, else
//            v_mfma_f32_16x16x4f32).  Group g consumes the g-th of KG equal
//            k ranges of every K-tile; the groups' accumulators are summed
//            through LDS at the end (two waves per SIMD hide each other's
//            waits).  Lane group g feeds k = kk + VEC*g + v (v < VEC) to both
//            operands, so one VEC-wide LDS read of A serves VEC MFMA steps.
// A split (ks > 1) stores its partial C tile; a reduce kernel sums the splits
// into C in split order.
#include <utility>

#include "kern_common.h"

namespace ds {

namespace {

#define DS_GLOBAL(p) ((const __attribute__((address_space(1))) void *)(p))
#define DS_LOCAL(p) ((__attribute__((address_space(3))) void *)(p))

// Tiles in groups of a.gm tile rows (chosen on the host: the XCD's range of
// tiles square in elements), column-major inside a group, so the contiguous
// tile range of one XCD touches few rows of A and columns of B.
__device__ __forceinline__ void mm_tile_coords(const MatmulArgs &a, int &mt, int &nt, int &z) {
    const int tiles = a.tiles_m * a.tiles_n;
    const int t = xcd_tile(blockIdx.x, gridDim.x);
    z = t / tiles;
    const int r = t - z * tiles;
    const int gm = a.gm;
    const int gsz = gm * a.tiles_n;
    const int g = r / gsz, first = g * gm;
    const int rows = min(a.tiles_m - first, gm);
    const int rg = r - g * gsz;
    mt = first + rg % rows;
    nt = rg / rows;
}

// Lane exchange inside quads of lanes (DPP quad_perm).
template <int CTRL>
__device__ __forceinline__ float quad_perm(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}

// 4x4 transpose across the four lanes of a quad: lane b's x[j] becomes lane
// j's x[b].  Two rounds of 2x2 swaps: lanes b, b^1 on register pairs (0,1),
// (2,3), then lanes b, b^2 on pairs (0,2), (1,3).
__device__ __forceinline__ void quad_transpose(float (&x)[4], int b) {
    const bool o1 = b & 1, o2 = b & 2;
#pragma unroll
    for (int p = 0; p < 4; p += 2) {
        const float r = quad_perm<0xB1>(o1 ? x[p] : x[p + 1]);   // lanes [1,0,3,2]
        x[p] = o1 ? r : x[p];
        x[p + 1] = o1 ? x[p + 1] : r;
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const float r = quad_perm<0x4E>(o2 ? x[p] : x[p + 2]);   // lanes [2,3,0,1]
        x[p] = o2 ? r : x[p];
        x[p + 2] = o2 ? x[p + 2] : r;
    }
}

// Slot permutation of A row r (BK/4 slots per row).
template <int BK>
__device__ __forceinline__ int a_swz(int r) {
    constexpr int SPR = BK / 4;
    if constexpr (SPR >= 8) return r & 7;
    else return ((r * SPR) >> 3) & (SPR - 1);
}

// Float offset of A element (row, k) inside a stage.
template <int BK>
__device__ __forceinline__ int a_off(int row, int k) {
    return row * BK + (((k >> 2) ^ a_swz<BK>(row)) << 2) + (k & 3);
}

// Waits for every vector-memory operation of the wave, then for LDS, then
// barriers the workgroup without a memory fence (the waits above make the LDS
// writes of every wave complete before any wave passes).
// s_waitcnt immediate for vmcnt(n) (expcnt, lgkmcnt not waited on).
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | 0x70 | 0xF00; }

template <int VM = 0>
__device__ __forceinline__ void stage_barrier() {
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(VM));
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Global -> LDS copy of one full, aligned K-tile (16 bytes per lane per
// instruction; the LDS destination of a wave's instruction is contiguous).
template <int BM, int BN, int BK, int NT>
__device__ __forceinline__ void direct_load(const MatmulArgs &a, int m0, int n0, int kt, float *As,
                                            float *Bs) {
    constexpr int SPR = BK / 4, A4 = BM * SPR, B4 = BK * BN / 4;
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < (A4 + NT - 1) / NT; ++j) {
        const int base = j * NT + wid * 64;
        const int c = base + lane;
        if (A4 % NT == 0 || c < A4) {
            const int row = c / SPR, slot = c % SPR;
            const float *src = a.A + (size_t)(m0 + row) * a.K + kt * BK + 4 * (slot ^ a_swz<BK>(row));
            __builtin_amdgcn_global_load_lds(DS_GLOBAL(src), DS_LOCAL(As + base * 4), 16, 0, 0);
        }
    }
#pragma unroll
    for (int j = 0; j < (B4 + NT - 1) / NT; ++j) {
        const int base = j * NT + wid * 64;
        const int c = base + lane;
        if (B4 % NT == 0 || c < B4) {
            const int k = c / (BN / 4), n4 = c % (BN / 4);
            const float *src = a.B + (size_t)(kt * BK + k) * a.N + n0 + 4 * n4;
            __builtin_amdgcn_global_load_lds(DS_GLOBAL(src), DS_LOCAL(Bs + base * 4), 16, 0, 0);
        }
    }
}

// Global -> register staging of one K-tile (float4 slots; zero outside A, B).
template <int BM, int BN, int BK, int NT>
struct Stager {
    static constexpr int A4 = BM * BK / 4, B4 = BK * BN / 4;
    static constexpr int AL = (A4 + NT - 1) / NT, BL = (B4 + NT - 1) / NT;
    floatx4 ra[AL], rb[BL];

    __device__ __forceinline__ void load(const MatmulArgs &a, int m0, int n0, int kt) {
        const int tid = threadIdx.x;
#pragma unroll
        for (int u = 0; u < AL; ++u) {
            const int e = tid + NT * u;
            floatx4 v = {0.f, 0.f, 0.f, 0.f};
            if (A4 % NT == 0 || e < A4) {
                const int m = e / (BK / 4), k4 = e - m * (BK / 4);
                const int gm = m0 + m, gk = kt * BK + 4 * k4;
                if (gm < a.M) {
                    const float *src = a.A + (size_t)gm * a.K + gk;
                    if (a.vecA && gk + 3 < a.K) {
                        v = *reinterpret_cast<const floatx4 *>(src);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (gk + i < a.K) v[i] = src[i];
                    }
                }
            }
            ra[u] = v;
        }
#pragma unroll
        for (int u = 0; u < BL; ++u) {
            const int e = tid + NT * u;
            floatx4 v = {0.f, 0.f, 0.f, 0.f};
            if (B4 % NT == 0 || e < B4) {
                const int k = e / (BN / 4), n4 = e - k * (BN / 4);
                const int gk = kt * BK + k, gn = n0 + 4 * n4;
                if (gk < a.K) {
                    const float *src = a.B + (size_t)gk * a.N + gn;
                    if (a.vecB && gn + 3 < a.N) {
                        v = *reinterpret_cast<const floatx4 *>(src);
                    } else {
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (gn + i < a.N) v[i] = src[i];
                    }
                }
            }
            rb[u] = v;
        }
    }

    __device__ __forceinline__ void store(float *As, float *Bs) const {
        const int tid = threadIdx.x;
#pragma unroll
        for (int u = 0; u < AL; ++u) {
            const int e = tid + NT * u;
            if (A4 % NT == 0 || e < A4) {
                const int m = e / (BK / 4), k4 = e - m * (BK / 4);
                *reinterpret_cast<floatx4 *>(As + a_off<BK>(m, 4 * k4)) = ra[u];
            }
        }
#pragma unroll
        for (int u = 0; u < BL; ++u) {
            const int e = tid + NT * u;
            if (B4 % NT == 0 || e < B4) {
                const int k = e / (BN / 4), n4 = e - k * (BN / 4);
                *reinterpret_cast<floatx4 *>(Bs + k * BN + 4 * n4) = rb[u];
            }
        }
    }
};

// The K-loop shared by both families: stages K-tiles [kt0, kt1) through LDS
// and calls compute(As, Bs) on each.  NT threads; ST LDS stages (1: stage,
// barrier, compute; >= 2: the next tiles are in flight during compute).
template <int BM, int BN, int BK, int ST, int NT, class F>
__device__ __forceinline__ void k_loop(const MatmulArgs &a, int m0, int n0, int kt0, int kt1,
                                       float *smem, F &&compute) {
    constexpr int STAGE = BM * BK + BK * BN;
    if (a.direct) {
        if constexpr (ST >= 2) {
            // Each thread issues the same L copies per tile when the tile
            // divides into whole rounds of NT threads; then waiting until at
            // most L*(ST-2) copies are outstanding means tile kt has landed.
            constexpr int A4 = BM * BK / 4, B4 = BK * BN / 4;
            constexpr bool EXACT = A4 % NT == 0 && B4 % NT == 0;
            constexpr int L = A4 / NT + B4 / NT;
#pragma unroll
            for (int p = 0; p < ST - 1; ++p)
                if (kt0 + p < kt1)
                    direct_load<BM, BN, BK, NT>(a, m0, n0, kt0 + p, smem + p * STAGE,
                                                smem + p * STAGE + BM * BK);
            int s = 0;
            for (int kt = kt0; kt < kt1; ++kt) {
                if (EXACT && ST > 2 && kt + ST - 2 < kt1) stage_barrier<EXACT ? L * (ST - 2) : 0>();
                else stage_barrier<0>();
                if (kt + ST - 1 < kt1) {
                    int sn = s + ST - 1;
                    if (sn >= ST) sn -= ST;
                    float *nx = smem + sn * STAGE;
                    direct_load<BM, BN, BK, NT>(a, m0, n0, kt + ST - 1, nx, nx + BM * BK);
                }
                compute(smem + s * STAGE, smem + s * STAGE + BM * BK);
                if (++s == ST) s = 0;
            }
        } else {
            for (int kt = kt0; kt < kt1; ++kt) {
                stage_barrier();
                direct_load<BM, BN, BK, NT>(a, m0, n0, kt, smem, smem + BM * BK);
                stage_barrier();
                compute(smem, smem + BM * BK);
            }
        }
        return;
    }
    Stager<BM, BN, BK, NT> st;
    if constexpr (ST >= 2) {
        st.load(a, m0, n0, kt0);
        st.store(smem, smem + BM * BK);
        __syncthreads();
        for (int kt = kt0; kt < kt1; ++kt) {
            const int s = (kt - kt0) & 1;
            const bool more = kt + 1 < kt1;
            if (more) st.load(a, m0, n0, kt + 1);
            compute(smem + s * STAGE, smem + s * STAGE + BM * BK);
            if (more) st.store(smem + (s ^ 1) * STAGE, smem + (s ^ 1) * STAGE + BM * BK);
            __syncthreads();
        }
    } else {
        for (int kt = kt0; kt < kt1; ++kt) {
            st.load(a, m0, n0, kt);
            __syncthreads();
            st.store(smem, smem + BM * BK);
            __syncthreads();
            compute(smem, smem + BM * BK);
        }
    }
}

template <int RM, int RN, int BK, int UF, int DB>
__global__ __launch_bounds__(256) void mm_valu(MatmulArgs a) {
    constexpr int BM = 16 * RM, BN = 16 * RN;
    constexpr int ST = mm_stages(BM, BN, BK, DB);
    constexpr int U4 = UF >= 4 ? UF / 4 : 1;
    extern __shared__ float smem[];
    int mt, nt, z;
    mm_tile_coords(a, mt, nt, z);
    const int kt0 = z * a.kps, kt1 = min(kt0 + a.kps, a.nkt);
    if (kt0 >= kt1) return;
    const int m0 = mt * BM, n0 = nt * BN;
    const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;

    float acc[RM][RN];
#pragma unroll
    for (int i = 0; i < RM; ++i)
#pragma unroll
        for (int j = 0; j < RN; ++j) acc[i][j] = 0.f;

    auto compute = [&](const float *As, const float *Bs) {
#pragma unroll U4
        for (int kk = 0; kk < BK; kk += 4) {
            floatx4 av[RM];
#pragma unroll
            for (int i = 0; i < RM; ++i)
                av[i] = *reinterpret_cast<const floatx4 *>(As + a_off<BK>(ty * RM + i, kk));
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float bv[RN];
                const float *brow = Bs + (kk + v) * BN + tx * RN;
                if constexpr (RN >= 4) {
#pragma unroll
                    for (int j = 0; j < RN; j += 4) {
                        const floatx4 b4 = *reinterpret_cast<const floatx4 *>(brow + j);
                        bv[j] = b4[0];
                        bv[j + 1] = b4[1];
                        bv[j + 2] = b4[2];
                        bv[j + 3] = b4[3];
                    }
                } else {
#pragma unroll
                    for (int j = 0; j < RN; ++j) bv[j] = brow[j];
                }
#pragma unroll
                for (int i = 0; i < RM; ++i)
#pragma unroll
                    for (int j = 0; j < RN; ++j) acc[i][j] = fmaf(av[i][v], bv[j], acc[i][j]);
            }
        }
    };
    k_loop<BM, BN, BK, ST, 256>(a, m0, n0, kt0, kt1, smem, compute);

    float *cbase = a.ks > 1 ? a.part + (size_t)z * a.M * a.N : a.C;
#pragma unroll
    for (int i = 0; i < RM; ++i) {
        const int gm = m0 + ty * RM + i;
        if (gm >= a.M) continue;
        float *crow = cbase + (size_t)gm * a.N;
#pragma unroll
        for (int j = 0; j < RN; ++j) {
            const int gn = n0 + tx * RN + j;
            if (gn < a.N) crow[gn] = acc[i][j];
        }
    }
}

// Geometry of one wave group's MFMA work on a K-tile.
template <int WM, int WN, int BK, int KG>
struct MfmaShape {
    static constexpr bool BIG = WM >= 32 && WN >= 32;
    static constexpr int IM = BIG ? 32 : 16;          // MFMA output tile edge
    static constexpr int NG = 64 / IM;                // lane groups along k
    static constexpr int KR = BK / KG;                // k of every K-tile per wave group
    static constexpr int VEC = cmin(4, KR / NG);      // k values per lane per LDS read
    static constexpr int KGS = NG * VEC;              // k consumed per chunk
    static constexpr int NCH = KR / KGS;              // chunks per K-tile
    static constexpr int MB = WM / IM, NB = WN / IM;
    static constexpr int NV = BIG ? 16 : 4;           // accumulator values per lane
};

// Whether the direct path runs software-pipelined (mm_mfma_pipe): at least
// two stages, every thread issuing the same number of copies per K-tile, and
// at least two chunks per K-tile.
template <int WM, int WN, int BK, int DB, int KG>
constexpr bool mm_pipelined() {
    using S = MfmaShape<WM, WN, BK, KG>;
    constexpr int BM = 2 * WM, BN = 2 * WN, NT = 256 * KG;
    return mm_stages(BM, BN, BK, DB) >= 2 && (BM * BK / 4) % NT == 0 && (BK * BN / 4) % NT == 0 &&
           S::NCH >= 2;
}

// Direct (global -> LDS) K-loop with the LDS operand reads software-pipelined
// across MFMA chunks.  A chunk is one k step of every MFMA block of the wave
// (KGS k values).  The operands of chunk c + D are read while the MFMAs of
// chunk c run, from a ring of D + 1 operand sets (D = 3 with unroll >= 16 when
// the chunks of a K-tile divide into whole rings, else 1).  The stage barrier
// sits before the last D chunks of every K-tile: past it every wave has
// finished reading the current tile and the next tile has landed, so the next
// tile's first reads overlap the current tile's last MFMAs, and the stage of
// the tile just consumed is refilled in the next iteration.  Each K-tile's
// copies are spread over the chunks before the barrier.  Past the end of the
// split the last K-tile is loaded again into a stage nobody reads, so every
// iteration has the same copies in flight and the wait counts are constants.
template <int WM, int WN, int BK, int UF, int DB, int KG, class Acc, int MB, int NB>
__device__ __forceinline__ void mm_mfma_pipe(const MatmulArgs &a, int m0, int n0, int kt0, int kt1,
                                             float *smem, Acc (&acc)[MB][NB]) {
    using S = MfmaShape<WM, WN, BK, KG>;
    constexpr int BM = 2 * WM, BN = 2 * WN, NT = 256 * KG;
    constexpr int ST = mm_stages(BM, BN, BK, DB);
    constexpr int STAGE = BM * BK + BK * BN;
    constexpr int SPR = BK / 4, A4 = BM * SPR, B4 = BK * BN / 4;
    constexpr int AL = A4 / NT, BL = B4 / NT, L = AL + BL;
    constexpr int IM = S::IM, VEC = S::VEC, KGS = S::KGS, NCH = S::NCH;
    constexpr int D = UF >= 16 && NCH % 4 == 0 ? 3 : 1;
    constexpr int RG = D + 1;
    constexpr bool RING = NCH % RG == 0;   // chunk c always uses ring slot c % RG
    constexpr int PRE = NCH - D;           // chunks before the stage barrier
    constexpr int PER = (L + PRE - 1) / PRE;
    static_assert(PRE >= 1, "the copies of a tile are issued before its barrier");

    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int wsc = __builtin_amdgcn_readfirstlane(wid);
    const int kg = wid >> 2, wq = wid & 3;
    const int wr = wq >> 1, wc = wq & 1;
    const int li = lane % IM, lg = lane / IM;

    // per-thread sources of K-tile 0; a tile adds kt*BK (A) or kt*BK*N (B)
    const float *pa[AL], *pb[BL];
#pragma unroll
    for (int j = 0; j < AL; ++j) {
        const int c = j * NT + wid * 64 + lane;
        const int row = c / SPR, slot = c % SPR;
        pa[j] = a.A + (size_t)(m0 + row) * a.K + 4 * (slot ^ a_swz<BK>(row));
    }
#pragma unroll
    for (int j = 0; j < BL; ++j) {
        const int c = j * NT + wid * 64 + lane;
        const int k = c / (BN / 4), n4 = c % (BN / 4);
        pb[j] = a.B + (size_t)k * a.N + n0 + 4 * n4;
    }
    // copy j of K-tile kt into the stage at st (the LDS slot is wave-uniform)
    auto copy = [&](int kt, float *st, int j) {
        if (j < AL) {
            __builtin_amdgcn_global_load_lds(DS_GLOBAL(pa[j] + (size_t)kt * BK),
                                             DS_LOCAL(st + (j * NT + wsc * 64) * 4), 16, 0, 0);
        } else {
            const int jb = j - AL;
            __builtin_amdgcn_global_load_lds(DS_GLOBAL(pb[jb] + (size_t)kt * BK * a.N),
                                             DS_LOCAL(st + BM * BK + (jb * NT + wsc * 64) * 4), 16,
                                             0, 0);
        }
    };

    struct Ops {
        float a[MB][VEC];
        float b[VEC][NB];
    };
    const int arow = wr * WM + li;
    const int bcol = BM * BK + wc * WN + li;
    auto read = [&](const float *st, int c, Ops &o) {
        const int k = kg * S::KR + c * KGS + VEC * lg;
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            const float *src = st + a_off<BK>(arow + i * IM, k);
            if constexpr (VEC == 4) {
                const floatx4 t = *reinterpret_cast<const floatx4 *>(src);
                o.a[i][0] = t[0];
                o.a[i][1] = t[1];
                o.a[i][2] = t[2];
                o.a[i][3] = t[3];
            } else if constexpr (VEC == 2) {
                const float2 t = *reinterpret_cast<const float2 *>(src);
                o.a[i][0] = t.x;
                o.a[i][1] = t.y;
            } else {
                o.a[i][0] = src[0];
            }
        }
#pragma unroll
        for (int v = 0; v < VEC; ++v)
#pragma unroll
            for (int j = 0; j < NB; ++j) o.b[v][j] = st[bcol + (k + v) * BN + j * IM];
    };
    auto mma = [&](const Ops &o) {
#pragma unroll
        for (int v = 0; v < VEC; ++v)
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    if constexpr (S::BIG)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(o.a[i][v], o.b[v][j],
                                                                        acc[i][j], 0, 0, 0);
                    else
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[i][v], o.b[v][j],
                                                                        acc[i][j], 0, 0, 0);
                }
    };
    // one LDS read between consecutive MFMAs of a chunk
    auto interleave = [&]() {
        constexpr int NM = VEC * MB * NB, NDS = MB + (VEC * NB + 1) / 2;
#pragma unroll
        for (int t = 0; t < NM; ++t) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (t < NDS && t + 1 < NM) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
    };

    // prologue: K-tiles kt0 .. kt0+ST-2, then wait for the first
#pragma unroll
    for (int p = 0; p < ST - 1; ++p)
#pragma unroll
        for (int j = 0; j < L; ++j) copy(min(kt0 + p, kt1 - 1), smem + p * STAGE, j);
    stage_barrier<L * (ST - 2)>();
    Ops o[RG];
#pragma unroll
    for (int c = 0; c < D; ++c) read(smem, c, o[c]);

    int s = 0;
    for (int kt = kt0; kt < kt1; ++kt) {
        int sp = s + ST - 1;
        if (sp >= ST) sp -= ST;
        int sn = s + 1;
        if (sn == ST) sn = 0;
        const float *cur = smem + s * STAGE, *nxt = smem + sn * STAGE;
        float *fill = smem + sp * STAGE;
        const int ktf = min(kt + ST - 1, kt1 - 1);
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            if (c == PRE) stage_barrier<L * (ST - 2)>();
            Ops &rd = RING ? o[(c + D) % RG] : o[D];
            if (c + D < NCH) read(cur, c + D, rd);
            else read(nxt, c + D - NCH, rd);
            mma(RING ? o[c % RG] : o[0]);
            if (c < PRE) {
#pragma unroll
                for (int q = 0; q < PER; ++q)
                    if (c * PER + q < L) copy(ktf, fill, c * PER + q);
            }
            interleave();
            if constexpr (!RING) {
#pragma unroll
                for (int r = 0; r < D; ++r) o[r] = o[r + 1];
            }
        }
        s = sn;
    }
    // the reloads past the end are still in flight
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
}

template <int WM, int WN, int BK, int UF, int DB, int KG>
__global__ __launch_bounds__(256 * KG) void mm_mfma(MatmulArgs a) {
    constexpr int BM = 2 * WM, BN = 2 * WN;
    constexpr int ST = mm_stages(BM, BN, BK, DB);
    constexpr int KR = BK / KG;                // k of every K-tile per wave group
    constexpr bool BIG = WM >= 32 && WN >= 32;
    constexpr int IM = BIG ? 32 : 16;          // MFMA output tile edge
    constexpr int NG = 64 / IM;                // lane groups along k
    static_assert(KR >= NG, "every wave group needs one k step per lane group");
    constexpr int VEC = cmin(4, KR / NG);      // k values per lane per LDS read
    constexpr int KGS = NG * VEC;              // k consumed per group step
    constexpr int MB = WM / IM, NB = WN / IM;
    constexpr int KSTEP = BIG ? 2 : 4;
    constexpr int UG = cmax(1, UF * KSTEP / KGS);
    using Acc = typename std::conditional<BIG, floatx16, floatx4>::type;

    extern __shared__ float smem[];
    int mt, nt, z;
    mm_tile_coords(a, mt, nt, z);
    const int kt0 = z * a.kps, kt1 = min(kt0 + a.kps, a.nkt);
    if (kt0 >= kt1) return;
    const int m0 = mt * BM, n0 = nt * BN;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int kg = wid >> 2, wq = wid & 3;
    const int wr = wq >> 1, wc = wq & 1;
    const int li = lane % IM, lg = lane / IM;

    Acc acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) acc[i][j] = Acc{};

    auto compute = [&](const float *As, const float *Bs) {
#pragma unroll UG
        for (int kk = kg * KR; kk < (kg + 1) * KR; kk += KGS) {
            float av[MB][VEC];
#pragma unroll
            for (int i = 0; i < MB; ++i) {
                const float *src = As + a_off<BK>(wr * WM + i * IM + li, kk + VEC * lg);
                if constexpr (VEC == 4) {
                    const floatx4 t = *reinterpret_cast<const floatx4 *>(src);
                    av[i][0] = t[0];
                    av[i][1] = t[1];
                    av[i][2] = t[2];
                    av[i][3] = t[3];
                } else if constexpr (VEC == 2) {
                    const float2 t = *reinterpret_cast<const float2 *>(src);
                    av[i][0] = t.x;
                    av[i][1] = t.y;
                } else {
                    av[i][0] = src[0];
                }
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                float bv[NB];
                const float *brow = Bs + (kk + VEC * lg + v) * BN + wc * WN + li;
#pragma unroll
                for (int j = 0; j < NB; ++j) bv[j] = brow[j * IM];
#pragma unroll
                for (int i = 0; i < MB; ++i)
#pragma unroll
                    for (int j = 0; j < NB; ++j) {
                        if constexpr (BIG)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][v], bv[j],
                                                                            acc[i][j], 0, 0, 0);
                        else
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i][v], bv[j],
                                                                            acc[i][j], 0, 0, 0);
                    }
            }
        }
    };
    if constexpr (mm_pipelined<WM, WN, BK, DB, KG>()) {
        if (a.direct) mm_mfma_pipe<WM, WN, BK, UF, DB, KG>(a, m0, n0, kt0, kt1, smem, acc);
        else k_loop<BM, BN, BK, ST, 256 * KG>(a, m0, n0, kt0, kt1, smem, compute);
    } else {
        k_loop<BM, BN, BK, ST, 256 * KG>(a, m0, n0, kt0, kt1, smem, compute);
    }

    constexpr int NV = BIG ? 16 : 4;
    if constexpr (KG > 1) {
        // group 1 hands its partial tile to group 0 through LDS (16 bytes
        // per lane per access: value quad q of block b at ((b*NV/4 + q)*64 + lane)*4)
        __syncthreads();
        float *rb = smem + wq * (WM * WN);
        if (kg == 1) {
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < NB; ++j)
#pragma unroll
                    for (int q = 0; q < NV / 4; ++q)
                        *reinterpret_cast<floatx4 *>(rb + (((i * NB + j) * (NV / 4) + q) * 64 + lane) * 4) =
                            floatx4{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                    acc[i][j][4 * q + 3]};
        }
        __syncthreads();
        if (kg == 1) return;
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int j = 0; j < NB; ++j)
#pragma unroll
                for (int q = 0; q < NV / 4; ++q) {
                    const floatx4 t = *reinterpret_cast<const floatx4 *>(
                        rb + (((i * NB + j) * (NV / 4) + q) * 64 + lane) * 4);
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[i][j][4 * q + e] += t[e];
                }
    }

    // Output layout: 32x32 block, lane holds rows 8*(v/4) + 4*lg + v%4 of
    // column li (v < 16); 16x16 block, rows 4*lg + v of column li (v < 4).
    float *cbase = a.ks > 1 ? a.part + (size_t)z * a.M * a.N : a.C;
    if constexpr (!BIG && NB % 4 == 0) {
        // Four 16x16 blocks side by side: lane 4q+b holds columns 16j + 4q + b
        // (j < 4) of a row; a 4x4 transpose inside each lane quad leaves it
        // columns 16b + 4q .. +3, so every lane stores 16 contiguous bytes and
        // a row's 64 columns go out as whole 256-byte segments (non-temporal,
        // like the 32x32 blocks).  Full aligned tiles only.
        if (a.direct && (reinterpret_cast<uintptr_t>(cbase) & 15) == 0) {
            const int b = li & 3, q4 = li >> 2;
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int v = 0; v < NV; ++v) {
                    const int gm = m0 + wr * WM + i * IM + 4 * lg + v;
#pragma unroll
                    for (int jq = 0; jq < NB / 4; ++jq) {
                        float x[4] = {acc[i][4 * jq][v], acc[i][4 * jq + 1][v],
                                      acc[i][4 * jq + 2][v], acc[i][4 * jq + 3][v]};
                        quad_transpose(x, b);
                        const int gn = n0 + wc * WN + jq * 64 + 16 * b + 4 * q4;
                        __builtin_nontemporal_store(
                            floatx4{x[0], x[1], x[2], x[3]},
                            reinterpret_cast<floatx4 *>(cbase + (size_t)gm * a.N + gn));
                    }
                }
            return;
        }
    }
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int gn = n0 + wc * WN + j * IM + li;
            if (gn >= a.N) continue;
#pragma unroll
            for (int v = 0; v < NV; ++v) {
                const int row = BIG ? 8 * (v / 4) + 4 * lg + (v % 4) : 4 * lg + v;
                const int gm = m0 + wr * WM + i * IM + row;
                if (gm >= a.M) continue;
                // 32x32 blocks write whole 128-byte row segments per half-wave:
                // those go out with the non-temporal hint; the 64-byte segments of
                // 16x16 blocks stay in L2 to be merged (with the hint they cost
                // up to 1.5x the HBM writes)
                if constexpr (BIG) store_out(cbase + (size_t)gm * a.N + gn, acc[i][j][v]);
                else cbase[(size_t)gm * a.N + gn] = acc[i][j][v];
            }
        }
}

}  // namespace

extern const void *g_mm_valu[kMmValuSlots];
extern const void *g_mm_mfma[kMmMfmaSlots];

#ifndef DS_SLICE
#define DS_SLICE 0
#define DS_NSLICES 1
#endif

namespace {

constexpr int kMmBkList[5] = {4, 8, 16, 32, 64};
constexpr int kMmWaveList[4] = {16, 32, 64, 128};

// slot = (((log2 RM * 5 + log2 RN) * 5 + ibk) * 7 + log2 UF) * 2 + DB
template <int I>
void reg_mm_valu() {
    constexpr int DB = I % 2, iuf = (I / 2) % 7, ibk = (I / 14) % 5, irn = (I / 70) % 5,
                  irm = I / 350;
    constexpr int RM = 1 << irm, RN = 1 << irn, BK = kMmBkList[ibk], UF = 1 << iuf;
    constexpr int lds = mm_stages(16 * RM, 16 * RN, BK, DB) * (16 * RM * BK + BK * 16 * RN) * 4;
    if constexpr (RM * RN <= 128 && UF <= BK && lds <= kLdsLimit &&
                  mm_uf_reachable(BK, RM * RN, UF) && I % DS_NSLICES == DS_SLICE)
        g_mm_valu[I] = reinterpret_cast<const void *>(&mm_valu<RM, RN, BK, UF, DB>);
}

// slot = ((((iwm * 4 + iwn) * 5 + ibk) * 7 + log2 UF) * 2 + DB) * 2 + (KG - 1)
template <int I>
void reg_mm_mfma() {
    constexpr int KG = 1 + I % 2, DB = (I / 2) % 2, iuf = (I / 4) % 7, ibk = (I / 28) % 5,
                  iwn = (I / 140) % 4, iwm = I / 560;
    constexpr int WM = kMmWaveList[iwm], WN = kMmWaveList[iwn], BK = kMmBkList[ibk],
                  UF = 1 << iuf;
    constexpr bool BIG = WM >= 32 && WN >= 32;
    constexpr int KSTEP = BIG ? 2 : 4;
    constexpr int blocks = BIG ? (WM / 32) * (WN / 32) : (WM / 16) * (WN / 16);
    constexpr int lds = mm_stages(2 * WM, 2 * WN, BK, DB) * (2 * WM * BK + BK * 2 * WN) * 4;
    if constexpr (lds <= kLdsLimit && UF <= BK / KSTEP && mm_uf_reachable(BK / KSTEP, blocks, UF) &&
                  (KG == 1 || BK >= 8) && I % DS_NSLICES == DS_SLICE)
        g_mm_mfma[I] = reinterpret_cast<const void *>(&mm_mfma<WM, WN, BK, UF, DB, KG>);
}

template <size_t... I>
void reg_all_valu(std::index_sequence<I...>) {
    (reg_mm_valu<int(I)>(), ...);
}
// in halves: one fold over every slot would exceed the compiler's nesting limit
template <size_t Off, size_t... I>
void reg_all_mfma(std::index_sequence<I...>) {
    (reg_mm_mfma<int(Off + I)>(), ...);
}

struct Registrar {
    Registrar() {
        reg_all_valu(std::make_index_sequence<kMmValuSlots>{});
        reg_all_mfma<0>(std::make_index_sequence<kMmMfmaSlots / 2>{});
        reg_all_mfma<kMmMfmaSlots / 2>(std::make_index_sequence<kMmMfmaSlots - kMmMfmaSlots / 2>{});
    }
};
const Registrar registrar;

}  // namespace

}  // namespace ds
