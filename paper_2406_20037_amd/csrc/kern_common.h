// Device-side helpers shared by the kernel families (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>

#include "ds_internal.h"

namespace ds {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

// Workgroups are dispatched to the 8 XCDs of the chip round-robin by
// workgroup id.  Renumber them so that each XCD receives one contiguous range
// of tiles: neighbouring tiles share operands, and each XCD has its own L2.
__device__ __forceinline__ int xcd_tile(int b, int nwg) {
    const int q = nwg >> 3, r = nwg & 7;
    const int x = b & 7, j = b >> 3;
    return x * q + (x < r ? x : r) + j;
}

// Output store with the non-temporal hint.  The matmul's 32x32-block epilogue
// uses it: no kernel reads its own outputs back, and for whole 128-byte row
// segments it shortens the time from one launch to the next by 1-2% (measured
// at 1024^3).  Partly coalesced stores (the convolutions', 64-byte segments)
// run slower or write more with it and store normally.
__device__ __forceinline__ void store_out(float *p, float v) { __builtin_nontemporal_store(v, p); }

// Instance table sizes (one slot per template-parameter tuple).
constexpr int kConvValuSlots = 7 * 5 * 5 * 2;   // KPT, PPT, UF, LDS
constexpr int kConvMfmaSlots = 3 * 7 * 3 * 2;   // TKB, NPB, D, LDS
constexpr int kConvMfma2Slots = 3 * 6 * 3 * 3 * 2;  // TKB, NPB, U, KG, RC
constexpr int kMmValuSlots = 5 * 5 * 5 * 7 * 2; // RM, RN, BK, UF, DB
constexpr int kMmMfmaSlots = 4 * 4 * 5 * 7 * 2 * 2; // WM, WN, BK, UF, DB, KG

constexpr int ilog2(int v) { return v <= 1 ? 0 : 1 + ilog2(v / 2); }
constexpr int cmin(int a, int b) { return a < b ? a : b; }
constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int p2floor(int v) { return v < 2 ? 1 : 2 * p2floor(v / 2); }

// Unroll factors the lattice can produce for a reduction loop of `body`
// accumulator updates per step: conv caps at 16 steps (runtime trip count);
// matmul unrolls up to its compile-time trip count.
constexpr bool conv_uf_reachable(int body, int uf) {
    if (uf == 1) return true;
    const int us[3] = {16, 64, 512};
    for (int u : us)
        if (cmin(16, p2floor(cmax(1, u / body))) == uf) return true;
    return false;
}

// Read-ahead depth of the MFMA conv's group loop for an unroll factor u of
// conv_uf (1..16): 1 below 4, 2 below 16, 3 at 16.
constexpr int conv_mfma_depth(int u) { return u >= 16 ? 3 : (u >= 4 ? 2 : 1); }

// Depths the lattice can produce for TKB x NPB blocks, and that fit: the
// D+1 operand sets (4 TKB + 4 NPB floats each) stay within 96 registers.
constexpr bool conv_mfma_depth_ok(int tkb, int npb, int d) {
    if ((d + 1) * 4 * (tkb + npb) > 96) return d == 1;
    const int body = tkb * npb;
    if (d == 1) return true;
    const int us[3] = {16, 64, 512};
    for (int u : us)
        if (conv_mfma_depth(cmin(16, p2floor(cmax(1, u / body)))) == d) return true;
    return false;
}

constexpr bool mm_uf_reachable(int trip, int body, int uf) {
    if (uf == 1) return true;
    const int us[3] = {16, 64, 512};
    for (int u : us) {
        const int e = trip * body <= u ? trip : cmin(trip, p2floor(cmax(1, u / body)));
        if (e == uf) return true;
    }
    return false;
}

}  // namespace ds
