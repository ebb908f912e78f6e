"""Reference schedule lattice (test infrastructure only).

Definition 1 of the paper: a sketch fixes a sequence of transformations; an
annotation assigns a value to each of its parameters; the kernel search space
of a sketch is the set of every *valid* annotation.  Section 2.2 (Example 3)
arranges those parameters as coordinates, one axis per varying parameter, and
defines the neighbours of a point as the points one step away along a single
axis.  This module is a plain restatement of the lattice the HIP library
exposes; the C++ side is written separately and must agree with it bit for
bit on every integer it produces.

The paper's rule figures (sketch, initialisation, mutation) are missing, so the
two lattices below are readings:

conv2d (op 1), shape (N, C, H, W, K, R, S, stride, pad), axes in order
    tk, th, tw, tc in {1, 2, 4, ..., 64}: output-tile extent along K, P, Q and
        the input-channel chunk of one reduction step; kept if <= K, P, Q, C
        (the smallest value is always kept), and th, tw also keep the smallest
        value >= P, Q (only band tiles, mfma 3, may reach past the output);
    unroll in {0, 16, 64, 512}: maximum unrolled steps of the reduction loop;
    lds in {0, 1}: stage input and weight tiles in LDS;
    ks in {1, 2, 4, 8, 16, 32}: reduction split over C across workgroups (kept
        if <= C);
    mfma in {0, 1, 2, 3}: contract on VALU FMA (0) or fp32 MFMA (implicit
        GEMM): 1 steps through 16-step groups of the (c, r, s) reduction, 2
        through (tap, channel quad) steps over rectangular tiles (a second MFMA
        sketch, LDS staging only), 3 the same over band tiles (the pixel loops
        fused over image, row and column before tiling);
    vec in {1, 4}: floats per lane of the global -> LDS copies (4 or 16 bytes).

matmul (op 2), shape (M, N, K), axes in order
    bm, bn in {16, 32, 64, 128, 256}: workgroup tile, kept if <= M, N;
    bk in {4, 8, 16, 32, 64}: K-step of one LDS stage, kept if <= K;
    unroll in {0, 16, 64, 512};  dbuf in {0, 1}: LDS double buffer;
    mfma in {0, 1};  ks in {1, 2, 4, 8}: split-K across workgroups (kept if <= K);
    vec in {1, 4}: floats per lane of the operand loads (4 or 16 bytes).

Validity is the hardware and register budget of the kernel family: at most
1024 threads and 163840 bytes of LDS per workgroup, an accumulator budget per
lane, register budgets of the operand rings and unrolled loops (the limits at
which the compiled instances start to spill), MFMA tile minima, a VALU conv
tile of at least one wave (64 outputs, or the largest tile of a smaller
shape), at most 2**31 - 1 workgroups, a split no finer than the number of
reduction steps, and for vec = 4 an operand that can move 16 bytes per lane.

The unroll knob is TVM's auto_unroll_max_step reading: the VALU loops and the
matmul unroll their reduction loop by the largest power of two <= unroll /
(accumulator updates per step) (capped at 16 for conv, at the trip count for
matmul); the MFMA conv turns that factor u into the read-ahead depth D of its
16-step group loop (D = 3 from u = 16, 2 from u = 4, else 1).  Unroll values
that give the same factor select the same compiled program (the saturation of
auto_unroll_max_step).

Pins: the neighbourhood reproduces Example 3 of Section 2.2
(tests/golden/droplet_example3.txt); value lists, counts and hand-computed
geometry of named points are checked in tests/test_oracle_space.py.  The
validity half (register, LDS and thread budgets) is pinned against the
compiled kernels on the GPU (tests/test_gpu_instances.py): every instance a
valid point of the five workloads can select launches bit-exact, spills
nothing, and fits its launch bound and LDS.  The paper prints no launch
geometry (grid, threads, LDS bytes, accumulators), so against the paper that
half is parity unpinned; its pins are the hand-computed points and the
compiled kernels above.
"""
from __future__ import annotations

import math

OP_CONV = 1
OP_MATMUL = 2

LDS_LIMIT = 163840
THREADS_LIMIT = 1024
GRID_LIMIT = 2 ** 31 - 1

POW2_64 = [1, 2, 4, 8, 16, 32, 64]
UNROLL = [0, 16, 64, 512]
SPLITK = [1, 2, 4, 8]
CONV_SPLIT = [1, 2, 4, 8, 16, 32]
MM_TILE = [16, 32, 64, 128, 256]
MM_BK = [4, 8, 16, 32, 64]

VEC = [1, 4]

CONV_AXES = ["tk", "th", "tw", "tc", "unroll", "lds", "ks", "mfma", "vec"]
MM_AXES = ["bm", "bn", "bk", "unroll", "dbuf", "mfma", "ks", "vec"]


def _clip(values, extent):
    kept = [v for v in values if v <= extent]
    return kept if kept else [min(values)]


def _cover(values, extent):
    """The clipped list plus the smallest value >= extent when that value
    is larger than every kept one (a tile spanning a whole output row or
    column)."""
    kept = _clip(values, extent)
    above = [v for v in values if v >= extent]
    if above and min(above) > kept[-1]:
        kept = kept + [min(above)]
    return kept


def _cdiv(a, b):
    return -(-a // b)


def _pow2floor(v):
    p = 1
    while p * 2 <= v:
        p *= 2
    return p


def conv_out(shape):
    N, C, H, W, K, R, S, st, pd = shape
    return (H + 2 * pd - R) // st + 1, (W + 2 * pd - S) // st + 1


def check_shape(op, shape):
    """Shapes the library accepts (raises ValueError otherwise)."""
    if op == OP_CONV:
        if len(shape) != 9:
            raise ValueError("conv shape has 9 entries")
        N, C, H, W, K, R, S, st, pd = shape
        if N < 0 or min(C, H, W, K, R, S, st) < 1 or pd < 0:
            raise ValueError("bad conv shape")
        if H + 2 * pd < R or W + 2 * pd < S:
            raise ValueError("conv shape has no output")
    elif op == OP_MATMUL:
        if len(shape) != 3:
            raise ValueError("matmul shape has 3 entries")
        M, N, K = shape
        if M < 0 or N < 1 or K < 1:
            raise ValueError("bad matmul shape")
    else:
        raise ValueError("unknown op")


class Lattice:
    """A product of ordered value lists with an optional validity predicate
    (Definition 1: every valid annotation of one sketch)."""

    def __init__(self, values, names=None, predicate=None):
        self.values = [list(v) for v in values]
        self.names = list(names) if names else [f"p{a}" for a in range(len(self.values))]
        self.sizes = [len(v) for v in self.values]
        self._pred = predicate

    def size(self):
        return math.prod(self.sizes)

    def knobs(self, idx):
        return {n: self.values[a][i] for a, (n, i) in enumerate(zip(self.names, idx))}

    def key(self, idx):
        """Mixed radix, axis 0 least significant."""
        k, radix = 0, 1
        for a, i in enumerate(idx):
            k += i * radix
            radix *= self.sizes[a]
        return k

    def from_key(self, key):
        idx = []
        for n in self.sizes:
            idx.append(key % n)
            key //= n
        return tuple(idx)

    def in_range(self, idx):
        return len(idx) == len(self.sizes) and all(0 <= i < n for i, n in zip(idx, self.sizes))

    def valid(self, idx):
        if not self.in_range(idx):
            return False
        return True if self._pred is None else bool(self._pred(tuple(idx)))

    def neighbors(self, idx):
        """Example 3 of Section 2.2: one index step along one axis.  Axis order
        ascending, the -1 step before the +1 step; out-of-range and invalid
        points are left out."""
        out = []
        for a in range(len(self.sizes)):
            for d in (-1, 1):
                j = idx[a] + d
                if 0 <= j < self.sizes[a]:
                    nb = tuple(idx[:a]) + (j,) + tuple(idx[a + 1:])
                    if self.valid(nb):
                        out.append(nb)
        return out

    def origin(self):
        """'Parameters that implement no optimization' (Section 2.2, step 1):
        index 0 on every axis -- the smallest tile and chunk, no unrolling, no
        LDS, no split, no MFMA.  If that point is invalid, the first valid
        point in key order."""
        z = tuple(0 for _ in self.sizes)
        if self.valid(z):
            return z
        for k in range(self.size()):
            p = self.from_key(k)
            if self.valid(p):
                return p
        return None

    def valid_points(self):
        return [p for p in map(self.from_key, range(self.size())) if self.valid(p)]


class Space(Lattice):
    """The lattice of one kernel family at one shape."""

    def __init__(self, op, shape):
        shape = tuple(int(v) for v in shape)
        check_shape(op, shape)
        self.op = op
        self.shape = shape
        if op == OP_CONV:
            N, C, H, W, K, R, S, st, pd = shape
            P, Q = conv_out(shape)
            values = [
                _clip(POW2_64, K), _cover(POW2_64, P), _cover(POW2_64, Q), _clip(POW2_64, C),
                list(UNROLL), [0, 1], _clip(CONV_SPLIT, C), [0, 1, 2, 3], list(VEC),
            ]
            names = CONV_AXES
        else:
            M, N, K = shape
            values = [
                _clip(MM_TILE, M), _clip(MM_TILE, N), _clip(MM_BK, K),
                list(UNROLL), [0, 1], [0, 1], _clip(SPLITK, K), list(VEC),
            ]
            names = MM_AXES
        super().__init__(values, names, predicate=lambda idx: self.geometry(idx)["valid"])

    def geometry(self, idx):
        """Launch geometry and derived template parameters; ``valid`` says
        whether the point belongs to the search space."""
        v = self.knobs(idx)
        return conv_geometry(self.shape, v) if self.op == OP_CONV else matmul_geometry(self.shape, v)


def conv_geometry(shape, v):
    if v["mfma"] >= 2:
        return conv_quad_geometry(shape, v)
    N, C, H, W, K, R, S, st, pd = shape
    P, Q = conv_out(shape)
    tk, th, tw, tc = v["tk"], v["th"], v["tw"], v["tc"]
    if th > P or tw > Q:
        # tiles past the output's height or width exist only as mfma = 3 bands
        return dict(valid=False, grid=0, threads=0, lds_bytes=0, acc=0, unroll_eff=1, t0=0,
                    t1=0, red=0, chunks=0)
    npx = th * tw
    outs = tk * npx
    if v["mfma"] == 0:
        # Lanes cover pixels first, then channel groups; a tile must fill at
        # least one wave, or be the largest tile the shape allows.
        biggest = _clip(POW2_64, K)[-1] * _clip(POW2_64, P)[-1] * _clip(POW2_64, Q)[-1]
        ok = outs >= min(64, biggest)
        if npx >= 256:
            threads, ppt, kpt = 256, npx // 256, tk
        else:
            threads = min(256, outs)
            kpt = max(1, tk // max(1, threads // npx))
            ppt = 1
        acc = kpt * ppt
        body = acc
        ok = ok and acc <= 64
        red = tc * R * S
        wrow = red
        t0, t1 = kpt, ppt           # template parameters: channels and pixels per thread
    else:
        # Up to four waves split the pixels (one per 16-pixel block for tiles
        # under 64 pixels); each wave covers all tk channels in 16x16 blocks
        # (v_mfma_f32_16x16x4f32).
        waves = min(4, max(1, npx // 16))
        threads = 64 * waves
        ok = tk >= 16 and npx >= 16
        tkb = max(1, tk // 16)
        npb = max(1, npx // (16 * waves))
        acc = 4 * tkb * npb
        body = tkb * npb
        ok = ok and acc <= 128
        red = _cdiv(tc * R * S, 16) * 16
        wrow = red + 4
        t0, t1 = tkb, npb           # template parameters: channel blocks, pixel blocks per wave
    hs = (th - 1) * st + R
    # aligned halo layout (image rows of whole 16-byte groups, tiles of at
    # least 16 input columns): rows start at the 16-byte boundary at or before
    # the tile's first column, up to 3 more columns, rounded to 4
    # (only with 16-byte copies, vec = 4)
    halo16 = v["vec"] == 4 and W % 4 == 0 and tw * st >= 16
    if halo16:
        ws = _cdiv((tw - 1) * st + S + 3, 4) * 4
    else:
        ws = (tw - 1) * st + S
    chunks = max(1, _cdiv(C, tc))
    if v["lds"]:
        # weights + halo (+ one zero float) per buffer, rounded to 16 bytes; two
        # buffers when a workgroup walks more than one chunk; then the table.
        nbuf = 2 if _cdiv(chunks, v["ks"]) > 1 else 1
        # + the reduction table and one source offset per staged position
        lds = 4 * (nbuf * _cdiv(tk * wrow + tc * hs * ws + 1, 4) * 4 + red + tk * wrow + tc * hs * ws)
    else:
        lds = 8 * red
    grid = N * v["ks"] * _cdiv(K, tk) * _cdiv(P, th) * _cdiv(Q, tw)
    uf = 1 if v["unroll"] == 0 else min(16, _pow2floor(max(1, v["unroll"] // body)))
    if v["mfma"]:
        # The MFMA family's unroll is its read-ahead depth D: 3 from 16, 2 from
        # 4, else 1; D+1 operand sets of 4 (tkb + npb) floats must fit 96
        # registers (192 when D = 1), the budget of its compiled instances.
        uf = 3 if uf >= 16 else (2 if uf >= 4 else 1)
        ring = (uf + 1) * 4 * (t0 + t1)
        ok = ok and (ring <= 96 or (uf == 1 and ring <= 192))
    else:
        # 64 accumulators on the global path do not fit an unroll of 8 or more
        ok = ok and not (v["lds"] == 0 and acc == 64 and uf >= 8)
    # vec = 4 (16-byte copies into LDS) needs staging by whole waves and one
    # operand whose staged rows are whole 16-byte groups
    if v["vec"] == 4:
        w16 = (C * R * S) % 4 == 0 and (tc * R * S) % 4 == 0 and wrow % 4 == 0
        h16 = halo16 and (tk * wrow) % 4 == 0
        ok = ok and v["lds"] == 1 and threads % 64 == 0 and (w16 or h16)
    valid = (ok and lds <= LDS_LIMIT and threads <= THREADS_LIMIT and v["ks"] <= chunks
             and grid <= GRID_LIMIT)
    return dict(valid=valid, grid=grid, threads=threads, lds_bytes=lds, acc=acc,
                unroll_eff=uf, t0=t0, t1=t1, red=red, chunks=chunks)


def conv_quad_geometry(shape, v):
    """mfma = 2 and 3: implicit GEMM whose k-steps each take one channel quad (four
    consecutive input channels) at one tap (r, s), over LDS-staged weights and
    input halo.  Waves split the tile's pixels as for mfma = 1 (16x16 blocks,
    up to four pixel waves); the unroll knob gives the depth D (3 from 16
    unrolled steps, 2 from 4, else 1) and a step takes U = 2^(D-1) quads.  A
    reduction split ks first goes to KG wave groups of one workgroup (the
    largest of 4, 2, 1 not above ks whose U-blocks of quads divide the chunk's
    quads and that keeps 1024 threads), the rest across workgroups.

    mfma = 2 tiles are th x tw rectangles of one image (th <= P, tw <= Q).
    mfma = 3 tiles are bands: th * tw consecutive pixels of the output
    flattened over (image, row, column), the pixel loops fused before tiling
    (a sketch of its own).
    Image n's output row p reads padded rows n * hp + p * st + r with
    hp = (P - 1) * st + R, so a band's halo is one range of padded rows, each
    one output row wide; the grid is ks / KG * (K / tk) * (N P Q / (th tw))
    rounded up.  A band spans at most D = min(N P, 1 + ceil((npx - 1) / Q))
    output rows (at least one) with at most X = min(N - 1, ceil((D - 1) / P)) image
    boundaries among them: consecutive rows are st padded rows apart, R across
    a boundary, so hs = (D - 1) st + X max(0, R - st) + R.

    LDS per buffer: tk weight rows of wrow floats (the smallest 4 * odd >=
    4 * quads * R * S with 16-byte weight copies, else the smallest 2 * odd)
    and 4 * quads halo channels of cs floats (the smallest >= hs * ws that is
    16 mod 32); two buffers when a workgroup walks more than one chunk; the
    wave groups' partial tiles and the output staging rows (16 x 68 floats
    per pixel wave) reuse it.  Validity adds: at least one 16x16
    block, chunks of whole channel quads (tc >= 4, or tc = 1 standing for all
    channels of an image with fewer than four), LDS staging, the register
    budget of the compiled instances (at most 32, 16, 4 blocks per wave and
    20, 12, 8 channel plus pixel blocks for KG = 1, 2, 4), at most 12 copy
    units per thread per kind for a full chunk (4-byte units, or 16-byte ones
    where rows allow: vec), and copy offsets below 2^29 floats.
    """
    N, C, H, W, K, R, S, st, pd = shape
    P, Q = conv_out(shape)
    tk, th, tw, tc = v["tk"], v["th"], v["tw"], v["tc"]
    band = v["mfma"] == 3
    npx = th * tw
    waves = min(4, max(1, npx // 16))
    tkb, npb = max(1, tk // 16), max(1, npx // (16 * waves))
    blocks = tkb * npb
    uf = 1 if v["unroll"] == 0 else min(16, _pow2floor(max(1, v["unroll"] // blocks)))
    depth = 3 if uf >= 16 else (2 if uf >= 4 else 1)
    quads_per_step = 2 ** (depth - 1)
    chan = C if C < 4 else tc                  # real channels of a full chunk
    quads = _cdiv(chan, 4)
    ok = tk >= 16 and npx >= 16 and (tc >= 4 or (C < 4 and tc == 1))
    ok = ok and (band or (th <= P and tw <= Q))
    kg = min(v["ks"], 4)
    while kg > 1 and (quads % (kg * quads_per_step) or 64 * waves * kg > THREADS_LIMIT):
        kg //= 2
    ksw = v["ks"] // kg
    ok = ok and 4 * blocks <= 128 and quads % (kg * quads_per_step) == 0
    ok = ok and blocks <= {1: 32, 2: 16, 4: 4}[kg] and tkb + npb <= {1: 20, 2: 12, 4: 8}[kg]
    chunks = _cdiv(C, chan)
    cps = _cdiv(chunks, ksw)
    ok = ok and ksw <= chunks
    if band:
        d = max(1, min(N * P, 1 + _cdiv(npx - 1, Q)))
        x = min(N - 1, _cdiv(d - 1, P))
        hs = (d - 1) * st + max(0, x) * max(0, R - st) + R
        cols = Q
    else:
        hs = (th - 1) * st + R
        cols = tw
    halo16 = v["vec"] == 4 and W % 4 == 0 and cols * st >= 16
    ws = _cdiv((cols - 1) * st + S + 3, 4) * 4 if halo16 else (cols - 1) * st + S
    cs = hs * ws
    while cs % 32 != 16:
        cs += 1
    w16 = v["vec"] == 4 and (C * R * S) % 4 == 0 and (chan * R * S) % 4 == 0
    unit = 4 if w16 else 2
    odd = _cdiv(4 * quads * R * S, unit)
    if odd % 2 == 0:
        odd += 1
    wrow = unit * odd
    ok = ok and (v["vec"] == 1 or w16 or halo16)
    threads = 64 * waves * kg
    units_w = tk * wrow // 4 if w16 else tk * wrow
    units_h = quads * cs if halo16 else 4 * quads * cs
    per_thread = max(_cdiv(units_w, threads), _cdiv(units_h, threads))
    ok = ok and (C < 4 or per_thread <= 12)
    nbuf = 2 if cps > 1 else 1
    buf = tk * wrow + 4 * quads * cs
    # buffers; the wave groups' partial tiles; the output staging rows (16
    # rows of 68 floats per pixel wave)
    lds = max(4 * nbuf * buf, 16 * (kg - 1) * waves * 64 * blocks, 4 * 16 * 68 * waves)
    if band:
        grid = ksw * _cdiv(K, tk) * _cdiv(N * P * Q, npx)
        images = min(N, 1 + _cdiv(npx - 1, P * Q))
        ok = ok and (images * C + 4 * quads) * H * W < 2 ** 29
    else:
        grid = N * ksw * _cdiv(K, tk) * _cdiv(P, th) * _cdiv(Q, tw)
        ok = ok and 4 * quads * H * W < 2 ** 29
    ok = ok and tk * C * R * S < 2 ** 29
    valid = (ok and v["lds"] == 1 and lds <= LDS_LIMIT and threads <= THREADS_LIMIT
             and grid <= GRID_LIMIT)
    return dict(valid=valid, grid=grid, threads=threads, lds_bytes=lds, acc=4 * blocks,
                unroll_eff=depth, t0=tkb, t1=npb, red=4 * quads * R * S, chunks=chunks)


def matmul_geometry(shape, v):
    M, N, K = shape
    bm, bn, bk = v["bm"], v["bn"], v["bk"]
    if v["mfma"] == 0:
        rm, rn = bm // 16, bn // 16
        acc = rm * rn
        body = acc
        kstep = 1
        ok = acc <= 128
        t0, t1 = rm, rn
    else:
        ok = bm >= 32 and bn >= 32
        wm, wn = bm // 2, bn // 2
        if wm >= 32 and wn >= 32:
            kstep = 2
            blocks = (wm // 32) * (wn // 32)
            acc = 16 * blocks
        else:
            kstep = 4
            blocks = max(1, wm // 16) * max(1, wn // 16)
            acc = 4 * blocks
        body = blocks
        ok = ok and acc <= 256
        t0, t1 = wm, wn
    trip = max(1, bk // kstep)
    if v["unroll"] == 0:
        uf = 1
    elif trip * body <= v["unroll"]:
        uf = trip
    else:
        uf = min(trip, _pow2floor(max(1, v["unroll"] // body)))
    # LDS stages: one without dbuf; with dbuf three when they fit, else two.
    stage = bm * bk + bk * bn
    stages = 1 if not v["dbuf"] else (3 if 3 * stage * 4 <= LDS_LIMIT else 2)
    # A reduction split first splits every K-tile between two wave groups of
    # one MFMA workgroup (when the K-tile has at least 8 steps); the rest of
    # the split goes across workgroups.
    kg = 2 if v["mfma"] and v["ks"] >= 2 and bk >= 8 else 1
    wgs = v["ks"] // kg
    # Register budget of the compiled instances: two wave groups leave room
    # for 64 accumulators per lane; a 128x128 wave tile with 16-deep K-tiles
    # unrolled 8 times on one LDS stage does not fit; a VALU tile that stages
    # the next K-tile in registers (dbuf) fits (rm + rn) * unroll <= 512.
    if v["mfma"]:
        ok = ok and (kg == 1 or acc <= 64) and not (
            acc == 256 and not v["dbuf"] and bk == 16 and uf == 8)
    else:
        ok = ok and (not v["dbuf"] or (t0 + t1) * uf <= 512)
    # vec = 4 (16-byte operand loads) needs rows of A (K) or B (N) in whole
    # 16-byte groups
    ok = ok and (v["vec"] == 1 or K % 4 == 0 or N % 4 == 0)
    lds = max(stages * stage, bm * bn if kg > 1 else 0) * 4
    nkt = _cdiv(K, bk)
    grid = _cdiv(M, bm) * _cdiv(N, bn) * wgs
    threads = 256 * kg
    valid = (ok and lds <= LDS_LIMIT and threads <= THREADS_LIMIT and wgs <= nkt
             and grid <= GRID_LIMIT)
    return dict(valid=valid, grid=grid, threads=threads, lds_bytes=lds, acc=acc,
                unroll_eff=uf, t0=t0, t1=t1, red=kstep, chunks=nkt)
