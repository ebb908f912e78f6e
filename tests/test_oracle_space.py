"""Pins of the reference lattice: the paper's worked neighbourhood example,
hand-computed value lists and geometry, and structural invariants."""
import math

import pytest

from oracle import space as sp


def read_golden(path):
    rows = {}
    axes = []
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        head, *rest = line.split()
        if head == "axis":
            axes.append([int(v) for v in rest[1:]])
        else:
            rows[head] = rest
    return axes, rows


def test_example3_neighbors(golden_dir):
    axes, rows = read_golden(f"{golden_dir}/droplet_example3.txt")
    lat = sp.Lattice(axes, ["unroll", "tile"])
    point = tuple(axes[a].index(int(v)) for a, v in enumerate(rows["point"]))
    got = [tuple(axes[a][i] for a, i in enumerate(nb)) for nb in lat.neighbors(point)]
    expect = [tuple(int(t) for t in s.split(",")) for s in rows["neighbors"]]
    assert got == expect
    # (1,1) is a corner: two neighbours; the origin applies no optimisation.
    assert lat.neighbors((0, 0)) == [(1, 0), (0, 1)]
    assert lat.origin() == (0, 0)
    assert lat.size() == 25


def test_invalid_neighbors_skipped_not_hopped():
    lat = sp.Lattice([[1, 2, 3], [1, 2, 4]], predicate=lambda p: p != (1, 1))
    assert lat.neighbors((1, 0)) == [(0, 0), (2, 0)]
    assert (1, 1) not in lat.valid_points() and len(lat.valid_points()) == 8
    lat2 = sp.Lattice([[1, 2]], predicate=lambda p: p != (0,))
    assert lat2.origin() == (1,)


def test_key_mixed_radix():
    lat = sp.Lattice([[0, 1, 2], [0, 1], [0, 1, 2, 3]])
    assert lat.key((2, 1, 3)) == 2 + 1 * 3 + 3 * 6
    keys = [lat.key(lat.from_key(k)) for k in range(lat.size())]
    assert keys == list(range(24))


def test_value_lists_named_shapes():
    s0 = sp.Space(sp.OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1))
    assert s0.values[0] == [1, 2, 4, 8, 16, 32, 64]
    # P = Q = 56: tile heights and widths up to 32, and 64 that covers a row
    # (for band tiles)
    assert s0.values[1] == [1, 2, 4, 8, 16, 32, 64] == s0.values[2]
    assert s0.values[3] == [1, 2, 4, 8, 16, 32, 64]
    # conv splits reach 32 (C = 64 keeps all six)
    assert s0.values[4:] == [[0, 16, 64, 512], [0, 1], [1, 2, 4, 8, 16, 32], [0, 1, 2, 3],
                             [1, 4]]
    assert s0.size() == 7 * 7 * 7 * 7 * 4 * 2 * 6 * 4 * 2
    s14 = sp.Space(sp.OP_CONV, (16, 512, 14, 14, 512, 3, 3, 1, 1))
    assert s14.values[1] == [1, 2, 4, 8, 16] == s14.values[2]
    s32 = sp.Space(sp.OP_CONV, (1, 8, 32, 32, 16, 3, 3, 1, 1))
    assert s32.values[1] == [1, 2, 4, 8, 16, 32] == s32.values[2]   # 32 covers 32
    assert s32.values[6] == [1, 2, 4, 8]                  # C = 8 clips the splits
    s2 = sp.Space(sp.OP_CONV, (1, 3, 224, 224, 64, 7, 7, 2, 3))
    assert s2.values[1] == [1, 2, 4, 8, 16, 32, 64]       # P = 112: nothing covers it
    assert s2.values[3] == [1, 2] and s2.values[6] == [1, 2]
    m = sp.Space(sp.OP_MATMUL, (1024, 1024, 1024))
    assert m.values == [[16, 32, 64, 128, 256]] * 2 + [[4, 8, 16, 32, 64], [0, 16, 64, 512],
                                                         [0, 1], [0, 1], [1, 2, 4, 8], [1, 4]]
    fc = sp.Space(sp.OP_MATMUL, (1, 1000, 2048))
    assert fc.values[0] == [16]                          # smallest value kept
    tiny = sp.Space(sp.OP_MATMUL, (3, 5, 2))
    assert tiny.values[2] == [4] and tiny.values[6] == [1, 2] and tiny.values[7] == [1, 4]


def idx_of(space, **kv):
    return tuple(space.values[a].index(kv[n]) for a, n in enumerate(space.names))


def test_conv_geometry_hand_computed():
    s = sp.Space(sp.OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1))
    g = s.geometry(idx_of(s, tk=16, th=8, tw=8, tc=16, unroll=64, lds=1, ks=1, mfma=1, vec=4))
    # 64 pixels -> one 16-pixel block per wave; 16 channels -> one block.
    # reduction 16*9 = 144 (a multiple of 16); weight rows padded to 148; halo
    # 10x10 (8 columns wide: no aligned layout); 4 chunks in one split -> two
    # buffers of 16*148 + 16*100 + 1 -> 3972 floats, + table, + one staging
    # source per weight and halo position (2368 + 1600).  Unroll 64 over one
    # block per step -> u = 16 -> read-ahead depth 3 (ring 4 * 4 * 2 = 32).
    assert g == dict(valid=True, grid=4 * 7 * 7, threads=256,
                     lds_bytes=4 * (2 * 3972 + 144 + 2368 + 1600), acc=4,
                     unroll_eff=3, t0=1, t1=1, red=144, chunks=4)
    # 4-byte copies: the same layout here (the halo is narrower than 16 columns)
    assert s.geometry(idx_of(s, tk=16, th=8, tw=8, tc=16, unroll=64, lds=1, ks=1, mfma=1,
                             vec=1)) == g
    # unroll 16 with two 16x16 blocks per step -> u = 8 -> depth 2
    g = s.geometry(idx_of(s, tk=32, th=8, tw=8, tc=16, unroll=16, lds=1, ks=1, mfma=1, vec=4))
    assert g["valid"] and g["unroll_eff"] == 2 and (g["t0"], g["t1"]) == (2, 1)
    g = s.geometry(idx_of(s, tk=4, th=4, tw=32, tc=8, unroll=16, lds=0, ks=2, mfma=0, vec=1))
    # 128 pixels x 4 channels -> 256 threads, 2 channel groups of 2; unroll 16//2 = 8.
    assert g == dict(valid=True, grid=2 * 16 * 14 * 2, threads=256, lds_bytes=8 * 72, acc=2,
                     unroll_eff=8, t0=2, t1=1, red=72, chunks=8)
    # One pixel, 64 channels: one wave, one channel per lane; 32 chunks -> two
    # buffers of 64*18 + 2*3*3 + 1 = 1171 -> 1172 floats, + table, + sources.
    g = s.geometry(idx_of(s, tk=64, th=1, tw=1, tc=2, unroll=0, lds=1, ks=1, mfma=0, vec=1))
    assert g == dict(valid=True, grid=56 * 56, threads=64, lds_bytes=4 * (2 * 1172 + 18 + 1152 + 18),
                     acc=1, unroll_eff=1, t0=1, t1=1, red=18, chunks=32)
    # 16-byte copies need an operand in whole 16-byte rows: chunk rows of
    # 2 * 9 = 18 weights are not, and a one-column halo is not
    assert not s.valid(idx_of(s, tk=64, th=1, tw=1, tc=2, unroll=0, lds=1, ks=1, mfma=0, vec=4))
    # nor without LDS staging
    assert not s.valid(idx_of(s, tk=4, th=4, tw=32, tc=8, unroll=16, lds=0, ks=2, mfma=0, vec=4))
    # Fewer than 64 outputs: not a full wave.
    assert not s.valid(idx_of(s, tk=2, th=4, tw=4, tc=1, unroll=0, lds=0, ks=1, mfma=0, vec=1))
    # MFMA reduction padded to a multiple of 16: 4 channels x 9 taps = 36 -> 48;
    # 16 columns wide on an image of 56 (a multiple of 4): aligned halo layout,
    # rows of 18 + 3 -> 24 floats; 16 chunks -> two buffers of
    # 32*52 + 4*6*24 + 1 = 2241 -> 2244 floats.
    g = s.geometry(idx_of(s, tk=32, th=4, tw=16, tc=4, unroll=0, lds=1, ks=1, mfma=1, vec=4))
    assert g["red"] == 48 and g["lds_bytes"] == 4 * (2 * 2244 + 48 + 1664 + 576)
    # with 4-byte copies the rows keep exactly the tile's 18 input columns:
    # 32*52 + 4*6*18 + 1 = 2097 -> 2100 floats per buffer
    g = s.geometry(idx_of(s, tk=32, th=4, tw=16, tc=4, unroll=0, lds=1, ks=1, mfma=1, vec=1))
    assert g["lds_bytes"] == 4 * (2 * 2100 + 48 + 1664 + 432)
    # acc budget: 64 channels x 4 pixels per thread (1024 px / 256) = 256 > 64.
    assert not s.geometry(idx_of(s, tk=64, th=32, tw=32, tc=1, unroll=0, lds=0, ks=1, mfma=0,
                                 vec=1))["valid"]
    # MFMA needs >= 16 channels and >= 16 pixels (one 16x16 block per wave).
    assert not s.valid(idx_of(s, tk=8, th=8, tw=8, tc=4, unroll=0, lds=0, ks=1, mfma=1, vec=1))
    assert not s.valid(idx_of(s, tk=16, th=2, tw=4, tc=4, unroll=0, lds=0, ks=1, mfma=1, vec=1))
    assert s.valid(idx_of(s, tk=16, th=4, tw=8, tc=4, unroll=0, lds=0, ks=1, mfma=1, vec=1))
    # LDS limit: 64-channel chunk of a 34-row halo in the aligned layout (rows
    # of 34 + 3 -> 40 floats) does not fit (one chunk, one buffer of
    # 16*576 + 64*34*40 + 1 -> 96260 floats).
    g = s.geometry(idx_of(s, tk=16, th=32, tw=32, tc=64, unroll=0, lds=1, ks=1, mfma=0, vec=4))
    assert g["lds_bytes"] == 4 * (96260 + 576 + 9216 + 87040) and not g["valid"]
    # split finer than the chunk count.
    assert not s.valid(idx_of(s, tk=16, th=8, tw=8, tc=64, unroll=0, lds=0, ks=2, mfma=0, vec=1))
    # register budgets of the compiled kernels: one 16-channel block x 32
    # pixel blocks per wave (2048 pixels over four waves, on VGG-16 layer 2)
    # needs two operand sets of 4 * 33 floats = 264 > 192; 2 x 16 blocks fit
    v = sp.Space(sp.OP_CONV, (16, 64, 224, 224, 64, 3, 3, 1, 1))
    assert not v.valid(idx_of(v, tk=16, th=64, tw=32, tc=4, unroll=0, lds=1, ks=1, mfma=1, vec=4))
    g = v.geometry(idx_of(v, tk=32, th=64, tw=16, tc=4, unroll=0, lds=1, ks=1, mfma=1, vec=4))
    assert g["valid"] and (g["t0"], g["t1"]) == (2, 16)
    # a third operand set (unroll 64 over 32 blocks -> u = 2, depth 1) is not
    # reachable there; depth 2 needs 3 * 4 * (tkb + npb) <= 96
    g = v.geometry(idx_of(v, tk=64, th=8, tw=16, tc=4, unroll=64, lds=1, ks=1, mfma=1, vec=4))
    assert (g["t0"], g["t1"], g["unroll_eff"]) == (4, 2, 2) and g["valid"]
    # 64 accumulators (256 pixels, one per thread, x 64 channels) on the
    # global path with an 8-fold unroll (512 / 64)
    g = s.geometry(idx_of(s, tk=64, th=16, tw=16, tc=8, unroll=512, lds=0, ks=1, mfma=0, vec=1))
    assert g["acc"] == 64 and g["unroll_eff"] == 8 and not g["valid"]
    assert s.valid(idx_of(s, tk=64, th=16, tw=16, tc=8, unroll=64, lds=0, ks=1, mfma=0, vec=1))


def test_conv_mfma_small_tile_geometry():
    # 7x7 outputs: a 4x4 tile (16 pixels) runs on one wave.  Reduction chunk
    # 16 channels x 9 taps = 144 (a multiple of 16), weight row 148; halo 6x6;
    # 32 chunks over 8 splits -> two LDS buffers of
    # ceil((16*148 + 16*36 + 1) / 4) * 4 = 2948 floats, then the 144-entry table
    # and the staging sources (2368 + 576).
    s = sp.Space(sp.OP_CONV, (1, 512, 7, 7, 512, 3, 3, 1, 1))
    g = s.geometry(idx_of(s, tk=16, th=4, tw=4, tc=16, unroll=64, lds=1, ks=8, mfma=1, vec=4))
    assert g == dict(valid=True, grid=8 * 32 * 2 * 2, threads=64,
                     lds_bytes=4 * (2 * 2948 + 144 + 2368 + 576),
                     acc=4, unroll_eff=3, t0=1, t1=1, red=144, chunks=32)
    # two 16-channel blocks on the one wave
    g = s.geometry(idx_of(s, tk=32, th=4, tw=4, tc=16, unroll=0, lds=0, ks=4, mfma=1, vec=1))
    assert g["valid"] and g["threads"] == 64 and g["t0"] == 2 and g["t1"] == 1
    # 8 pixels: less than one 16-pixel block
    assert not s.valid(idx_of(s, tk=32, th=4, tw=2, tc=16, unroll=0, lds=0, ks=4, mfma=1, vec=1))
    # 32 pixels: two waves, one block each.
    c = sp.Space(sp.OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1))
    g = c.geometry(idx_of(c, tk=16, th=4, tw=8, tc=16, unroll=0, lds=1, ks=1, mfma=1, vec=4))
    assert g["valid"] and g["threads"] == 128 and g["t1"] == 1


def test_conv_quad_geometry_hand_computed():
    """mfma = 2 (channel-quad steps, rectangular tiles) and mfma = 3 (the same
    over band tiles), worked by hand from the layout rules."""
    s = sp.Space(sp.OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1))
    # 64 pixels over four waves, one 16x16 block each; unroll 64 over one
    # block -> u = 16 -> depth 3 -> 4 quads per step.  All 64 channels in one
    # chunk: 16 quads; ks = 2 -> two wave groups (16 % (2 * 4) == 0, 512
    # threads), no split across workgroups.  Halo 6 rows of 24 (aligned:
    # 15 + 3 + 3 -> 24), channel stride 144 (= 16 mod 32); weight rows of
    # 16 * 9 = 144 -> 145 (odd) * 4 = 580 floats.  One buffer of
    # 16 * 580 + 64 * 144 = 18496 floats.  Copy units per thread:
    # 2320 / 512 and 2304 / 512 -> 5.  Grid 4 x 14 x 4 (16 columns cover 56
    # as 64).
    g = s.geometry(idx_of(s, tk=16, th=4, tw=16, tc=64, unroll=64, lds=1, ks=2, mfma=2, vec=4))
    assert g == dict(valid=True, grid=4 * 14 * 4, threads=512, lds_bytes=4 * 18496, acc=4,
                     unroll_eff=3, t0=1, t1=1, red=576, chunks=1)
    # The same knobs as a band (mfma = 3): 64 consecutive pixels spanning at
    # most 1 + ceil(63 / 56) = 3 rows of one image: 2 + 3 = 5 padded rows of
    # 55 + 3 + 3 -> 64 floats (aligned), channel stride 320 -> 336.  One buffer
    # of 16 * 580 + 64 * 336 = 30784 floats; copy units 2320 / 512 -> 5 and
    # 16 * 336 / 512 -> 11.  Grid 4 x ceil(3136 / 64): no padded pixel.
    g = s.geometry(idx_of(s, tk=16, th=4, tw=16, tc=64, unroll=64, lds=1, ks=2, mfma=3, vec=4))
    assert g == dict(valid=True, grid=4 * 49, threads=512, lds_bytes=4 * 30784, acc=4,
                     unroll_eff=3, t0=1, t1=1, red=576, chunks=1)
    # 4 x 8 tiles with 32-channel chunks: two waves of one block, 8 quads, two
    # chunks and two buffers; ks = 2 -> two wave groups (8 % (2 * 4) == 0, 256
    # threads).  Halo 6 rows of 7 + 3 = 10 (8 columns: no aligned layout),
    # channel stride 60 -> 80; weight rows 32 * 9 = 288 -> 72 (even) -> 73 * 4
    # = 292.  Buffer 16 * 292 + 32 * 80 = 7232 floats; copy units 1168 / 256
    # -> 5 and (4-byte halo copies) 2560 / 256 -> 10.  Grid 4 * 14 * 7.
    g = s.geometry(idx_of(s, tk=16, th=4, tw=8, tc=32, unroll=64, lds=1, ks=2, mfma=2, vec=4))
    assert g == dict(valid=True, grid=4 * 14 * 7, threads=256, lds_bytes=4 * 2 * 7232, acc=4,
                     unroll_eff=3, t0=1, t1=1, red=288, chunks=2)
    # the 4 x 16 tile with unroll 0 (one quad per step) and ks = 4: four wave
    # groups of four waves, 64 * 4 * 4 = 1024 threads
    g = s.geometry(idx_of(s, tk=16, th=4, tw=16, tc=64, unroll=0, lds=1, ks=4, mfma=2, vec=4))
    assert g["valid"] and g["threads"] == 1024 and g["grid"] == 224
    # 8-channel chunks hold 2 quads: unroll 64 (4 quads per step) does not fit
    # them; with one quad per step and ks = 4 the groups fall back to two
    # (2 % 4 != 0), the remaining factor 2 splits across workgroups
    assert not s.valid(idx_of(s, tk=16, th=4, tw=16, tc=8, unroll=64, lds=1, ks=1, mfma=2, vec=4))
    g = s.geometry(idx_of(s, tk=16, th=4, tw=16, tc=8, unroll=0, lds=1, ks=4, mfma=2, vec=4))
    assert g["valid"] and g["threads"] == 512 and g["grid"] == 2 * 224 and g["chunks"] == 8
    # chunks of whole quads: tc = 2 on 64 channels is not; LDS staging only
    assert not s.valid(idx_of(s, tk=16, th=4, tw=16, tc=2, unroll=0, lds=1, ks=1, mfma=2, vec=4))
    assert not s.valid(idx_of(s, tk=16, th=4, tw=16, tc=64, unroll=0, lds=0, ks=1, mfma=2, vec=1))
    # register budget of four wave groups: at most 4 blocks per wave (4 x 2
    # blocks do not fit, 2 x 2 do)
    assert not s.valid(idx_of(s, tk=64, th=8, tw=16, tc=64, unroll=0, lds=1, ks=4, mfma=2, vec=4))
    assert s.valid(idx_of(s, tk=32, th=8, tw=16, tc=64, unroll=0, lds=1, ks=4, mfma=2, vec=4))
    # rectangular tiles stay inside the output: 64 columns on 56 are bands only
    assert not s.valid(idx_of(s, tk=16, th=1, tw=64, tc=64, unroll=0, lds=1, ks=4, mfma=2, vec=4))
    assert s.valid(idx_of(s, tk=16, th=1, tw=64, tc=64, unroll=0, lds=1, ks=4, mfma=3, vec=4))
    # The 3-channel stem: tc = 1 stands for the single chunk of all three
    # channels (one quad, channel 3 zero); 256 pixels -> four blocks per wave;
    # halo 7 * 2 + 7 = 21 rows of 31 * 2 + 7 + 3 -> 72 (aligned), channel
    # stride 1512 -> 1520 (= 16 mod 32); 3 * 49 weights per filter are not
    # whole 16-byte groups, so weight rows take 4-byte copies and are
    # 2 * odd floats: 4 * 49 = 196 -> 98 (even) -> 99 * 2 = 198.
    st = sp.Space(sp.OP_CONV, (1, 3, 224, 224, 64, 7, 7, 2, 3))
    g = st.geometry(idx_of(st, tk=16, th=8, tw=32, tc=1, unroll=0, lds=1, ks=1, mfma=2, vec=4))
    assert g == dict(valid=True, grid=4 * 14 * 4, threads=256, lds_bytes=4 * (16 * 198 + 4 * 1520),
                     acc=16, unroll_eff=1, t0=1, t1=4, red=196, chunks=1)
    # the same knobs as a band: 256 pixels spanning at most 1 + ceil(255 /
    # 112) = 4 rows: 3 * 2 + 7 = 13 padded rows of 111 * 2 + 7 + 3 -> 232
    # floats, channel stride 3016 -> 3024; grid 4 x ceil(12544 / 256)
    g = st.geometry(idx_of(st, tk=16, th=8, tw=32, tc=1, unroll=0, lds=1, ks=1, mfma=3, vec=4))
    assert g == dict(valid=True, grid=4 * 49, threads=256, lds_bytes=4 * (16 * 198 + 4 * 3024),
                     acc=16, unroll_eff=1, t0=1, t1=4, red=196, chunks=1)
    assert not st.valid(idx_of(st, tk=16, th=8, tw=32, tc=2, unroll=0, lds=1, ks=1, mfma=2, vec=4))


def test_conv_band_geometry_hand_computed():
    """mfma = 3 band tiles, worked by hand."""
    # VGG-16 L11 (16 images of 512 x 14 x 14): a band of 8 * 16 = 128
    # consecutive output pixels.  Four waves
    # of two 16-pixel blocks, four channel blocks; 8-channel chunks: 2 quads,
    # 64 chunks, two buffers.  A band spans at most 1 + ceil(127 / 14) = 11
    # output rows with at most one image boundary among them: 10 + 1 * 2 + 3
    # = 15 padded rows of 13 + 3 = 16 floats (W % 4 != 0: 4-byte halo
    # copies), channel stride 240 (= 16 mod 32).  Weight rows: 8 * 9 = 72
    # floats -> 18 (even) -> 19 * 4 = 76 (16-byte copies).  Buffer 64 * 76 +
    # 8 * 240 = 6784 floats; copy units per thread: 1216 / 256 -> 5 and
    # 1920 / 256 -> 8.  Grid: 8 channel tiles x ceil(3136 / 128) = 25 bands.
    v = sp.Space(sp.OP_CONV, (16, 512, 14, 14, 512, 3, 3, 1, 1))
    g = v.geometry(idx_of(v, tk=64, th=8, tw=16, tc=8, unroll=0, lds=1, ks=1, mfma=3, vec=4))
    assert g == dict(valid=True, grid=200, threads=256, lds_bytes=4 * 2 * 6784, acc=32,
                     unroll_eff=1, t0=4, t1=2, red=72, chunks=64)
    # a band depends on th * tw only: 16 x 8 is the same 128-pixel band
    g16 = v.geometry(idx_of(v, tk=64, th=16, tw=8, tc=8, unroll=0, lds=1, ks=1, mfma=3, vec=4))
    assert g16 == g
    # as rectangles, neither fits inside 14 x 14
    assert not v.valid(idx_of(v, tk=64, th=8, tw=16, tc=8, unroll=0, lds=1, ks=1, mfma=2, vec=4))
    assert not v.valid(idx_of(v, tk=64, th=16, tw=8, tc=8, unroll=0, lds=1, ks=1, mfma=2, vec=4))
    # the other families have no tiles past the output at all
    g = v.geometry(idx_of(v, tk=64, th=8, tw=16, tc=8, unroll=0, lds=1, ks=1, mfma=1, vec=4))
    assert g == dict(valid=False, grid=0, threads=0, lds_bytes=0, acc=0, unroll_eff=1, t0=0,
                     t1=0, red=0, chunks=0)
    # Stride 2, 1 x 1 (ResNet-50 downsampling, one image of 256 x 56 x 56 to
    # 28 x 28): tw = 32 covers 28; bands of 4 * 32 = 128 pixels span at most
    # 1 + ceil(127 / 28) = 6 rows of one image: 5 * 2 + 1 = 11 padded rows of
    # 27 * 2 + 1 + 3 -> 60 floats (aligned, 16-byte copies), channel stride
    # 660 -> 688.  Weight rows 16 -> 4 (even) -> 5 * 4 = 20.  Copy units per
    # thread: 160 / 256 -> 1 and 4 * 688 / 256 -> 11.  Buffer 32 * 20 +
    # 16 * 688 = 11648 floats, two of them; grid 16 x ceil(784 / 128) = 7.
    r = sp.Space(sp.OP_CONV, (1, 256, 56, 56, 512, 1, 1, 2, 0))
    g = r.geometry(idx_of(r, tk=32, th=4, tw=32, tc=16, unroll=0, lds=1, ks=1, mfma=3, vec=4))
    assert g == dict(valid=True, grid=112, threads=256, lds_bytes=4 * 2 * 11648, acc=16,
                     unroll_eff=1, t0=2, t1=2, red=16, chunks=16)



def test_matmul_geometry_hand_computed():
    m = sp.Space(sp.OP_MATMUL, (1024, 1024, 1024))
    g = m.geometry(idx_of(m, bm=64, bn=64, bk=16, unroll=64, dbuf=1, mfma=1, ks=1, vec=4))
    # dbuf: three stages of 8 KiB fit.
    assert g == dict(valid=True, grid=256, threads=256, lds_bytes=3 * (64 * 16 + 16 * 64) * 4,
                     acc=16, unroll_eff=8, t0=32, t1=32, red=2, chunks=64)
    g = m.geometry(idx_of(m, bm=32, bn=128, bk=32, unroll=16, dbuf=0, mfma=1, ks=4, vec=4))
    # wave tile 16x64 -> 16x16x4 blocks: 1*4, acc 16; trip 8, 8*4 > 16 -> 16//4 = 4.
    # ks 4: two wave groups (512 threads) x two workgroup splits; LDS holds the
    # larger of one stage (5120 floats) and the 32x128 partial tile (4096).
    assert g == dict(valid=True, grid=32 * 8 * 2, threads=512, lds_bytes=(32 * 32 + 32 * 128) * 4,
                     acc=16, unroll_eff=4, t0=16, t1=64, red=4, chunks=32)
    # dbuf with 2 x 64 KiB stages: three do not fit, two do.
    g = m.geometry(idx_of(m, bm=128, bn=128, bk=64, unroll=0, dbuf=1, mfma=1, ks=1, vec=4))
    assert g["valid"] and g["lds_bytes"] == 2 * (128 * 64 + 64 * 128) * 4
    # ks 2 with a K-tile of 4 steps stays a two-workgroup split of 256 threads.
    g = m.geometry(idx_of(m, bm=64, bn=64, bk=4, unroll=0, dbuf=0, mfma=1, ks=2, vec=4))
    assert g["threads"] == 256 and g["grid"] == 16 * 16 * 2
    # ks 2 with 256x256 tiles: the partial tile (256 KiB) does not fit in LDS.
    assert not m.valid(idx_of(m, bm=256, bn=256, bk=8, unroll=0, dbuf=0, mfma=1, ks=2, vec=4))
    g = m.geometry(idx_of(m, bm=128, bn=64, bk=8, unroll=512, dbuf=0, mfma=0, ks=1, vec=4))
    assert g == dict(valid=True, grid=8 * 16, threads=256, lds_bytes=(128 * 8 + 8 * 64) * 4,
                     acc=32, unroll_eff=8, t0=8, t1=4, red=1, chunks=128)
    assert not m.valid(idx_of(m, bm=256, bn=256, bk=4, unroll=0, dbuf=0, mfma=0, ks=1, vec=4))  # acc 256
    assert m.valid(idx_of(m, bm=256, bn=256, bk=4, unroll=0, dbuf=0, mfma=1, ks=1, vec=4))      # AGPRs
    assert not m.valid(idx_of(m, bm=256, bn=256, bk=64, unroll=0, dbuf=1, mfma=1, ks=1, vec=4))  # LDS
    assert not m.valid(idx_of(m, bm=16, bn=64, bk=8, unroll=0, dbuf=0, mfma=1, ks=1, vec=4))    # MFMA min
    # register budgets of the compiled kernels: two wave groups (ks 2, bk >= 8)
    # hold at most 64 accumulators (64x128 wave tile: 128)
    assert not m.valid(idx_of(m, bm=128, bn=256, bk=8, unroll=0, dbuf=0, mfma=1, ks=2, vec=4))
    assert m.valid(idx_of(m, bm=128, bn=256, bk=8, unroll=0, dbuf=0, mfma=1, ks=1, vec=4))
    # 128x128 wave tile, 16-deep K-tile unrolled 8 times (trip 8 * 16 blocks <= 512), one stage
    assert not m.valid(idx_of(m, bm=256, bn=256, bk=16, unroll=512, dbuf=0, mfma=1, ks=1, vec=4))
    assert m.valid(idx_of(m, bm=256, bn=256, bk=16, unroll=512, dbuf=1, mfma=1, ks=1, vec=4))
    # VALU 1x16 per thread, 32-deep K-tile fully unrolled (16 * 32 <= 512), staged
    # through registers: (1 + 16) * 32 = 544 > 512
    assert not m.valid(idx_of(m, bm=16, bn=256, bk=32, unroll=512, dbuf=1, mfma=0, ks=1, vec=4))
    assert m.valid(idx_of(m, bm=16, bn=256, bk=32, unroll=512, dbuf=0, mfma=0, ks=1, vec=4))
    # 16-byte loads need K or N in whole 16-byte groups
    o = sp.Space(sp.OP_MATMUL, (33, 45, 7))
    assert not o.valid(idx_of(o, bm=16, bn=16, bk=4, unroll=0, dbuf=0, mfma=0, ks=1, vec=4))
    assert o.valid(idx_of(o, bm=16, bn=16, bk=4, unroll=0, dbuf=0, mfma=0, ks=1, vec=1))


@pytest.mark.parametrize("op,shape", [
    (sp.OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1)),
    (sp.OP_CONV, (1, 3, 224, 224, 64, 7, 7, 2, 3)),
    (sp.OP_MATMUL, (1024, 1024, 1024)),
    (sp.OP_MATMUL, (1, 1000, 2048)),
])
def test_invariants(op, shape):
    s = sp.Space(op, shape)
    pts = s.valid_points()
    assert pts and s.origin() == min(pts, key=s.key)
    if op == sp.OP_MATMUL:
        assert s.origin() == tuple(0 for _ in s.sizes)
    for p in pts[:: max(1, len(pts) // 500)]:
        g = s.geometry(p)
        assert g["lds_bytes"] <= sp.LDS_LIMIT and g["threads"] <= 1024 and g["threads"] % 64 == 0
        assert 1 <= g["unroll_eff"] <= 64 and g["grid"] >= 1
        for nb in s.neighbors(p):
            assert s.valid(nb) and sum(a != b for a, b in zip(nb, p)) == 1
            assert sum(abs(a - b) for a, b in zip(nb, p)) == 1


def test_shape_errors():
    with pytest.raises(ValueError):
        sp.Space(sp.OP_CONV, (1, 0, 4, 4, 1, 3, 3, 1, 1))
    with pytest.raises(ValueError):
        sp.Space(sp.OP_CONV, (1, 1, 2, 2, 1, 5, 5, 1, 0))
    with pytest.raises(ValueError):
        sp.Space(sp.OP_MATMUL, (4, 0, 4))
    with pytest.raises(ValueError):
        sp.Space(3, (4, 4, 4))
    assert sp.Space(sp.OP_MATMUL, (0, 4, 4)).size() > 0     # empty output is a legal shape
    assert math.prod(sp.Space(sp.OP_CONV, (0, 2, 4, 4, 2, 3, 3, 1, 1)).sizes) > 0
