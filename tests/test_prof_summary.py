"""Host logic of the profile summaries (no GPU): kernel-name shortening and the
pairing of a split schedule's conv dispatches with the reduce launch that
follows each of them in a kernel trace (dispatches of the same instance and
grid that no reduce follows belong to another task)."""
import sqlite3

from paper_2406_20037_amd import prof_summary as ps

CONV = "void ds::(anonymous namespace)::conv_mfma2<2, 8, 2, 1>(ds::Conv2Args)"
RED = "void ds::(anonymous namespace)::split_reduce_kernel<8>(float const*, float*, long)"
OTHER = "void ds::(anonymous namespace)::conv_mfma2<4, 4, 1, 1>(ds::Conv2Args)"


def trace(rows, with_start=True):
    cur = sqlite3.connect(":memory:").cursor()
    if with_start:
        cur.execute("create table kernels(name text, start int, duration int, grid_x int, "
                    "grid_y int, grid_z int)")
        cur.executemany("insert into kernels values (?,?,?,?,?,?)",
                        [(n, s, d, g, 1, 1) for n, s, d, g in rows])
    else:
        cur.execute("create table kernels(name text, duration int, grid_x int, grid_y int, "
                    "grid_z int)")
        cur.executemany("insert into kernels values (?,?,?,?,?)",
                        [(n, d, g, 1, 1) for n, _, d, g in rows])
    return cur


def test_short_names():
    assert ps.short(CONV) == "conv_mfma2<2, 8, 2, 1>"
    assert ps.short(RED) == "split_reduce_kernel<8>"


def test_reduce_paired_with_the_dispatch_before_it():
    rows = [(CONV, 0, 590, 819200), (RED, 600, 40, 1048576),
            (OTHER, 650, 500, 802816), (RED, 1200, 100, 1048576),   # another task's reduce
            (CONV, 2000, 595, 819200), (RED, 2600, 45, 1048576),
            (CONV, 3000, 597, 409600), (RED, 3600, 70, 1048576)]    # other grid
    rows += [(CONV, 4000, 70, 819200), (OTHER, 4100, 500, 802816)]   # same grid, no reduce
    cur = trace(rows)
    want = [(590, 40), (595, 45)]
    assert ps.paired_reduce(cur, "conv_mfma2<2, 8, 2, 1>", 819200, "split_reduce_kernel<8>") == want
    # rows inserted out of time order pair the same way
    cur = trace(list(reversed(rows)))
    assert ps.paired_reduce(cur, "conv_mfma2<2, 8, 2, 1>", 819200, "split_reduce_kernel<8>") == want


def test_no_start_times_gives_no_pairs():
    cur = trace([(CONV, 0, 590, 819200), (RED, 600, 40, 1048576)], with_start=False)
    assert ps.paired_reduce(cur, "conv_mfma2<2, 8, 2, 1>", 819200, "split_reduce_kernel<8>") == []


def test_code_digest_ignores_comments_not_code(tmp_path):
    a = tmp_path / "a.hip"
    a.write_text("// header\nint f(int x) {\n    return x + 1;   /* one */\n}\n")
    d0 = ps.code_digest([a])
    a.write_text("// header, reworded\n/* a block\n   comment */\nint f(int x) {\n  return x + 1;\n}\n")
    assert ps.code_digest([a]) == d0
    a.write_text("int f(int x) {\n    return x + 2;\n}\n")
    assert ps.code_digest([a]) != d0
    # file boundaries count: the same files in another order are another digest
    b = tmp_path / "b.hip"
    b.write_text("")
    assert ps.code_digest([a, b]) != ps.code_digest([b, a])


def test_traffic_key_band_tiles_by_pixel_count():
    sh = (16, 256, 56, 56, 256, 3, 3, 1, 1)
    a = ps.traffic_key("conv_mfma2<4, 4, 1, 1, 4>",
                       "tk=64,th=64,tw=4,tc=4,unroll=16,lds=1,ks=4,mfma=3,vec=4", sh)
    b = ps.traffic_key("conv_mfma2<4, 4, 1, 1, 4>",
                       "tk=64,th=8,tw=32,tc=4,unroll=0,lds=1,ks=4,mfma=3,vec=4", sh)
    assert a == b and "npx=256" in a and "th=" not in a and "*" in a
    # rectangular tiles keep th and tw: the same product is another tile
    c = ps.traffic_key("conv_mfma2<4, 4, 1, 1, 4>",
                       "tk=64,th=8,tw=32,tc=4,unroll=0,lds=1,ks=1,mfma=2,vec=4", sh)
    d = ps.traffic_key("conv_mfma2<4, 4, 1, 1, 4>",
                       "tk=64,th=16,tw=16,tc=4,unroll=0,lds=1,ks=1,mfma=2,vec=4", sh)
    assert c != d and "th=8,tw=32" in c
