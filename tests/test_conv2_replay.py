"""The channel-quad conv kernel's index arithmetic, replayed on the CPU.

`tests/replay/conv2_replay.cpp` walks every workgroup, thread and lane of
conv_mfma2 (conv mfma 2: rectangular tiles, conv mfma 3: band tiles) with the
launch geometry of the library's own set-up, and checks what a GPU run cannot
report: global reads inside their tensors, LDS accesses inside the geometry's
LDS size and inside their buffer, 16-byte copies and stores on 16-byte
boundaries, no unwritten LDS word feeding a kept output, every output written
once per split, one arrival per non-empty split on every output tile, a
workgroup order that is a permutation, and the fp64 result of the replayed
multiply-adds equal to a direct convolution.  It pins the geometry (LDS size,
grid, split rows) against the kernel's own addressing, from the side the
oracle's hand-worked pins do not cover.

Shapes: bands crossing image boundaries, several images per band, strides 2,
3 input channels, no padding, 5x5 filters, W not a multiple of 4, ragged K.
Points: sampled valid mfma 2 and 3 points of each shape; a third of them also
replayed with both operands 4 bytes off a 16-byte boundary.  Split shapes:
batch-1 layers with many channels and few output pixels, replayed at 16 and
32 reduction splits only (including splits left empty by the chunk count).
"""
import os
import random
import shutil
import subprocess

import pytest

from oracle import space as sp

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

SHAPES = [
    (2, 16, 14, 14, 32, 3, 3, 1, 1),
    (3, 8, 7, 7, 16, 3, 3, 1, 1),
    (1, 16, 28, 28, 32, 1, 1, 2, 0),
    (2, 16, 28, 28, 16, 3, 3, 2, 1),
    (2, 3, 20, 20, 16, 7, 7, 2, 3),
    (2, 12, 13, 13, 20, 3, 3, 1, 1),
    (2, 20, 9, 9, 24, 3, 3, 1, 0),
    (4, 8, 6, 6, 16, 3, 3, 1, 1),
    (2, 32, 16, 16, 32, 3, 3, 1, 1),
    (1, 8, 5, 40, 16, 3, 3, 1, 1),
    (2, 4, 30, 30, 17, 5, 5, 1, 2),
]
PER_SHAPE = 14
SPLIT_SHAPES = [
    (1, 128, 7, 7, 32, 3, 3, 1, 1),
    (1, 256, 14, 14, 32, 3, 3, 2, 1),
    (1, 96, 6, 6, 16, 1, 1, 1, 0),
]


@pytest.fixture(scope="module")
def replay_bin(tmp_path_factory):
    gxx = shutil.which("g++")
    if not gxx or not os.path.exists(os.path.join(ROCM, "include", "hip")):
        pytest.skip("needs g++ and the ROCm headers")
    out = str(tmp_path_factory.mktemp("replay") / "conv2_replay")
    subprocess.run([gxx, "-O2", "-std=c++17", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
                    "-I", os.path.join(ROOT, "paper_2406_20037_amd", "csrc"),
                    os.path.join(HERE, "replay", "conv2_replay.cpp"), "-o", out], check=True)
    return out


def _replay(replay_bin, s, sh, pick):
    lines = []
    for i, p in enumerate(pick):
        v, g = s.knobs(p), s.geometry(p)
        row = list(sh) + [v["tk"], v["th"], v["tw"], v["tc"], g["unroll_eff"], v["ks"], v["vec"],
                          1 if i % 3 == 0 else 0, 1 if v["mfma"] == 3 else 0]
        lines.append(" ".join(map(str, row)))
    r = subprocess.run([replay_bin], input="\n".join(lines) + "\n", capture_output=True, text=True,
                       timeout=600)
    out = r.stdout.strip().splitlines()
    assert r.returncode == 0 and len(out) == len(lines) and all(o.startswith("ok") for o in out), (
        f"{lines[len(out) - 1] if out else lines[0]}: {out[-1:] } {r.stderr[-2000:]}")


@pytest.mark.parametrize("sh", SHAPES, ids=["x".join(map(str, s)) for s in SHAPES])
def test_conv2_index_replay(replay_bin, sh):
    s = sp.Space(sp.OP_CONV, sh)
    pts = [p for p in s.valid_points() if s.knobs(p)["mfma"] >= 2]
    assert pts
    rng = random.Random(hash(sh) & 0xFFFF)
    band = [p for p in pts if s.knobs(p)["mfma"] == 3]
    rect = [p for p in pts if s.knobs(p)["mfma"] == 2]
    pick = rng.sample(band, min(PER_SHAPE, len(band))) + rng.sample(rect, min(PER_SHAPE // 2, len(rect)))
    _replay(replay_bin, s, sh, pick)


@pytest.mark.parametrize("sh", SPLIT_SHAPES, ids=["x".join(map(str, s)) for s in SPLIT_SHAPES])
def test_conv2_index_replay_many_splits(replay_bin, sh):
    s = sp.Space(sp.OP_CONV, sh)
    pts = [p for p in s.valid_points() if s.knobs(p)["mfma"] >= 2 and s.knobs(p)["ks"] >= 16]
    # 96 channels make 24 quad chunks: 16 splits leave some empty, 32 are invalid
    assert {s.knobs(p)["ks"] for p in pts} == ({16} if sh[1] == 96 else {16, 32})
    rng = random.Random(hash(sh) & 0xFFFF)
    _replay(replay_bin, s, sh, rng.sample(pts, min(PER_SHAPE, len(pts))))
