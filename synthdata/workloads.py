"""Workload shapes (no method arithmetic): the single kernels and the layer
lists whose schedules are tuned.

The paper tunes ONNX-zoo models (Section 3, "Benchmarks"); their graphs and
trained weights are not available here, so the model workloads are the layer
*shapes* of ResNet-50 (torchvision v1.5 layout: the stride sits on the 3x3 of
the first block of a stage) at batch 1 and of VGG-16 at batch 16, with
seeded synthetic values (He-normal weights, N(0,1) inputs).  Kernel time has
no data-dependent control flow, so synthetic values do not change timing.

conv shape = (N, C, H, W, K, R, S, stride, pad); matmul shape = (M, N, K).
"""
from __future__ import annotations

OP_CONV = 1
OP_MATMUL = 2

SINGLE = {
    "conv3x3_c64_56": (OP_CONV, (1, 64, 56, 56, 64, 3, 3, 1, 1)),
    "matmul_1024": (OP_MATMUL, (1024, 1024, 1024)),
    "conv7x7_s2_c3_224": (OP_CONV, (1, 3, 224, 224, 64, 7, 7, 2, 3)),
}


def _c(C, K, H, R, st=1, N=1):
    return (N, C, H, H, K, R, R, st, R // 2)


# (name, op, shape, count in the network)
RESNET50 = [
    ("stem_7x7_3_64", OP_CONV, _c(3, 64, 224, 7, 2), 1),
    ("s1_1x1_64_64", OP_CONV, _c(64, 64, 56, 1), 1),
    ("s1_3x3_64_64", OP_CONV, _c(64, 64, 56, 3), 3),
    ("s1_1x1_64_256", OP_CONV, _c(64, 256, 56, 1), 4),
    ("s1_1x1_256_64", OP_CONV, _c(256, 64, 56, 1), 2),
    ("s2_1x1_256_128", OP_CONV, _c(256, 128, 56, 1), 1),
    ("s2_3x3_128_128_s2", OP_CONV, _c(128, 128, 56, 3, 2), 1),
    ("s2_1x1_128_512", OP_CONV, _c(128, 512, 28, 1), 4),
    ("s2_ds_256_512_s2", OP_CONV, _c(256, 512, 56, 1, 2), 1),
    ("s2_1x1_512_128", OP_CONV, _c(512, 128, 28, 1), 3),
    ("s2_3x3_128_128", OP_CONV, _c(128, 128, 28, 3), 3),
    ("s3_1x1_512_256", OP_CONV, _c(512, 256, 28, 1), 1),
    ("s3_3x3_256_256_s2", OP_CONV, _c(256, 256, 28, 3, 2), 1),
    ("s3_1x1_256_1024", OP_CONV, _c(256, 1024, 14, 1), 6),
    ("s3_ds_512_1024_s2", OP_CONV, _c(512, 1024, 28, 1, 2), 1),
    ("s3_1x1_1024_256", OP_CONV, _c(1024, 256, 14, 1), 5),
    ("s3_3x3_256_256", OP_CONV, _c(256, 256, 14, 3), 5),
    ("s4_1x1_1024_512", OP_CONV, _c(1024, 512, 14, 1), 1),
    ("s4_3x3_512_512_s2", OP_CONV, _c(512, 512, 14, 3, 2), 1),
    ("s4_1x1_512_2048", OP_CONV, _c(512, 2048, 7, 1), 3),
    ("s4_ds_1024_2048_s2", OP_CONV, _c(1024, 2048, 14, 1, 2), 1),
    ("s4_1x1_2048_512", OP_CONV, _c(2048, 512, 7, 1), 2),
    ("s4_3x3_512_512", OP_CONV, _c(512, 512, 7, 3), 2),
    ("fc_2048_1000", OP_MATMUL, (1, 1000, 2048), 1),
]

VGG16 = [
    (f"L{i + 1}_{C}_{K}_{H}", OP_CONV, _c(C, K, H, 3, 1, N=16), 1)
    for i, (C, K, H) in enumerate([
        (3, 64, 224), (64, 64, 224), (64, 128, 112), (128, 128, 112), (128, 256, 56),
        (256, 256, 56), (256, 256, 56), (256, 512, 28), (512, 512, 28), (512, 512, 28),
        (512, 512, 14), (512, 512, 14), (512, 512, 14)])
]

BASE_SEED = 240620037


def sampler_seed(config: int, layer: int = 0) -> int:
    return BASE_SEED + 1000 * config + layer


def flops(op, shape) -> int:
    if op == OP_CONV:
        N, C, H, W, K, R, S, st, pd = shape
        P = (H + 2 * pd - R) // st + 1
        Q = (W + 2 * pd - S) // st + 1
        return 2 * N * K * P * Q * C * R * S
    M, N, K = shape
    return 2 * M * N * K


def algorithmic_bytes(op, shape) -> int:
    """Compulsory fp32 traffic: inputs read once, output written once."""
    if op == OP_CONV:
        N, C, H, W, K, R, S, st, pd = shape
        P = (H + 2 * pd - R) // st + 1
        Q = (W + 2 * pd - S) // st + 1
        return 4 * (N * C * H * W + K * C * R * S + N * K * P * Q)
    M, N, K = shape
    return 4 * (M * K + K * N + M * N)
