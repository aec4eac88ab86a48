"""Seeded synthetic inputs shared by the tests, the smoke check and the
benchmark. No arithmetic of the method lives here: only random draws with
the shapes and distributions of the workloads.

Images are N(0,1) float32 in NCHW, labels uniform integers in [0, C): they
stand in for CIFAR-100 (32x32x3, 100 classes) and ImageNet (3x224x224 after
cropping, 1000 classes), whose pixel values do not change the work done.
"""
import numpy as np


def images(seed, n, h, w):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, 3, h, w), dtype=np.float32)


def labels(seed, n, num_classes):
    rng = np.random.default_rng(seed + 1_000_003)
    return rng.integers(0, num_classes, n, dtype=np.int32)


def tensor(seed, shape, scale=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(scale)).astype(np.float32)


# The training configurations: (name, arch, classes, precision, [(N, H)], lr)
CONFIGS = {
    "tiny_fp32": ("tiny", 10, "fp32", [(8, 16)]),
    "cifar_fp32_b128_32": ("cifar", 100, "fp32", [(128, 32)]),
    "cifar_cyclic_fp32": ("cifar", 100, "fp32", [(512, 16), (256, 24), (128, 32)]),
    "imagenet_bf16_b256_224": ("imagenet", 1000, "bf16", [(256, 224)]),
    "imagenet_hybrid_bf16": ("imagenet", 1000, "bf16", [(1024, 128), (640, 160), (448, 192), (256, 224)]),
}
SMALL_WORKER_BATCH = 64
