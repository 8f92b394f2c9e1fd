"""Shared test helpers (golden-file parsing, small case builders). No method arithmetic."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line


def rand_bits(rng, shape, scale=1.0):
    from workloads import draw_bf16
    return draw_bf16(rng, shape, scale)


# Tolerance of the FP8 variant against exact attention (the fp64 oracle): the
# bf16 bounds (max|err| <= 1e-2 * max|V|, mean|err| <= 1e-3) scaled by the
# ratio of the two formats' unit roundoffs, 2^-4 (e4m3, 4 significant bits)
# over 2^-8 (bf16, 8 significant bits) = 16, and by 2 for the number of
# rounded operands: the FP8 step codes Q, K, V and the weights, the bf16 step
# rounds only Q and the weights (its K and V are the stored values
# themselves).
FP8_MAX_REL_V = 0.32
FP8_MEAN = 3.2e-2


def e4m3_exact_case_values(rng, shape, lo, hi, step):
    """bf16 bit patterns of values step * k, k uniform in [lo/step, hi/step], chosen
    so that both bf16 and e4m3 represent every value exactly."""
    from workloads import f32_to_bf16_bits
    k = rng.integers(int(round(lo / step)), int(round(hi / step)), shape, endpoint=True)
    return f32_to_bf16_bits((k * step).astype(np.float32))
