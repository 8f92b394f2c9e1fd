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
