"""Pins for the oracle's bf16 emulation and draft-initialisation generator."""
import os

import numpy as np
import pytest
import torch

from oracle.jacobi import GOLDEN, MASK64, pad_id, splitmix64
from oracle.numerics import bf16_bits_to_float, round_bf16

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_round_bf16_golden_cases():
    for line in open(os.path.join(GOLD, "bf16_rne.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        src, want = line.split()
        x = np.array([eval(src)], dtype=np.float64)
        assert round_bf16(x)[0] == eval(want), line
        assert round_bf16(x.astype(np.float32))[0] == np.float32(eval(want)), line


def test_round_bf16_matches_torch_cast():
    """torch's float32 -> bfloat16 conversion is round-to-nearest-even."""
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(200000) * 10.0 ** rng.integers(-6, 6, 200000)).astype(np.float32)
    # add exact ties: bit 15 set, bits 0..14 clear
    ties = (rng.integers(0, 2**31, 5000).astype(np.uint32) & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    x = np.concatenate([x, ties.view(np.float32)])
    x = x[np.isfinite(x) & (np.abs(x) < 1e30) & (np.abs(x) > 1e-37)]  # normal range
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(round_bf16(x), want)
    # the float64 path agrees on float32-representable inputs
    np.testing.assert_array_equal(round_bf16(x.astype(np.float64)), want.astype(np.float64))


def test_bf16_decode():
    bits = np.array([0x3F80, 0xBF80, 0x4049, 0x0000], dtype=np.uint16)
    np.testing.assert_array_equal(bf16_bits_to_float(bits), [1.0, -1.0, 3.140625, 0.0])


def test_splitmix64_published_vector():
    rows = [l.split() for l in open(os.path.join(GOLD, "splitmix64.txt")) if l[0] != "#"]
    for i, (state, out) in enumerate(rows):
        assert splitmix64((int(state) + i * GOLDEN) & MASK64) == int(out)


def test_pad_id_range_and_spread():
    v = [pad_id(2, p, 1024) for p in range(20000)]
    assert min(v) >= 0 and max(v) < 1024
    counts = np.bincount(v, minlength=1024)
    assert counts.min() > 0            # every id reachable
    assert abs(np.mean(v) - 511.5) < 15
