"""Seeded input generator: determinism, rounding to the storage formats, shapes."""
import numpy as np
import pytest
import torch

from paper_2609_16389_amd import workloads as wl


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(0, 1, 100000), rng.uniform(-1e30, 1e30, 1000),
                        rng.normal(0, 1e-30, 1000), [0.0, -0.0, 1.0, 1.00390625, 1.01171875]])
    x32 = x.astype(np.float32)
    ours = wl.to_bits(x32, "bf16")
    ref = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_bf16_ties_round_to_even():
    # 1 + 2^-8 lies halfway between bf16 1.0 (0x3f80) and 1 + 2^-7 (0x3f81): goes to even 0x3f80.
    # 1 + 3*2^-8 lies halfway between 0x3f81 and 0x3f82: goes to even 0x3f82.
    got = wl.to_bits(np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8]), "bf16")
    assert got.tolist() == [0x3F80, 0x3F82]


def test_fp16_uses_ieee_half():
    got = wl.to_bits(np.array([1.0, -2.0, 65504.0, 2.0 ** -24]), "fp16")
    assert got.tolist() == [0x3C00, 0xC000, 0x7BFF, 0x0001]


@pytest.mark.parametrize("name", sorted(wl.WORKLOADS))
def test_workload_table(name):
    w = wl.WORKLOADS[name]
    assert w.flops == 2 * w.M * w.N * w.K
    assert w.dtype in ("bf16", "fp16")


def test_seeded_inputs_are_deterministic_and_ordered():
    A1, B1 = wl.make_inputs(64, 48, 32, "bf16", "uniform", seed=2)
    A2, B2 = wl.make_inputs(64, 48, 32, "bf16", "uniform", seed=2)
    assert np.array_equal(A1, A2) and np.array_equal(B1, B2)
    # A is drawn before B from one generator
    rng = np.random.default_rng(2)
    a = rng.uniform(-1, 1, size=(64, 32))
    b = rng.uniform(-1, 1, size=(32, 48))
    assert np.array_equal(A1, wl.to_bits(a, "bf16")) and np.array_equal(B1, wl.to_bits(b, "bf16"))
    assert wl.sha256_bits(A1, B1) == wl.sha256_bits(A2, B2)


def test_normal_fp16_has_subnormals():
    A, _ = wl.make_inputs(512, 1, 512, "fp16", "normal", seed=3, param=0.02)
    e = (A >> 10) & 31
    frac = np.count_nonzero((e == 0) & ((A & 1023) != 0)) / A.size
    assert 0.0005 < frac < 0.01


def test_int_inputs_exact():
    A, B = wl.make_int_inputs(20, 30, 40, "fp16", seed=1)
    Av = A.view(np.float16).astype(np.float64)
    assert np.all(Av == np.round(Av)) and Av.min() >= -8 and Av.max() <= 8
