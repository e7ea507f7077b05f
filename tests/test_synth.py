"""The seeded generator shared by the oracle and the GPU path."""
import os

import numpy as np
import pytest
import torch

import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def _kat_rows():
    rows = []
    with open(os.path.join(HERE, "golden", "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            v = [int(x, 16) for x in line.split()]
            rows.append((tuple(v[0:4]), tuple(v[4:6]), tuple(v[6:10])))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat_rows())
def test_philox_known_answers(ctr, key, expect):
    assert synth.philox4x32(ctr, key, 10) == expect


def test_normal_moments_and_determinism():
    a = synth.normal(7, 123, (2_000_000,), 0.0, 1.0, "f32")
    b = synth.normal(7, 123, (2_000_000,), 0.0, 1.0, "f32")
    assert np.array_equal(a, b)
    assert abs(a.mean()) < 3e-3
    assert abs(a.std() - 1.0) < 3e-3
    assert abs((a.astype(np.float64) ** 4).mean() - 3.0) < 3e-2  # normal kurtosis
    # the standard normal CDF at 1 is 0.8413
    assert abs((a < 1.0).mean() - 0.841344746) < 2e-3
    c = synth.normal(8, 123, (1000,), 0.0, 1.0, "f32")
    assert not np.array_equal(a[:1000], c)


def test_offset_fill_matches_full_draw():
    full = synth.normal(3, 9, (10007,), 0.5, 2.0, "f32")
    part = np.empty(5000, np.float32)
    synth.fill_normal(3, 9, 5000, 0.5, 2.0, "f32", part.ctypes.data, offset=4097)
    assert np.array_equal(part, full[4097:9097])


def test_fp16_rounding_is_round_to_nearest_even():
    f32 = synth.normal(11, 1, (30_000,), 0.0, 3.0, "f32")
    edge = np.array([65504.0, 65519.0, 65520.0, 1e6, 6e-8, 2.0 ** -25, 2.0 ** -24, 3 * 2.0 ** -26,
                     2.0 ** -14, 2.0 ** -14 * (1 - 2.0 ** -11), -0.0, 1e-30, 1.0 + 2.0 ** -11,
                     1.0 + 3 * 2.0 ** -11, np.inf, -np.inf], np.float32)
    xs = np.concatenate([f32[::7], f32[::7] * 1e-5, f32[::7] * 3e4, edge])
    got = np.array([synth.f32_to_f16_bits(float(x)) for x in xs], np.uint16)
    with np.errstate(over="ignore"):
        ref = xs.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref)


def test_bf16_rounding_is_round_to_nearest_even():
    f32 = synth.normal(12, 1, (50_000,), 0.0, 3.0, "f32")
    ref = torch.from_numpy(f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([synth.f32_to_bf16_bits(float(x)) for x in f32], np.uint16)
    assert np.array_equal(got, ref)


def test_storage_draws_are_rounded_float_draws():
    f32 = synth.normal(5, 77, (40_000,), 0.0, 0.02, "f32")
    f16 = synth.normal(5, 77, (40_000,), 0.0, 0.02, "f16")
    bf = synth.normal(5, 77, (40_000,), 0.0, 0.02, "bf16")
    assert np.array_equal(f16, f32.astype(np.float16).view(np.uint16))
    ref = torch.from_numpy(f32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf, ref)


def test_tokens_in_range():
    w = synth.WORKLOADS["opt-1.3b"]
    t = synth.tokens(w)
    assert t.shape == (1, 512)
    assert t.min() >= 2 and t.max() < w.vocab
    t2 = synth.tokens(w)
    assert np.array_equal(t, t2)


def test_workload_sizes_match_stated_model_sizes():
    # parameter totals of the OPT shapes (fp16 bytes): about 2.6, 13.4, 26 and 132 GB
    gb = {n: synth.WORKLOADS[n].storage_bytes() / 1e9 for n in
          ("opt-1.3b", "opt-6.7b", "opt-13b", "opt-66b")}
    assert abs(gb["opt-1.3b"] - 2.63) < 0.05
    assert abs(gb["opt-6.7b"] - 13.3) < 0.2
    assert abs(gb["opt-13b"] - 25.7) < 0.3
    assert abs(gb["opt-66b"] - 131.4) < 1.0
