"""The tolerance rule of the parity tests (host only): the absolute bound
covers entries below |ref| = 4, where a bf16 output can meet it, and the
relative bound covers every entry."""
import numpy as np
import pytest

from parity_util import assert_parity, parity_stats
from paper_2504_09345_amd import workloads as W


def _bf16(x):
    return W.bf16_bits_to_f32(W.f32_to_bf16_bits(np.asarray(x, np.float32)))


def test_correctly_rounded_large_entry_passes():
    # 4.013821 rounds to 4.0 in bf16 (values from 4 on are 1/32 apart)
    ref = np.array([[[4.013821, 1.0, -0.5, 0.25]]])
    got = _bf16(ref)
    st = parity_stats(got, ref)
    assert st["max_abs_all"] > 1e-2 and st["max_abs"] < 1e-2
    assert_parity(got, ref, strict=False)


def test_small_entry_off_by_more_than_the_absolute_bound_fails():
    ref = np.array([[[3.0, 3.0, 3.0, 3.0]]])
    got = ref + np.array([[[0.011, 0.0, 0.0, 0.0]]])
    with pytest.raises(AssertionError):
        assert_parity(got, ref, strict=False)


def test_large_entry_off_by_more_than_the_relative_bound_fails():
    ref = np.array([[[6.0, 6.0, 6.0, 6.0]]])
    got = ref + np.array([[[0.04, 0.0, 0.0, 0.0]]])  # 6.7e-3 relative
    with pytest.raises(AssertionError):
        assert_parity(got, ref, strict=False)


def test_every_bf16_rounding_of_unit_scale_outputs_passes():
    rng = np.random.default_rng(3)
    ref = rng.normal(0, 1.5, (64, 8, 128)).astype(np.float64)
    assert_parity(_bf16(ref).astype(np.float64), ref, strict=False)
