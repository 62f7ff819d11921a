"""Pins of the oracle's several-model functions (Sections 5, 6.2 and 6.3)
against exact arithmetic, independent of the GPU path."""
import numpy as np
import pytest

import oracle
from paper_1605_04809_amd.workloads import CONFIGS, draw_params


def _params(seed, cfg=CONFIGS["tiny"]):
    return draw_params(cfg.replace(seed=seed), np.random.default_rng(seed))


def test_average_of_one_model_is_the_model():
    p = _params(1)
    a = oracle.average_params([p], coef=[1.0])
    for n in oracle.PARAM_FIELDS:
        np.testing.assert_array_equal(a[n], p[n])


def test_average_of_copies_is_the_model():
    p = _params(2)
    for K in (2, 4):  # 1/K exact in binary
        a = oracle.average_params([p] * K)
        for n in oracle.PARAM_FIELDS:
            np.testing.assert_array_equal(a[n], p[n])


def test_average_is_exact_on_small_values():
    names = oracle.PARAM_FIELDS
    x = {n: np.array([1.0, 2.0, -3.0], np.float32) for n in names}
    y = {n: np.array([3.0, 5.0, 1.0], np.float32) for n in names}
    a = oracle.average_params([x, y])
    np.testing.assert_array_equal(a["out_b"], np.array([2.0, 3.5, -1.0], np.float32))
    w = oracle.average_params([x, y], coef=[0.25, 0.75])
    np.testing.assert_array_equal(w["g1_W"], np.array([2.5, 4.25, 0.0], np.float32))


def test_average_bf16_rounds_ties_to_even():
    names = oracle.PARAM_FIELDS
    # bf16 keeps 7 fraction bits: 1 + 2^-8 and 1 + 3*2^-8 are ties.
    x = {n: np.array([1.0, 1.0078125], np.float32) for n in names}
    y = {n: np.array([1.0078125, 1.015625], np.float32) for n in names}
    a = oracle.average_params([x, y], bf16=True)
    np.testing.assert_array_equal(a["att_v"], np.array([1.0, 1.015625], np.float32))
    f = oracle.average_params([x, y], bf16=False)
    np.testing.assert_array_equal(f["att_v"], np.array([1.00390625, 1.01171875], np.float32))


def test_average_is_symmetric_and_between_members():
    p, q, r = _params(3), _params(4), _params(5)
    a = oracle.average_params([p, q, r])
    b = oracle.average_params([r, p, q])
    for n in oracle.PARAM_FIELDS:
        np.testing.assert_array_equal(a[n], b[n])
        lo = np.minimum(np.minimum(p[n], q[n]), r[n])
        hi = np.maximum(np.maximum(p[n], q[n]), r[n])
        assert np.all(a[n] >= lo - 1e-7) and np.all(a[n] <= hi + 1e-7)


def test_log_linear_weights():
    lp = np.array([[-1.0, -2.0], [-3.0, -0.5]])
    np.testing.assert_array_equal(oracle.log_linear(lp), [-4.0, -2.5])
    np.testing.assert_array_equal(oracle.log_linear(lp, [0.5, 2.0]), [-6.5, -2.0])
