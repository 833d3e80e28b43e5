"""Pins of the oracle's prediction values and ensemble mean (Section 3.5: an
ensemble averages its members' predictions, probabilities for classification)
against library routines and hand-computed values."""
import math

import numpy as np
import torch

from oracle.online import ensemble_predict
from oracle.pack import prediction, prediction_values


def test_regression_values_are_the_outputs():
    Y = np.array([[1.5], [-2.0], [0.0]])
    np.testing.assert_array_equal(prediction_values(Y, "reg"), Y)


def test_binary_values_hand_computed_and_torch_sigmoid():
    # sigma(0) = 1/2, sigma(ln 3) = 3/4, sigma(-ln 3) = 1/4
    Y = np.array([[0.0], [math.log(3.0)], [-math.log(3.0)]])
    np.testing.assert_allclose(prediction_values(Y, "bin")[:, 0], [0.5, 0.75, 0.25], rtol=0, atol=1e-15)
    Z = np.random.default_rng(0).normal(0, 4, (50, 1))
    np.testing.assert_allclose(prediction_values(Z, "bin"), torch.sigmoid(torch.from_numpy(Z)).numpy(),
                               rtol=1e-14, atol=0)


def test_multiclass_values_hand_computed_and_torch_softmax():
    # logits (0, ln 3) -> (1/4, 3/4); (ln 2, ln 2, ln 4) -> (1/4, 1/4, 1/2)
    Y = np.array([[0.0, math.log(3.0), -np.inf]])
    np.testing.assert_allclose(prediction_values(Y, "multi"), [[0.25, 0.75, 0.0]], rtol=0, atol=1e-15)
    Y = np.array([[math.log(2.0), math.log(2.0), math.log(4.0)]]) + 100.0  # shift invariance, no overflow
    np.testing.assert_allclose(prediction_values(Y, "multi"), [[0.25, 0.25, 0.5]], rtol=0, atol=1e-15)
    # rows are samples, columns classes (N != d_out so a wrong axis cannot pass)
    Z = np.random.default_rng(1).normal(0, 3, (37, 10))
    P = prediction_values(Z, "multi")
    np.testing.assert_allclose(P, torch.softmax(torch.from_numpy(Z), dim=1).numpy(), rtol=1e-13, atol=1e-16)
    np.testing.assert_allclose(P.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    # the candidate value of a row is its true class's probability
    lab = np.random.default_rng(2).integers(0, 10, 37)
    np.testing.assert_array_equal(prediction(Z, lab, "multi"), P[np.arange(37), lab])


def test_ensemble_predict_is_the_mean_over_instances():
    # three instances with constant predictions 1, 2, 6 (rows 2, outputs 3): mean 3
    consts = {"a": 1.0, "b": 2.0, "c": 6.0}
    out = ensemble_predict(["a", "b", "c"], lambda inst: np.full((2, 3), consts[inst]))
    np.testing.assert_array_equal(out, np.full((2, 3), 3.0))
    # a repeated instance counts twice: (1 + 1 + 6) / 3
    out = ensemble_predict(["a", "a", "c"], lambda inst: np.full((2, 3), consts[inst]))
    np.testing.assert_allclose(out, np.full((2, 3), 8.0 / 3.0), rtol=1e-15)
    # per element, not over rows or outputs
    rng = np.random.default_rng(3)
    vals = {i: rng.normal(size=(4, 10)) for i in range(5)}
    out = ensemble_predict(list(range(5)), lambda i: vals[i])
    np.testing.assert_allclose(out, sum(vals.values()) / 5.0, rtol=1e-14)
    assert out.shape == (4, 10)
