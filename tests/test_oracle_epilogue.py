"""Pins of the oracle's forward epilogue (per-channel affine, ReLU and the
batch-normalization statistics of the stored output; arXiv 2204.01701
section 4.2, model construction: batch normalization after the quadratic
layers, an activation in deeper networks): a hand-worked example, PyTorch's
batch_norm in evaluation mode (the folded affine) and in training mode (the
statistics), and relu."""
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden():
    vals = {}
    with open(os.path.join(GOLDEN, "epilogue_worked_example.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, *v = line.split()
            vals[k] = np.array([float(t) for t in v])
    return vals


def test_epilogue_worked_example():
    g = _golden()
    y = g["y"].reshape(2, 2, 1, 2)
    yo, s, s2 = oracle.epilogue(y, g["scale"], g["shift"], relu=True)
    assert np.array_equal(yo.ravel(), g["yo"])
    assert np.array_equal(s, g["sum"]) and np.array_equal(s2, g["sumsq"])
    yo, s, s2 = oracle.epilogue(y)
    assert np.array_equal(yo, y)
    assert np.array_equal(s, g["plain_sum"]) and np.array_equal(s2, g["plain_sumsq"])


@pytest.mark.parametrize("shape", [(3, 5, 4, 6), (7, 9), (1, 2, 1, 1)])
@pytest.mark.parametrize("relu", [False, True])
def test_affine_is_eval_mode_batch_norm(shape, relu):
    """scale = gamma / sqrt(var + eps), shift = beta - mean scale: F.batch_norm with running statistics."""
    rng = np.random.default_rng(11)
    y = rng.standard_normal(shape)
    O = shape[1]
    rm, rv = rng.standard_normal(O), rng.uniform(0.5, 2.0, O)
    gamma, beta, eps = rng.standard_normal(O), rng.standard_normal(O), 1e-5
    scale = gamma / np.sqrt(rv + eps)
    shift = beta - rm * scale
    yo, _, _ = oracle.epilogue(y, scale, shift, relu=relu)
    t = torch.from_numpy(y)
    ref = F.batch_norm(t, torch.from_numpy(rm), torch.from_numpy(rv), torch.from_numpy(gamma),
                       torch.from_numpy(beta), training=False, eps=eps)
    if relu:
        ref = F.relu(ref)
    np.testing.assert_allclose(yo, ref.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", [(4, 6, 5, 3), (16, 10)])
@pytest.mark.parametrize("relu", [False, True])
def test_statistics_give_training_mode_batch_norm(shape, relu):
    """mean = sum / M and the biased variance sumsq / M - mean^2 equal torch's, and
    normalizing with them reproduces F.batch_norm in training mode."""
    rng = np.random.default_rng(12)
    y = rng.standard_normal(shape) * 3 + 1
    axes = (0,) + tuple(range(2, len(shape)))
    M = int(np.prod([shape[a] for a in axes]))
    scale = rng.standard_normal(shape[1]) if relu else None
    yo, s, s2 = oracle.epilogue(y, scale, None, relu=relu)
    t = torch.from_numpy(yo)
    var, mean = torch.var_mean(t, dim=axes, unbiased=False)
    np.testing.assert_allclose(s / M, mean.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(s2 / M - (s / M) ** 2, var.numpy(), rtol=1e-10, atol=1e-12)
    eps = 1e-5
    ref = F.batch_norm(t, None, None, training=True, eps=eps)
    bshape = (1, -1) + (1,) * (len(shape) - 2)
    mine = (yo - (s / M).reshape(bshape)) / np.sqrt((s2 / M - (s / M) ** 2).reshape(bshape) + eps)
    np.testing.assert_allclose(mine, ref.numpy(), rtol=1e-9, atol=1e-9)


def test_relu_alone_is_library_relu():
    rng = np.random.default_rng(13)
    y = rng.standard_normal((2, 3, 4, 4))
    yo, s, _ = oracle.epilogue(y, relu=True)
    assert np.array_equal(yo, F.relu(torch.from_numpy(y)).numpy())
    assert np.allclose(s, F.relu(torch.from_numpy(y)).sum(dim=(0, 2, 3)).numpy(), rtol=1e-13)
