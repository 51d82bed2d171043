"""Consensus distance of the workers' models (test infrastructure only).

Section 4's analysis tracks how far the workers' iterates are from their
average: the consensus distance, the mean over workers of the squared
Euclidean distance to the average.  Here it is taken over the models
themselves with the uniform average as centre,

    Xi = (1/n) * sum_i ||x_i - xbar||^2,   xbar = (1/n) * sum_i x_i,

together with the largest coordinate deviation max_{i,c} |x_ic - xbar_c|.
(The analysis weighs an extended state of delayed copies by the stationary
vector of its mixing matrix; on the models alone, with every worker weighted
alike, that weighting is the uniform one.)  Plain numpy in float64: a
reader can check it against the definition by eye.

Only ``tests/`` may import this module; the product library never does.
"""
from __future__ import annotations

import numpy as np


def consensus_distance(x) -> tuple[float, float]:
    """(Xi, max deviation) of the rows of x ([n, d], any float type), in float64."""
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[0]
    if x.size == 0:
        return 0.0, 0.0
    xbar = x.sum(axis=0) / n
    dev = x - xbar
    return float((dev * dev).sum() / n), float(np.abs(dev).max())
