"""Oracle for the BASE layer gate (Sec. 3.1, BASE Layer): balanced assignment.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The BASE layer assigns each of N tokens to one expert so that the summed score
x_i . w_{a_i} is largest while every expert receives exactly N / E tokens (a
linear assignment problem).  Here the score of token i for expert e is the gate
logit L[i, e] = x_i . W[:, e] (+ bias), so the expert embeddings are the gate's
columns.  Readings: R22 N must be a multiple of E; R23 a kept token's weight is
sigmoid(L[i, a_i]), the scaling of the BASE layer's expert output.

The optimum is computed exactly by the library routine for the assignment
problem (scipy's linear_sum_assignment) on the N x N matrix that repeats each
expert's column N / E times.  Several assignments can be optimal; the optimal
total score is unique.
"""

import numpy as np
from scipy.optimize import linear_sum_assignment


def base_assign(L):
    """Optimal balanced assignment for scores L [N, E] (float64).

    Returns (ids [N] int32, total score float64).
    """
    L = np.asarray(L, dtype=np.float64)
    N, E = L.shape
    if N % E != 0:
        raise ValueError("the BASE layer needs N to be a multiple of E")
    c = N // E
    cost = np.repeat(L, c, axis=1)          # column e * c + j is copy j of expert e
    rows, cols = linear_sum_assignment(cost, maximize=True)
    ids = np.empty(N, dtype=np.int32)
    ids[rows] = cols // c
    return ids, float(L[np.arange(N), ids].sum())


def base_weights(L, ids):
    """Weight of each token's expert (R23): sigmoid of its score, float64 [N]."""
    L = np.asarray(L, dtype=np.float64)
    v = L[np.arange(L.shape[0]), np.asarray(ids)]
    return 1.0 / (1.0 + np.exp(-v))
