"""Balanced k-means of neuron feature rows -- CPU oracle in fp64.
TEST INFRASTRUCTURE ONLY (tests, the smoke check and the CPU-baseline leg of
the benchmark); it shares nothing with the HIP library.

MoEfication's clustering step (Sec. 2.2): the d_ff intermediate neurons are
grouped by balanced k-means (constrained k-means, the method the paper cites)
into E clusters of exactly d_ff / E neurons, which gives the permutation Pi of
Eq. (permuted_weights).  Lloyd's iteration with the balance constraint:

  assignment: minimise sum_i ||x_i - mu_a(i)||^2 over assignments a with
              |a^-1(j)| = m = n / k for every cluster j -- a transportation
              problem, solved exactly here as a linear assignment over the
              n x n matrix in which every cluster's column is repeated m times
              (scipy.optimize.linear_sum_assignment);
  update:     mu_j = mean of the rows assigned to j;
  Pi:         clusters in index order, each cluster's rows ascending.

The feature rows, the initial centroids and the iteration count are inputs
(any random draw happens outside).  Squared distances are written out as
explicit differences.
"""
import numpy as np
from scipy.optimize import linear_sum_assignment


def sq_dist(X, mu):
    """[n, k] squared Euclidean distances, fp64, from explicit differences."""
    X = np.asarray(X, np.float64)
    mu = np.asarray(mu, np.float64)
    return ((X[:, None, :] - mu[None, :, :]) ** 2).sum(axis=-1)


def balanced_assign(X, mu):
    """Optimal balanced assignment for fixed centroids: (a [n] int64, cost)."""
    S = sq_dist(X, mu)
    n, k = S.shape
    if n % k:
        raise ValueError("n must be a multiple of k")
    m = n // k
    rows, cols = linear_sum_assignment(np.repeat(S, m, axis=1))
    a = np.empty(n, np.int64)
    a[rows] = cols // m
    return a, float(S[np.arange(n), a].sum())


def update(X, a, k):
    """Centroids: the mean of each cluster's rows (fp64)."""
    X = np.asarray(X, np.float64)
    return np.stack([X[a == j].mean(axis=0) for j in range(k)])


def perm_from(a, k):
    """Pi as a row index list: cluster 0's rows ascending, then cluster 1's, ..."""
    return np.concatenate([np.nonzero(a == j)[0] for j in range(k)]).astype(np.int32)


def balanced_kmeans(X, init_mu, iters):
    """iters Lloyd iterations from init_mu.  Returns dict(assign, perm, centroids
    (after the last update), objective [iters]: the assignment cost of each
    iteration, computed with the centroids that assignment used)."""
    mu = np.asarray(init_mu, np.float64)
    k = mu.shape[0]
    objective = []
    a = None
    for _ in range(iters):
        a, cost = balanced_assign(X, mu)
        objective.append(cost)
        mu = update(X, a, k)
    return dict(assign=a, perm=perm_from(a, k), centroids=mu, objective=np.array(objective))
