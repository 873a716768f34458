"""Router: logits, top-k and routing weights (oracle; test infrastructure only).

The paper's introduction and Native Serving Path section say only that the
router selects each token's routed experts, and that this selection is what
drives materialisation.  Readings used here:

* logits z = x W_r with W_r stored [hidden, n_experts] row-major, fp32 inputs,
  evaluated exactly in fp64;
* experts ranked by (-z_e, e): higher logit first, the lower id wins exact ties;
  the routed set is the first k, returned in that order;
* weights are the softmax restricted to the routed set (softmax over all
  experts followed by renormalisation over the k chosen ones is the same);
* the decision gap z_(k) - z_(k+1) (k-th minus (k+1)-th largest) flags
  near-ties, where either set is accepted.
"""
import numpy as np


def logits(x, router_w):
    """z [T, E] fp64 from x [T, H] and W_r [H, E] (both taken as given fp32 values)."""
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    return x @ np.asarray(router_w, dtype=np.float64)


def rank(z_row):
    """Expert ids ordered by (-z_e, e)."""
    z_row = np.asarray(z_row, dtype=np.float64)
    return np.lexsort((np.arange(z_row.size), -z_row))


def topk(z, k):
    """(idx [T,k] int32 in rank order, w [T,k] fp64, gap [T] fp64)."""
    z = np.atleast_2d(z)
    T, E = z.shape
    idx = np.empty((T, k), np.int32)
    w = np.empty((T, k), np.float64)
    gap = np.full(T, np.inf)
    for t in range(T):
        order = rank(z[t])
        sel = order[:k]
        idx[t] = sel
        zs = z[t, sel]
        ex = np.exp(zs - zs.max())
        w[t] = ex / ex.sum()
        if k < E:
            gap[t] = z[t, order[k - 1]] - z[t, order[k]]
    return idx, w, gap


def route(x, router_w, k):
    """Routes of a layer call: (idx, w, gap) for tokens x [T, H]."""
    return topk(logits(x, router_w), k)
