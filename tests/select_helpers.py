"""Retained-axis selection for very large Lambda in the tests: the same
order as the oracle's full sort (Lambda desc, flat index asc), found with a
partition for the m-th largest value and a sort of the candidates only.
Pinned against oracle.select_retained in test_oracle_pins.py."""
import numpy as np

import oracle as O


def select_large(lam: np.ndarray, damping: float, m: int) -> O.Retained:
    flat_lam = np.asarray(lam, np.float64).ravel()
    d_in = lam.shape[1]
    thr = np.partition(flat_lam, flat_lam.size - m)[flat_lam.size - m]
    above = np.flatnonzero(flat_lam > thr)
    ties = np.flatnonzero(flat_lam == thr)[: m - above.size]
    cand = np.concatenate([above, ties])
    order = np.lexsort((cand, -flat_lam[cand]))
    flat = cand[order].astype(np.int64)
    lam_r = flat_lam[flat]
    return O.Retained(flat=flat, j=flat // d_in, k=flat % d_in, lam=lam_r,
                      w=1.0 / np.sqrt(lam_r + damping))


def restrict(ret: O.Retained, coords: np.ndarray):
    """The retained axes at positions `coords`, with row and column indices
    relabelled to positions in the sorted distinct rows J and columns K they
    use (so the oracle needs only Q_S[:, J] and Q_A[:, K])."""
    J, jinv = np.unique(ret.j[coords], return_inverse=True)
    K, kinv = np.unique(ret.k[coords], return_inverse=True)
    sub = O.Retained(flat=ret.flat[coords], j=jinv.astype(np.int64), k=kinv.astype(np.int64),
                     lam=ret.lam[coords], w=ret.w[coords])
    return sub, J, K
