"""OBD saliency and the global keep-mask (test infrastructure only).

Section 4.1 (background): removing weight i costs rho_i = theta_i^2 / (2 [F^-1]_ii)
under the local quadratic model; the lowest saliencies are pruned first, and
the pruning is global over all blocks. The keep-mask marks the k largest
saliencies, ties broken by the lower coordinate index, all in float64.
"""

import numpy as np


def scores(theta, diag):
    """rho_j = theta_j^2 / (2 * diag_j) in float64."""
    t = np.asarray(theta, dtype=np.float64)
    return t * t / (2.0 * np.asarray(diag, dtype=np.float64))


def keep_mask(s, keep):
    """uint8 mask with ones on the ``keep`` largest scores (score desc, index asc)."""
    s = np.asarray(s, dtype=np.float64)
    d = s.shape[0]
    order = np.lexsort((np.arange(d), -s))  # primary: -s ascending; secondary: index
    mask = np.zeros(d, np.uint8)
    mask[order[:keep]] = 1
    return mask


def keep_count(d, keep_frac):
    """Number of kept coordinates for a keep fraction (floor of d * frac)."""
    return int(np.floor(d * keep_frac))
