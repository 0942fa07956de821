"""Brute-force ridge least squares.  TEST INFRASTRUCTURE ONLY (see the
package header).

The test-time-regression objective of Sec. 2.3 (Eq. ttr_obj):

    S_t = argmin_S  1/2 sum_{i<=t} ||S k_i - v_i||^2 + lam/2 ||S||_F^2

solved directly as an ordinary least-squares problem on the stacked system
[K_t; sqrt(lam) I] S^T = [V_t; 0] with numpy's SVD-based `lstsq`, i.e.
without forming the normal equations (Eq. normal_eqs) or any recurrence.
"""
from __future__ import annotations

import numpy as np


def ridge_map(K, V, lam):
    """K (t, dk), V (t, dv) -> S (dv, dk)."""
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    dk = K.shape[1]
    Xa = np.vstack([K, np.sqrt(lam) * np.eye(dk)])
    Ya = np.vstack([V, np.zeros((dk, V.shape[1]))])
    St, *_ = np.linalg.lstsq(Xa, Ya, rcond=None)
    return St.T


def ridge_maps(K, V, lam):
    """The ridge map after every prefix: (T, dv, dk)."""
    return np.stack([ridge_map(K[:t + 1], V[:t + 1], lam)
                     for t in range(K.shape[0])])
