"""The benchmark's work accounting against the oracle.

`workload.visible_pairs` counts the (row, key) pairs the causal mask over
compressed positions (Sec. III-B, Eq. 5) lets through; it sets the prefill's
algorithmic FLOPs.  Here the count is read off the oracle's attention instead
of its formula: with q = 0 every visible key gets the same weight, and with
one-hot value rows (V[c] = e_c) each output row is 1/n_vis(p) on exactly the
visible keys, so the nonzeros of row p are its visible keys.
"""
import numpy as np
import pytest

import oracle
from paper_2607_06827_amd.workload import visible_pairs


@pytest.mark.parametrize("P,T,N,w", [(3, 7, 2, 4), (0, 5, 0, 2), (4, 0, 3, 4), (2, 9, 1, 3),
                                     (1, 8, 0, 4), (5, 3, 4, 1), (0, 1, 2, 4)])
def test_visible_pairs_matches_oracle_mask(P, T, N, w):
    layer, l0 = 1, 0  # compressed layer
    L = oracle.compressed_len(P, T, N, w, layer, l0)
    D = max(L, 1)
    S = P + T + N
    q = np.zeros((1, S, 1, D))
    k = np.zeros((1, L, 1, D))
    v = np.eye(L, D).reshape(1, L, 1, D)
    out, _ = oracle.attention(q, k, v, [P], [T], [N], w, layer, l0, 0, 1.0)
    counted = int((np.abs(out[0, :, 0, :]) > 1e-12).sum())
    assert counted == visible_pairs(P, T, N, w)
