"""Oracle: token-to-expert bucketing.  TEST INFRASTRUCTURE ONLY.

Section 3.1 keeps the dense structure of each surviving expert, so the layer
runs every expert as one dense matrix product over the tokens routed to it.
Bucketing groups the (token, slot) assignments by expert:

* ``counts[e]`` = number of assignments to expert ``e``;
* ``offsets`` = exclusive prefix sum of ``counts`` over ``e = 0..E-1``, with
  ``offsets[E] = n * k``;
* ``perm[p] = t * k + j`` lists every assignment, ordered by expert ascending,
  then by token ascending.  A token's ``k`` experts are distinct, so this order
  is unique, and it is exactly a stable sort of the flattened ``idx`` by value;
* ``active`` = experts with ``counts > 0``, ascending.
"""
import numpy as np


def bucket(idx, n_experts):
    """idx int ``[n, k]`` -> (offsets int32 ``[E+1]``, perm int32 ``[n*k]``, active int32)."""
    flat = np.asarray(idx, dtype=np.int64).ravel()
    perm = np.argsort(flat, kind="stable").astype(np.int32)
    counts = np.bincount(flat, minlength=n_experts)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    active = np.nonzero(counts)[0].astype(np.int32)
    return offsets, perm, active
