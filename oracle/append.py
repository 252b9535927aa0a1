"""Appending one decoded token to the paged cache (oracle).

Test infrastructure: see the package docstring.
"""
from __future__ import annotations

import numpy as np


def append_token(k_pool: np.ndarray, v_pool: np.ndarray, table_row: np.ndarray, n_tokens: int,
                 k_new: np.ndarray, v_new: np.ndarray, block_size: int) -> int:
    """Write the new token's key and value [H_kv, d] at logical position
    n_tokens (physical block table[n // bs], slot n % bs) of the pools
    (K pool [P, H_kv, bs, d], V pool [P, H_kv, d, bs]) in place, and return
    the new length.  The memory state of the paged cache grows by one token
    per decode step (Section 3, the state's memory component)."""
    p = int(table_row[n_tokens // block_size])
    slot = n_tokens % block_size
    k_pool[p, :, slot, :] = k_new
    v_pool[p, :, :, slot] = v_new
    return n_tokens + 1
