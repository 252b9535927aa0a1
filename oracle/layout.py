"""Reading the library's buffer layouts into float64 logical arrays (oracle side).

Paged cache layout, as the library defines it:
  K pool  [P, H_kv, bs, d]   token-major tile per (physical block, KV head)
  V pool  [P, H_kv, d, bs]   dim-major tile per (physical block, KV head)
  block table row [MAXB] of physical block ids; logical token i of a
  sequence lives in physical block table[i // bs], slot i % bs.
bf16 data arrives as uint16 bit patterns; float32 data as float32.
"""
from __future__ import annotations

import numpy as np


def to_f64(a: np.ndarray) -> np.ndarray:
    """Exact promotion of bf16 bit patterns (uint16) or float32 values to float64."""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


def gather_sequence(k_pool: np.ndarray, v_pool: np.ndarray, table_row: np.ndarray,
                    n_tokens: int, block_size: int):
    """Logical keys and values [n_tokens, H_kv, d] (float64) of one sequence."""
    nb = -(-n_tokens // block_size)
    phys = np.asarray(table_row[:nb], dtype=np.int64)
    kt = to_f64(k_pool[phys])                      # [nb, Hkv, bs, d]
    vt = to_f64(v_pool[phys])                      # [nb, Hkv, d, bs]
    K = kt.transpose(0, 2, 1, 3).reshape(nb * block_size, kt.shape[1], kt.shape[3])
    V = vt.transpose(0, 3, 1, 2).reshape(nb * block_size, vt.shape[1], vt.shape[2])
    return K[:n_tokens], V[:n_tokens]
