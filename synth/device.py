"""Device residency of synthetic inputs (torch tensors), and the library
configuration fields of a workload.  Plumbing only: no arithmetic of the method."""
from __future__ import annotations

from dataclasses import dataclass
from typing import Optional

import numpy as np

from .gen import Inputs
from .params import Params
from .workloads import Workload


def config_fields(w: Workload, p: Params, num_pool_blocks: int,
                  max_batch: Optional[int] = None, max_blocks: Optional[int] = None) -> dict:
    """Field values of the library's ent_config for workload `w` and parameters `p`."""
    return dict(
        max_batch=w.batch if max_batch is None else max_batch,
        num_q_heads=w.num_q_heads, num_kv_heads=w.num_kv_heads, head_dim=w.head_dim,
        block_size=w.block_size,
        max_blocks_per_seq=w.max_blocks_per_seq if max_blocks is None else max_blocks,
        num_pool_blocks=max(1, num_pool_blocks), vocab=w.vocab,
        kv_dtype=1 if w.kv_dtype == "bf16" else 0,
        scale=p.scale, eta=p.eta, h_target=p.h_target, t_min=p.t_min, t_max=p.t_max,
        eps_h=p.eps_h, h_min=p.h_min, kappa_min=p.kappa_min, b_min=p.b_min, log_v=p.log_v,
        estimator=p.estimator, est_k=p.est_k, t_cal=p.t_cal, rho_t=p.rho_t, dkappa=p.dkappa,
        h_bias=p.h_bias, scoring=p.scoring, keep_first=p.keep_first, keep_last=p.keep_last)


def _tensor(a: np.ndarray, device):
    import torch
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


@dataclass
class DeviceInputs:
    """Inputs of one workload resident in device memory, plus output buffers."""
    ctx_lens: object
    block_tables: object
    k_pool: object
    v_pool: object
    q: object          # [S, B, Hq, d]
    logits: object     # [S, B, V]
    uniforms: object   # [S, B]
    h_prev: object
    tau: object
    temp: object
    k_new: object
    v_new: object
    # outputs
    ksum: object
    h: object
    temp_used: object
    row_stats: object
    kept: object
    n_kept: object
    scores: object
    theta: object
    out: object
    lse: object
    tokens: object
    kappa: object      # kept-fraction state (NaN: no previous step)


def upload(x: Inputs, device="cuda", copies: int = 1) -> DeviceInputs:
    """Copy `x` to the device and allocate the step's outputs."""
    import torch
    w = x.workload
    B, Hq, d, Hkv = w.batch, w.num_q_heads, w.head_dim, w.num_kv_heads
    C = -(-w.vocab // 4096)
    maxb = x.block_tables.shape[1]
    f32 = dict(dtype=torch.float32, device=device)
    i32 = dict(dtype=torch.int32, device=device)
    return DeviceInputs(
        ctx_lens=_tensor(x.ctx_lens, device), block_tables=_tensor(x.block_tables, device),
        k_pool=_tensor(x.k_pool, device), v_pool=_tensor(x.v_pool, device),
        q=_tensor(x.q, device), logits=_tensor(x.logits, device),
        uniforms=_tensor(x.uniforms, device), h_prev=_tensor(x.h_prev, device),
        tau=_tensor(x.tau, device), temp=_tensor(x.temp, device),
        k_new=None if x.k_new is None else _tensor(x.k_new, device),
        v_new=None if x.v_new is None else _tensor(x.v_new, device),
        ksum=torch.zeros((max(1, x.num_pool_blocks), Hkv, d), **f32),
        h=torch.zeros(B, **f32), temp_used=torch.zeros(B, **f32),
        row_stats=torch.zeros((B, C, 2), **f32),
        kept=torch.full((B, maxb), -1, **i32), n_kept=torch.zeros(B, **i32),
        scores=torch.zeros((B, maxb), **f32), theta=torch.zeros(B, **f32),
        out=torch.zeros((B, Hq, d), **f32), lse=torch.zeros((B, Hq), **f32),
        tokens=torch.zeros(B, **i32), kappa=torch.full((B,), float("nan"), **f32))
