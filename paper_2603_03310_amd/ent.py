"""ctypes binding of libent.so: the entropic-time decode step on MI355X.

Argument marshalling only.  Every computation runs in the library's HIP
kernels; this module converts tensors to device pointers and checks return
codes.  Names follow the C ABI declared in include/ent.h.  The library must
have been built (``python -m paper_2603_03310_amd.build``); importing this
module without it raises immediately: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libent.so")

ENT_OK, ENT_E_INVAL, ENT_E_NOMEM, ENT_E_HIP, ENT_E_UNSUPPORTED = 0, -1, -2, -3, -4
ENT_F32, ENT_BF16 = 0, 1
ENT_EST_EXACT, ENT_EST_TOPK, ENT_EST_TAIL = 0, 1, 2
ENT_EST_MAX_K = 512
ENT_SCORE_MEANKEY, ENT_SCORE_EXACT = 0, 1
ENT_ROW_CHUNK = 4096
ENT_BLOCK_SIZE = 16
ENT_DEV_BAD_TABLE, ENT_DEV_BAD_CTXLEN, ENT_DEV_CACHE_FULL = 1, 2, 4

EXPORTED = ("ent_default_config", "ent_check_config", "ent_row_stats_chunks", "ent_init",
            "ent_destroy", "ent_last_error", "ent_device_status", "ent_entropy_temperature",
            "ent_block_summary", "ent_block_select", "ent_sparse_paged_decode", "ent_sample",
            "ent_kv_append", "ent_decode_step", "ent_schedule", "ent_entropy_temperature_noalloc",
            "ent_decode_step_append")
ENT_NOALLOC_SCRATCH_BYTES = 2 << 20
ENT_SCHED_MAX_POOL = 8192


class ent_config(ctypes.Structure):
    _fields_ = [
        ("max_batch", ctypes.c_int), ("num_q_heads", ctypes.c_int),
        ("num_kv_heads", ctypes.c_int), ("head_dim", ctypes.c_int),
        ("block_size", ctypes.c_int), ("max_blocks_per_seq", ctypes.c_int),
        ("num_pool_blocks", ctypes.c_int), ("vocab", ctypes.c_int), ("kv_dtype", ctypes.c_int),
        ("scale", ctypes.c_float), ("eta", ctypes.c_float), ("h_target", ctypes.c_float),
        ("t_min", ctypes.c_float), ("t_max", ctypes.c_float), ("eps_h", ctypes.c_float),
        ("h_min", ctypes.c_float), ("kappa_min", ctypes.c_float), ("b_min", ctypes.c_int),
        ("log_v", ctypes.c_float), ("estimator", ctypes.c_int), ("est_k", ctypes.c_int),
        ("t_cal", ctypes.c_float), ("rho_t", ctypes.c_float), ("dkappa", ctypes.c_float),
        ("h_bias", ctypes.c_float), ("scoring", ctypes.c_int), ("keep_first", ctypes.c_int),
        ("keep_last", ctypes.c_int),
    ]


class ent_sched_params(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("gamma", ctypes.c_float),
                ("slo", ctypes.c_float), ("slack_floor", ctypes.c_float),
                ("gain_floor", ctypes.c_float), ("ewma_rate", ctypes.c_float)]


class ent_state(ctypes.Structure):
    _fields_ = [("h_prev", ctypes.c_void_p), ("tau", ctypes.c_void_p), ("temp", ctypes.c_void_p),
                ("kappa", ctypes.c_void_p)]


class EntError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libent error {code}: {msg}")
        self.code = code


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libent.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2603_03310_amd.build`")
    # torch first: its HIP runtime is then the one the library binds to (torch's
    # libraries name the runtime without a version, so a runtime loaded first
    # for the library would not be shared and the process would hold two).
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    vp, i, ll = ctypes.c_void_p, ctypes.c_int, ctypes.c_longlong
    cfgp = ctypes.POINTER(ent_config)
    sig = {
        "ent_default_config": (None, [cfgp]),
        "ent_check_config": (i, [cfgp, ctypes.c_char_p, i]),
        "ent_row_stats_chunks": (i, [i]),
        "ent_init": (i, [cfgp, ctypes.POINTER(vp)]),
        "ent_destroy": (i, [vp]),
        "ent_last_error": (ctypes.c_char_p, [vp]),
        "ent_device_status": (i, [vp, vp, ctypes.POINTER(ctypes.c_uint)]),
        "ent_entropy_temperature": (i, [vp, i, vp, ll, ent_state, vp, vp, vp, vp]),
        "ent_entropy_temperature_noalloc": (i, [cfgp, i, vp, ll, ent_state, vp, vp, vp, vp]),
        "ent_block_summary": (i, [vp, i, vp, vp, vp, vp, vp]),
        "ent_block_select": (i, [vp, i] + [vp] * 12),
        "ent_sparse_paged_decode": (i, [vp, i, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "ent_sample": (i, [vp, i, vp, ll, vp, vp, vp, vp, vp]),
        "ent_kv_append": (i, [vp, i, vp, vp, vp, vp, vp, vp, vp, vp]),
        "ent_decode_step": (i, [vp, i, vp, ll, ent_state] + [vp] * 18),
        "ent_decode_step_append": (i, [vp, i, vp, ll, ent_state] + [vp] * 20),
        "ent_schedule": (i, [vp, i, ctypes.POINTER(ent_sched_params)] + [vp] * 6
                         + [i] + [vp] * 4),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def ptr(x) -> Optional[int]:
    """Device (or host) address of a tensor, an int address, or None for NULL."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def ent_default_config() -> ent_config:
    cfg = ent_config()
    load().ent_default_config(ctypes.byref(cfg))
    return cfg


def ent_check_config(cfg: ent_config):
    buf = ctypes.create_string_buffer(256)
    code = load().ent_check_config(ctypes.byref(cfg), buf, 256)
    return code, buf.value.decode()


def ent_row_stats_chunks(vocab: int) -> int:
    return load().ent_row_stats_chunks(vocab)


def _check(ctx, code: int):
    if code != ENT_OK:
        msg = load().ent_last_error(ctx)
        raise EntError(code, (msg or b"").decode())


def ent_init(cfg: ent_config) -> int:
    h = ctypes.c_void_p()
    code = load().ent_init(ctypes.byref(cfg), ctypes.byref(h))
    _check(None, code)
    return h.value


def ent_destroy(ctx: int) -> None:
    _check(None, load().ent_destroy(ctx))


def ent_last_error(ctx: Optional[int]) -> str:
    return (load().ent_last_error(ctx) or b"").decode()


def ent_device_status(ctx: int, stream=None) -> int:
    flags = ctypes.c_uint(0)
    _check(ctx, load().ent_device_status(ctx, _stream(stream), ctypes.byref(flags)))
    return flags.value


def ent_entropy_temperature(ctx, B, logits, ld, h_prev, tau, temp, h_out, temp_used,
                            row_stats=None, stream=None):
    st = ent_state(ptr(h_prev), ptr(tau), ptr(temp), None)
    _check(ctx, load().ent_entropy_temperature(ctx, B, ptr(logits), ld, st, ptr(h_out),
                                               ptr(temp_used), ptr(row_stats), _stream(stream)))


def ent_entropy_temperature_noalloc(cfg: ent_config, B, logits, ld, h_prev, tau, temp, h_out,
                                    temp_used, row_stats=None, stream=None):
    """ent_entropy_temperature without a context: no device allocation."""
    st = ent_state(ptr(h_prev), ptr(tau), ptr(temp), None)
    _check(None, load().ent_entropy_temperature_noalloc(ctypes.byref(cfg), B, ptr(logits), ld, st,
                                                        ptr(h_out), ptr(temp_used),
                                                        ptr(row_stats), _stream(stream)))


def ent_block_summary(ctx, B, k_cache, block_tables, ctx_lens, ksum, stream=None):
    _check(ctx, load().ent_block_summary(ctx, B, ptr(k_cache), ptr(block_tables), ptr(ctx_lens),
                                         ptr(ksum), _stream(stream)))


def ent_block_select(ctx, B, q, ksum, block_tables, ctx_lens, h, kept, n_kept, scores=None,
                     theta=None, stream=None, kappa=None, k_cache=None):
    _check(ctx, load().ent_block_select(ctx, B, ptr(q), ptr(ksum), ptr(k_cache),
                                        ptr(block_tables), ptr(ctx_lens), ptr(h), ptr(kept),
                                        ptr(n_kept), ptr(scores), ptr(theta), ptr(kappa),
                                        _stream(stream)))


def ent_sparse_paged_decode(ctx, B, q, k_cache, v_cache, block_tables, ctx_lens, kept, n_kept,
                            out, lse=None, stream=None):
    _check(ctx, load().ent_sparse_paged_decode(ctx, B, ptr(q), ptr(k_cache), ptr(v_cache),
                                               ptr(block_tables), ptr(ctx_lens), ptr(kept),
                                               ptr(n_kept), ptr(out), ptr(lse), _stream(stream)))


def ent_sample(ctx, B, logits, ld, row_stats, temp_used, uniforms, tokens, stream=None):
    _check(ctx, load().ent_sample(ctx, B, ptr(logits), ld, ptr(row_stats), ptr(temp_used),
                                  ptr(uniforms), ptr(tokens), _stream(stream)))


def ent_kv_append(ctx, B, k_new, v_new, block_tables, ctx_lens, k_cache, v_cache, ksum,
                  stream=None):
    _check(ctx, load().ent_kv_append(ctx, B, ptr(k_new), ptr(v_new), ptr(block_tables),
                                     ptr(ctx_lens), ptr(k_cache), ptr(v_cache), ptr(ksum),
                                     _stream(stream)))


def ent_decode_step(ctx, B, logits, ld, h_prev, tau, temp, q, k_cache, v_cache, ksum,
                    block_tables, ctx_lens, uniforms, h_out, temp_used, kept, n_kept, out,
                    tokens, row_stats=None, lse=None, scores=None, theta=None, stream=None,
                    kappa=None):
    st = ent_state(ptr(h_prev), ptr(tau), ptr(temp), ptr(kappa))
    _check(ctx, load().ent_decode_step(ctx, B, ptr(logits), ld, st, ptr(q), ptr(k_cache),
                                       ptr(v_cache), ptr(ksum), ptr(block_tables), ptr(ctx_lens),
                                       ptr(uniforms), ptr(h_out), ptr(temp_used), ptr(row_stats),
                                       ptr(kept), ptr(n_kept), ptr(out), ptr(lse), ptr(tokens),
                                       ptr(scores), ptr(theta), _stream(stream)))


def ent_decode_step_append(ctx, B, logits, ld, h_prev, tau, temp, q, k_cache, v_cache, ksum,
                           block_tables, ctx_lens, uniforms, k_new, v_new, h_out, temp_used, kept,
                           n_kept, out, tokens, row_stats=None, lse=None, scores=None, theta=None,
                           stream=None, kappa=None):
    st = ent_state(ptr(h_prev), ptr(tau), ptr(temp), ptr(kappa))
    _check(ctx, load().ent_decode_step_append(
        ctx, B, ptr(logits), ld, st, ptr(q), ptr(k_cache), ptr(v_cache), ptr(ksum),
        ptr(block_tables), ptr(ctx_lens), ptr(uniforms), ptr(k_new), ptr(v_new), ptr(h_out),
        ptr(temp_used), ptr(row_stats), ptr(kept), ptr(n_kept), ptr(out), ptr(lse), ptr(tokens),
        ptr(scores), ptr(theta), _stream(stream)))


def ent_schedule(ctx, N, prm: ent_sched_params, tau, n_kept, ctx_lens, tau_last, gain, age,
                 b_sel, selected, n_selected, priority=None, stream=None):
    _check(ctx, load().ent_schedule(ctx, N, ctypes.byref(prm), ptr(tau), ptr(n_kept),
                                    ptr(ctx_lens), ptr(tau_last), ptr(gain), ptr(age), b_sel,
                                    ptr(selected), ptr(n_selected), ptr(priority),
                                    _stream(stream)))
