"""A thin driver of the C ABI: one context, and the entry points of a decode
step issued in order on one stream.  Marshalling only; all work is in libent."""
from __future__ import annotations

from . import ent


def make_config(**fields) -> ent.ent_config:
    """ent_config from the library defaults overridden by `fields`."""
    cfg = ent.ent_default_config()
    for k, v in fields.items():
        if not hasattr(cfg, k):
            raise KeyError(k)
        setattr(cfg, k, v)
    return cfg


class Decoder:
    """Owns one library context; `step` runs the whole decode step, either as
    ent_entropy_temperature -> ent_block_select -> ent_sparse_paged_decode ->
    ent_sample (fused=False) or as the single call ent_decode_step (fused=True,
    the default); the two give bit-identical results."""

    def __init__(self, **fields):
        self.cfg = make_config(**fields)
        self.ctx = ent.ent_init(self.cfg)

    def close(self):
        if self.ctx:
            ent.ent_destroy(self.ctx)
            self.ctx = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def summarize(self, B, k_cache, block_tables, ctx_lens, ksum, stream=None):
        ent.ent_block_summary(self.ctx, B, k_cache, block_tables, ctx_lens, ksum, stream)

    def step(self, B, *, logits, h_prev, tau, temp, q, k_cache, v_cache, block_tables, ctx_lens,
             ksum, uniforms, h, temp_used, row_stats, kept, n_kept, out, tokens, lse=None,
             scores=None, theta=None, stream=None, fused=True, kappa=None):
        ld = logits.stride(0)
        if fused:
            ent.ent_decode_step(self.ctx, B, logits, ld, h_prev, tau, temp, q, k_cache, v_cache,
                                ksum, block_tables, ctx_lens, uniforms, h, temp_used, kept,
                                n_kept, out, tokens, row_stats, lse, scores, theta, stream, kappa)
            return
        ent.ent_entropy_temperature(self.ctx, B, logits, ld, h_prev, tau, temp, h, temp_used,
                                    row_stats, stream)
        ent.ent_block_select(self.ctx, B, q, ksum, block_tables, ctx_lens, h, kept, n_kept,
                             scores, theta, stream, kappa, k_cache)
        ent.ent_sparse_paged_decode(self.ctx, B, q, k_cache, v_cache, block_tables, ctx_lens,
                                    kept, n_kept, out, lse, stream)
        ent.ent_sample(self.ctx, B, logits, ld, row_stats, temp_used, uniforms, tokens, stream)

    def append(self, B, k_new, v_new, block_tables, ctx_lens, k_cache, v_cache, ksum, stream=None):
        ent.ent_kv_append(self.ctx, B, k_new, v_new, block_tables, ctx_lens, k_cache, v_cache,
                          ksum, stream)

    def device_status(self, stream=None) -> int:
        return ent.ent_device_status(self.ctx, stream)

    def schedule(self, N, prm, tau, n_kept, ctx_lens, tau_last, gain, age, b_sel, selected,
                 n_selected, priority=None, stream=None):
        ent.ent_schedule(self.ctx, N, prm, tau, n_kept, ctx_lens, tau_last, gain, age, b_sel,
                         selected, n_selected, priority, stream)
