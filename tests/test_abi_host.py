"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol include/ent.h declares, and rejects bad configurations."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "ent.h")).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\*)\s+(ent_\w+)\s*\(", src, re.M)))


def test_header_declares_the_binding_names():
    from paper_2603_03310_amd import ent
    assert _declared() == sorted(ent.EXPORTED)


def test_library_exports_every_declared_symbol():
    from paper_2603_03310_amd import ent
    lib = ent.load()
    for name in _declared():
        assert hasattr(lib, name), name


def test_default_config_is_valid_and_checks_reject_bad_ones():
    from paper_2603_03310_amd import ent
    cfg = ent.ent_default_config()
    cfg.num_pool_blocks = 100
    assert ent.ent_check_config(cfg) == (ent.ENT_OK, "")
    assert abs(cfg.eta + 0.05) < 1e-7 and cfg.block_size == 16
    bad = [("block_size", 32, ent.ENT_E_INVAL), ("num_kv_heads", 3, ent.ENT_E_INVAL),
           ("head_dim", 96, ent.ENT_E_UNSUPPORTED), ("t_min", 0.0, ent.ENT_E_INVAL),
           ("log_v", 1.0, ent.ENT_E_INVAL), ("kappa_min", 1.5, ent.ENT_E_INVAL),
           ("max_batch", 0, ent.ENT_E_INVAL), ("max_blocks_per_seq", 20000, ent.ENT_E_UNSUPPORTED),
           ("vocab", 2_000_000, ent.ENT_E_UNSUPPORTED), ("kv_dtype", 7, ent.ENT_E_INVAL),
           ("estimator", 3, ent.ENT_E_INVAL), ("scoring", 2, ent.ENT_E_INVAL),
           ("keep_first", -1, ent.ENT_E_INVAL), ("keep_last", -2, ent.ENT_E_INVAL)]
    for field, val, code in bad:
        c = ent.ent_default_config()
        c.num_pool_blocks = 100
        setattr(c, field, val)
        got, msg = ent.ent_check_config(c)
        assert got == code and msg, (field, got, msg)
    c = ent.ent_default_config()
    c.num_pool_blocks = 100
    c.num_q_heads = 48          # G = 6
    assert ent.ent_check_config(c)[0] == ent.ENT_E_UNSUPPORTED
    # Estimator k: checked only when an estimator is configured.
    for est, k, code in [(ent.ENT_EST_TOPK, 0, ent.ENT_E_INVAL),
                         (ent.ENT_EST_TAIL, ent.ENT_EST_MAX_K + 1, ent.ENT_E_INVAL),
                         (ent.ENT_EST_TAIL, ent.ENT_EST_MAX_K, ent.ENT_OK),
                         (ent.ENT_EST_EXACT, 0, ent.ENT_OK)]:
        c = ent.ent_default_config()
        c.num_pool_blocks = 100
        c.estimator, c.est_k = est, k
        assert ent.ent_check_config(c)[0] == code, (est, k)
    d = ent.ent_default_config()
    assert d.estimator == ent.ENT_EST_EXACT and d.est_k == 256


def test_row_stats_chunks():
    from paper_2603_03310_amd import ent
    assert ent.ent_row_stats_chunks(128256) == 32
    assert ent.ent_row_stats_chunks(4096) == 1
    assert ent.ent_row_stats_chunks(4097) == 2
    assert ent.ent_row_stats_chunks(0) == 0


def test_init_rejects_bad_config_without_a_device():
    from paper_2603_03310_amd import ent
    c = ent.ent_default_config()
    c.block_size = 8
    with pytest.raises(ent.EntError) as e:
        ent.ent_init(c)
    assert e.value.code == ent.ENT_E_INVAL and "block_size" in str(e.value)


def test_schedule_rejects_null_context_without_a_device():
    from paper_2603_03310_amd import ent
    lib = ent.load()
    prm = ent.ent_sched_params(1.0, 0.25, 4.0, 16.0, 0.5, 1e-3, 0.25)
    code = lib.ent_schedule(None, 4, ctypes.byref(prm), *([None] * 6), 2, None, None, None, None)
    assert code == ent.ENT_E_INVAL
