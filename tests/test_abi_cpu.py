"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every entry point include/lede.h declares, and validates configurations."""
import ctypes
import os
import re

import pytest

import lede_inputs as li
from lede_inputs.configs import WORKLOADS, TINY, shrink

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    from paper_2606_03113_amd import lede
    if not os.path.exists(lede.LIB_PATH):
        from paper_2606_03113_amd import build
        build.build()
    return lede.load()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "lede.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lede_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(lib, n), n


# the boundary's calls, named after the steps of the MDP transition (Section
# 3.1): weights in, prefill, draft at (l, k), verify, the whole step, KV
# rollback and state read-back, the logits behind a decision, errors
BOUNDARY = ["lede_create", "lede_destroy", "lede_last_error", "lede_load_weights", "lede_prefill", "lede_draft",
            "lede_verify", "lede_step", "lede_truncate", "lede_get_kv_state", "lede_debug_logits"]


def test_boundary_calls_declared_and_exported(lib):
    names = declared_functions()
    for n in BOUNDARY:
        assert n in names, n
        assert hasattr(lib, n), n


def test_load_weights_rejects_bad_arguments(lib):
    from paper_2606_03113_amd import lede
    assert lib.lede_load_weights(None, None, None) == lede.LEDE_E_ARG
    assert lib.lede_debug_logits(None, 0, None, 0, None, None) == lede.LEDE_E_ARG
    assert lib.lede_debug_inject_failure(None, 0) == lede.LEDE_E_ARG


def test_weights_struct_matches_header():
    """The binding's lede_weights mirrors the header's field order and size."""
    from paper_2606_03113_amd import lede
    text = open(os.path.join(ROOT, "include", "lede.h")).read()
    body = re.search(r"typedef struct \{([^{}]*)\} lede_weights;", text).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"\*?\s*(\w+)\s*[,;]", body)
    assert fields == [f for f, _ in lede.LedeWeights._fields_]
    assert ctypes.sizeof(lede.LedeWeights) == 3 * 8 + 8 + 8 + 8 * 8
    assert re.search(r"#define LEDE_LAYER_TENSORS (\d+)", text).group(1) == str(lede.LAYER_TENSORS)
    assert len(lede.LAYER_ORDER) == lede.LAYER_TENSORS


def test_binding_names_match_header():
    from paper_2606_03113_amd import lede
    assert sorted(lede.EXPORTED) == declared_functions()


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_region_bytes_for_every_workload(lib, name):
    from paper_2606_03113_amd import lede
    w = WORKLOADS[name]
    m = w.model
    cfg = lede.make_config(m, w.max_ctx)
    wb, kvb, wsb = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.lede_region_bytes(ctypes.byref(cfg), ctypes.byref(wb), ctypes.byref(kvb), ctypes.byref(wsb)) == 0
    model_bytes = m.n_layers * m.layer_weight_bytes() + m.head_weight_bytes() + m.vocab * m.d_model * m.wbytes
    assert model_bytes <= wb.value <= model_bytes * 1.02 + (1 << 20) + m.qnet_bytes() * 2
    pages = -(-w.max_ctx // 64)
    assert kvb.value >= 2 * m.n_layers * pages * 64 * m.kv_dim * m.wbytes


@pytest.mark.parametrize("bad", [dict(head_dim=96, d_model=384), dict(ffn_dim=690), dict(vocab=1000),
                                 dict(n_kv_heads=3)])
def test_unsupported_shapes_are_rejected(lib, bad):
    from paper_2606_03113_amd import lede
    m = shrink(TINY, **bad)
    cfg = lede.make_config(m, 128)
    wb = ctypes.c_size_t()
    assert lib.lede_region_bytes(ctypes.byref(cfg), ctypes.byref(wb), None, None) == lede.LEDE_E_UNSUPPORTED


def test_bad_page_size_and_kmax_rejected(lib):
    from paper_2606_03113_amd import lede
    cfg = lede.make_config(TINY, 128)
    cfg.page_size = 32
    assert lib.lede_region_bytes(ctypes.byref(cfg), None, None, None) == lede.LEDE_E_UNSUPPORTED
    cfg = lede.make_config(TINY, 128, k_max=16)
    assert lib.lede_region_bytes(ctypes.byref(cfg), None, None, None) == lede.LEDE_E_UNSUPPORTED


def test_null_arguments(lib):
    from paper_2606_03113_amd import lede
    assert lib.lede_region_bytes(None, None, None, None) == lede.LEDE_E_ARG
    out = ctypes.c_void_p()
    assert lib.lede_create(None, None, 0, None, 0, None, 0, ctypes.byref(out)) == lede.LEDE_E_ARG
    assert lib.lede_last_error(None) == b"null context"


def test_pipelined_step_null_arguments(lib):
    import re
    from paper_2606_03113_amd import lede
    act = lede.LedeAction(1, 2)
    rec = lede.LedeStepRecord()
    assert lib.lede_step_submit(None, ctypes.byref(act), 0, 8, None) == lede.LEDE_E_ARG
    assert lib.lede_step_collect(None, None, ctypes.byref(rec)) == lede.LEDE_E_ARG
    text = open(os.path.join(ROOT, "include", "lede.h")).read()
    assert int(re.search(r"#define LEDE_MAX_IN_FLIGHT (\d+)", text).group(1)) == lede.MAX_IN_FLIGHT


def test_read_probe_rejects_bad_arguments(lib):
    from paper_2606_03113_amd import lede
    sink = ctypes.c_void_p(16)
    src = ctypes.c_void_p(4096)
    assert lib.lede_op_read_probe(None, 1024, sink, 4, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_probe(src, 1000, sink, 4, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_probe(src, 0, sink, 4, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_probe(src, 1024, sink, 0, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_probe(src, 1024, sink, 65536, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_probe(src, 1024, None, 4, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_groups(None, 4, 8, sink, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_groups(src, 0, 8, sink, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_groups(src, 65536, 8, sink, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_groups(src, 4, 0, sink, None, None) == lede.LEDE_E_ARG
    assert lib.lede_op_read_groups(src, 4, 8, None, None, None) == lede.LEDE_E_ARG


def test_sampling_entry_points_reject_bad_arguments(lib):
    from paper_2606_03113_amd import lede
    tok = ctypes.c_int32()
    x = ctypes.c_void_p(4096)
    assert lib.lede_op_sample(None, 16, 0.6, 0.5, ctypes.byref(tok), None) == lede.LEDE_E_ARG
    assert lib.lede_op_sample(x, 0, 0.6, 0.5, ctypes.byref(tok), None) == lede.LEDE_E_ARG
    for t in (0.0, -1.0, float("inf"), float("nan")):
        assert lib.lede_op_sample(x, 16, t, 0.5, ctypes.byref(tok), None) == lede.LEDE_E_ARG
    for u in (1.0, -0.1, float("nan")):
        assert lib.lede_op_sample(x, 16, 0.6, u, ctypes.byref(tok), None) == lede.LEDE_E_ARG
    assert lib.lede_op_sample(x, 16, 0.6, 0.5, None, None) == lede.LEDE_E_ARG
    u = (ctypes.c_float * lede.SAMPLE_STRIDE)()
    assert lib.lede_step_sampled(None, None, 0, 4, 0.6, u, None, None) == lede.LEDE_E_ARG


def test_exit_policy_config_and_entry_points(lib):
    from paper_2606_03113_amd import lede
    wb0, wb1 = ctypes.c_size_t(), ctypes.c_size_t()
    cfg = lede.make_config(TINY, 128)
    assert lib.lede_region_bytes(ctypes.byref(cfg), ctypes.byref(wb0), None, None) == 0
    cfg = lede.make_config(TINY, 128, exit_hidden=16)
    assert lib.lede_region_bytes(ctypes.byref(cfg), ctypes.byref(wb1), None, None) == 0
    assert wb1.value >= wb0.value + 4 * (16 * 3 + 16 + 2 * 16 + 2)
    for bad in (-1, 1025):
        cfg = lede.make_config(TINY, 128, exit_hidden=bad)
        assert lib.lede_region_bytes(ctypes.byref(cfg), None, None, None) == lede.LEDE_E_UNSUPPORTED
    m = shrink(TINY, qnet_hidden=0, exits=(3, 2))
    cfg = lede.make_config(m, 128, exit_hidden=8)       # candidates must ascend
    assert lib.lede_region_bytes(ctypes.byref(cfg), None, None, None) == lede.LEDE_E_UNSUPPORTED
    rec = lede.LedeStepRecord()
    assert lib.lede_step_policy(None, 4, None, ctypes.byref(rec)) == lede.LEDE_E_ARG
    assert lib.lede_set_trace(None, None, 0, None) == lede.LEDE_E_ARG
    n = ctypes.c_int32()
    assert lib.lede_get_trace(None, None, ctypes.byref(n), None) == lede.LEDE_E_ARG


def _dqn_cfg(**kw):
    from paper_2606_03113_amd import lede
    base = dict(hidden=16, capacity=1000, batch=32, n_step=3, gamma=0.99, lr=6.25e-5, beta1=0.9, beta2=0.999,
                adam_eps=1.5e-4, sigma0=0.1)
    base.update(kw)
    return lede.LedeDqnConfig(*[base[f] for f, _ in lede.LedeDqnConfig._fields_])


def test_dqn_region_bytes(lib):
    """Four parameter sets of 2 (6H + 2) floats and the ring of 8-float slots,
    each 256-byte aligned, plus the loss."""
    def up(x):
        return (x + 255) // 256 * 256
    for H, cap in ((16, 1000), (1, 2), (128, 1 << 20)):
        n = lib.lede_dqn_region_bytes(ctypes.byref(_dqn_cfg(hidden=H, capacity=cap, batch=16)))
        assert n == 4 * up(2 * (6 * H + 2) * 4) + up(cap * 32) + 256


@pytest.mark.parametrize("bad,code", [(dict(hidden=0), -6), (dict(hidden=129), -6), (dict(capacity=1), -6),
                                      (dict(capacity=(1 << 24) + 1), -6), (dict(batch=0), -6),
                                      (dict(batch=257), -6), (dict(batch=64, hidden=128), -6),
                                      (dict(n_step=0), -6), (dict(n_step=17), -6), (dict(gamma=1.5), -1),
                                      (dict(gamma=float("nan")), -1), (dict(lr=0.0), -1),
                                      (dict(lr=float("inf")), -1), (dict(beta1=1.0), -1),
                                      (dict(beta2=-0.1), -1), (dict(adam_eps=0.0), -1),
                                      (dict(sigma0=-1.0), -1)])
def test_dqn_config_checks(lib, bad, code):
    cfg = _dqn_cfg(**bad)
    assert lib.lede_dqn_region_bytes(ctypes.byref(cfg)) == 0
    h = ctypes.c_void_p()
    assert lib.lede_dqn_create(ctypes.byref(cfg), 256, 1 << 30, ctypes.byref(h)) == code
    assert not h.value


def test_dqn_null_and_region_checks(lib):
    cfg = _dqn_cfg()
    n = lib.lede_dqn_region_bytes(ctypes.byref(cfg))
    h = ctypes.c_void_p()
    assert lib.lede_dqn_create(None, 256, n, ctypes.byref(h)) == -1
    assert lib.lede_dqn_create(ctypes.byref(cfg), None, n, ctypes.byref(h)) == -1
    assert lib.lede_dqn_create(ctypes.byref(cfg), 256, n - 1, ctypes.byref(h)) == -1     # too small
    assert lib.lede_dqn_create(ctypes.byref(cfg), 256 + 4, n, ctypes.byref(h)) == -1     # misaligned
    assert lib.lede_dqn_create(ctypes.byref(cfg), 256, n, None) == -1
    for f in ("lede_dqn_init", "lede_dqn_end_episode", "lede_dqn_sync_target"):
        assert getattr(lib, f)(*([None] * len(getattr(lib, f).argtypes))) == -1
    assert lib.lede_dqn_update(None, None, None, None, None) == -1
    assert lib.lede_dqn_push(None, None, 0, None) == -1
    assert lib.lede_dqn_record(None, None, 0, None) == -1
    assert lib.lede_dqn_act(None, None, None, None) == -1
    assert lib.lede_dqn_read(None, 0, None, 0, None, None) == -1
    assert lib.lede_dqn_last_error(None) == b"null handle"
    lib.lede_dqn_destroy(None)
