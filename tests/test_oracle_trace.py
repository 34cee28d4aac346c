"""Pin of the oracle's confidence-trace feed (Section 3.1.1: C_trace is the
mean of -log max p of the full model's next-token distribution over the last
20 committed tokens) against an independent computation: the torch-fp64
no-cache brute force (tests/torch_reference.py) run once over the prompt and
the committed output.  Row P - 1 + i of that pass is the full model's
distribution at the position of committed token i, so the trace must hold
-log max softmax of the last 20 such rows after any mix of greedy,
sampled and exit-policy steps.

Two plausible wrong feeds are planted in copies of oracle/model.py (pushing
the draft heads' rows, and pushing verify rows 1..a+1 instead of 0..a); the
pin must reject both.  Also pins the Section 4.1 run metrics E, d and the
acceptance rate on a hand-worked record list."""
import importlib.util
import math
import os
import sys

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from tests.torch_reference import TorchReference

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MODEL_SRC = os.path.join(ROOT, "oracle", "model.py")

MICRO = shrink(TINY, name="micro-f32", n_layers=4, d_model=32, n_heads=4, n_kv_heads=4, head_dim=8,
               ffn_dim=40, vocab=48, exits=(1, 2, 3))
MICRO_BF16 = shrink(MICRO, name="micro-bf16", dtype="bf16")


def _weights(model):
    """Seeded weights with a final-norm gain of 8, so that the next-token
    distributions spread and their confidences differ row to row."""
    w = li.weights(model)
    if model.dtype == "bf16":
        w["final_norm"] = np.full_like(w["final_norm"], 0x4100)  # 8.0 in bf16
    else:
        w["final_norm"] = np.full_like(w["final_norm"], 8.0)
    return w


def _threshold_policy(c5_ref, h_ref, scale=50.0):
    w1 = np.array([[1, 0, 0], [0, 1, 0], [-1, 0, 0], [0, -1, 0]], dtype=np.float32)
    b1 = np.array([-c5_ref, -h_ref, c5_ref, h_ref], dtype=np.float32)
    w2 = np.array([[scale, scale, 0, 0], [0, 0, scale, scale]], dtype=np.float32)
    return {"w1": w1, "b1": b1, "w2": w2, "b2": np.zeros(2, dtype=np.float32)}


def _run_mixed(om, model, weights, prompt, n_total=48):
    """Prefill, then a fixed cycle of greedy steps (early and last-layer
    exits), sampled steps and exit-policy steps; returns the state."""
    max_ctx = 128
    dec = om.OracleDecoder(model, weights, max_ctx)
    st = om.SSDState(dec, -(-max_ctx // 64), 64)
    st.prefill(prompt)
    z = dec.head(dec.forward([st.pending], st.c, 1))[0]
    f = om.exit_features(z, 0.0)
    pol = _threshold_policy(f[0], f[1])
    L = model.n_layers
    i = 0
    while len(st.out) < n_total:
        kind = i % 5
        if kind == 0:
            st.step(1, 3, n_total)
        elif kind == 1:
            st.step(L, 3, n_total)          # last-layer exit: every draft is accepted
        elif kind == 2:
            st.step_sampled(2, 3, n_total, 0.6, li.step_uniforms(i))
        elif kind == 3:
            st.step_paper(n_total, pol, k_cap=4)
        else:
            st.step(2, 0, n_total)          # one autoregressive step
        i += 1
    return st


def _expected_trace(model, weights, prompt, out):
    """-log max p of the brute-force full model at every committed position."""
    ref = TorchReference(model, weights)
    z = ref.logits(list(prompt) + list(out[:-1]))   # row P-1+i predicts out[i]
    rows = z[len(prompt) - 1:]
    assert rows.shape[0] == len(out)
    vals = -F.log_softmax(rows, dim=-1).max(dim=-1).values
    return vals.numpy()


def _check_trace(om, model):
    w = _weights(model)
    prompt = li.uniform_int(1, 40, 9, 0, model.vocab - 1)
    st = _run_mixed(om, model, w, prompt)
    want = _expected_trace(model, w, prompt, st.out)
    got = np.array(list(st.trace.vals))
    n = min(len(st.out), om.POLICY_TRACE)
    assert len(got) == n
    # the oracle's fp64 logits against the fp64 brute force (the two round to
    # bf16 at the same points); observed agreement is about 1e-15
    tol = 1e-6
    np.testing.assert_allclose(got, want[-n:], rtol=0, atol=tol)
    assert st.trace.value() == pytest.approx(float(np.mean(want[-n:])), abs=tol)
    return want


@pytest.mark.parametrize("model", [MICRO, MICRO_BF16], ids=lambda m: m.name)
def test_trace_is_full_model_confidence_at_committed_positions(model):
    from oracle import model as om
    want = _check_trace(om, model)
    # the confidences differ from row to row well beyond the tolerance, so a
    # feed of other rows is visible
    assert np.ptp(want) > 0.5


def test_trace_before_and_after_prefill():
    from oracle import model as om
    w = _weights(MICRO)
    prompt = li.uniform_int(1, 41, 6, 0, MICRO.vocab - 1)
    dec = om.OracleDecoder(MICRO, w, 64)
    st = om.SSDState(dec, 1, 64)
    assert st.trace.value() == 0.0 and len(st.trace.vals) == 0
    st.prefill(prompt)
    want = _expected_trace(MICRO, w, prompt, st.out)
    assert list(st.trace.vals) == pytest.approx(list(want), abs=1e-6)


# planted wrong feeds: (name, [(old, new), ...]) replaced everywhere in model.py
TRACE_MUTANTS = [
    ("pushes_draft_rows",
     [("self.trace.push_logits(z[j])", "self.trace.push_logits(dz[j] if j < len(dz) else z[j])"),
      ("self.trace.push_logits(zv[j])", "self.trace.push_logits(dz[j] if j < len(dz) else zv[j])")]),
    ("pushes_rows_one_later",
     [("self.trace.push_logits(z[j])", "self.trace.push_logits(z[min(j + 1, len(z) - 1)])"),
      ("self.trace.push_logits(zv[j])", "self.trace.push_logits(zv[min(j + 1, len(zv) - 1)])")]),
]


def _load_mutant(tmp_path, name, edits):
    text = open(MODEL_SRC).read()
    for old, new in edits:
        assert old in text, "mutation anchor not found: %r" % old
        text = text.replace(old, new)
    path = tmp_path / ("model_mut_%s.py" % name)
    path.write_text(text)
    # a submodule of the real package, so that its relative imports resolve
    spec = importlib.util.spec_from_file_location("oracle._mut_%s" % name, str(path))
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod  # the module's dataclasses look themselves up there
    try:
        spec.loader.exec_module(mod)
    except Exception:
        del sys.modules[spec.name]
        raise
    return mod


@pytest.mark.parametrize("name,edits", TRACE_MUTANTS, ids=[m[0] for m in TRACE_MUTANTS])
def test_trace_pin_catches_planted_feed(tmp_path, name, edits):
    om = _load_mutant(tmp_path, name, edits)
    for model in (MICRO, MICRO_BF16):
        with pytest.raises(AssertionError):
            _check_trace(om, model)


def test_metrics_hand_worked():
    """Section 4.1: E = mean exit layer and d = mean draft length over the
    steps that drafted, acceptance = accepted / drafted.  Records worked by
    hand: (l, k_eff, a) = (4, 3, 1), (8, 5, 5), (4, 0, 0) [autoregressive,
    not counted], (12, 2, 0)."""
    from oracle.model import StepRecord, metrics
    rows = [(4, 3, 1), (8, 5, 5), (4, 0, 0), (12, 2, 0)]
    recs = [StepRecord(l=l, k_req=k, k_eff=k, accepted=a, emitted=[0] * (a + 1), drafts=[0] * k,
                       verify=[0] * (k + 1), reward=0.0, seq_len=0) for l, k, a in rows]
    m = metrics(recs)
    assert m["E"] == pytest.approx(8.0)          # (4 + 8 + 12) / 3
    assert m["d"] == pytest.approx(10.0 / 3.0)   # (3 + 5 + 2) / 3
    assert m["acc"] == pytest.approx(0.6)        # (1 + 5 + 0) / (3 + 5 + 2)
    assert m["tokens"] == 2 + 6 + 1 + 1
    assert m["steps"] == 4
    assert math.isnan(metrics(recs[2:3])["E"])
