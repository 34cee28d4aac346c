"""Pins of the oracle's implementation of the paper's exit policy (Sections
3.1.1, 3.1.2, 3.3): the state features against library routines, the
2-action Q-network against a library MLP, the confidence-trace window in
closed form, the control flow against the already-pinned fixed-action step
in its two limits (always exit, always continue), and greedy SSD = greedy AR
under a policy whose decisions vary."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle.model import (POLICY_MAX_DRAFT, POLICY_TRACE, ConfidenceTrace, OracleDecoder, SSDState, exit_features,
                          exit_qnet, greedy_ar)

MICRO = shrink(TINY, name="micro-f32", n_layers=4, d_model=32, n_heads=4, n_kv_heads=4, head_dim=8,
               ffn_dim=40, vocab=48, exits=(1, 2, 3))
MICRO_BF16 = shrink(MICRO, name="micro-bf16", dtype="bf16")


def test_features_match_library_routines():
    rng = np.random.default_rng(0)
    for V in (5, 48, 1000):
        z = rng.standard_normal(V) * rng.choice([0.1, 1.0, 5.0])
        f = exit_features(z, 0.7)
        t = torch.from_numpy(z)
        lp = F.log_softmax(t, dim=0)
        c5 = -torch.topk(lp, 5).values.mean().item()
        ent = torch.distributions.Categorical(logits=t).entropy().item()
        assert abs(f[0] - c5) < 1e-12 and abs(f[1] - ent) < 1e-12 and f[2] == 0.7
    # uniform over V: C5 = H = log V
    f = exit_features(np.zeros(64), 0.0)
    assert abs(f[0] - math.log(64)) < 1e-12 and abs(f[1] - math.log(64)) < 1e-12


def test_exit_qnet_matches_library_mlp():
    w = li.exit_qnet_weights(16, seed=5)
    rng = np.random.default_rng(1)
    for _ in range(5):
        s = rng.standard_normal(3) * 3
        want = F.linear(F.relu(F.linear(torch.from_numpy(s), torch.from_numpy(w["w1"]).double(),
                                        torch.from_numpy(w["b1"]).double())),
                        torch.from_numpy(w["w2"]).double(), torch.from_numpy(w["b2"]).double()).numpy()
        assert np.allclose(exit_qnet(s, w), want, rtol=0, atol=1e-12)


def test_trace_window_closed_form():
    tr = ConfidenceTrace()
    assert tr.value() == 0.0
    pm = [0.5, 0.4, 0.9, 0.6]      # each the largest of (p, (1-p)/2, (1-p)/2)
    vals = []
    for i in range(POLICY_TRACE + 7):
        p = pm[i % 4]
        z = np.log(np.array([p, (1 - p) / 2, (1 - p) / 2]))
        tr.push_logits(z)
        vals.append(-math.log(p))
        want = np.mean(vals[-POLICY_TRACE:])
        assert abs(tr.value() - want) < 1e-12


def _threshold_policy(c5_ref, h_ref, scale=50.0):
    """'exit' when the state's confidence and entropy are below the refs,
    'continue' above, as an MLP of the policy's form."""
    w1 = np.array([[1, 0, 0], [0, 1, 0], [-1, 0, 0], [0, -1, 0]], dtype=np.float32)
    b1 = np.array([-c5_ref, -h_ref, c5_ref, h_ref], dtype=np.float32)
    w2 = np.array([[scale, scale, 0, 0], [0, 0, scale, scale]], dtype=np.float32)
    return {"w1": w1, "b1": b1, "w2": w2, "b2": np.zeros(2, dtype=np.float32)}


def _const_policy(action):
    b2 = np.array([0.0, 0.0], dtype=np.float32)
    b2[action] = 1.0
    return {"w1": np.zeros((4, 3), np.float32), "b1": np.zeros(4, np.float32), "w2": np.zeros((2, 4), np.float32),
            "b2": b2}


def _states(model, prompt, n=2, max_ctx=128):
    w = li.weights(model)
    out = []
    for _ in range(n):
        dec = OracleDecoder(model, w, max_ctx)
        st = SSDState(dec, -(-max_ctx // 64), 64)
        st.prefill(prompt)
        out.append(st)
    return out


@pytest.mark.parametrize("model", [MICRO, MICRO_BF16], ids=lambda m: m.name)
def test_always_exit_is_the_fixed_first_layer_policy(model):
    prompt = li.uniform_int(1, 30, 9, 0, model.vocab - 1)
    a, b = _states(model, prompt)
    n_total, k_cap = 30, 4
    while len(a.out) < n_total:
        ra = a.step_paper(n_total, _const_policy(1), k_cap=k_cap)
        rb = b.step(min(model.exits), k_cap, n_total)
        assert (ra.l, ra.k_eff, ra.accepted, ra.emitted, ra.seq_len) == (rb.l, rb.k_eff, rb.accepted, rb.emitted,
                                                                         rb.seq_len)
        assert [d[0] for d in ra.decisions] == ["layer"] + ["draft"] * (ra.k_eff - 1)
        assert all(d[4] == 1 for d in ra.decisions)
    assert a.out == b.out and a.pager.table == b.pager.table


@pytest.mark.parametrize("model", [MICRO, MICRO_BF16], ids=lambda m: m.name)
def test_always_continue_is_the_last_layer_with_one_draft(model):
    prompt = li.uniform_int(1, 31, 9, 0, model.vocab - 1)
    a, b = _states(model, prompt)
    n_total = 20
    while len(a.out) < n_total:
        ra = a.step_paper(n_total, _const_policy(0))
        rb = b.step(max(model.exits), 1, n_total)
        assert (ra.l, ra.k_eff, ra.emitted) == (rb.l, rb.k_eff, rb.emitted)
        if ra.k_eff:
            kinds = [d[0] for d in ra.decisions]
            # every candidate visited (the last forced), then one draft pass ended by 'continue'
            assert kinds == ["layer"] * len(model.exits) + (["draft"] if n_total - len(a.out) + len(ra.emitted) > 2
                                                           else [])
    assert a.out == b.out


@pytest.mark.parametrize("model", [MICRO, MICRO_BF16], ids=lambda m: m.name)
def test_policy_ssd_equals_greedy_ar_and_decisions_vary(model):
    prompt = li.uniform_int(1, 32, 11, 0, model.vocab - 1)
    (st,) = _states(model, prompt, 1)
    n_total = 40
    want, _ = greedy_ar(st.dec, prompt, n_total)
    (st,) = _states(model, prompt, 1)
    # references at the median of the states this model produces
    z = st.dec.head(st.dec.forward([st.pending], st.c, 1))[0]
    f = exit_features(z, 0.0)
    pol = _threshold_policy(f[0], f[1], scale=50.0)
    layers, ks, acts = [], [], []
    while len(st.out) < n_total:
        r = st.step_paper(n_total, pol)
        layers.append(r.l)
        ks.append(r.k_eff)
        acts += [d[4] for d in r.decisions]
        assert r.k_eff <= POLICY_MAX_DRAFT
    assert st.out == want
    assert 0 < sum(acts) < len(acts)          # both actions taken
    assert len(set(ks)) > 1 or len(set(layers)) > 1


def test_trace_follows_committed_tokens():
    model = MICRO
    prompt = li.uniform_int(1, 33, 7, 0, model.vocab - 1)
    (st,) = _states(model, prompt, 1)
    assert len(st.trace.vals) == 1            # the prompt's next token
    n = 1
    while len(st.out) < 30:
        r = st.step_paper(30, _const_policy(1), k_cap=3)
        n += len(r.emitted)
        assert len(st.trace.vals) == min(n, POLICY_TRACE)
    # the values themselves are pinned against the brute-force full model in
    # tests/test_oracle_trace.py
