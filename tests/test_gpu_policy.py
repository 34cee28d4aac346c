"""The paper's exit policy (Sections 3.1.1, 3.1.2, 3.3) on the GPU, through
the C ABI, against the oracle's step_paper: every decision's state (top-5
confidence, entropy, confidence trace) and Q-values within tolerance, the
same actions except at near ties, and then the same drafts, acceptance,
tokens, KV state and trace; the two fixed-policy limits (always exit =
first candidate with the longest drafts, always continue = last candidate
with one draft) bit-exact against the GPU's fixed-action steps; policy
decoding equal to greedy autoregressive decoding on the GPU."""
import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle.model import OracleDecoder, SSDState, exit_features
from tests.parity import Report, check_policy, say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TINY_BF16 = shrink(TINY, name="tiny-bf16", dtype="bf16")
GQA_128 = shrink(TINY, name="gqa-hd128-f32", n_layers=4, d_model=512, n_heads=8, n_kv_heads=2,
                 head_dim=128, ffn_dim=704, vocab=1024, dtype="f32", qnet_hidden=32, exits=(1, 2, 3),
                 lengths=(1, 3, 5))
MAX_CTX = 200


def _peaky(w):
    """Sharper next-token distributions (final-norm gain 8), so that the
    features vary between layers and tokens."""
    w = dict(w)
    g = np.asarray(w["final_norm"])
    if g.dtype == np.uint16:
        w["final_norm"] = np.full_like(g, 0x4100)      # bf16 8.0
    else:
        w["final_norm"] = np.full_like(g, 8.0)
    return w


def _threshold_policy(c5_ref, h_ref, scale=20.0):
    w1 = np.array([[1, 0, 0], [0, 1, 0], [-1, 0, 0], [0, -1, 0]], dtype=np.float32)
    b1 = np.array([-c5_ref, -h_ref, c5_ref, h_ref], dtype=np.float32)
    w2 = np.array([[scale, scale, 0, 0], [0, 0, scale, scale]], dtype=np.float32)
    return {"w1": w1, "b1": b1, "w2": w2, "b2": np.zeros(2, dtype=np.float32)}


def _const_policy(action):
    b2 = np.zeros(2, dtype=np.float32)
    b2[action] = 1.0
    return {"w1": np.zeros((4, 3), np.float32), "b1": np.zeros(4, np.float32), "w2": np.zeros((2, 4), np.float32),
            "b2": b2}


def _engine(model, w, policy, debug=1):
    from paper_2606_03113_amd import Engine
    eng = Engine(model, max_ctx=MAX_CTX, k_max=15, exit_hidden=policy["w1"].shape[0])
    eng.load_weights(w, li.qnet_weights(model))
    eng.load_exit_qnet(policy)
    eng.lede_set_options(0, debug)
    return eng


def _prompt(model):
    return li.uniform_int(1, 40, 37, 0, model.vocab - 1)


def _oracle(model, w, prompt):
    dec = OracleDecoder(model, w, MAX_CTX)
    st = SSDState(dec, -(-MAX_CTX // 64), 64)
    st.prefill(prompt)
    return dec, st


@pytest.mark.parametrize("model", [TINY, GQA_128, TINY_BF16], ids=lambda m: m.name)
def test_policy_steps_match_oracle(model):
    say("exit policy parity", model.name)
    w = _peaky(li.weights(model))
    prompt = _prompt(model)
    dec, st = _oracle(model, w, prompt)
    z = dec.head(dec.forward([st.pending], st.c, model.exits[len(model.exits) // 2]))[0]
    f = exit_features(z, 0.0)
    pol = _threshold_policy(f[0], f[1])
    eng = _engine(model, w, pol)
    g = eng.lede_prefill(prompt)
    if g != st.pending:
        eng.lede_set_pending(st.pending)
    eps = 1e-4 if model.dtype == "f32" else 2e-2 * float(z.max() - z.min())
    tr = eng.lede_get_trace()
    assert len(tr) == 1 and abs(tr[0] - st.trace.vals[0]) <= 4 * eps + 1e-4
    rep = Report()
    check_policy(eng, st, model, 1 + 45, pol, rep, logit_eps=eps)
    say("  steps=%d rows=%d max_err/tol=%.3g subs=%d" % (rep.steps, rep.rows, rep.max_err_rel, rep.substitutions))
    assert rep.substitutions <= rep.steps // 2


@pytest.mark.parametrize("action", [1, 0], ids=["always-exit", "always-continue"])
def test_policy_limits_equal_fixed_steps_on_gpu(action):
    model = TINY_BF16
    w = li.weights(model)
    prompt = _prompt(model)
    pol = _const_policy(action)
    a = _engine(model, w, pol, debug=0)
    b = _engine(model, w, pol, debug=0)
    assert a.lede_prefill(prompt) == b.lede_prefill(prompt)
    n_total = 40
    out_a = out_b = 1
    l_fixed, k_fixed = (min(model.exits), 12) if action == 1 else (max(model.exits), 1)
    while out_a < n_total:
        ra = a.lede_step_policy(n_remaining=n_total - out_a)
        rb = b.lede_step((l_fixed, k_fixed), n_remaining=n_total - out_b, log_qnet=False)
        assert (ra.k_eff, ra.accepted, ra.emitted, ra.seq_len) == \
               (rb.k_eff, rb.accepted, rb.emitted, rb.seq_len), (ra, rb)
        if ra.k_eff:                     # with no drafts no exit layer is used
            assert ra.l == rb.l
        out_a += len(ra.emitted)
        out_b += len(rb.emitted)
        kinds = a.policy_log()[:, 0].astype(int).tolist()
        if ra.k_eff:
            n_layers = 1 if action == 1 else len(model.exits)
            assert kinds[:n_layers] == [0] * n_layers
    assert a.lede_get_kv_state() == b.lede_get_kv_state()


def test_policy_decoding_equals_ar_on_gpu():
    model = TINY_BF16
    w = _peaky(li.weights(model))
    prompt = _prompt(model)
    dec, st = _oracle(model, w, prompt)
    z = dec.head(dec.forward([st.pending], st.c, 2))[0]
    f = exit_features(z, 0.0)
    pol = _threshold_policy(f[0], f[1])
    eng = _engine(model, w, pol, debug=0)
    n = 50
    ar = [eng.lede_prefill(prompt)]
    while len(ar) < n:
        ar += eng.lede_verify()[1]
    eng.lede_truncate(len(prompt))
    eng.lede_set_pending(ar[0])
    out, ks, ls = [ar[0]], [], []
    while len(out) < n:
        r = eng.lede_step_policy(n_remaining=n - len(out))
        out += r.emitted
        ks.append(r.k_eff)
        ls.append(r.l)
    assert out == ar
    say("  exit layers %s, draft lengths %s" % (sorted(set(ls)), sorted(set(ks))))


def test_trace_set_get_and_errors():
    from paper_2606_03113_amd import LedeError
    model = TINY
    w = li.weights(model)
    eng = _engine(model, w, _const_policy(1), debug=0)
    vals = np.arange(1, 26, dtype=np.float32) / 10
    with pytest.raises(LedeError):
        eng.lede_set_trace(vals)                 # more than 20
    eng.lede_set_trace(vals[:7])
    assert np.array_equal(eng.lede_get_trace(), vals[:7])
    eng.lede_set_trace(vals[:20])
    assert np.array_equal(eng.lede_get_trace(), vals[:20])
    with pytest.raises(LedeError):
        eng.lede_step_policy(n_remaining=5)      # no prefill yet
    from paper_2606_03113_amd import Engine
    plain = Engine(model, max_ctx=MAX_CTX, k_max=8)
    plain.load_weights(w)
    plain.lede_prefill(_prompt(model))
    with pytest.raises(LedeError):
        plain.lede_step_policy(n_remaining=5)    # no exit policy configured
