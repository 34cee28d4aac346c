"""Verify reuse on the GPU (the verify pass starts at the exit layer, on the
hidden states and KV the draft passes computed) against the oracle's
self-speculative step, which recomputes every layer: in exact arithmetic the
two are the same function, so every verify row must agree within the logit
tolerance and the committed tokens, acceptance, KV length and page table
must match except at near ties (after which the GPU is resynchronised onto
the oracle's state).  Covers fixed actions and seeded schedules including
exits at layer 1 and at the last layer, the Q-network policy, the paper's
exit policy, speculative sampling and the draft / verify entry points."""
import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle.model import SSDState, exit_features
from tests.parity import Report, check_policy, check_sampled, check_ssd, make_decoder, near_tie_bound, say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TINY_BF16 = shrink(TINY, name="tiny-bf16", dtype="bf16")
SMALL_128 = shrink(TINY, name="small-hd128-bf16", n_layers=3, d_model=512, n_heads=4, n_kv_heads=4,
                   head_dim=128, ffn_dim=1376, vocab=4096, dtype="bf16", qnet_hidden=64,
                   exits=(1, 2, 3), lengths=tuple(range(1, 9)))
SMALL_GQA = shrink(TINY, name="small-gqa-bf16", n_layers=3, d_model=512, n_heads=8, n_kv_heads=2,
                   head_dim=64, ffn_dim=1408, vocab=2048, dtype="bf16", rope_base=500000.0,
                   qnet_hidden=32, exits=(1, 2, 3), lengths=(1, 2, 4, 8))
MODELS = [TINY, TINY_BF16, SMALL_128, SMALL_GQA]
MAX_CTX = 200


def _setup(model, exit_hidden=0, n_pages=None, order=None):
    from paper_2606_03113_amd import Engine
    eng = Engine(model, max_ctx=MAX_CTX, n_pages=n_pages, k_max=12, exit_hidden=exit_hidden)
    w = li.weights(model)
    q = li.qnet_weights(model)
    eng.load_weights(w, q)
    eng.lede_set_options(0, 1)
    if order is not None:
        eng.lede_set_free_list(order)
    eng.lede_set_verify_reuse(True)
    dec = make_decoder(model, w, q, MAX_CTX)
    st = SSDState(dec, n_pages or -(-MAX_CTX // 64), 64, order)
    prompt = li.uniform_int(1, 50, 70, 0, model.vocab - 1)
    g = eng.lede_prefill(prompt)
    st.prefill(prompt)
    rep = Report()
    if g != st.pending:
        rep.token(model.dtype, g, dec.head(dec.forward(prompt, 0, model.n_layers)[-1:])[0])
        eng.lede_set_pending(st.pending)
    return eng, w, st, rep


@pytest.mark.parametrize("model", MODELS, ids=lambda m: m.name)
def test_reuse_steps_match_oracle(model):
    say("verify reuse parity", model.name)
    n_pages = 5
    order = list(np.random.default_rng(7).permutation(n_pages))
    eng, _, st, rep = _setup(model, n_pages=n_pages, order=order)
    L = model.n_layers
    acts = [(1, 3), (L, 4), (2, 8), (1, 1), (L, 8), (2, 12)]
    sched = np.stack([li.uniform_int(2, 60, 64, 1, L), li.uniform_int(2, 61, 64, 1, 12)], 1)
    check_ssd(eng, st, model, 1 + 24, acts, rep, qnet_log=True)
    check_ssd(eng, st, model, 1 + 24 + 30, sched, rep)
    say("  steps=%d rows=%d max_err/tol=%.3g subs=%d" % (rep.steps, rep.rows, rep.max_err_rel, rep.substitutions))
    assert rep.steps >= 8


@pytest.mark.parametrize("model", [TINY_BF16, SMALL_GQA], ids=lambda m: m.name)
def test_reuse_with_qnet_policy(model):
    eng, _, st, rep = _setup(model)
    check_ssd(eng, st, model, 30, [(1, 1)], rep, qnet_policy=True)
    say("  qnet policy with reuse: steps=%d subs=%d" % (rep.steps, rep.substitutions))


@pytest.mark.parametrize("model", [TINY, TINY_BF16], ids=lambda m: m.name)
def test_reuse_sampled_steps_match_oracle(model):
    eng, _, st, rep = _setup(model)
    L = model.n_layers
    check_sampled(eng, st, model, 30, [(1, 3), (L, 2), (2, 5)], 0.6, rep)
    say("  sampled with reuse: steps=%d subs=%d (expected %.2f)"
        % (rep.steps, rep.substitutions, rep.expected_substitutions))
    assert rep.substitutions <= near_tie_bound(rep.expected_substitutions)


def test_reuse_exit_policy_matches_oracle():
    """The exit policy with reuse: a pass that ended drafting with 'continue'
    already took the last draft through layers 1..l*; otherwise one more pass
    does (both endings occur)."""
    model = shrink(TINY_BF16, exits=(1, 2, 3))
    eng, w, st, rep = _setup(model, exit_hidden=4)
    z = st.dec.head(st.dec.forward([st.pending], st.c, 2))[0]
    f = exit_features(z, 0.0)
    w1 = np.array([[1, 0, 0], [0, 1, 0], [-1, 0, 0], [0, -1, 0]], dtype=np.float32)
    pol = {"w1": w1, "b1": np.array([-f[0], -f[1], f[0], f[1]], np.float32),
           "w2": np.array([[20, 20, 0, 0], [0, 0, 20, 20]], np.float32), "b2": np.zeros(2, np.float32)}
    eng.load_exit_qnet(pol)
    eps = 2e-2 * float(z.max() - z.min())        # the bf16 logit tolerance of this model's rows
    check_policy(eng, st, model, 40, pol, rep, logit_eps=eps)
    say("  exit policy with reuse: steps=%d subs=%d" % (rep.steps, rep.substitutions))


@pytest.mark.parametrize("model", [TINY_BF16, SMALL_128], ids=lambda m: m.name)
def test_draft_verify_entry_points_equal_step_with_reuse(model):
    """lede_draft + lede_verify launch what lede_step does: the same tokens
    and the same verify logits, bit for bit."""
    from paper_2606_03113_amd import Engine
    prompt = li.uniform_int(1, 51, 40, 0, model.vocab - 1)
    outs, logits = [], []
    for split in (False, True):
        eng = Engine(model, max_ctx=MAX_CTX, k_max=12)
        eng.load_weights(li.weights(model), li.qnet_weights(model))
        eng.lede_set_options(0, 1)
        eng.lede_set_verify_reuse(True)
        out = [eng.lede_prefill(prompt)]
        zs = []
        for l, k in [(1, 4), (2, 6), (model.n_layers, 3), (2, 1)] * 3:
            if split:
                eng.lede_draft(l, k)
                _, em, _ = eng.lede_verify()
            else:
                em = eng.lede_step((l, k), log_qnet=False).emitted
            out += em
            zs.append(eng.logits(0)[:k + 1].copy())
        outs.append(out)
        logits.append(zs)
        eng.close()
    assert outs[0] == outs[1]
    for a, b in zip(*logits):
        assert np.array_equal(a, b)


def test_reuse_at_the_last_layer_accepts_the_drafts():
    """At l* = L the verify runs no layer: the head reads the hidden states
    the draft passes produced, so the drafts are accepted unless the one-row
    and matrix-core heads round a near tie apart."""
    model = TINY_BF16
    from paper_2606_03113_amd import Engine
    eng = Engine(model, max_ctx=MAX_CTX, k_max=12)
    eng.load_weights(li.weights(model), li.qnet_weights(model))
    eng.lede_set_verify_reuse(True)
    eng.lede_prefill(li.uniform_int(1, 52, 33, 0, model.vocab - 1))
    acc = drafted = 0
    for _ in range(6):
        rec = eng.lede_step((model.n_layers, 8), n_remaining=1000)
        acc += rec.accepted
        drafted += rec.k_eff
    assert acc >= drafted - 1, (acc, drafted)


def test_reuse_switch_needs_no_outstanding_draft():
    from paper_2606_03113_amd import Engine, LedeError
    model = TINY_BF16
    eng = Engine(model, max_ctx=MAX_CTX, k_max=12)
    eng.load_weights(li.weights(model), li.qnet_weights(model))
    eng.lede_prefill(li.uniform_int(1, 53, 20, 0, model.vocab - 1))
    eng.lede_draft(1, 2)
    with pytest.raises(LedeError, match="E_STATE"):
        eng.lede_set_verify_reuse(True)
    eng.lede_verify()
    eng.lede_set_verify_reuse(True)
    eng.lede_set_verify_reuse(False)
