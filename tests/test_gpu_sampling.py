"""Speculative sampling on the GPU (Section 4.1: sampling at temperature T
with speculative-sampling acceptance) against the oracle, through the C ABI:

* the sampling kernel alone: every draw is the inverse-CDF draw of its
  uniform (up to fp32 rounding of the running sums), and the draws of a
  stratified grid of uniforms reproduce the softmax frequencies;
* sampled self-speculative steps on small models: every draft, acceptance
  and final draw follows the rule on the GPU's own logits and equals the
  oracle's decision except at near ties; integers are bit-exact;
* the method's guarantee: from a fixed state, the first token a sampled step
  emits follows the full model's distribution (chi-square against the
  oracle's probabilities over 4000 steps);
* error paths leave the state unchanged."""
import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle import model as om
from oracle.model import OracleDecoder, SSDState
from tests.parity import CDF_EPS, Report, check_sampled, draw_consistent, near_tie_bound, say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TINY_BF16 = shrink(TINY, name="tiny-bf16", dtype="bf16")
SMALL_GQA = shrink(TINY, name="small-gqa-bf16", n_layers=3, d_model=512, n_heads=8, n_kv_heads=2,
                   head_dim=64, ffn_dim=1408, vocab=2048, dtype="bf16", rope_base=500000.0,
                   qnet_hidden=32, exits=(1, 2, 3), lengths=(1, 2, 4, 8))


@pytest.mark.parametrize("V", [1, 7, 1000, 1024, 1025, 32000, 128256])
@pytest.mark.parametrize("T", [0.6, 0.05])
def test_sample_kernel_is_inverse_cdf(V, T):
    from paper_2606_03113_amd import op_sample
    say("sample kernel V=%d T=%g" % (V, T))
    z = (li.normal(7, 50, V, 1.0, "f32") * 0.3).astype(np.float32)
    zt = torch.from_numpy(z).to("cuda")
    p = om.probs_at(z.astype(np.float64), T)
    us = list((np.arange(256) + 0.5) / 256) + [0.0, 1.0 - 2 ** -24] + list(li.uniform01(9, 51, 64))
    for u in us:
        g = op_sample(zt, T, float(np.float32(u)))
        assert draw_consistent(p, g, float(np.float32(u)), CDF_EPS), (u, g)
    if V <= 1025:
        n = 2048
        grid = (np.arange(n) + 0.5) / n
        counts = np.bincount([op_sample(zt, T, float(np.float32(u))) for u in grid], minlength=V)
        assert np.max(np.abs(counts / n - p)) <= 1.0 / n + 1e-4


def _setup(model, prompt_len=40, max_ctx=160):
    from paper_2606_03113_amd import Engine
    eng = Engine(model, max_ctx=max_ctx, k_max=8)
    w = li.weights(model)
    eng.load_weights(w, li.qnet_weights(model))
    eng.lede_set_options(0, 1)
    prompt = li.uniform_int(1, 20, prompt_len, 0, model.vocab - 1)
    dec = OracleDecoder(model, w, max_ctx)
    st = SSDState(dec, -(-max_ctx // 64), 64)
    st.prefill(prompt)
    g = eng.lede_prefill(prompt)
    if g != st.pending:
        eng.lede_set_pending(st.pending)
    return eng, dec, st, prompt


@pytest.mark.parametrize("model", [TINY, TINY_BF16, SMALL_GQA], ids=lambda m: m.name)
@pytest.mark.parametrize("T", [0.6, 0.05])
def test_sampled_ssd_matches_oracle(model, T):
    say("sampled ssd", model.name, T)
    eng, dec, st, prompt = _setup(model)
    L = model.n_layers
    acts = [(1, 4), (L, 3), (2 if L > 2 else 1, 8), (1, 1), (1, 0), (L, 6)]
    rep = Report()
    check_sampled(eng, st, model, 1 + 40, acts, T, rep)
    say("  steps=%d rows=%d max_err/tol=%.3g subs=%d (expected %.2f)"
        % (rep.steps, rep.rows, rep.max_err_rel, rep.substitutions, rep.expected_substitutions))
    assert rep.substitutions <= near_tie_bound(rep.expected_substitutions)


def test_first_emitted_token_follows_the_full_model():
    """From one fixed state, N sampled steps with draft layer 1 and k = 3 (so
    the drafts come from a different distribution): the first emitted token
    must be distributed as softmax(z_full / T) (the guarantee of speculative
    sampling), checked by chi-square against the oracle's probabilities."""
    from scipy.stats import chi2
    model = TINY_BF16
    T = 0.1
    eng, dec, st, prompt = _setup(model)
    P = len(prompt)
    z = dec.head(dec.forward([st.pending], P, model.n_layers))[0]
    p = om.probs_at(z, T)
    N = 4000
    counts = np.zeros(model.vocab)
    n_acc = 0
    for i in range(N):
        eng.lede_truncate(P)
        eng.lede_set_pending(st.pending)
        rec = eng.lede_step_sampled((1, 3), T, li.step_uniforms(10000 + i), n_remaining=100)
        counts[rec.emitted[0]] += 1
        n_acc += rec.accepted > 0
    exp = N * p
    big = exp >= 5
    obs = np.append(counts[big], counts[~big].sum())
    ex = np.append(exp[big], exp[~big].sum())
    if ex[-1] < 5:
        obs, ex = obs[:-1], ex[:-1]
    stat = float(np.sum((obs - ex) ** 2 / ex))
    pval = float(chi2.sf(stat, len(obs) - 1))
    say("  bins=%d chi2=%.1f p=%.3g first-draft accepted in %d of %d" % (len(obs), stat, pval, n_acc, N))
    assert pval > 1e-4
    assert 0 < n_acc < N        # both branches (accepted draft, residual draw) were taken


def test_sampled_step_error_paths_leave_state_unchanged():
    from paper_2606_03113_amd import LedeError
    eng, dec, st, prompt = _setup(TINY)
    before = eng.lede_get_kv_state()
    u = li.step_uniforms(0)
    for T, uu in ((0.0, u), (-1.0, u), (float("nan"), u), (0.6, np.append(u[:-1], 1.0))):
        with pytest.raises(LedeError):
            eng.lede_step_sampled((1, 4), T, uu, n_remaining=10)
        assert eng.lede_get_kv_state() == before
    rec = eng.lede_step_sampled((1, 4), 0.6, u, n_remaining=10)
    assert rec.k_eff == 4 and rec.seq_len == len(prompt) + rec.accepted + 1
