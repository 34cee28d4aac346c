"""Pins of the oracle's speculative sampling (Section 4.1: sampling at
temperature 0.6 with speculative-sampling acceptance) against facts fixed
outside it: the frequency property of inverse-CDF sampling, the guarantee of
speculative sampling that every emitted token follows the target
distribution, the limits T -> 0 (greedy decoding) and draft = target
(every draft accepted), and the support of the residual distribution."""
import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle.model import (OracleDecoder, SSDState, greedy_ar, probs_at, sample_inverse_cdf,
                          speculative_accept)

MICRO = shrink(TINY, name="micro-f32", n_layers=2, d_model=32, n_heads=4, n_kv_heads=4,
               head_dim=8, ffn_dim=40, vocab=48)
MICRO_BF16 = shrink(MICRO, name="micro-bf16", dtype="bf16")


def test_generator_uniforms_are_exact_24_bit_floats():
    u = li.uniform01(4, 40, 100000)
    assert u.dtype == np.float32 and u.min() >= 0.0 and u.max() < 1.0
    assert np.all((u.astype(np.float64) * 2 ** 24) % 1 == 0)
    assert abs(u.mean() - 0.5) < 0.005 and abs(u.var() - 1 / 12) < 0.002
    assert np.array_equal(li.step_uniforms(3), li.uniform01(4, 40, 33, offset=99))


def test_inverse_cdf_frequencies_on_a_stratified_grid():
    """With u on the grid (i + 0.5) / N, index v is drawn for a fraction of
    the grid equal to w_v / sum(w) up to 1 / N: the defining property of
    inverse-CDF sampling."""
    rng = np.random.default_rng(1)
    N = 4000
    grid = (np.arange(N) + 0.5) / N
    for V in (1, 2, 7, 33):
        w = rng.random(V) * (rng.random(V) < 0.7)
        if w.sum() == 0:
            w[0] = 1.0
        w *= rng.choice([1e-3, 1.0, 50.0])      # any scale
        counts = np.bincount([sample_inverse_cdf(w, u) for u in grid], minlength=V)
        assert np.all(np.abs(counts / N - w / w.sum()) <= 1.0 / N + 1e-12)
        assert np.all(counts[w == 0] == 0)


def test_inverse_cdf_special_cases():
    w = np.zeros(9)
    w[4] = 2.0
    assert {sample_inverse_cdf(w, u) for u in (0.0, 0.3, 0.999999)} == {4}
    w = np.array([0.0, 0.0, 1.0, 1.0])
    assert sample_inverse_cdf(w, 0.0) == 2            # u = 0: the first index of positive weight
    assert sample_inverse_cdf(w, 0.5) == 3
    assert sample_inverse_cdf(w, 1.0 - 2 ** -24) == 3
    assert sample_inverse_cdf(np.array([1.0, 0.0]), 0.9999) == 0   # never an index of zero weight


def test_probs_at_temperature():
    z = np.array([1.0, 2.0, 3.0])
    assert np.allclose(probs_at(z, 1.0), np.exp(z) / np.exp(z).sum(), rtol=1e-15)
    assert np.allclose(probs_at(z, 0.5), np.exp(2 * z) / np.exp(2 * z).sum(), rtol=1e-15)
    assert probs_at(z, 1e-3)[2] == 1.0
    assert abs(probs_at(np.array([0.0, 0.0, 0.0, 0.0]), 0.6).sum() - 1.0) < 1e-15


def _dists(rng, V, k):
    """Random target rows p_0..p_k and draft rows q_0..q_{k-1}, with a few
    exact zeros and a few equal entries."""
    def one():
        x = rng.random(V) ** 3
        x[rng.random(V) < 0.15] = 0.0
        x[0] += 1e-3
        return x / x.sum()
    return [one() for _ in range(k + 1)], [one() for _ in range(k)]


def _first_token_error(accept, seed=2, trials=4, n=36):
    """Largest deviation of the first emitted token's distribution from p_0
    over a stratified grid of the three uniforms of a k = 1 step."""
    rng = np.random.default_rng(seed)
    grid = (np.arange(n) + 0.5) / n
    worst = 0.0
    for _ in range(trials):
        V = 5
        p, q = _dists(rng, V, 1)
        counts = np.zeros(V)
        for ud in grid:
            d = sample_inverse_cdf(q[0], ud)
            for ua in grid:
                for ur in grid:
                    a, y = accept(p, q, [d], [ua], ur)
                    counts[d if a == 1 else y] += 1
        worst = max(worst, float(np.max(np.abs(counts / n ** 3 - p[0]))))
    return worst


def test_speculative_sampling_first_token_follows_the_target():
    """k = 1 on a stratified grid of all three uniforms: the first emitted
    token has distribution p_0 (the guarantee of speculative sampling)."""
    assert _first_token_error(speculative_accept) < 3.0 / 36


def _mutant(kind):
    """Copies of the acceptance rule with one plausible mistake each."""
    def accept(p_rows, q_rows, drafts, u_acc, u_res):
        k = len(drafts)
        a = 0
        while a < k:
            d = int(drafts[a])
            p, q = p_rows[a][d], q_rows[a][d]
            ok = {"ratio_inverted": u_acc[a] * p < q, "always": True}.get(kind, u_acc[a] * q < p)
            if not ok:
                break
            a += 1
        if a < k:
            r = {"residual_q_minus_p": np.maximum(q_rows[a] - p_rows[a], 0.0),
                 "residual_is_target": p_rows[a],
                 "residual_unclipped": p_rows[a] - q_rows[a] + 1.0 / len(p_rows[a])}.get(
                     kind, np.maximum(p_rows[a] - q_rows[a], 0.0))
            y = sample_inverse_cdf(r, u_res)
        else:
            y = sample_inverse_cdf(p_rows[0] if kind == "bonus_from_first_row" else p_rows[k], u_res)
        return a, y
    return accept


@pytest.mark.parametrize("kind", ["ratio_inverted", "always", "residual_q_minus_p", "residual_is_target",
                                  "residual_unclipped"])
def test_first_token_check_catches_mutants(kind):
    assert _first_token_error(_mutant(kind), trials=3, n=24) > 3.0 / 24


def test_speculative_sampling_chain_marginals():
    """k = 3 by Monte Carlo: the j-th emitted token, given that j - 1 drafts
    were accepted before it, follows p_{j-1}; acceptance counts follow the
    closed form P(accept draft i) = sum_v min(p_i(v), q_i(v))."""
    rng = np.random.default_rng(3)
    V, k, n = 6, 3, 40000
    p, q = _dists(rng, V, k)
    acc_mass = [np.minimum(p[i], q[i]).sum() for i in range(k)]
    counts = np.zeros((k + 1, V))
    reached = np.zeros(k + 1)
    n_acc = np.zeros(k + 1)
    u = rng.random((n, 2 * k + 1))
    for s in range(n):
        drafts = [sample_inverse_cdf(q[i], u[s, i]) for i in range(k)]
        a, y = speculative_accept(p, q, drafts, u[s, k:2 * k], u[s, 2 * k])
        out = drafts[:a] + [y]
        for j, t in enumerate(out):
            counts[j, t] += 1
            reached[j] += 1
        n_acc[a] += 1
    for j in range(k + 1):
        if reached[j] > 2000:
            got = counts[j] / reached[j]
            sd = np.sqrt(p[j] * (1 - p[j]) / reached[j])
            assert np.all(np.abs(got - p[j]) <= 5 * sd + 1e-3), (j, got, p[j])
    # P(a >= i + 1 | a >= i) = acc_mass[i]
    survive = n
    for i in range(k):
        passed = n - n_acc[:i + 1].sum()
        rate = passed / survive
        sd = np.sqrt(acc_mass[i] * (1 - acc_mass[i]) / survive)
        assert abs(rate - acc_mass[i]) <= 5 * sd + 1e-3, (i, rate, acc_mass[i])
        survive = passed


def test_chain_check_catches_a_bonus_from_the_wrong_row():
    """After k acceptances the bonus must come from p_k: drawing it from p_0
    shifts the last marginal."""
    rng = np.random.default_rng(3)
    V, k, n = 6, 3, 20000
    p, q = _dists(rng, V, k)
    q = [p[i].copy() for i in range(k)]            # drafts = targets: every draft accepted
    bad = _mutant("bonus_from_first_row")
    u = rng.random((n, 2 * k + 1))
    counts = np.zeros(V)
    for s in range(n):
        drafts = [sample_inverse_cdf(q[i], u[s, i]) for i in range(k)]
        a, y = bad(p, q, drafts, u[s, k:2 * k], u[s, 2 * k])
        assert a == k
        counts[y] += 1
    sd = np.sqrt(p[k] * (1 - p[k]) / n)
    assert np.any(np.abs(counts / n - p[k]) > 5 * sd + 1e-3)


def test_residual_token_has_more_target_than_draft_mass():
    rng = np.random.default_rng(4)
    for _ in range(300):
        p, q = _dists(rng, 8, 1)
        d = int(np.argmax(q[0] - p[0]))            # a draft the target likes less
        a, y = speculative_accept(p, q, [d], [0.999999], float(rng.random()))
        assert a == 0 and p[0][y] > q[0][y]


def _state(model, prompt, max_ctx=96):
    w = li.weights(model)
    dec = OracleDecoder(model, w, max_ctx)
    st = SSDState(dec, -(-max_ctx // 64), 64)
    st.prefill(prompt)
    return dec, st


@pytest.mark.parametrize("model", [MICRO, MICRO_BF16], ids=lambda m: m.name)
def test_sampling_at_vanishing_temperature_is_greedy_decoding(model):
    """As T -> 0 the draft and target distributions become one-hot on the
    argmax: self-speculative sampling then emits greedy decoding's tokens."""
    prompt = li.uniform_int(1, 20, 11, 0, model.vocab - 1)
    n_total = 24
    dec, st = _state(model, prompt)
    want, _ = greedy_ar(dec, prompt, n_total)
    _, st = _state(model, prompt)
    acts = [(1, 3), (2, 4), (1, 1), (2, 2)]
    i = 0
    while len(st.out) < n_total:
        l, k = acts[i % len(acts)]
        st.step_sampled(l, k, n_total, 1e-5, li.step_uniforms(i))
        i += 1
    assert st.out == want


def test_draft_equal_to_target_accepts_every_draft():
    """At l = L the draft rows are computed exactly as the verify rows, so
    p = q and u < 1 accepts every draft."""
    model = MICRO
    prompt = li.uniform_int(1, 21, 9, 0, model.vocab - 1)
    _, st = _state(model, prompt)
    for i in range(4):
        rec = st.step_sampled(model.n_layers, 4, 100, 0.6, li.step_uniforms(i))
        assert rec.accepted == rec.k_eff == 4
        assert all(np.array_equal(pr, qr) for pr, qr in zip(st.last_p_rows, st.last_q_rows))


def test_sampled_step_bookkeeping():
    """Invariant c = P + n_gen - 1, KV truncation and k clamping hold for
    sampled steps as for greedy ones."""
    model = MICRO_BF16
    prompt = li.uniform_int(1, 22, 13, 0, model.vocab - 1)
    _, st = _state(model, prompt)
    n_total = 30
    i = 0
    while len(st.out) < n_total:
        rec = st.step_sampled(1, 5, n_total, 0.6, li.step_uniforms(i))
        assert rec.k_eff == min(5, n_total - (len(st.out) - len(rec.emitted)) - 1)
        assert st.c == len(prompt) + len(st.out) - 1 == rec.seq_len
        assert len(st.pager.table) == -(-st.c // 64)
        i += 1
    assert len(st.out) == n_total
