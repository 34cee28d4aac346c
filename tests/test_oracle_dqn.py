"""Pins of the oracle's offline policy optimisation (Section 3.2, training
hyperparameters of Section 4.1) against facts fixed outside it: the loss
gradient against torch autograd and central differences, the Adam step
against torch.optim.Adam, noisy-layer statistics against their closed forms,
n-step returns against closed-form geometric sums, the sampling map by
exhaustive enumeration, the per-decision rewards against the already-pinned
step reward, and learning itself on MDPs whose Q-values are known.  Every
planted mistake in a copy of the oracle must fail at least one pin."""
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
from oracle import dqn
from oracle.model import OracleDecoder, SSDState, exit_features

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MICRO = shrink(TINY, name="micro-f32", n_layers=4, d_model=32, n_heads=4, n_kv_heads=4, head_dim=8,
               ffn_dim=40, vocab=48, exits=(1, 2, 3))


def _replay(mod, rng, n, capacity=None, p_done=0.15):
    rep = mod.Replay(capacity or n)
    for _ in range(n):
        rep.push(rng.standard_normal(3) * 2, int(rng.integers(0, 2)), float(rng.standard_normal()),
                 bool(rng.random() < p_done))
    return rep


def _uniforms(rng, n):
    return rng.integers(0, 1 << 24, n) / float(1 << 24)


# ------------------------------------------------------------------ pins

def check_noise_statistics(mod):
    """f keeps the sign and f(x)^2 = |x|.  For standard normal factors
    E[f(x)^2] = E|x| = sqrt(2/pi), so a noisy weight has mean mu and variance
    sigma^2 * 2/pi."""
    x = np.array([-4.0, -0.25, 0.0, 0.36, 9.0])
    assert np.allclose(mod.factor(x), [-2.0, -0.5, 0.0, 0.6, 3.0], rtol=0, atol=1e-15)
    H = 4
    rng = np.random.default_rng(11)
    theta = mod.noisy_init(H, 0.5, _uniforms(rng, mod.param_count(H)))
    mu = mod.effective(theta, H, None)
    n = 40000
    draws = np.stack([mod.effective(theta, H, rng.standard_normal(mod.noise_count(H)))[0] for _ in range(n)])
    sig = mod.split(theta[mod.param_count(H):], H)[0]
    assert np.all(np.abs(draws.mean(0) - mu[0]) < 5 * sig * math.sqrt(2 / math.pi) / math.sqrt(n))
    var = draws.var(0)
    assert np.all(np.abs(var / (sig ** 2 * 2 / math.pi) - 1) < 0.05)


def check_init(mod):
    """mu ~ U(-1/sqrt(p), 1/sqrt(p)), sigma = sigma0 / sqrt(p), p = fan-in."""
    H = 64
    P = mod.param_count(H)
    u = _uniforms(np.random.default_rng(3), P)
    theta = mod.noisy_init(H, 0.1, u)
    w1, b1, w2, b2 = mod.split(theta[:P], H)
    s1, sb1, s2, sb2 = mod.split(theta[P:], H)
    for m, p in ((w1, 3), (b1, 3), (w2, H), (b2, H)):
        assert np.all(np.abs(m) <= 1 / math.sqrt(p))
    assert abs(np.var(np.concatenate([w1.ravel(), b1])) * 3 * 3 - 1) < 0.15     # Var U(-a, a) = a^2 / 3
    assert abs(np.var(w2) * 3 * H - 1) < 0.2
    assert np.allclose(s1, 0.1 / math.sqrt(3)) and np.allclose(sb1, 0.1 / math.sqrt(3))
    assert np.allclose(s2, 0.1 / math.sqrt(H)) and np.allclose(sb2, 0.1 / math.sqrt(H))
    # u = 1/2 gives mu = 0 everywhere
    assert np.all(mod.noisy_init(H, 0.1, np.full(P, 0.5))[:P] == 0)


def _torch_loss(theta, target, states, actions, rboot, sboot, gammas, eps_on, eps_tg, H):
    """The same loss written with torch's own layers, from the definitions:
    noisy weights mu + sigma * outer(f(eps_out), f(eps_in)), an MLP, the
    greedy target value, the mean square error."""
    P = 6 * H + 2

    def weights(th, eps):
        e = torch.from_numpy(eps)
        f = lambda x: torch.sign(x) * torch.sqrt(torch.abs(x))   # noqa: E731
        fi1, fo1, fi2, fo2 = f(e[:3]), f(e[3:3 + H]), f(e[3 + H:3 + 2 * H]), f(e[3 + 2 * H:])
        mu, sg = th[:P], th[P:]
        W1 = mu[:3 * H].view(H, 3) + sg[:3 * H].view(H, 3) * torch.outer(fo1, fi1)
        b1 = mu[3 * H:4 * H] + sg[3 * H:4 * H] * fo1
        W2 = mu[4 * H:6 * H].view(2, H) + sg[4 * H:6 * H].view(2, H) * torch.outer(fo2, fi2)
        b2 = mu[6 * H:] + sg[6 * H:] * fo2
        return W1, b1, W2, b2

    def q(w, s):
        return F.linear(F.relu(F.linear(s, w[0], w[1])), w[2], w[3])

    with torch.no_grad():
        qbar = q(weights(torch.from_numpy(target), eps_tg), torch.from_numpy(sboot)).max(dim=1).values
    y = torch.from_numpy(rboot) + torch.from_numpy(gammas) * qbar
    qa = q(weights(theta, eps_on), torch.from_numpy(states)).gather(1, torch.from_numpy(actions)[:, None])[:, 0]
    return F.mse_loss(qa, y)


def check_gradient_against_autograd(mod):
    rng = np.random.default_rng(5)
    for H, B, n in ((8, 32, 3), (5, 7, 1), (16, 32, 5)):
        hp = mod.Hyper(hidden=H, batch=B, n_step=n, gamma=0.9)
        theta = mod.noisy_init(H, 0.3, _uniforms(rng, mod.param_count(H)))
        target = mod.noisy_init(H, 0.3, _uniforms(rng, mod.param_count(H)))
        rep = _replay(mod, rng, 60, capacity=50)         # wrapped ring
        eo, et = rng.standard_normal(mod.noise_count(H)), rng.standard_normal(mod.noise_count(H))
        res = mod.loss_and_grad(theta, target, rep, _uniforms(rng, B), eo, et, hp)
        # targets from the ring, gathered here by logical position
        s, a, r, d = rep.logical()
        states = s[res.positions]
        actions = a[res.positions]
        rboot, sboot, gam = np.zeros(B), np.zeros((B, 3)), np.zeros(B)
        for b, j in enumerate(res.positions):
            for k in range(n):
                rboot[b] += hp.gamma ** k * r[j + k]
                if d[j + k]:
                    break
            else:
                sboot[b], gam[b] = s[j + n], hp.gamma ** n
        th = torch.from_numpy(theta.copy()).requires_grad_(True)
        loss = _torch_loss(th, target, states, actions, rboot, sboot, gam, eo, et, H)
        loss.backward()
        assert abs(loss.item() - res.loss) <= 1e-12 * max(1.0, abs(res.loss))
        assert np.allclose(res.grad, th.grad.numpy(), rtol=1e-10, atol=1e-12)


def check_central_differences(mod):
    rng = np.random.default_rng(6)
    H, B = 6, 16
    hp = mod.Hyper(hidden=H, batch=B, n_step=2, gamma=0.95)
    theta = mod.noisy_init(H, 0.3, _uniforms(rng, mod.param_count(H)))
    rep = _replay(mod, rng, 40)
    u = _uniforms(rng, B)
    eo, et = rng.standard_normal(mod.noise_count(H)), rng.standard_normal(mod.noise_count(H))
    target = theta.copy()
    g = mod.loss_and_grad(theta, target, rep, u, eo, et, hp).grad
    h = 1e-6
    for i in rng.choice(len(theta), 24, replace=False):
        tp, tm = theta.copy(), theta.copy()
        tp[i] += h
        tm[i] -= h
        fd = (mod.loss_and_grad(tp, target, rep, u, eo, et, hp).loss -
              mod.loss_and_grad(tm, target, rep, u, eo, et, hp).loss) / (2 * h)
        assert abs(fd - g[i]) <= 1e-6 * max(1.0, abs(g[i])), (i, fd, g[i])


def check_adam_against_torch(mod):
    rng = np.random.default_rng(7)
    H = 8
    hp = mod.Hyper(hidden=H, batch=16, n_step=3, lr=1e-3, adam_eps=1e-3)
    tr = mod.Trainer(hp, 64, _uniforms(rng, mod.param_count(H)))
    tr.replay = _replay(mod, rng, 64)
    p = torch.nn.Parameter(torch.from_numpy(tr.theta.copy()))
    opt = torch.optim.Adam([p], lr=hp.lr, betas=(hp.beta1, hp.beta2), eps=hp.adam_eps)
    for step in range(6):
        u = _uniforms(rng, hp.batch)
        eo, et = rng.standard_normal(mod.noise_count(H)), rng.standard_normal(mod.noise_count(H))
        res = tr.update(u, eo, et)
        opt.zero_grad()
        p.grad = torch.from_numpy(res.grad.copy())
        opt.step()
        assert np.allclose(tr.theta, p.detach().numpy(), rtol=0, atol=1e-13), step
        if step == 2:
            tr.sync_target()


def check_n_step_closed_forms(mod):
    g = 0.9
    rep = mod.Replay(16)
    for i in range(12):
        rep.push([i, 0, 0], 1, 1.0, done=(i == 7))
    # constant reward 1 with no terminal: R = (1 - g^n) / (1 - g), bootstrap from j + n
    for n in (1, 2, 3, 4):
        R, sb, gn = mod.n_step_return(rep, 0, n, g)
        assert abs(R - (1 - g ** n) / (1 - g)) < 1e-14 and sb[0] == n and abs(gn - g ** n) < 1e-15
    # a terminal at offset d < n: R = (1 - g^(d+1)) / (1 - g) and no bootstrap
    R, sb, _ = mod.n_step_return(rep, 5, 4, g)
    assert sb is None and abs(R - (1 - g ** 3) / (1 - g)) < 1e-14
    # the terminal transition itself: R = r
    R, sb, _ = mod.n_step_return(rep, 7, 3, g)
    assert sb is None and R == 1.0
    # gamma = 0: R = r_j
    rep2 = mod.Replay(8)
    for i in range(8):
        rep2.push([i, 0, 0], 0, float(i + 1))
    R, sb, gn = mod.n_step_return(rep2, 2, 3, 0.0)
    assert R == 3.0 and gn == 0.0 and sb[0] == 5
    # wrapped ring: logical order survives overwriting
    rep3 = mod.Replay(5)
    for i in range(13):
        rep3.push([i, 0, 0], 0, float(i))
    assert [rep3.s[rep3.slot(j)][0] for j in range(5)] == [8, 9, 10, 11, 12]
    R, sb, _ = mod.n_step_return(rep3, 1, 2, 0.5)
    assert R == 9 + 0.5 * 10 and sb[0] == 11


def check_sampling_map(mod):
    m = np.arange(1 << 24, dtype=np.int64)
    u = m / float(1 << 24)
    assert np.all(mod.sample_positions(u[::4099], 1) == 0)
    for nv in (3, (1 << 20) + 7):
        pos = mod.sample_positions(u, nv)
        c = np.bincount(pos, minlength=nv)
        assert len(c) == nv and c.min() >= (1 << 24) // nv and c.max() <= -(-(1 << 24) // nv)
        assert np.all(np.diff(pos) >= 0)


def check_rewards_against_step_reward(mod):
    """Section 3.1.3 per decision: continue -0.01; an exit scores its draft.
    Summed over the kept drafts up to and including the first rejection, the
    exit rewards give the step reward already pinned in closed form."""
    w = li.weights(MICRO)
    dec = OracleDecoder(MICRO, w, 96)
    st = SSDState(dec, 2, 64)
    st.prefill(li.uniform_int(1, 31, 10, 0, MICRO.vocab - 1))
    # 'exit' below the confidence and entropy of the first state, 'continue' above
    f = exit_features(dec.head(dec.forward([st.pending], st.c, 1))[0], 0.0)
    pol = {"w1": np.array([[1.0, 0, 0], [0, 1, 0], [-1, 0, 0], [0, -1, 0]]),
           "b1": np.array([-f[0], -f[1], f[0], f[1]]),
           "w2": np.array([[50.0, 50, 0, 0], [0, 0, 50, 50]]), "b2": np.zeros(2)}
    seen = set()
    for _ in range(14):
        rec = st.step_paper(200, pol)
        lam = (MICRO.n_layers - rec.l) / MICRO.n_layers
        tr = mod.step_transitions(rec.decisions, rec.accepted, rec.l, MICRO.n_layers)
        assert len(tr) == len(rec.decisions)
        exits = [(kind, where) for (kind, where, *_), (_, a, _) in zip(rec.decisions, tr) if a == 1]
        assert len([e for e in exits if e[0] == "layer"]) == 1 and exits[0] == ("layer", rec.l)
        assert 1 + len([e for e in exits if e[0] == "draft"]) == rec.k_eff
        kept = 0
        total = 0.0
        for (kind, where, *_), (_, a, r) in zip(rec.decisions, tr):
            if a == 0:
                assert r == -0.01
                continue
            kept += 1
            assert r == (1 + lam if kept <= rec.accepted else -2 + lam)
            if kept <= rec.accepted + 1:
                total += r
        assert abs(total - rec.reward) < 1e-12
        seen.update((kind, a) for (kind, *_), (_, a, _) in zip(rec.decisions, tr))
    assert seen == {("layer", 0), ("layer", 1), ("draft", 0), ("draft", 1)}


def check_learning_on_a_bandit(mod):
    """Terminal one-step transitions with a reward that depends on (s, a):
    training drives Q(s, a) to the reward (the regression optimum)."""
    rng = np.random.default_rng(8)
    hp = mod.Hyper(hidden=16, batch=32, n_step=3, lr=3e-3, sigma0=0.01)
    tr = mod.Trainer(hp, 400, _uniforms(rng, mod.param_count(16)))
    for _ in range(400):
        s = rng.standard_normal(3)
        a = int(rng.integers(0, 2))
        tr.replay.push(s, a, (0.8 * s[0] - 0.3 * s[1] + 0.5) if a == 1 else -0.01, done=True)
    losses = []
    for i in range(1500):
        res = tr.update(_uniforms(rng, 32), rng.standard_normal(mod.noise_count(16)),
                        rng.standard_normal(mod.noise_count(16)))
        losses.append(res.loss)
    assert np.mean(losses[-100:]) < 0.1 * np.mean(losses[:100])
    _, q = mod.forward(mod.effective(tr.theta, 16), np.array([[2.0, 0, 0], [-2.0, 0, 0]]))
    assert abs(q[0, 1] - 2.1) < 0.25 and abs(q[1, 1] + 1.1) < 0.25 and abs(q[0, 0] + 0.01) < 0.25


def check_learning_bootstraps_through_the_target(mod):
    """Two-decision episodes A -continue-> B -exit-> end with rewards -0.01
    and 1.5, n = 1: Q(A, continue) -> -0.01 + gamma * max_a Q(B, a)."""
    rng = np.random.default_rng(9)
    hp = mod.Hyper(hidden=16, batch=32, n_step=1, gamma=0.9, lr=3e-3, sigma0=0.01)
    tr = mod.Trainer(hp, 512, _uniforms(rng, mod.param_count(16)))
    A, Bs = np.array([1.0, -1.0, 0.5]), np.array([-1.0, 1.0, 0.5])
    for _ in range(256):
        tr.replay.push(A, 0, -0.01)
        tr.replay.push(Bs, 1, 1.5, done=True)
    for i in range(2500):
        tr.update(_uniforms(rng, 32), rng.standard_normal(mod.noise_count(16)),
                  rng.standard_normal(mod.noise_count(16)))
        if i % 100 == 99:
            tr.sync_target()
    _, q = mod.forward(mod.effective(tr.theta, 16), np.stack([A, Bs]))
    assert abs(q[1, 1] - 1.5) < 0.1
    assert abs(q[0, 0] - (-0.01 + 0.9 * 1.5)) < 0.15


PINS = [check_noise_statistics, check_init, check_gradient_against_autograd, check_central_differences,
        check_adam_against_torch, check_n_step_closed_forms, check_rewards_against_step_reward,
        check_learning_on_a_bandit, check_learning_bootstraps_through_the_target, check_sampling_map]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(dqn)


# ------------------------------------------------------------------ mutants

SRC = os.path.join(ROOT, "oracle", "dqn.py")
MUTANTS = [
    ("bootstrap_without_gamma_n", "return R, rep.s[rep.slot(j + n)], gamma ** n",
     "return R, rep.s[rep.slot(j + n)], 1.0"),
    ("bootstrap_through_terminal", "        if rep.done[i]:\n            return R, None, gamma ** n\n", ""),
    ("discount_off_by_one", "R += gamma ** k * rep.r[i]", "R += gamma ** (k + 1) * rep.r[i]"),
    ("noise_without_f", "fi1, fo1 = factor(e[:N_FEATURES]), factor(e[N_FEATURES:N_FEATURES + H])",
     "fi1, fo1 = e[:N_FEATURES], e[N_FEATURES:N_FEATURES + H]"),
    ("sigma_grad_without_noise", "g_sigma = np.concatenate([(g * z).ravel() for g, z in zip(g_eff, nz)])",
     "g_sigma = np.concatenate([g.ravel() for g in g_eff])"),
    ("relu_mask_dropped", "d_pre = (dq @ w2) * (pre > 0)", "d_pre = dq @ w2"),
    ("td_sign", "delta = qa - y", "delta = y - qa"),
    ("loss_not_averaged", "dq[np.arange(B), a] = 2.0 * delta / B", "dq[np.arange(B), a] = 2.0 * delta"),
    ("adam_no_bias_correction", "m_hat = self.m / (1.0 - hp.beta1 ** self.t)", "m_hat = self.m"),
    ("target_is_online", "_, qbar = forward(effective(target, H, eps_target), s_boot)",
     "_, qbar = forward(effective(theta, H, eps_target), s_boot)"),
    ("target_mean_not_max", "y[b] += g_n * qbar[0].max()", "y[b] += g_n * qbar[0].mean()"),
    ("forced_exit_stored_as_continue", "executed = 1 if where == l_star else int(act)", "executed = int(act)"),
    ("reward_counts_first_rejection_accepted", "r = (1.0 + lam) if draft <= accepted else (-2.0 + lam)",
     "r = (1.0 + lam) if draft <= accepted + 1 else (-2.0 + lam)"),
    ("init_fan_in_swapped", "np.full(N_ACTIONS * hidden + N_ACTIONS, float(hidden))",
     "np.full(N_ACTIONS * hidden + N_ACTIONS, float(N_FEATURES))"),
    ("sampling_off_by_one", "return (m * n_valid) >> U_BITS", "return (m * (n_valid + 1)) >> U_BITS"),
    ("ring_order", "return (self.head - self.count + j) % self.capacity", "return j % self.capacity"),
]


def _load_mutant(name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, name
    spec = importlib.util.spec_from_loader("dqn_mutant_" + name, loader=None)
    mod = importlib.util.module_from_spec(spec)
    mod.__dict__["__name__"] = spec.name
    sys.modules[spec.name] = mod      # dataclasses look the module up by name
    try:
        exec(compile(text.replace(old, new), SRC + ":" + name, "exec"), mod.__dict__)
    finally:
        del sys.modules[spec.name]
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(name, old, new):
    mod = _load_mutant(name, old, new)
    caught = []
    for pin in PINS:
        try:
            pin(mod)
        except (AssertionError, IndexError, ValueError):
            caught.append(pin.__name__)
            break
    assert caught, "no pin failed for mutant " + name
