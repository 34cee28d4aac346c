"""CPU ORACLE -- test infrastructure only (see the package docstring).

Offline optimisation of the exit policy's Q-network (Section 3.2, with the
training hyperparameters of Section 4.1), written plainly in fp64 numpy:

* experience: every decision of the exit policy (Section 3.3: one per
  candidate layer visited, one per further draft pass) becomes a transition
  (s_t, a_t, r_t) with the reward of Section 3.1.3; s_{t+1} is the state of
  the next decision;
* the Q-network is the 3 -> H -> 2 MLP of the exit policy with factorised
  Gaussian noisy layers (NoisyNet, Fortunato et al. 2018): every weight is
  mu + sigma * f(eps_out) f(eps_in), f(x) = sgn(x) sqrt(|x|), with the
  standard-normal eps supplied by the caller;
* one learning update: a mini-batch of replay positions drawn from supplied
  uniforms, the n-step target y = sum_{k<n} gamma^k r_{t+k} +
  gamma^n max_a' Qbar(s_{t+n}, a') from the target network, the mean square
  error to Q(s_t, a_t), its gradient with respect to every mu and sigma, and
  one Adam step (Kingma and Ba 2015);
* the target network is a copy of the online parameters, refreshed on
  request.

Readings where the paper is silent:
* an episode is one generation; its decisions are stored in decoding order
  and the last one is terminal; the n-step sum stops after a terminal
  transition and does not bootstrap past it;
* the action stored for the last candidate layer is 'exit' (the executed,
  forced action);
* reward of an exit: at a candidate layer it scores draft 1, at a further
  draft pass it scores the draft that pass keeps; +1 + (L - l*)/L when the
  draft is among the accepted ones, -2 + (L - l*)/L otherwise (a draft after
  the first rejection is never emitted, so it counts as rejected); every
  'continue' gets -0.01;
* a transition can be sampled once its n successors are stored: position j
  of the count stored ones (oldest first) for j < count - n, chosen as
  floor(m * (count - n) / 2^24) from a uniform u = m / 2^24;
* both networks draw fresh noise at every update; the acting network used
  during exploration is the online one with its own noise, the evaluation
  network its means;
* initialisation (NoisyNet, factorised): mu ~ U(-1/sqrt(p), 1/sqrt(p)) and
  sigma = sigma0 / sqrt(p) with p the layer's fan-in, from supplied uniforms;
* Adam's epsilon, unstated in the paper, is a parameter (the bench takes
  1.5e-4, the value published with the same learning rate, batch and n).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

N_FEATURES = 3            # C_k, H, C_trace (Section 3.1.1)
N_ACTIONS = 2             # continue, exit (Section 3.1.2)
CONTINUE_PENALTY = -0.01  # Section 3.1.3
U_BITS = 24               # uniforms are m / 2^24


def param_count(hidden: int) -> int:
    """Entries of one parameter set: W1 [H][3], b1 [H], W2 [2][H], b2 [2]."""
    return N_FEATURES * hidden + hidden + N_ACTIONS * hidden + N_ACTIONS


def noise_count(hidden: int) -> int:
    """Standard normals one network draws: eps_in and eps_out of each layer."""
    return N_FEATURES + hidden + hidden + N_ACTIONS


def split(vec: np.ndarray, hidden: int):
    """(W1, b1, W2, b2) views of a flat parameter set."""
    H = hidden
    o1 = N_FEATURES * H
    o2 = o1 + H
    o3 = o2 + N_ACTIONS * H
    return vec[:o1].reshape(H, N_FEATURES), vec[o1:o2], vec[o2:o3].reshape(N_ACTIONS, H), vec[o3:o3 + N_ACTIONS]


def factor(x: np.ndarray) -> np.ndarray:
    """f(x) = sgn(x) sqrt(|x|) of factorised noisy layers."""
    x = np.asarray(x, dtype=np.float64)
    return np.sign(x) * np.sqrt(np.abs(x))


def noisy_init(hidden: int, sigma0: float, u: np.ndarray) -> np.ndarray:
    """theta = [mu (param_count), sigma (param_count)] from param_count
    uniforms in [0, 1)."""
    P = param_count(hidden)
    u = np.asarray(u, dtype=np.float64)
    assert u.shape == (P,)
    fan_in = np.concatenate([np.full(N_FEATURES * hidden + hidden, float(N_FEATURES)),
                             np.full(N_ACTIONS * hidden + N_ACTIONS, float(hidden))])
    mu = (2.0 * u - 1.0) / np.sqrt(fan_in)
    sigma = sigma0 / np.sqrt(fan_in)
    return np.concatenate([mu, sigma])


def noise_matrices(hidden: int, eps: Optional[np.ndarray]):
    """The factorised noise of W1, b1, W2, b2 (zeros without eps)."""
    H = hidden
    if eps is None:
        return (np.zeros((H, N_FEATURES)), np.zeros(H), np.zeros((N_ACTIONS, H)), np.zeros(N_ACTIONS))
    e = np.asarray(eps, dtype=np.float64)
    assert e.shape == (noise_count(H),)
    fi1, fo1 = factor(e[:N_FEATURES]), factor(e[N_FEATURES:N_FEATURES + H])
    fi2, fo2 = factor(e[N_FEATURES + H:N_FEATURES + 2 * H]), factor(e[N_FEATURES + 2 * H:])
    return np.outer(fo1, fi1), fo1, np.outer(fo2, fi2), fo2


def effective(theta: np.ndarray, hidden: int, eps: Optional[np.ndarray] = None):
    """Weights of the network for one noise draw: mu + sigma * noise."""
    P = param_count(hidden)
    mu = split(np.asarray(theta[:P], dtype=np.float64), hidden)
    sg = split(np.asarray(theta[P:], dtype=np.float64), hidden)
    nz = noise_matrices(hidden, eps)
    return tuple(m + s * n for m, s, n in zip(mu, sg, nz))


def forward(net, states: np.ndarray):
    """Pre-activations [B][H] and Q-values [B][2] of W2 ReLU(W1 s + b1) + b2."""
    w1, b1, w2, b2 = net
    s = np.asarray(states, dtype=np.float64).reshape(-1, N_FEATURES)
    pre = s @ w1.T + b1
    return pre, np.maximum(pre, 0.0) @ w2.T + b2


# ---------------------------------------------------------------- experience

def step_transitions(decisions, accepted: int, l_star: int, n_layers: int) -> List[Tuple[np.ndarray, int, float]]:
    """(state, action, reward) of each decision of one policy step, in order
    (Section 3.1.3 rewards; ``decisions`` as the oracle's step_paper lists
    them: (kind, layer or draft index, state, Q-values, chosen action))."""
    lam = (n_layers - l_star) / n_layers
    out = []
    for kind, where, state, _, act in decisions:
        if kind == "layer":
            executed = 1 if where == l_star else int(act)   # the last candidate exits by force
            draft = 1
        else:
            executed = int(act)
            draft = int(where)
        if executed == 0:
            r = CONTINUE_PENALTY
        else:
            r = (1.0 + lam) if draft <= accepted else (-2.0 + lam)
        out.append((np.asarray(state, dtype=np.float64), executed, r))
    return out


class Replay:
    """Ring of the last ``capacity`` transitions (state, action, reward,
    terminal), oldest first in logical order."""

    def __init__(self, capacity: int):
        self.capacity = capacity
        self.s = np.zeros((capacity, N_FEATURES))
        self.a = np.zeros(capacity, dtype=np.int64)
        self.r = np.zeros(capacity)
        self.done = np.zeros(capacity, dtype=bool)
        self.head = 0      # next slot written
        self.count = 0

    def push(self, state, action: int, reward: float, done: bool = False):
        i = self.head
        self.s[i] = state
        self.a[i] = action
        self.r[i] = reward
        self.done[i] = done
        self.head = (i + 1) % self.capacity
        self.count = min(self.count + 1, self.capacity)

    def end_episode(self):
        """Marks the newest stored transition terminal."""
        if self.count:
            self.done[(self.head - 1) % self.capacity] = True

    def slot(self, j: int) -> int:
        """Ring slot of logical position j (0 = oldest)."""
        return (self.head - self.count + j) % self.capacity

    def n_valid(self, n: int) -> int:
        return max(0, self.count - n)

    def logical(self):
        idx = [self.slot(j) for j in range(self.count)]
        return self.s[idx], self.a[idx], self.r[idx], self.done[idx]


def sample_positions(u: np.ndarray, n_valid: int) -> np.ndarray:
    """floor(m * n_valid / 2^24) for u = m / 2^24, in integers."""
    m = np.round(np.asarray(u, dtype=np.float64) * (1 << U_BITS)).astype(np.int64)
    assert np.all((m >= 0) & (m < (1 << U_BITS)))
    assert np.array_equal(m.astype(np.float64) / (1 << U_BITS), np.asarray(u, dtype=np.float64))
    return (m * n_valid) >> U_BITS


def n_step_return(rep: Replay, j: int, n: int, gamma: float):
    """(sum_{k<m} gamma^k r_{j+k}, bootstrap state or None, gamma^n): m = n,
    or fewer when a terminal transition comes first."""
    R = 0.0
    for k in range(n):
        i = rep.slot(j + k)
        R += gamma ** k * rep.r[i]
        if rep.done[i]:
            return R, None, gamma ** n
    return R, rep.s[rep.slot(j + n)], gamma ** n


@dataclass
class Hyper:
    hidden: int = 16
    batch: int = 32
    n_step: int = 3
    gamma: float = 0.99
    lr: float = 6.25e-5
    beta1: float = 0.9
    beta2: float = 0.999
    adam_eps: float = 1.5e-4
    sigma0: float = 0.1


@dataclass
class UpdateResult:
    loss: float
    positions: np.ndarray
    targets: np.ndarray
    q_taken: np.ndarray
    grad: np.ndarray          # d loss / d theta, [mu, sigma]


def loss_and_grad(theta: np.ndarray, target: np.ndarray, rep: Replay, u_batch, eps_online, eps_target,
                  hp: Hyper) -> UpdateResult:
    """The n-step TD loss of one mini-batch and its gradient (Section 3.2)."""
    H = hp.hidden
    nv = rep.n_valid(hp.n_step)
    assert nv >= 1
    pos = sample_positions(u_batch, nv)
    B = len(pos)
    s = np.zeros((B, N_FEATURES))
    a = np.zeros(B, dtype=np.int64)
    y = np.zeros(B)
    for b, j in enumerate(pos):
        i = rep.slot(int(j))
        s[b], a[b] = rep.s[i], rep.a[i]
        R, s_boot, g_n = n_step_return(rep, int(j), hp.n_step, hp.gamma)
        y[b] = R
        if s_boot is not None:
            _, qbar = forward(effective(target, H, eps_target), s_boot)
            y[b] += g_n * qbar[0].max()
    net = effective(theta, H, eps_online)
    pre, q = forward(net, s)
    qa = q[np.arange(B), a]
    delta = qa - y
    loss = float(np.mean(delta ** 2))
    # backward through the mean square error, the output layer and the ReLU
    dq = np.zeros((B, N_ACTIONS))
    dq[np.arange(B), a] = 2.0 * delta / B
    w1, b1, w2, b2 = net
    hid = np.maximum(pre, 0.0)
    g_w2 = dq.T @ hid
    g_b2 = dq.sum(axis=0)
    d_pre = (dq @ w2) * (pre > 0)
    g_w1 = d_pre.T @ s
    g_b1 = d_pre.sum(axis=0)
    g_eff = [g_w1, g_b1, g_w2, g_b2]
    nz = noise_matrices(H, eps_online)
    g_mu = np.concatenate([g.ravel() for g in g_eff])
    g_sigma = np.concatenate([(g * z).ravel() for g, z in zip(g_eff, nz)])
    return UpdateResult(loss, pos, y, qa, np.concatenate([g_mu, g_sigma]))


class Trainer:
    """Online and target parameters, Adam moments and the replay ring."""

    def __init__(self, hp: Hyper, capacity: int, u_init: np.ndarray):
        self.hp = hp
        self.theta = noisy_init(hp.hidden, hp.sigma0, u_init)
        self.target = self.theta.copy()
        self.m = np.zeros_like(self.theta)
        self.v = np.zeros_like(self.theta)
        self.t = 0
        self.replay = Replay(capacity)

    def sync_target(self):
        self.target = self.theta.copy()

    def update(self, u_batch, eps_online, eps_target) -> UpdateResult:
        """One learning update: loss, gradient and an Adam step."""
        hp = self.hp
        res = loss_and_grad(self.theta, self.target, self.replay, u_batch, eps_online, eps_target, hp)
        g = res.grad
        self.t += 1
        self.m = hp.beta1 * self.m + (1.0 - hp.beta1) * g
        self.v = hp.beta2 * self.v + (1.0 - hp.beta2) * g * g
        m_hat = self.m / (1.0 - hp.beta1 ** self.t)
        v_hat = self.v / (1.0 - hp.beta2 ** self.t)
        self.theta = self.theta - hp.lr * m_hat / (np.sqrt(v_hat) + hp.adam_eps)
        return res

    def record_step(self, decisions, accepted: int, l_star: int, n_layers: int, episode_end: bool = False):
        for s, a, r in step_transitions(decisions, accepted, l_star, n_layers):
            self.replay.push(s, a, r)
        if episode_end:
            self.replay.end_episode()

    def acting_weights(self, eps: Optional[np.ndarray] = None) -> dict:
        """The exit policy's Q-network weights for one noise draw (the means
        without one)."""
        w1, b1, w2, b2 = effective(self.theta, self.hp.hidden, eps)
        return {"w1": w1, "b1": b1, "w2": w2, "b2": b2}
