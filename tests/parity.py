"""GPU-vs-oracle parity protocol shared by the GPU tests.

Logits agree within max-abs 1e-4 for fp32 models and within 2e-2 x (logit
range of the oracle's row) for bf16 models, times sqrt(depth / 40) for models
deeper than 40 layers (oracle.model.Tolerance).  Every GPU argmax g must satisfy
z_oracle[g] >= max(z_oracle) - tol; if g is not the oracle's argmax the step
is a near-tie substitution and the GPU is forced onto the oracle's tokens (the
oracle never takes an input from the GPU).  Integers (acceptance, emitted
tokens, KV length, page table) must then be bit-exact.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass, field
from typing import List

import numpy as np

from oracle import model as om
from oracle.model import OracleDecoder, SSDState, Tolerance

TOL = Tolerance()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def tol_of(dtype: str, z: np.ndarray, depth: int = 0) -> float:
    return TOL.of(dtype, float(z.max() - z.min()), depth)


@dataclass
class Report:
    rows: int = 0
    max_err_rel: float = 0.0     # max |dz| / tol over rows
    max_err_abs: float = 0.0
    substitutions: int = 0
    steps: int = 0
    # sampled steps: summed probability (over the shared uniforms) that a
    # decision taken on the GPU's logits differs from the oracle's
    expected_substitutions: float = 0.0
    notes: List[str] = field(default_factory=list)
    depth: int = 0               # model depth (scales the bf16 bound past the paper's depths)

    def row(self, dtype, z_gpu, z_orc):
        t = tol_of(dtype, z_orc, self.depth)
        err = float(np.max(np.abs(z_gpu.astype(np.float64) - z_orc)))
        self.rows += 1
        self.max_err_abs = max(self.max_err_abs, err)
        self.max_err_rel = max(self.max_err_rel, err / t)
        assert err <= t, "logit error %.3g exceeds tolerance %.3g" % (err, t)

    def token(self, dtype, g: int, z_orc: np.ndarray) -> bool:
        """True if g is the oracle's argmax; False for an allowed near-tie."""
        t = tol_of(dtype, z_orc, self.depth)
        best = int(np.argmax(z_orc))
        assert z_orc[g] >= z_orc[best] - t, "token %d is not within tolerance of the argmax %d" % (g, best)
        if g != best:
            self.substitutions += 1
            return False
        return True


def make_decoder(model, weights, qnet, max_ctx):
    return OracleDecoder(model, weights, max_ctx, qnet)


def check_ar(eng, dec, model, prompt, n_gen, rep: Report):
    """Greedy AR on the GPU (verify with k = 0) against the oracle, teacher-
    forced on the oracle's tokens."""
    L = model.n_layers
    g = eng.lede_prefill(prompt)
    h = dec.forward(prompt, 0, L)
    z = dec.head(h[-1:])[0]
    rep.row(model.dtype, eng.logits(0)[-1], z)
    want = int(np.argmax(z))
    if not rep.token(model.dtype, g, z):
        eng.lede_set_pending(want)
    toks = [want]
    pos = len(prompt)
    gpu_toks = [g]
    while len(toks) < n_gen:
        a, emitted, ver = eng.lede_verify()
        assert a == 0 and len(emitted) == 1
        h = dec.forward([toks[-1]], pos, L)
        pos += 1
        z = dec.head(h)[0]
        rep.row(model.dtype, eng.logits(0)[0], z)
        want = int(np.argmax(z))
        gpu_toks.append(emitted[0])
        if not rep.token(model.dtype, emitted[0], z):
            eng.lede_set_pending(want)
        toks.append(want)
        sl, pend, _ = eng.lede_get_kv_state()
        assert sl == pos and pend == want
    rep.steps += n_gen - 1
    return toks, gpu_toks


def check_ssd(eng, st: SSDState, model, n_total, actions, rep: Report, qnet_log=False, qnet_policy=False,
              check_drafts=True):
    """Self-speculative steps on the GPU against the oracle's SSD loop, step by
    step (needs the engine in debug mode).  A near-tie substitution
    resynchronises the GPU onto the oracle's committed state."""
    dt = model.dtype
    i = 0
    while len(st.out) < n_total:
        l, k = actions[min(i, len(actions) - 1)]
        i += 1
        c0, pending0 = st.c, st.pending
        n_rem = n_total - len(st.out)
        orc = st.step(int(l), int(k), n_total, qnet=(qnet_log or qnet_policy), use_qnet_action=qnet_policy)
        rec = eng.lede_step(None if qnet_policy else (int(l), int(k)), n_remaining=n_rem, log_qnet=qnet_log)
        rep.steps += 1
        diverged = False
        if orc.q_values is not None:
            assert rec.q_action >= 0
            qv, _ = eng.lede_debug_read(1, len(orc.q_values))
            qtol = TOL.of(dt, float(orc.q_values.max() - orc.q_values.min()))
            assert np.max(np.abs(qv - orc.q_values)) <= qtol
            if rec.q_action != orc.q_action:
                assert orc.q_values[rec.q_action] >= orc.q_values.max() - qtol
                rep.substitutions += 1
                diverged = qnet_policy
        if not diverged:
            assert rec.k_eff == orc.k_eff, (rec, orc.l, orc.k_eff)
            if orc.k_eff:  # with no drafts no exit layer is used
                assert rec.l == orc.l, (rec, orc.l)
            n_same = 0
            while n_same < orc.k_eff and rec.drafts[n_same] == orc.drafts[n_same]:
                n_same += 1
            if orc.k_eff:
                zd = eng.logits(3)
                for j in range(min(n_same + 1, orc.k_eff)):
                    if check_drafts:
                        rep.row(dt, zd[j], st.last_draft_logits[j])
                    if rec.drafts[j] != orc.drafts[j]:
                        rep.token(dt, rec.drafts[j], st.last_draft_logits[j])
                        diverged = True
            zv = eng.logits(0)
            for j in range(min(n_same, orc.k_eff) + 1):
                rep.row(dt, zv[j], st.last_verify_logits[j])
                g = int(np.argmax(zv[j]))
                if g != orc.verify[j]:
                    rep.token(dt, g, st.last_verify_logits[j])
                    diverged = True
        if not diverged:
            assert rec.accepted == orc.accepted and rec.emitted == orc.emitted, (rec, orc)
            assert rec.seq_len == orc.seq_len and rec.pending == st.pending
            sl, pend, table = eng.lede_get_kv_state()
            assert (sl, pend) == (orc.seq_len, st.pending)
            assert table == orc.block_table, (table, orc.block_table)
            assert abs(rec.reward - orc.reward) < 1e-5
        else:
            eng.lede_truncate(c0)
            eng.lede_prefill([pending0] + orc.emitted[:-1])
            eng.lede_set_pending(st.pending)
            sl, pend, table = eng.lede_get_kv_state()
            assert (sl, pend) == (st.c, st.pending)
            assert table == orc.block_table
    return rep


# ---- speculative sampling -------------------------------------------------------

CDF_EPS = 2e-5   # fp32 running sums against the fp64 CDF


def _cdf_interval(w, v):
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    c = c / c[-1]
    return (c[v - 1] if v > 0 else 0.0), c[v]


def draw_consistent(w, v, u, delta):
    """v is an inverse-CDF draw of u from weights w up to delta in the CDF."""
    if v < 0 or v >= len(w) or w[v] <= 0:
        return False
    lo, hi = _cdf_interval(w, v)
    return lo - delta <= u <= hi + delta


def draw_split(wa, wb):
    """Probability over a shared uniform u that the inverse-CDF draws from
    the weights wa and wb differ: the measure of the u for which they do.
    Between consecutive points of the two CDFs both draws are constant."""
    ca = np.cumsum(np.asarray(wa, dtype=np.float64))
    cb = np.cumsum(np.asarray(wb, dtype=np.float64))
    if not (ca[-1] > 0 and cb[-1] > 0):
        return 1.0  # an empty residual: the draw falls back to another rule
    ca, cb = ca / ca[-1], cb / cb[-1]
    pts = np.unique(np.concatenate([[0.0, 1.0], ca, cb]))
    mid = 0.5 * (pts[:-1] + pts[1:])
    differ = np.searchsorted(ca, mid, side="right") != np.searchsorted(cb, mid, side="right")
    return float(np.sum(np.diff(pts)[differ]))


def near_tie_bound(mu, alpha=1e-3):
    """Largest substitution count consistent at level alpha with decisions
    whose divergence probabilities sum to mu: the Poisson(mu) upper quantile,
    whose tail bounds that of any sum of independent Bernoulli variables with
    that mean."""
    n, term = 0, np.exp(-mu)
    cdf = term
    while 1.0 - cdf > alpha:
        n += 1
        term *= mu / n
        cdf += term
    return n


def _spread(eps, T):
    """Bound on how far a CDF or a probability ratio moves when every logit
    moves by at most eps (softmax at temperature T)."""
    return 2.0 * (np.exp(2.0 * eps / T) - 1.0) + CDF_EPS


def _decisions(zd, zv, drafts, u, T):
    """The acceptance count and the draw weights of the token after it, from
    one set of logits (rows of drafts, rows of verify)."""
    k = len(drafts)
    p = [om.probs_at(zv[j], T) for j in range(k + 1)]
    q = [om.probs_at(zd[i], T) for i in range(k)]
    a = 0
    while a < k and u[om.SAMPLE_SLOTS + a] * q[a][drafts[a]] < p[a][drafts[a]]:
        a += 1
    w = np.maximum(p[a] - q[a], 0.0) if a < k else p[a]
    return a, w, p, q


def check_sampled(eng, st: SSDState, model, n_total, actions, T, rep: Report, step0=0):
    """Self-speculative sampling on the GPU against the oracle, step by step,
    with the same uniforms.  Every GPU decision must follow the rule on the
    GPU's own logits (to fp32 rounding); it must equal the oracle's decision
    unless the oracle's margin is within what the logit tolerance allows (a
    near-tie substitution, after which the GPU is resynchronised onto the
    oracle's committed state).  Integers are bit-exact otherwise."""
    import lede_inputs as li
    dt = model.dtype
    i = 0
    while len(st.out) < n_total:
        l, k = actions[i % len(actions)]
        u = li.step_uniforms(step0 + i)
        i += 1
        c0, pending0 = st.c, st.pending
        n_rem = n_total - len(st.out)
        orc = st.step_sampled(int(l), int(k), n_total, T, u)
        rec = eng.lede_step_sampled((int(l), int(k)), T, u, n_remaining=n_rem)
        rep.steps += 1
        assert rec.k_eff == orc.k_eff
        ke = orc.k_eff
        zd = eng.logits(3)[:ke] if ke else np.zeros((0, model.vocab))
        zv = eng.logits(0)
        assert len(zv) == ke + 1
        diverged = False
        eps = 0.0
        # drafts: each row compared while the token histories agree
        for j in range(ke):
            rep.row(dt, zd[j], st.last_draft_logits[j])
            eps = max(eps, float(np.max(np.abs(zd[j] - st.last_draft_logits[j]))))
            g = rec.drafts[j]
            assert draw_consistent(om.probs_at(zd[j], T), g, u[j], CDF_EPS), ("draft draw", j)
            rep.expected_substitutions += draw_split(om.probs_at(zd[j], T), st.last_q_rows[j])
            if g != orc.drafts[j]:
                assert draw_consistent(st.last_q_rows[j], g, u[j], _spread(eps, T)), ("draft", j)
                diverged = True
                break
        if not diverged:
            for j in range(ke + 1):
                rep.row(dt, zv[j], st.last_verify_logits[j])
                eps = max(eps, float(np.max(np.abs(zv[j] - st.last_verify_logits[j]))))
            a_g, w_g, p_g, q_g = _decisions(zd, zv, rec.drafts, u, T)
            assert a_g == rec.accepted, ("acceptance on the GPU's own logits", a_g, rec.accepted)
            assert draw_consistent(w_g, rec.emitted[-1], u[2 * om.SAMPLE_SLOTS], CDF_EPS), "final draw"
            a_o, w_o, p_o, q_o = _decisions(st.last_draft_logits, st.last_verify_logits, orc.drafts, u, T)
            assert a_o == orc.accepted
            # acceptance tests up to the first rejection on either side: u < p / q
            for j in range(min(a_g, a_o, ke - 1) + 1 if ke else 0):
                d = orc.drafts[j]
                rep.expected_substitutions += abs(min(1.0, p_g[j][d] / q_g[j][d]) - min(1.0, p_o[j][d] / q_o[j][d]))
            if a_g == a_o:
                rep.expected_substitutions += draw_split(w_g, w_o)
            if a_g != a_o:
                j = min(a_g, a_o)
                d = orc.drafts[j]
                margin = abs(u[om.SAMPLE_SLOTS + j] * q_o[j][d] - p_o[j][d])
                assert margin <= _spread(eps, T) * (p_o[j][d] + q_o[j][d]), ("acceptance", j, margin)
                diverged = True
            elif rec.emitted[-1] != orc.emitted[-1]:
                assert draw_consistent(w_o, rec.emitted[-1], u[2 * om.SAMPLE_SLOTS], _spread(eps, T)), "final"
                diverged = True
        if not diverged:
            assert rec.accepted == orc.accepted and rec.emitted == orc.emitted, (rec, orc)
            sl, pend, table = eng.lede_get_kv_state()
            assert (sl, pend) == (orc.seq_len, st.pending)
            assert table == orc.block_table
            assert abs(rec.reward - orc.reward) < 1e-5
        else:
            rep.substitutions += 1
            eng.lede_truncate(c0)
            eng.lede_prefill([pending0] + orc.emitted[:-1])
            eng.lede_set_pending(st.pending)
            sl, pend, table = eng.lede_get_kv_state()
            assert (sl, pend) == (st.c, st.pending)
            assert table == orc.block_table
    return rep


# ---- the paper's exit policy ------------------------------------------------------

def _qnet_lipschitz(w):
    """|dQ| <= lip * max |ds| for the policy MLP (ReLU is 1-Lipschitz)."""
    l1 = np.abs(w["w1"].astype(np.float64)).sum(axis=1)
    return float(np.max(np.abs(w["w2"].astype(np.float64)) @ l1))


def check_policy(eng, st: SSDState, model, n_total, policy, rep: Report, logit_eps=None):
    """Greedy steps under the paper's exit policy on the GPU against the
    oracle's step_paper: decision by decision the kind and index must match,
    the state within the feature tolerance and the Q-values within what the
    network turns it into; an action may differ only where the oracle's
    Q-margin is within that tolerance (a near tie: the GPU is resynchronised
    onto the oracle's committed state and trace).  Without a near tie the
    drafts, acceptance, tokens, KV state and trace must match."""
    dt = model.dtype
    lip = _qnet_lipschitz(policy)
    i = 0
    while len(st.out) < n_total:
        i += 1
        c0, pending0 = st.c, st.pending
        n_rem = n_total - len(st.out)
        orc = st.step_paper(n_total, policy)
        rec = eng.lede_step_policy(n_remaining=n_rem)
        log = eng.policy_log()
        rep.steps += 1
        diverged = False
        for j, d in enumerate(orc.decisions):
            kind, idx, s_o, q_o, a_o = d
            if kind == "draft":
                # its input tokens are drafts 1 .. idx-1: a near tie in one of
                # them changes every later state
                for t in range(idx - 1):
                    if rec.drafts[t] != orc.drafts[t]:
                        rep.token(dt, rec.drafts[t], st.last_draft_logits[t])
                        diverged = True
                        break
                if diverged:
                    break
            assert j < len(log), ("GPU made fewer decisions", j, len(log))
            g = log[j]
            assert int(g[0]) == (0 if kind == "layer" else 1) and int(g[1]) == idx, (j, g, d)
            eps = logit_eps if logit_eps is not None else 1e-4
            f_tol = 4.0 * eps + 1e-4 * (1 + np.abs(s_o))
            assert np.all(np.abs(g[2:5] - s_o) <= f_tol), ("state", j, g[2:5], s_o)
            q_tol = lip * float(np.max(f_tol)) + 1e-3 * (1 + np.max(np.abs(q_o)))
            assert np.all(np.abs(g[5:7] - q_o) <= q_tol), ("Q", j, g[5:7], q_o)
            if int(g[7]) != a_o:
                assert abs(q_o[1] - q_o[0]) <= 2 * q_tol, ("action", j, q_o, g)
                diverged = True
                break
        if not diverged:
            assert len(log) == len(orc.decisions)
            assert (rec.l, rec.k_eff) == (orc.l, orc.k_eff), (rec, orc.l, orc.k_eff)
            n_same = 0
            while n_same < orc.k_eff and rec.drafts[n_same] == orc.drafts[n_same]:
                n_same += 1
            if n_same < orc.k_eff:          # a near tie inside the draft argmax
                zd = eng.logits(3)
                rep.token(dt, rec.drafts[n_same], st.last_draft_logits[n_same])
                diverged = True
        if not diverged:
            zv = eng.logits(0)
            for j in range(orc.k_eff + 1):
                rep.row(dt, zv[j], st.last_verify_logits[j])
                gtok = int(np.argmax(zv[j]))
                if gtok != orc.verify[j]:
                    rep.token(dt, gtok, st.last_verify_logits[j])
                    diverged = True
                    break
        if not diverged:
            assert rec.accepted == orc.accepted and rec.emitted == orc.emitted
            sl, pend, table = eng.lede_get_kv_state()
            assert (sl, pend) == (orc.seq_len, st.pending) and table == orc.block_table
            tr = eng.lede_get_trace()
            assert len(tr) == len(st.trace.vals)
            assert np.allclose(tr, np.array(st.trace.vals), atol=4 * (logit_eps or 1e-4) + 1e-4)
        else:
            rep.substitutions += 1
            eng.lede_truncate(c0)
            eng.lede_prefill([pending0] + orc.emitted[:-1])
            eng.lede_set_pending(st.pending)
            eng.lede_set_trace(np.array(st.trace.vals, dtype=np.float32))
    return rep
