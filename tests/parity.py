"""GPU-vs-oracle parity protocol shared by the GPU tests.

Logits agree within max-abs 1e-4 for fp32 models and within 2e-2 x (logit
range of the oracle's row) for bf16 models.  Every GPU argmax g must satisfy
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

from oracle.model import OracleDecoder, SSDState, Tolerance

TOL = Tolerance()


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def tol_of(dtype: str, z: np.ndarray) -> float:
    return TOL.of(dtype, float(z.max() - z.min()))


@dataclass
class Report:
    rows: int = 0
    max_err_rel: float = 0.0     # max |dz| / tol over rows
    max_err_abs: float = 0.0
    substitutions: int = 0
    steps: int = 0
    notes: List[str] = field(default_factory=list)

    def row(self, dtype, z_gpu, z_orc):
        t = tol_of(dtype, z_orc)
        err = float(np.max(np.abs(z_gpu.astype(np.float64) - z_orc)))
        self.rows += 1
        self.max_err_abs = max(self.max_err_abs, err)
        self.max_err_rel = max(self.max_err_rel, err / t)
        assert err <= t, "logit error %.3g exceeds tolerance %.3g" % (err, t)

    def token(self, dtype, g: int, z_orc: np.ndarray) -> bool:
        """True if g is the oracle's argmax; False for an allowed near-tie."""
        t = tol_of(dtype, z_orc)
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
