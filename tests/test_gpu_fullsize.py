"""Parity at the full Llama-2-7B-shaped configuration, in the launch
configuration bench.py times (512-token prompt, exit layer 8, draft length
4, Q-network logged): the prefill's last-row logits and the first
self-speculative steps (every draft row, every verify row up to the
acceptance point, the Q-values, acceptance, KV length and page table)
against the fp64 oracle, then two steps with verify reuse; and, as a property that holds at any size, greedy
self-speculative output equal to greedy autoregressive output on the GPU."""
import time

import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import WORKLOADS
from oracle.model import OracleDecoder, SSDState, argmax_info
from tests.parity import Report, check_ssd, say

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
torch = pytest.importorskip("torch")

WL = WORKLOADS["llama2-7b"]


@pytest.fixture(scope="module")
def inputs():
    t = time.time()
    say("generating %s weights" % WL.model.name)
    w = li.weights(WL.model)
    q = li.qnet_weights(WL.model)
    say("  %.1f s" % (time.time() - t))
    return w, q, li.prompt(WL)


def _engine(w, q, debug=1):
    from paper_2606_03113_amd import Engine
    eng = Engine(WL.model, max_ctx=WL.max_ctx, k_max=8)
    eng.load_weights(w, q)
    eng.lede_set_options(0, debug)
    return eng


def test_fullsize_prefill_and_ssd_steps_match_oracle(inputs):
    w, q, prompt = inputs
    m = WL.model
    eng = _engine(w, q)
    say("gpu prefill", len(prompt))
    g = eng.lede_prefill(prompt)
    z_gpu = eng.logits(0)[-1]
    dec = OracleDecoder(m, w, WL.prompt_len + 64, q)
    st = SSDState(dec, -(-(WL.prompt_len + 64) // 64), 64)
    st.pager.ensure(len(prompt))
    h = None
    for off in range(0, len(prompt), 64):
        t = time.time()
        h = dec.forward(prompt[off:off + 64], off, m.n_layers)
        say("  oracle prefill rows %d..%d  %.1f s" % (off, off + len(h) - 1, time.time() - t))
    z = dec.head(h[-1:])[0]
    st.c, st.pending, st.out = len(prompt), argmax_info(z).token, [argmax_info(z).token]
    rep = Report()
    rep.row(m.dtype, z_gpu, z)
    if not rep.token(m.dtype, g, z):
        eng.lede_set_pending(st.pending)
    say("  prefill logits max err / tol = %.3g" % rep.max_err_rel)
    l, k = WL.fixed
    check_ssd(eng, st, m, 1 + 3 * (k + 1), [(l, k)], rep, qnet_log=True)
    say("  ssd steps=%d rows=%d max_err/tol=%.3g max_abs=%.3g substitutions=%d" %
        (rep.steps, rep.rows, rep.max_err_rel, rep.max_err_abs, rep.substitutions))
    assert rep.steps >= 3
    # two more steps with the verify starting at the exit layer
    eng.lede_set_verify_reuse(True)
    n0 = rep.steps
    check_ssd(eng, st, m, len(st.out) + 2 * (k + 1), [(l, k)], rep, qnet_log=True)
    say("  verify-reuse steps=%d max_err/tol=%.3g substitutions=%d" %
        (rep.steps - n0, rep.max_err_rel, rep.substitutions))
    assert rep.steps >= n0 + 2


def test_fullsize_ssd_equals_ar_on_gpu(inputs):
    w, q, prompt = inputs
    n = 24
    eng = _engine(w, q, debug=0)
    say("gpu greedy AR", n)
    ar = [eng.lede_prefill(prompt)]
    while len(ar) < n:
        a, em, _ = eng.lede_verify()
        ar += em
    eng.lede_truncate(len(prompt))
    eng.lede_set_pending(ar[0])
    say("gpu SSD (8, 4)")
    out = [ar[0]]
    while len(out) < n:
        rec = eng.lede_step(WL.fixed, n_remaining=n - len(out))
        out += rec.emitted
    assert out == ar
