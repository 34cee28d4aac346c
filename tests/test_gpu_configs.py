"""Parity at the full widths of the Llama-3-8B, Llama-2-13B and Llama-2-70B
shapes (every projection, head count, head dimension, vocabulary and prompt
length as in those workloads) with fewer layers, so that the fp64 oracle's
prefill stays within a minute:

* Llama-3-8B shape, 8 layers: GQA 32/8, FFN 14336, vocabulary 128256, RoPE
  base 5e5, 1024-token prompt, actions chosen by the Q-network
  (4096 -> 256 -> 4 exits x 4 lengths);
* Llama-2-13B shape, 4 layers: 4096-token prompt, so attention splits over
  64+ KV pages; seeded uniform (l, k) schedule;
* Llama-2-70B shape, 4 layers: d = 8192, GQA 64/8, FFN 28672, 2048-token
  prompt; seeded schedule.

Each case: prefill logits, then self-speculative steps against the oracle
(every draft row, every verify row up to the acceptance point, acceptance,
KV length, page table), and greedy SSD == greedy AR on the GPU.

The same shapes also run at full depth (32, 40 and 80 layers) with the
workloads' own action sets: the Llama-3-8B Q-network over its real grid
(16 exits x 8 lengths = 128 actions), the seeded schedules l 5..20 (13B) and
l 10..40 (70B).  There the prompts are short and four generated layer
weight sets (two for the 70B shape) repeat over the depth (layer j uses set
j mod 4, on the GPU and in the oracle alike), so that host generation and
the oracle's fp64 passes stay within minutes; every layer still has its own
KV cache, exit index and weights in the arena.  The 80-layer shape is past
the depths of the paper's models: its bf16 bound scales by sqrt(80 / 40)
(oracle.model.Tolerance)."""
import time

import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import WORKLOADS, shrink
from oracle.model import OracleDecoder, SSDState, argmax_info
from tests.parity import Report, check_ssd, say

pytestmark = [pytest.mark.gpu, pytest.mark.slow]
torch = pytest.importorskip("torch")

CASES = {
    "llama3-8b-L8": dict(wl="llama3-8b", layers=8, exits=(2, 4, 6, 8), policy="qnet", prompt=1024),
    "llama2-13b-L4": dict(wl="llama2-13b", layers=4, exits=(1, 2, 3, 4), policy="schedule", prompt=4096),
    "llama2-70b-L4": dict(wl="llama2-70b", layers=4, exits=(1, 2, 3, 4), policy="schedule", prompt=2048),
}
N_TOTAL = 16     # tokens per parity run: full draft lengths first, then k_eff clipped by the budget


def _setup(case):
    spec = CASES[case]
    wl = WORKLOADS[spec["wl"]]
    m = shrink(wl.model, name=case, n_layers=spec["layers"], exits=spec["exits"])
    t = time.time()
    w = li.weights(m)
    q = li.qnet_weights(m)
    prompt = li.prompt(wl, length=spec["prompt"])
    say("%s: weights %.1f s, prompt %d" % (case, time.time() - t, len(prompt)))
    return spec, wl, m, w, q, prompt


@pytest.mark.parametrize("case", list(CASES))
def test_config_shape_parity(case):
    from paper_2606_03113_amd import Engine
    spec, wl, m, w, q, prompt = _setup(case)
    max_ctx = len(prompt) + 64
    eng = Engine(m, max_ctx=max_ctx, k_max=8)
    eng.load_weights(w, q)
    eng.lede_set_options(0, 1)
    g = eng.lede_prefill(prompt)
    z_gpu = eng.logits(0)[-1]
    dec = OracleDecoder(m, w, max_ctx, q)
    st = SSDState(dec, -(-max_ctx // 64), 64)
    st.pager.ensure(len(prompt))
    h = None
    for off in range(0, len(prompt), 256):
        t = time.time()
        h = dec.forward(prompt[off:off + 256], off, m.n_layers)
        say("  oracle prefill rows %d..%d  %.1f s" % (off, off + len(h) - 1, time.time() - t))
    z = dec.head(h[-1:])[0]
    info = argmax_info(z)
    st.c, st.pending, st.out = len(prompt), info.token, [info.token]
    rep = Report()
    rep.row(m.dtype, z_gpu, z)
    if not rep.token(m.dtype, g, z):
        eng.lede_set_pending(st.pending)
    if spec["policy"] == "qnet":
        check_ssd(eng, st, m, N_TOTAL, [(1, 1)], rep, qnet_policy=True)
    else:
        sched = np.stack([li.uniform_int(li.SEED_SCHEDULE, li.STREAM_SCHED_L, 64, 1, m.n_layers),
                          li.uniform_int(li.SEED_SCHEDULE, li.STREAM_SCHED_K, 64, 1, 8)], 1)
        check_ssd(eng, st, m, N_TOTAL, sched, rep)
    say("  steps=%d rows=%d max_err/tol=%.3g max_abs=%.3g substitutions=%d" %
        (rep.steps, rep.rows, rep.max_err_rel, rep.max_err_abs, rep.substitutions))
    assert rep.steps >= 2

    # greedy SSD == greedy AR on the GPU (row-independent verify path)
    n_gen = 20
    eng.lede_truncate(len(prompt))
    eng.lede_set_pending(g)
    eng.lede_set_options(0, 0)
    ar = [g]
    while len(ar) < n_gen:
        a, em, _ = eng.lede_verify()
        ar += em
    eng.lede_truncate(len(prompt))
    eng.lede_set_pending(g)
    out = [g]
    i = 0
    while len(out) < n_gen:
        act = (m.exits[0], 1 + i % 8)
        rec = eng.lede_step(act, n_remaining=n_gen - len(out))
        out += rec.emitted
        i += 1
    assert out == ar


FULL = {
    "llama3-8b-L32": dict(wl="llama3-8b", prompt=16, n_total=10, distinct=4),
    "llama2-13b-L40": dict(wl="llama2-13b", prompt=16, n_total=8, distinct=4),
    "llama2-70b-L80": dict(wl="llama2-70b", prompt=8, n_total=4, distinct=2),
}


@pytest.mark.parametrize("case", list(FULL))
def test_config_full_depth_parity(case):
    from paper_2606_03113_amd import Engine
    spec = FULL[case]
    wl = WORKLOADS[spec["wl"]]
    m = wl.model
    t = time.time()
    nd = spec["distinct"]
    w4 = li.weights(shrink(m, n_layers=nd))
    w = dict(w4, layers=[w4["layers"][j % nd] for j in range(m.n_layers)])
    q = li.qnet_weights(m)
    prompt = li.prompt(wl, length=spec["prompt"])
    say("%s: %d layers (%d distinct), %d actions, weights %.1f s, prompt %d" %
        (case, m.n_layers, nd, m.n_actions, time.time() - t, len(prompt)))
    max_ctx = len(prompt) + 48
    eng = Engine(m, max_ctx=max_ctx, k_max=8)
    t = time.time()
    eng.load_weights(w, q)
    say("  loaded in %.1f s" % (time.time() - t))
    eng.lede_set_options(0, 1)
    g = eng.lede_prefill(prompt)
    dec = OracleDecoder(m, w, max_ctx, q)
    st = SSDState(dec, -(-max_ctx // 64), 64)
    t = time.time()
    st.pager.ensure(len(prompt))
    z = dec.head(dec.forward(prompt, 0, m.n_layers)[-1:])[0]
    info = argmax_info(z)
    st.c, st.pending, st.out = len(prompt), info.token, [info.token]
    say("  oracle prefill %.1f s" % (time.time() - t))
    rep = Report(depth=m.n_layers)
    rep.row(m.dtype, eng.logits(0)[-1], z)
    if not rep.token(m.dtype, g, z):
        eng.lede_set_pending(st.pending)
    t = time.time()
    if wl.policy == "qnet":
        check_ssd(eng, st, m, spec["n_total"], [(1, 1)], rep, qnet_policy=True)
    else:
        sched = np.stack([li.uniform_int(li.SEED_SCHEDULE, li.STREAM_SCHED_L, 64, *wl.sched_l),
                          li.uniform_int(li.SEED_SCHEDULE, li.STREAM_SCHED_K, 64, *wl.sched_k)], 1)
        check_ssd(eng, st, m, spec["n_total"], sched, rep)
    say("  steps=%d rows=%d max_err/tol=%.3g max_abs=%.3g substitutions=%d  %.1f s" %
        (rep.steps, rep.rows, rep.max_err_rel, rep.max_err_abs, rep.substitutions, time.time() - t))
    assert rep.steps >= 2
