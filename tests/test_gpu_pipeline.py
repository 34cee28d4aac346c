"""Pipelined steps (lede_step_submit / lede_step_collect: up to two forced
greedy steps in flight on one stream) against synchronous lede_step on a
twin engine.  Both make the same launches on the same device state, so every
record must be bit-identical: emitted tokens, acceptance, drafts, Q-network
action and maximum, reward, committed length and pending token.  The
schedule crosses page boundaries and covers k = 0, exits at the first and
last layer and draft lengths cut by n_remaining; a synchronous step after
the pipeline drains checks the KV and block table it left.  The pipelined
stream is also checked against the oracle's SSD loop (Sections 2.2, 3.3) up
to its first near tie."""
import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle.model import SSDState
from tests.parity import make_decoder, say, tol_of

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

TINY_BF16 = shrink(TINY, name="tiny-bf16", dtype="bf16")
SMALL_GQA = shrink(TINY, name="small-gqa-bf16", n_layers=3, d_model=512, n_heads=8, n_kv_heads=2,
                   head_dim=64, ffn_dim=1408, vocab=2048, dtype="bf16", rope_base=500000.0,
                   qnet_hidden=32, exits=(1, 2, 3), lengths=(1, 2, 4, 8))
MODELS = [TINY, TINY_BF16, SMALL_GQA]
MAX_CTX = 256
K_MAX = 12


def _engine(model, w, q, order):
    from paper_2606_03113_amd import Engine
    eng = Engine(model, max_ctx=MAX_CTX, n_pages=len(order), k_max=K_MAX)
    eng.load_weights(w, q)
    eng.lede_set_free_list(order)
    return eng


def _schedule(model, n):
    """(l, k, n_remaining) per step: seeded, with the special cases first."""
    L = model.n_layers
    big = 1 << 20
    sched = [(1, 3, big), (L, K_MAX, big), (2, 0, big), (1, 8, 1), (L, 5, 3), (1, 1, big), (L, 4, 2)]
    ls = li.uniform_int(3, 90, n, 1, L)
    ks = li.uniform_int(3, 91, n, 0, K_MAX)
    cut = li.uniform_int(3, 92, n, 0, 7)
    for i in range(n):
        sched.append((int(ls[i]), int(ks[i]), int(cut[i]) + 1 if cut[i] < 2 else big))
    return sched


def _fields(r):
    q_bits = int(np.float32(r.q_max).view(np.int32))
    return (r.l, r.k_req, r.k_eff, r.accepted, tuple(r.emitted), tuple(r.drafts), r.q_action, q_bits,
            float(r.reward), r.seq_len, r.pending)


def _near_tie(rows, dt):
    """Whether some row's top two logits are within twice the logit tolerance."""
    for z in rows:
        top = np.sort(np.asarray(z, dtype=np.float64))[-2:]
        if top[1] - top[0] <= 2 * tol_of(dt, np.asarray(z)):
            return True
    return False


@pytest.mark.parametrize("model", MODELS, ids=lambda m: m.name)
def test_pipelined_records_match_synchronous(model):
    from paper_2606_03113_amd.lede import MAX_IN_FLIGHT
    say("pipelined steps", model.name)
    w = li.weights(model)
    q = li.qnet_weights(model)
    n_pages = MAX_CTX // 64
    order = [int(x) for x in np.random.default_rng(11).permutation(n_pages)]
    sync, pipe = _engine(model, w, q, order), _engine(model, w, q, order)
    prompt = li.uniform_int(3, 50, 60, 0, model.vocab - 1)
    g = sync.lede_prefill(prompt)
    assert pipe.lede_prefill(prompt) == g
    # two steps in flight may each commit k + 1 tokens: stop well inside max_ctx
    sched = []
    c_hi = len(prompt)
    for l, k, n_rem in _schedule(model, 80):
        k_eff = max(0, min(k, n_rem - 1))
        if c_hi + (k_eff + 1) + MAX_IN_FLIGHT * (K_MAX + 1) > MAX_CTX:
            break
        sched.append((l, k, n_rem))
        c_hi += k_eff + 1
    want = [sync.lede_step((l, k), n_remaining=n, log_qnet=True) for l, k, n in sched]
    got = []
    for i, (l, k, n) in enumerate(sched):
        if i >= MAX_IN_FLIGHT:
            got.append(pipe.lede_step_collect())
        pipe.lede_step_submit((l, k), n_remaining=n, log_qnet=True)
    while len(got) < len(sched):
        got.append(pipe.lede_step_collect())
    for i, (a, b) in enumerate(zip(want, got)):
        assert _fields(a) == _fields(b), (i, sched[i], a, b)
    s_sync, s_pipe = sync.lede_get_kv_state(), pipe.lede_get_kv_state()
    assert s_sync[:2] == s_pipe[:2] and len(s_sync[2]) == len(s_pipe[2])
    crossed = want[-1].seq_len // 64 - len(prompt) // 64
    say("  %d steps, %d tokens, %d page boundaries" % (len(sched), want[-1].seq_len - len(prompt), crossed))
    assert crossed >= 1 and len(sched) >= 20
    # the pipeline drained: a synchronous step reads the KV and table it left
    assert _fields(sync.lede_step((1, 4), log_qnet=True)) == _fields(pipe.lede_step((1, 4), log_qnet=True))

    # the pipelined stream against the oracle, up to its first near tie
    dec = make_decoder(model, w, q, MAX_CTX)
    st = SSDState(dec, n_pages, 64, order)
    st.prefill(prompt)
    matched = 0
    for (l, k, n), r in zip(sched, got):
        orc = st.step(l, k, len(st.out) + n, qnet=True)
        same = (r.k_eff, r.accepted, r.emitted, r.drafts) == (orc.k_eff, orc.accepted, orc.emitted, orc.drafts)
        if not same:
            assert _near_tie(list(st.last_draft_logits) + list(st.last_verify_logits), model.dtype), \
                (matched, r, orc)
            break
        assert r.seq_len == orc.seq_len and r.pending == st.pending and abs(r.reward - orc.reward) < 1e-5
        if orc.q_values is not None and r.q_action >= 0:
            assert orc.q_values[r.q_action] >= orc.q_values.max() - tol_of(model.dtype, orc.q_values)
        matched += 1
    say("  oracle: %d of %d pipelined steps identical" % (matched, len(sched)))
    if model.dtype == "f32":
        assert matched == len(sched)


def test_pipeline_state_errors():
    from paper_2606_03113_amd.lede import LEDE_E_STATE, LedeError, MAX_IN_FLIGHT
    model = TINY
    w, q = li.weights(model), li.qnet_weights(model)
    eng = _engine(model, w, q, list(range(MAX_CTX // 64)))

    def code(f, *a, **kw):
        with pytest.raises(LedeError) as e:
            f(*a, **kw)
        return e.value.code

    assert code(eng.lede_step_submit, (1, 2)) == LEDE_E_STATE  # no prefill yet
    eng.lede_prefill(li.uniform_int(3, 51, 20, 0, model.vocab - 1))
    assert code(eng.lede_step_collect) == LEDE_E_STATE  # nothing submitted
    for _ in range(MAX_IN_FLIGHT):
        eng.lede_step_submit((1, 2), n_remaining=100)
    assert code(eng.lede_step_submit, (1, 2)) == LEDE_E_STATE  # pipeline full
    assert code(eng.lede_step, (1, 2)) == LEDE_E_STATE
    assert code(eng.lede_get_kv_state) == LEDE_E_STATE
    assert code(eng.lede_truncate, 20) == LEDE_E_STATE
    recs = [eng.lede_step_collect() for _ in range(MAX_IN_FLIGHT)]
    assert recs[1].seq_len == recs[0].seq_len + recs[1].accepted + 1
    assert eng.lede_get_kv_state()[0] == recs[1].seq_len
    eng.lede_set_options(1, 0)
    assert code(eng.lede_step_submit, (1, 2)) == LEDE_E_STATE  # graph replay is not pipelined
    eng.lede_set_options(0, 0)
    eng.lede_set_verify_reuse(True)
    assert code(eng.lede_step_submit, (1, 2)) == LEDE_E_STATE  # nor verify reuse


def test_steps_on_a_created_stream():
    """Forced steps with the Q-network logged (its hidden and output layers
    run on the library's second stream) on a stream the caller created, plain
    and pipelined, against the same steps on the default stream."""
    model = TINY_BF16
    w, q = li.weights(model), li.qnet_weights(model)
    order = list(range(MAX_CTX // 64))
    ref, eng = _engine(model, w, q, order), _engine(model, w, q, order)
    prompt = li.uniform_int(3, 52, 40, 0, model.vocab - 1)
    L = model.n_layers
    sched = [(1, 4), (L, 8), (2, 0), (L, 2), (1, 12), (2, 3)] * 3
    g = ref.lede_prefill(prompt)
    want = [ref.lede_step(a, log_qnet=True) for a in sched]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        assert eng.lede_prefill(prompt) == g
        half = len(sched) // 2
        got = [eng.lede_step(a, log_qnet=True) for a in sched[:half]]
        for i, a in enumerate(sched[half:]):
            if i >= 2:
                got.append(eng.lede_step_collect())
            eng.lede_step_submit(a, log_qnet=True)
        while len(got) < len(sched):
            got.append(eng.lede_step_collect())
    torch.cuda.synchronize()
    assert any(r.q_action >= 0 for r in want)
    for i, (a, b) in enumerate(zip(want, got)):
        assert _fields(a) == _fields(b), (i, sched[i], a, b)
