"""Decode parity at long contexts on small models: 1100 and 2200 positions
(18 and 35 KV pages), where the attention's page combine folds its pages in
two and three groups of 16 before folding the groups, and where a partial
block may take more than one page.  Greedy AR and self-speculative steps
against the CPU oracle, through the C ABI."""
import numpy as np
import pytest

import lede_inputs as li
from lede_inputs.configs import TINY, shrink
from oracle.model import SSDState
from tests.parity import Report, check_ar, check_ssd, make_decoder, say

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

LONG_BF16 = shrink(TINY, name="long-bf16", n_layers=2, dtype="bf16", exits=(1, 2))
LONG_128 = shrink(TINY, name="long-hd128-bf16", n_layers=2, d_model=512, n_heads=4, n_kv_heads=4,
                  head_dim=128, ffn_dim=704, vocab=1024, dtype="bf16", qnet_hidden=32,
                  exits=(1, 2), lengths=(1, 2, 4, 8))
LONG_GQA_F32 = shrink(TINY, name="long-gqa-f32", n_layers=2, d_model=256, n_heads=8, n_kv_heads=2,
                      head_dim=64, ffn_dim=512, vocab=512, dtype="f32", qnet_hidden=32,
                      exits=(1, 2), lengths=(1, 3, 5))
CASES = [(LONG_BF16, 1100), (LONG_128, 2200), (LONG_GQA_F32, 1100)]


@pytest.mark.parametrize("model,prompt_len", CASES, ids=lambda v: v.name if hasattr(v, "name") else str(v))
def test_long_context_ar_and_ssd(model, prompt_len):
    from paper_2606_03113_amd import Engine
    say("long context", model.name, prompt_len)
    max_ctx = prompt_len + 80
    w = li.weights(model)
    q = li.qnet_weights(model)
    prompt = li.uniform_int(3, 40, prompt_len, 0, model.vocab - 1)

    eng = Engine(model, max_ctx=max_ctx, k_max=8)
    eng.load_weights(w, q)
    eng.lede_set_options(0, 1)
    dec = make_decoder(model, w, q, max_ctx)
    rep = Report()
    check_ar(eng, dec, model, prompt, 6, rep)
    eng.close()

    eng = Engine(model, max_ctx=max_ctx, k_max=8)
    eng.load_weights(w, q)
    eng.lede_set_options(0, 1)
    dec = make_decoder(model, w, q, max_ctx)
    n_pages = -(-max_ctx // 64)
    st = SSDState(dec, n_pages, 64)
    g = eng.lede_prefill(prompt)
    st.prefill(prompt)
    if g != st.pending:
        rep.token(model.dtype, g, dec.head(dec.forward(prompt, 0, model.n_layers)[-1:])[0])
        eng.lede_set_pending(st.pending)
    L = model.n_layers
    check_ssd(eng, st, model, 1 + 16, [(1, 4), (L, 8), (1, 1), (L, 3)], rep, qnet_log=True)
    eng.close()
    say("  rows=%d steps=%d max_err/tol=%.3g subs=%d" % (rep.rows, rep.steps, rep.max_err_rel, rep.substitutions))
