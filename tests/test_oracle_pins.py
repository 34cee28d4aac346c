"""Pins of the CPU oracle against facts fixed outside it: library routines
(torch float64), closed forms, invariants, brute force on tiny inputs, and
the equivalences the method guarantees (Section 1 / 2.2: greedy
self-speculative decoding reproduces greedy autoregressive decoding; exit at
l = L is the full model)."""
import ctypes
import itertools
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import lede_inputs as li
from lede_inputs.configs import TINY, WORKLOADS, shrink
from oracle import model as om
from oracle.model import (OracleDecoder, Pager, accept_length, greedy_ar, metrics, reward,
                          ssd_generate)
from tests.torch_reference import TorchReference, round_bf16

MICRO_F32 = shrink(TINY, name="micro-f32", n_layers=2, d_model=32, n_heads=4, n_kv_heads=4,
                   head_dim=8, ffn_dim=40, vocab=48, qnet_hidden=16)
MICRO_BF16 = shrink(MICRO_F32, name="micro-bf16", dtype="bf16")
MICRO_GQA = shrink(MICRO_F32, name="micro-gqa", n_heads=4, n_kv_heads=2, rope_base=500000.0)
MICRO_GQA_BF16 = shrink(MICRO_GQA, name="micro-gqa-bf16", dtype="bf16")


def _ptr(a):
    return a.ctypes.data


def _random_gains(model, w, seed=11):
    """Replace the unit RMSNorm gains by random ones so that a gain mix-up is
    visible (the synthetic models use gains of 1)."""
    dt = model.dtype
    def g(stream):
        return li.normal(seed, stream, model.d_model, 0.5, dt)
    w = dict(w)
    w["final_norm"] = g(1)
    w["layers"] = [dict(lw, attn_norm=g(10 + 2 * j), ffn_norm=g(11 + 2 * j))
                   for j, lw in enumerate(w["layers"])]
    return w


def _dec(model, max_ctx=64, weights=None, qnet=False, library=None):
    w = weights if weights is not None else li.weights(model)
    q = li.qnet_weights(model) if qnet else None
    return OracleDecoder(model, w, max_ctx, q, library=library), w


# ---- scalar building blocks ------------------------------------------------

def test_round_bf16_matches_torch_on_fp32_values():
    L = om.lib()
    rng = np.random.default_rng(0)
    vals = np.concatenate([rng.standard_normal(4000).astype(np.float32) * 10.0 ** rng.integers(-6, 6, 4000),
                           np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0], dtype=np.float32)])
    got = np.array([L.oracle_round_bf16(float(v)) for v in vals])
    ref = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(got, ref)
    # ties to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> 1
    assert L.oracle_round_bf16(1.0 + 2 ** -8) == 1.0
    assert L.oracle_round_bf16(1.0 + 3 * 2 ** -8) == 1.0 + 2 ** -6


def _rope(v, pos, base):
    x = np.array(v, dtype=np.float64)
    om.lib().oracle_rope(_ptr(x), len(x), pos, base)
    return x


def test_rope_closed_form_values():
    # hd = 4, base = 10000: theta_0 = 1, theta_1 = 10000^(-1/2) = 0.01
    e0 = _rope([1, 0, 0, 0], 1, 10000.0)
    assert np.allclose(e0, [math.cos(1), 0, math.sin(1), 0], atol=1e-15)
    e1 = _rope([0, 1, 0, 0], 3, 10000.0)
    assert np.allclose(e1, [0, math.cos(0.03), 0, math.sin(0.03)], atol=1e-15)
    e3 = _rope([0, 0, 0, 1], 2, 10000.0)
    assert np.allclose(e3, [0, -math.sin(0.02), 0, math.cos(0.02)], atol=1e-15)


def test_rope_identity_at_zero_norm_and_relative_position():
    rng = np.random.default_rng(1)
    for hd in (8, 64, 128):
        q, k = rng.standard_normal(hd), rng.standard_normal(hd)
        assert np.array_equal(_rope(q, 0, 10000.0), q)
        for p in (1, 17, 4000):
            assert abs(np.linalg.norm(_rope(q, p, 10000.0)) - np.linalg.norm(q)) < 1e-12
        d1 = _rope(q, 9, 10000.0) @ _rope(k, 4, 10000.0)
        d2 = _rope(q, 105, 10000.0) @ _rope(k, 100, 10000.0)
        assert abs(d1 - d2) < 1e-10


def test_attend_matches_sdpa_and_special_cases():
    L = om.lib()
    rng = np.random.default_rng(2)
    hd, n = 16, 11
    q, K, V = rng.standard_normal(hd), rng.standard_normal((n, hd)), rng.standard_normal((n, hd))
    out, pr = np.empty(hd), np.empty(n)
    L.oracle_attend(_ptr(q), _ptr(K), _ptr(V), n, hd, _ptr(out), _ptr(pr))
    ref = F.scaled_dot_product_attention(torch.from_numpy(q)[None, None], torch.from_numpy(K)[None],
                                         torch.from_numpy(V)[None])[0, 0].numpy()
    assert np.allclose(out, ref, atol=1e-13)
    assert abs(pr.sum() - 1.0) < 1e-14
    # one key: the output is that value exactly
    out1, pr1 = np.empty(hd), np.empty(1)
    L.oracle_attend(_ptr(q), _ptr(K[:1].copy()), _ptr(V[:1].copy()), 1, hd, _ptr(out1), _ptr(pr1))
    assert np.array_equal(out1, V[0]) and pr1[0] == 1.0
    # zero query: uniform weights, the output is the mean value
    z = np.zeros(hd)
    L.oracle_attend(_ptr(z), _ptr(K), _ptr(V), n, hd, _ptr(out), _ptr(pr))
    assert np.allclose(out, V.mean(0), atol=1e-14)


def test_rmsnorm_matches_library_and_unit_rms():
    L = om.lib()
    rng = np.random.default_rng(3)
    x, g = rng.standard_normal(257) * 3, rng.standard_normal(257)
    out = np.empty(257)
    L.oracle_rmsnorm_f64(_ptr(x), _ptr(g), 257, 1e-5, _ptr(out))
    ref = F.rms_norm(torch.from_numpy(x), (257,), torch.from_numpy(g), eps=1e-5).numpy()
    assert np.allclose(out, ref, atol=1e-13)
    ones = np.ones(257)
    L.oracle_rmsnorm_f64(_ptr(x), _ptr(ones), 257, 0.0, _ptr(out))
    assert abs(np.sqrt(np.mean(out ** 2)) - 1.0) < 1e-14


# ---- decoder brute force (no KV cache, library ops) -------------------------

@pytest.mark.parametrize("model", [MICRO_F32, MICRO_BF16, MICRO_GQA, MICRO_GQA_BF16],
                         ids=lambda m: m.name)
def test_decoder_matches_torch_bruteforce(model):
    dec, w = _dec(model, weights=_random_gains(model, li.weights(model)))
    ref = TorchReference(model, w)
    prompt = li.uniform_int(7, 99, 9, 0, model.vocab - 1)
    toks, infos = greedy_ar(dec, prompt, 6)
    rtoks, rrows = ref.greedy(prompt, 6)
    assert toks == rtoks
    # logits of every generated position agree to fp64 rounding
    dec2, _ = _dec(model, weights=w)
    seq = list(prompt) + toks[:-1]
    h = dec2.forward(seq, 0, model.n_layers)
    z = dec2.head(h)
    zr = ref.logits(seq).numpy()
    assert np.max(np.abs(z - zr)) < 1e-10
    # early-exit logits at every layer agree too (shared final norm + head)
    for l in range(model.n_layers + 1):
        dec3, _ = _dec(model, weights=w)
        zl = dec3.head(dec3.forward(seq, 0, l))
        assert np.max(np.abs(zl - ref.logits(seq, l).numpy())) < 1e-10


def test_incremental_rows_equal_batched_rows_bitwise():
    """A row's result does not depend on how many rows share the call."""
    for model in (MICRO_F32, MICRO_BF16):
        w = li.weights(model)
        seq = li.uniform_int(7, 98, 12, 0, model.vocab - 1)
        a, _ = _dec(model, weights=w)
        ha = a.forward(seq, 0, model.n_layers)
        b, _ = _dec(model, weights=w)
        hb = np.concatenate([b.forward(seq[:5], 0, model.n_layers)] +
                            [b.forward([t], 5 + i, model.n_layers) for i, t in enumerate(seq[5:])])
        assert np.array_equal(ha, hb)


def test_gqa_equals_mha_with_duplicated_kv_heads():
    g = MICRO_GQA
    w = li.weights(g)
    mha = shrink(g, n_kv_heads=g.n_heads)
    group = g.n_heads // g.n_kv_heads
    w2 = {k: v for k, v in w.items() if k != "layers"}
    w2["layers"] = []
    for lw in w["layers"]:
        d = dict(lw)
        for name in ("wk", "wv"):
            heads = lw[name].reshape(g.n_kv_heads, g.head_dim, g.d_model)
            d[name] = np.ascontiguousarray(np.repeat(heads, group, axis=0).reshape(-1, g.d_model))
        w2["layers"].append(d)
    seq = li.uniform_int(7, 97, 10, 0, g.vocab - 1)
    a, _ = _dec(g, weights=w)
    b, _ = _dec(mha, weights=w2)
    assert np.array_equal(a.head(a.forward(seq, 0, g.n_layers)), b.head(b.forward(seq, 0, g.n_layers)))


# ---- the self-speculative loop ------------------------------------------------

def _tiny_variant(dtype):
    return TINY if dtype == "f32" else shrink(TINY, name="tiny-bf16", dtype="bf16")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ssd_equals_greedy_ar(dtype):
    model = _tiny_variant(dtype)
    w = li.weights(model)
    prompt = li.prompt(WORKLOADS["tiny"], length=20)
    n = 30
    ar, _ = greedy_ar(_dec(model, 96, weights=w)[0], prompt, n)
    acts = [(1, 1), (2, 4), (3, 8), (4, 3)]
    for l, k in acts:
        st, recs = ssd_generate(_dec(model, 96, weights=w)[0], prompt, n, [(l, k)], n_pages=4,
                                page_size=16)
        assert st.out == ar
        assert sum(len(r.emitted) for r in recs) == n - 1
    sched = li.uniform_int(5, 5, 64, 1, 4).reshape(-1, 1)
    ks = li.uniform_int(5, 6, 64, 1, 8).reshape(-1, 1)
    st, recs = ssd_generate(_dec(model, 96, weights=w)[0], prompt, n,
                            np.concatenate([sched, ks], 1), n_pages=4, page_size=16)
    assert st.out == ar


def test_exit_at_last_layer_accepts_every_draft():
    model = TINY
    w = li.weights(model)
    prompt = li.prompt(WORKLOADS["tiny"], length=16)
    st, recs = ssd_generate(_dec(model, 96, weights=w)[0], prompt, 25, [(model.n_layers, 4)],
                            n_pages=4, page_size=16)
    assert all(r.accepted == r.k_eff for r in recs)
    # and the exit-L draft logits equal the verify logits bitwise
    for r in recs:
        for di, vi in zip(r.draft_info, r.verify_info):
            assert di.token == vi.token and di.top == vi.top


@pytest.mark.parametrize("l", [1, 2, 3])
def test_zeroed_upper_layers_accept_every_draft(l):
    model = shrink(TINY, name="tiny-bf16", dtype="bf16")
    w = li.weights(model)
    for j in range(l, model.n_layers):
        w["layers"][j]["wo"] = np.zeros_like(w["layers"][j]["wo"])
        w["layers"][j]["wd"] = np.zeros_like(w["layers"][j]["wd"])
    prompt = li.prompt(WORKLOADS["tiny"], length=16)
    st, recs = ssd_generate(_dec(model, 96, weights=w)[0], prompt, 30, [(l, 5)], n_pages=4,
                            page_size=16)
    assert all(r.accepted == r.k_eff for r in recs)
    assert metrics(recs)["acc"] == 1.0


def test_acceptance_scan_exhaustive():
    for k in range(0, 5):
        for drafts in itertools.product(range(3), repeat=k):
            for verify in itertools.product(range(3), repeat=k + 1):
                eq = np.array([d == v for d, v in zip(drafts, verify)], dtype=np.int64)
                expect = int(np.cumprod(eq).sum()) if k else 0
                assert accept_length(list(drafts), list(verify)) == expect


def test_reward_closed_form_cases():
    """Section 3.1.3 reward, worked by hand in tests/golden/reward_cases.txt."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "reward_cases.txt")
    n = 0
    for line in open(path):
        line = line.split("#")[0].strip()
        if not line:
            continue
        a, k, l, L, r = line.split()
        assert reward(int(a), int(k), int(l), int(L)) == pytest.approx(float(r), abs=1e-12)
        n += 1
    assert n >= 6


def test_pager_invariants():
    rng = np.random.default_rng(4)
    order = list(rng.permutation(40))
    p = Pager(40, 8, order)
    c = 13
    p.ensure(c)
    for _ in range(300):
        k = int(rng.integers(0, 9))
        p.ensure(c + k + 1)
        assert len(p.table) * 8 >= c + k + 1
        a = int(rng.integers(0, k + 1))
        before = list(p.table)
        c += a + 1
        p.truncate(c)
        keep = -(-c // 8)
        assert p.table == before[:keep]
        assert len(set(p.table)) == len(p.table)
        assert set(p.table).isdisjoint(p.free)
        assert len(p.table) + len(p.free) == 40
        if c > 200:
            c = 13
            p.truncate(c)
    # freed pages come back to the same logical slots
    p2 = Pager(10, 4)
    p2.ensure(20)
    t0 = list(p2.table)
    p2.truncate(5)
    p2.ensure(20)
    assert p2.table == t0


def test_ssd_state_invariant_and_block_table():
    model = TINY
    w = li.weights(model)
    prompt = li.prompt(WORKLOADS["tiny"], length=20)
    st, recs = ssd_generate(_dec(model, 128, weights=w)[0], prompt, 40, [(2, 8)], n_pages=8,
                            page_size=16)
    for i, r in enumerate(recs):
        n_gen = 1 + sum(len(x.emitted) for x in recs[:i + 1])
        assert r.seq_len == len(prompt) + n_gen - 1
        assert len(r.block_table) == -(-r.seq_len // 16)


def test_qnet_matches_library_mlp():
    model = MICRO_F32
    dec, w = _dec(model, qnet=True)
    q = dec.qnet_w
    s = np.random.default_rng(5).standard_normal(model.d_model)
    got = dec.qnet(s)
    t = lambda a: torch.from_numpy(np.asarray(a, dtype=np.float64))
    ref = F.linear(torch.relu(F.linear(t(s), t(q["w1"]), t(q["b1"]))), t(q["w2"]), t(q["b2"])).numpy()
    assert np.allclose(got, ref, atol=1e-14)


def test_qnet_policy_picks_argmax_action():
    w = WORKLOADS["tiny"]
    model = w.model
    dec, W = _dec(model, 128, qnet=True)
    prompt = li.prompt(w, length=16)
    st, recs = ssd_generate(dec, prompt, 24, [(1, 1)], n_pages=8, page_size=16, qnet=True,
                            use_qnet_action=True)
    K = len(model.lengths)
    for r in recs:
        if r.k_eff == 0:
            continue
        assert r.q_action == int(np.argmax(r.q_values))
        assert r.l == model.exits[r.q_action // K]
        assert r.k_req == model.lengths[r.q_action % K]
    ar, _ = greedy_ar(_dec(model, 128, weights=W)[0], prompt, 24)
    assert st.out == ar
