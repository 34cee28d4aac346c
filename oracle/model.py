"""CPU ORACLE -- test infrastructure only (see the package docstring).

The decoding loop of self-speculative decoding with a learned (exit layer,
draft length) policy, written plainly in fp64 on top of ``lede_oracle.c``.

Paper references: Section 1 and 2.2 (self-speculative decoding: early layers
draft, the full model verifies in parallel); Section 3.1 (the MDP: a state
from the hidden state at a candidate exit layer, an action, the reward of
Section 3.1.3); Section 3.2 (greedy action from a small MLP Q-network);
Section 3.3 (exit layer chosen during the first forward pass of a step, then
drafting at that layer); Section 4.1 (batch 1, greedy decoding and sampling
at temperature 0.6, speculative-sampling acceptance, metrics E, d,
acceptance rate).

Readings where the paper is silent:
* the early-exit head is the shared final RMSNorm + LM head;
* acceptance is greedy: the longest prefix of drafts equal to the full
  model's argmax, plus the full model's token after it (the bonus token);
* verification recomputes all L layers for the k+1 rows and overwrites the
  drafted KV; positions past the committed length are discarded;
* the Q-network reads the final-normed hidden state of the pending token at
  the smallest candidate exit layer and scores the joint (exit, length) grid;
* argmax ties go to the lowest index; no EOS: exactly N tokens are produced,
  with k clamped to N - n_gen - 1;
* the reward is summed over the drafts up to and including the first
  rejected one; continue penalties do not arise with a joint action;
* the paper's exit policy: the confidence feature is the mean -log p of the
  5 most likely tokens, the entropy is in nats, both at temperature 1; the
  trace is the mean -log max p of the full model over the last 20 committed
  tokens (the prompt's next token included; 0 before any); a 'continue' after
  a draft pass ends drafting without keeping that pass's token; at most 12
  drafts;
* sampling: draws are inverse-CDF in index order from a uniform the caller
  supplies; acceptance keeps draft d while u < p(d) / q(d); the token after
  a rejection comes from the normalised max(0, p - q), after k acceptances
  from p (the speculative-sampling rule the paper cites).
"""
from __future__ import annotations

import ctypes
import math
from collections import deque
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

from .build import build, library_path

_lib = None


class _OracleModel(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int), ("d", ctypes.c_int), ("nq", ctypes.c_int),
        ("nkv", ctypes.c_int), ("hd", ctypes.c_int), ("ffn", ctypes.c_int),
        ("vocab", ctypes.c_int), ("is_bf16", ctypes.c_int), ("max_ctx", ctypes.c_int),
        ("eps", ctypes.c_double), ("rope_base", ctypes.c_double),
        ("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("head", ctypes.c_void_p),
        ("attn_norm", ctypes.POINTER(ctypes.c_void_p)), ("wq", ctypes.POINTER(ctypes.c_void_p)),
        ("wk", ctypes.POINTER(ctypes.c_void_p)), ("wv", ctypes.POINTER(ctypes.c_void_p)),
        ("wo", ctypes.POINTER(ctypes.c_void_p)), ("ffn_norm", ctypes.POINTER(ctypes.c_void_p)),
        ("wg", ctypes.POINTER(ctypes.c_void_p)), ("wu", ctypes.POINTER(ctypes.c_void_p)),
        ("wd", ctypes.POINTER(ctypes.c_void_p)),
        ("kcache", ctypes.c_void_p), ("vcache", ctypes.c_void_p),
    ]


def lib(path: Optional[str] = None):
    """The oracle C library (built on first use).  ``path`` loads another
    build of it (the tests use this to load deliberately broken copies)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        build()
        _lib = _bind(ctypes.CDLL(library_path()))
    return _lib


def _bind(L):
    vp, i, d = ctypes.c_void_p, ctypes.c_int, ctypes.c_double
    L.oracle_forward.argtypes = [ctypes.POINTER(_OracleModel), vp, i, i, i, vp]
    L.oracle_forward.restype = i
    L.oracle_head.argtypes = [ctypes.POINTER(_OracleModel), vp, i, vp, vp]
    L.oracle_head.restype = i
    L.oracle_linear_f32.argtypes = [vp, vp, i, i, vp, vp]
    L.oracle_rope.argtypes = [vp, i, i, d]
    L.oracle_rmsnorm_f64.argtypes = [vp, vp, i, d, vp]
    L.oracle_attend.argtypes = [vp, vp, vp, i, i, vp, vp]
    L.oracle_matvec.argtypes = [vp, i, i, i, vp, i, vp]
    L.oracle_round_bf16.argtypes = [d]
    L.oracle_round_bf16.restype = d
    return L


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


class OracleDecoder:
    """fp64 decoder with a position-indexed KV cache.

    ``weights`` is the dict from ``lede_inputs.weights`` (logical row-major
    arrays; bf16 as uint16).  ``qnet`` is the dict from
    ``lede_inputs.qnet_weights`` or None.
    """

    def __init__(self, model, weights: dict, max_ctx: int, qnet: Optional[dict] = None,
                 library=None):
        self.m = model
        self.w = weights
        self.qnet_w = qnet
        self.max_ctx = max_ctx
        self.L = library if library is not None else lib()
        kvd = model.n_kv_heads * model.head_dim
        self.kcache = np.zeros((model.n_layers, max_ctx, kvd), dtype=np.float64)
        self.vcache = np.zeros((model.n_layers, max_ctx, kvd), dtype=np.float64)
        n = model.n_layers
        arr = ctypes.c_void_p * n

        def per_layer(name):
            return arr(*[_ptr(weights["layers"][j][name]) for j in range(n)])

        self._keep = {name: per_layer(name) for name in
                      ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")}
        s = _OracleModel()
        s.n_layers, s.d, s.nq, s.nkv = n, model.d_model, model.n_heads, model.n_kv_heads
        s.hd, s.ffn, s.vocab = model.head_dim, model.ffn_dim, model.vocab
        s.is_bf16 = 1 if model.dtype == "bf16" else 0
        s.max_ctx, s.eps, s.rope_base = max_ctx, model.rms_eps, model.rope_base
        s.embed, s.final_norm, s.head = _ptr(weights["embed"]), _ptr(weights["final_norm"]), _ptr(weights["head"])
        for name, a in self._keep.items():
            setattr(s, name, ctypes.cast(a, ctypes.POINTER(ctypes.c_void_p)))
        s.kcache, s.vcache = _ptr(self.kcache), _ptr(self.vcache)
        self.s = s

    # -- decoder -----------------------------------------------------------
    def forward(self, tokens: Sequence[int], pos0: int, l_end: int) -> np.ndarray:
        """Hidden states [T][d] after layers [0, l_end) of tokens at positions
        pos0..pos0+T-1; writes their KV for those layers."""
        toks = np.ascontiguousarray(tokens, dtype=np.int32)
        out = np.empty((len(toks), self.m.d_model), dtype=np.float64)
        rc = self.L.oracle_forward(ctypes.byref(self.s), _ptr(toks), len(toks), pos0, l_end, _ptr(out))
        if rc != 0:
            raise ValueError("oracle_forward rejected its arguments")
        return out

    def head(self, hidden: np.ndarray, with_normed: bool = False):
        """Logits [T][V] of the shared final RMSNorm + LM head."""
        h = np.ascontiguousarray(hidden, dtype=np.float64)
        T = h.shape[0]
        logits = np.empty((T, self.m.vocab), dtype=np.float64)
        normed = np.empty_like(h) if with_normed else None
        rc = self.L.oracle_head(ctypes.byref(self.s), _ptr(h), T, _ptr(logits),
                                _ptr(normed) if with_normed else None)
        if rc != 0:
            raise ValueError("oracle_head failed")
        return (logits, normed) if with_normed else logits

    def qnet(self, state: np.ndarray) -> np.ndarray:
        """Q-values over the joint (exit, length) grid: W2 ReLU(W1 s + b1) + b2
        (Section 3.2: a small MLP; greedy action = argmax)."""
        q = self.qnet_w
        s = np.ascontiguousarray(state, dtype=np.float64)
        hdim = q["w1"].shape[0]
        hid = np.empty(hdim, dtype=np.float64)
        self.L.oracle_linear_f32(_ptr(q["w1"]), _ptr(q["b1"]), hdim, s.shape[0], _ptr(s), _ptr(hid))
        hid = np.maximum(hid, 0.0)
        out = np.empty(q["w2"].shape[0], dtype=np.float64)
        self.L.oracle_linear_f32(_ptr(q["w2"]), _ptr(q["b2"]), out.shape[0], hdim, _ptr(hid), _ptr(out))
        return out

    def qnet_state(self, token: int, pos: int, l_min: int) -> np.ndarray:
        """Final-RMSNorm'd layer-l_min hidden state of `token` at `pos` (the
        Q-network's observation; not rounded)."""
        h = self.forward([token], pos, l_min)
        _, normed = self.head(h, with_normed=True)
        return normed[0]


def matvec(W: np.ndarray, x: np.ndarray, is_bf16: bool) -> np.ndarray:
    """y[t][n] = sum_k W[n][k] x[t][k] in fp64 (W: uint16 bf16 bits or float32)."""
    W = np.ascontiguousarray(W)
    x = np.ascontiguousarray(x, dtype=np.float64)
    T, K = x.shape
    N = W.shape[0]
    y = np.empty((T, N), dtype=np.float64)
    lib().oracle_matvec(_ptr(W), int(is_bf16), N, K, _ptr(x), T, _ptr(y))
    return y


def argmax_lowest(z: np.ndarray) -> int:
    """Index of the maximum, lowest index on ties."""
    return int(np.argmax(z))  # numpy returns the first occurrence


@dataclass
class ArgmaxInfo:
    token: int
    top: float
    second: float
    lo: float

    @property
    def margin(self) -> float:
        return self.top - self.second

    @property
    def span(self) -> float:
        return self.top - self.lo


def argmax_info(z: np.ndarray) -> ArgmaxInfo:
    t = argmax_lowest(z)
    top = float(z[t])
    rest = np.delete(z, t)
    return ArgmaxInfo(t, top, float(rest.max()) if rest.size else -math.inf, float(z.min()))


@dataclass
class Tolerance:
    """Logit tolerance: absolute for fp32 models, relative to the row's logit
    range for bf16 models.  The bf16 bound is set for the depths of the
    paper's models (Section 4.1: LLaMA-2 7B and 13B, up to 40 layers).  A
    deeper bf16 model accumulates more rounding decisions that the fp32 GPU
    path and the fp64 oracle take differently at the same bf16 quantisation
    points, and the logit difference grows about as the square root of the
    depth, so past ref_depth layers the bound scales by sqrt(depth /
    ref_depth)."""
    abs_f32: float = 1e-4
    rel_bf16: float = 2e-2
    ref_depth: int = 40

    def of(self, dtype: str, span: float, depth: int = 0) -> float:
        if dtype == "f32":
            return self.abs_f32
        return self.rel_bf16 * span * math.sqrt(max(1.0, depth / self.ref_depth))


def accept_length(drafts: Sequence[int], verify: Sequence[int]) -> int:
    """Greedy acceptance: largest a <= k with drafts[m] == verify[m] for all
    m < a (drafts[m] is d_{m+1}, verify[m] is the full model's token after
    the m-th verify row)."""
    a = 0
    while a < len(drafts) and drafts[a] == verify[a]:
        a += 1
    return a


def reward(a: int, k_eff: int, l_star: int, n_layers: int) -> float:
    """Section 3.1.3: each accepted draft earns 1 + (L - l*)/L, the first
    rejected draft earns -2 + (L - l*)/L; later drafts are not scored."""
    if k_eff == 0:
        return 0.0
    lam = (n_layers - l_star) / n_layers
    return a * (1.0 + lam) + (0.0 if a == k_eff else (-2.0 + lam))


class Pager:
    """Page allocator of the paged KV cache (the paper is silent; this is the
    reading both implementations follow).  Page size S; a free list seeded
    with an order; allocation pops the front; truncation frees the pages
    wholly past the new length and pushes them back to the front in
    descending logical order, so they are reused in the same order."""

    def __init__(self, n_pages: int, page_size: int, order: Optional[Sequence[int]] = None):
        self.S = page_size
        self.free = deque(range(n_pages) if order is None else order)
        self.table: List[int] = []

    def ensure(self, n_positions: int):
        while len(self.table) * self.S < n_positions:
            if not self.free:
                raise MemoryError("KV pool exhausted")
            self.table.append(self.free.popleft())

    def truncate(self, new_len: int):
        keep = -(-new_len // self.S)
        for j in range(len(self.table) - 1, keep - 1, -1):
            self.free.appendleft(self.table[j])
        self.table = self.table[:keep]


@dataclass
class StepRecord:
    l: int
    k_req: int
    k_eff: int
    accepted: int
    emitted: List[int]
    drafts: List[int]
    verify: List[int]
    reward: float
    seq_len: int
    q_action: int = -1
    q_values: Optional[np.ndarray] = None
    draft_info: List[ArgmaxInfo] = field(default_factory=list)
    verify_info: List[ArgmaxInfo] = field(default_factory=list)
    block_table: List[int] = field(default_factory=list)
    decisions: list = field(default_factory=list)   # exit policy: (kind, layer / draft, state, Q, action)
    c_trace: float = 0.0


def greedy_ar(dec: OracleDecoder, prompt: Sequence[int], n_gen: int):
    """Plain greedy autoregressive decoding of the full model: the result the
    self-speculative loop must reproduce exactly.  Returns (tokens, infos)."""
    L = dec.m.n_layers
    h = dec.forward(prompt, 0, L)
    info = argmax_info(dec.head(h[-1:])[0])
    toks, infos = [info.token], [info]
    pos = len(prompt)
    while len(toks) < n_gen:
        h = dec.forward([toks[-1]], pos, L)
        pos += 1
        info = argmax_info(dec.head(h)[0])
        toks.append(info.token)
        infos.append(info)
    return toks, infos


# ---- speculative sampling (Section 4.1: sampling at temperature T with
# speculative-sampling acceptance) -------------------------------------------

SAMPLE_SLOTS = 16   # per-step uniforms: drafts [0, 16), acceptance [16, 32), residual / bonus [32]


def probs_at(z: np.ndarray, T: float) -> np.ndarray:
    """softmax(z / T) in fp64."""
    x = np.asarray(z, dtype=np.float64) / T
    e = np.exp(x - x.max())
    return e / e.sum()


def sample_inverse_cdf(w: np.ndarray, u: float) -> int:
    """Inverse-CDF draw from non-negative weights w (any scale): the smallest
    index v whose running sum in index order exceeds u * sum(w); if rounding
    leaves none, the last index of positive weight."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    hit = np.nonzero(c > float(u) * c[-1])[0]
    if len(hit):
        return int(hit[0])
    return int(np.nonzero(np.asarray(w) > 0)[0][-1])


def speculative_accept(p_rows: Sequence[np.ndarray], q_rows: Sequence[np.ndarray], drafts: Sequence[int],
                       u_acc: Sequence[float], u_res: float):
    """Speculative-sampling acceptance of k drafts.

    p_rows[j] is the target distribution after j drafts (j = 0..k), q_rows[i]
    the draft distribution draft i+1 was sampled from.  Draft i+1 is kept
    while u_acc[i] < p_i(d) / q_i(d); at the first rejection the next token is
    drawn from the normalised residual max(0, p_i - q_i), and after k
    acceptances from p_k.  Returns (accepted count, next token)."""
    k = len(drafts)
    a = 0
    while a < k:
        d = int(drafts[a])
        if float(u_acc[a]) * q_rows[a][d] < p_rows[a][d]:
            a += 1
        else:
            break
    if a < k:
        y = sample_inverse_cdf(np.maximum(p_rows[a] - q_rows[a], 0.0), u_res)
    else:
        y = sample_inverse_cdf(p_rows[k], u_res)
    return a, y


# ---- the paper's exit policy (Sections 3.1.1, 3.1.2, 3.3) -------------------

POLICY_TOPK = 5        # tokens in the confidence feature
POLICY_TRACE = 20      # window of the confidence trace
POLICY_MAX_DRAFT = 12  # longest speculation of the adaptive drafting


def log_probs(z: np.ndarray) -> np.ndarray:
    """log softmax(z) in fp64."""
    x = np.asarray(z, dtype=np.float64)
    x = x - x.max()
    return x - math.log(np.exp(x).sum())


def exit_features(z: np.ndarray, c_trace: float) -> np.ndarray:
    """State at a candidate exit layer (Section 3.1.1) from the next-token
    logits z at that layer: the mean negative log-probability of the top-k
    tokens, the entropy of the distribution, and the confidence trace."""
    lp = log_probs(z)
    top = np.sort(lp)[-POLICY_TOPK:]
    return np.array([-top.mean(), -float(np.sum(np.exp(lp) * lp)), float(c_trace)])


def exit_qnet(state: np.ndarray, w: dict) -> np.ndarray:
    """Q(s, continue), Q(s, exit): W2 ReLU(W1 s + b1) + b2 in fp64 (Section 3.2)."""
    hid = np.maximum(w["w1"].astype(np.float64) @ state + w["b1"].astype(np.float64), 0.0)
    return w["w2"].astype(np.float64) @ hid + w["b2"].astype(np.float64)


class ConfidenceTrace:
    """The last POLICY_TRACE values of -log max p of the full model's
    distribution at committed positions; C_trace is their mean, 0 while
    empty."""

    def __init__(self):
        self.vals: deque = deque(maxlen=POLICY_TRACE)

    def push_logits(self, z: np.ndarray):
        self.vals.append(-float(log_probs(z).max()))

    def value(self) -> float:
        return float(np.mean(self.vals)) if self.vals else 0.0


class SSDState:
    """(c, pending token, n_gen) plus the pager, the committed output and the
    confidence trace of the exit policy."""

    def __init__(self, dec: OracleDecoder, n_pages: int, page_size: int, order=None):
        self.dec = dec
        self.pager = Pager(n_pages, page_size, order)
        self.c = 0
        self.pending = -1
        self.out: List[int] = []
        self.last_draft_logits: List[np.ndarray] = []
        self.last_verify_logits: Optional[np.ndarray] = None
        self.trace = ConfidenceTrace()

    def prefill(self, prompt: Sequence[int]) -> ArgmaxInfo:
        self.pager.ensure(len(prompt))
        h = self.dec.forward(prompt, 0, self.dec.m.n_layers)
        z = self.dec.head(h[-1:])[0]
        info = argmax_info(z)
        self.c = len(prompt)
        self.pending = info.token
        self.out = [info.token]
        self.trace.push_logits(z)
        return info

    def step(self, l: int, k: int, n_total: int, qnet: bool = False, use_qnet_action: bool = False) -> StepRecord:
        """One draft / verify / accept / commit step (Sections 2.2, 3.3)."""
        dec, m = self.dec, self.dec.m
        L = m.n_layers
        n_gen = len(self.out)
        k_eff = max(0, min(k, n_total - n_gen - 1))
        q_values, q_action = None, -1
        if qnet and k_eff > 0:
            l_min = min(m.exits)
            q_values = dec.qnet(dec.qnet_state(self.pending, self.c, l_min))
            q_action = argmax_lowest(q_values)
            if use_qnet_action:
                l = m.exits[q_action // len(m.lengths)]
                k = m.lengths[q_action % len(m.lengths)]
                k_eff = max(0, min(k, n_total - n_gen - 1))
        if not 1 <= l <= L:
            raise ValueError("exit layer out of range")
        self.pager.ensure(self.c + k_eff + 1)
        drafts, dinfo, dz = [], [], []
        u = self.pending
        for i in range(1, k_eff + 1):
            h = dec.forward([u], self.c + i - 1, l)
            zi = dec.head(h)[0]
            info = argmax_info(zi)
            drafts.append(info.token)
            dinfo.append(info)
            dz.append(zi)
            u = info.token
        h = dec.forward([self.pending] + drafts, self.c, L)
        z = dec.head(h)
        self.last_draft_logits = dz
        self.last_verify_logits = z
        vinfo = [argmax_info(z[i]) for i in range(k_eff + 1)]
        verify = [v.token for v in vinfo]
        a = accept_length(drafts, verify)
        emitted = drafts[:a] + [verify[a]]
        self.c += a + 1
        self.pending = verify[a]
        self.out.extend(emitted)
        self.pager.truncate(self.c)
        for j in range(a + 1):
            self.trace.push_logits(z[j])
        return StepRecord(l=l, k_req=k, k_eff=k_eff, accepted=a, emitted=emitted, drafts=drafts,
                          verify=verify, reward=reward(a, k_eff, l, L), seq_len=self.c,
                          q_action=q_action, q_values=q_values, draft_info=dinfo, verify_info=vinfo,
                          block_table=list(self.pager.table))


    def step_sampled(self, l: int, k: int, n_total: int, T: float, uniforms: Sequence[float]) -> StepRecord:
        """One step of self-speculative sampling at temperature T: draft i
        is drawn from softmax(z_draft / T) with uniforms[i-1], the drafts are
        verified by speculative-sampling acceptance with uniforms[16 + i - 1],
        and the token after them comes from the residual (or, after k
        acceptances, the target) distribution with uniforms[32]."""
        dec, m = self.dec, self.dec.m
        L = m.n_layers
        n_gen = len(self.out)
        k_eff = max(0, min(k, n_total - n_gen - 1))
        if not 1 <= l <= L:
            raise ValueError("exit layer out of range")
        self.pager.ensure(self.c + k_eff + 1)
        drafts, dz, q_rows = [], [], []
        tok = self.pending
        for i in range(1, k_eff + 1):
            h = dec.forward([tok], self.c + i - 1, l)
            zi = dec.head(h)[0]
            qi = probs_at(zi, T)
            tok = sample_inverse_cdf(qi, uniforms[i - 1])
            drafts.append(tok)
            dz.append(zi)
            q_rows.append(qi)
        h = dec.forward([self.pending] + drafts, self.c, L)
        z = dec.head(h)
        self.last_draft_logits = dz
        self.last_verify_logits = z
        p_rows = [probs_at(z[j], T) for j in range(k_eff + 1)]
        a, y = speculative_accept(p_rows, q_rows, drafts, uniforms[SAMPLE_SLOTS:SAMPLE_SLOTS + k_eff],
                                  uniforms[2 * SAMPLE_SLOTS])
        emitted = drafts[:a] + [y]
        self.c += a + 1
        self.pending = y
        self.out.extend(emitted)
        self.pager.truncate(self.c)
        for j in range(a + 1):
            self.trace.push_logits(z[j])
        self.last_p_rows, self.last_q_rows = p_rows, q_rows
        return StepRecord(l=l, k_req=k, k_eff=k_eff, accepted=a, emitted=emitted, drafts=drafts,
                          verify=[argmax_lowest(z[j]) for j in range(k_eff + 1)],
                          reward=reward(a, k_eff, l, L), seq_len=self.c, block_table=list(self.pager.table))


    def step_paper(self, n_total: int, policy: dict, k_cap: int = POLICY_MAX_DRAFT) -> StepRecord:
        """One greedy step under the paper's exit policy (Section 3.3).

        Exit layer: the pending token goes up the candidate exit layers in
        order; at each, the state (exit_features of that layer's next-token
        logits, with the trace of committed confidences) is scored by the
        2-action Q-network, and the first 'exit' (forced at the last
        candidate) fixes l*.  Draft 1 is the argmax there.  Draft length:
        each further draft pass at l* is scored the same way; 'exit' keeps its
        argmax as the next draft, 'continue' ends drafting (that token is not
        kept), and at most k_cap drafts are made.  Then verify, greedy
        acceptance and commit as in step().  ``decisions`` lists
        (kind, layer or draft index, state, Q-values, action)."""
        dec, m = self.dec, self.dec.m
        L = m.n_layers
        cands = sorted(m.exits)
        n_gen = len(self.out)
        k_lim = max(0, min(k_cap, n_total - n_gen - 1))
        ct = self.trace.value()
        decisions = []
        drafts, dz = [], []
        l_star = cands[-1]
        if k_lim > 0:
            for ci, l in enumerate(cands):
                z = dec.head(dec.forward([self.pending], self.c, l))[0]
                st = exit_features(z, ct)
                q = exit_qnet(st, policy)
                act = argmax_lowest(q)
                decisions.append(("layer", l, st, q, act))
                if act == 1 or ci == len(cands) - 1:
                    l_star = l
                    break
            drafts.append(argmax_lowest(z))
            dz.append(z)
            while len(drafts) < k_lim:
                z = dec.head(dec.forward([drafts[-1]], self.c + len(drafts), l_star))[0]
                st = exit_features(z, ct)
                q = exit_qnet(st, policy)
                act = argmax_lowest(q)
                decisions.append(("draft", len(drafts) + 1, st, q, act))
                if act != 1:
                    break
                drafts.append(argmax_lowest(z))
                dz.append(z)
        k_eff = len(drafts)
        self.pager.ensure(self.c + k_eff + 1)
        h = dec.forward([self.pending] + drafts, self.c, L)
        zv = dec.head(h)
        self.last_draft_logits = dz
        self.last_verify_logits = zv
        vinfo = [argmax_info(zv[i]) for i in range(k_eff + 1)]
        verify = [v.token for v in vinfo]
        a = accept_length(drafts, verify)
        emitted = drafts[:a] + [verify[a]]
        self.c += a + 1
        self.pending = verify[a]
        self.out.extend(emitted)
        self.pager.truncate(self.c)
        for j in range(a + 1):
            self.trace.push_logits(zv[j])
        return StepRecord(l=l_star, k_req=k_cap, k_eff=k_eff, accepted=a, emitted=emitted, drafts=drafts,
                          verify=verify, reward=reward(a, k_eff, l_star, L), seq_len=self.c,
                          verify_info=vinfo, block_table=list(self.pager.table), decisions=decisions, c_trace=ct)


def ssd_generate(dec: OracleDecoder, prompt: Sequence[int], n_total: int, actions, n_pages: int,
                 page_size: int = 64, qnet: bool = False, use_qnet_action: bool = False):
    """Self-speculative greedy generation of n_total tokens.  ``actions`` is a
    sequence of (l, k) per step (ignored for the action when
    use_qnet_action).  Returns (state, records)."""
    st = SSDState(dec, n_pages, page_size)
    st.prefill(prompt)
    recs = []
    i = 0
    while len(st.out) < n_total:
        l, k = actions[min(i, len(actions) - 1)]
        recs.append(st.step(int(l), int(k), n_total, qnet=qnet, use_qnet_action=use_qnet_action))
        i += 1
    return st, recs


def metrics(records: Sequence[StepRecord]) -> dict:
    """Section 4.1 metrics over steps that drafted: E (mean exit layer),
    d (mean draft length), acceptance rate (accepted / drafted)."""
    drafted = [r for r in records if r.k_eff > 0]
    if not drafted:
        return {"E": float("nan"), "d": float("nan"), "acc": float("nan"), "steps": len(records)}
    return {"E": sum(r.l for r in drafted) / len(drafted),
            "d": sum(r.k_eff for r in drafted) / len(drafted),
            "acc": sum(r.accepted for r in drafted) / sum(r.k_eff for r in drafted),
            "steps": len(records),
            "tokens": sum(len(r.emitted) for r in records)}
