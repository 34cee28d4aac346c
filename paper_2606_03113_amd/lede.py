"""Thin ctypes binding of liblede (include/lede.h).

Argument marshalling only: every step of decoding runs in the library's HIP
kernels.  PyTorch provides device memory (the weight arena, KV pool,
workspace and weight staging buffers) and the stream handle.  There is no
fallback: if liblede.so is missing or no GPU is present, the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liblede.so")

LEDE_OK, LEDE_E_ARG, LEDE_E_STATE, LEDE_E_KV_FULL, LEDE_E_CTX_OVERFLOW, LEDE_E_HIP, LEDE_E_UNSUPPORTED = \
    0, -1, -2, -3, -4, -5, -6
STATUS = {0: "OK", -1: "E_ARG", -2: "E_STATE", -3: "E_KV_FULL", -4: "E_CTX_OVERFLOW", -5: "E_HIP",
          -6: "E_UNSUPPORTED"}

T_EMBED, T_FINAL_NORM, T_HEAD, T_ATTN_NORM, T_WQ, T_WK, T_WV, T_WO, T_FFN_NORM, T_WG, T_WU, T_WD, \
    T_QNET_W1, T_QNET_B1, T_QNET_W2, T_QNET_B2, T_EXIT_W1, T_EXIT_B1, T_EXIT_W2, T_EXIT_B2 = range(20)
LAYER_KINDS = {"attn_norm": T_ATTN_NORM, "wq": T_WQ, "wk": T_WK, "wv": T_WV, "wo": T_WO,
               "ffn_norm": T_FFN_NORM, "wg": T_WG, "wu": T_WU, "wd": T_WD}


class LedeConfig(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("max_ctx", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("n_pages", ctypes.c_int32), ("qnet_hidden", ctypes.c_int32), ("n_exits", ctypes.c_int32),
                ("n_lengths", ctypes.c_int32), ("exits", ctypes.c_int32 * 64), ("lengths", ctypes.c_int32 * 16),
                ("k_max", ctypes.c_int32), ("exit_qnet_hidden", ctypes.c_int32)]


class LedeProfEntry(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double), ("bytes", ctypes.c_double), ("launches", ctypes.c_int64)]


K_NCLASS = 10
K_NAMES = ["linear_vec", "linear_mfma", "attention", "norm", "qnet", "accept", "draft_phase", "verify_phase",
           "linear_vec_gx", "linear_mfma_lx"]
# rocprofv3 kernel symbol of each linear timing class (bf16 models)
K_SYMBOLS = {"linear_vec": "lede::k_linear<1, 0>", "linear_mfma": "lede::k_linear<1, 2>",
             "linear_vec_gx": "lede::k_linear<1, 1>", "linear_mfma_lx": "lede::k_linear<1, 3>"}


LAYER_TENSORS = 9  # LEDE_LAYER_TENSORS: attn_norm, wq, wk, wv, wo, ffn_norm, wg, wu, wd
LAYER_ORDER = ["attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"]
LOGITS_VERIFY, LOGITS_DRAFT = 0, 1


class LedeWeights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("head", ctypes.c_void_p),
                ("first_layer", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("layer", ctypes.POINTER(ctypes.c_void_p)),
                ("qnet_w1", ctypes.c_void_p), ("qnet_b1", ctypes.c_void_p), ("qnet_w2", ctypes.c_void_p),
                ("qnet_b2", ctypes.c_void_p), ("exit_w1", ctypes.c_void_p), ("exit_b1", ctypes.c_void_p),
                ("exit_w2", ctypes.c_void_p), ("exit_b2", ctypes.c_void_p)]


class LedeAction(ctypes.Structure):
    _fields_ = [("l", ctypes.c_int32), ("k", ctypes.c_int32)]


class LedeStepRecord(ctypes.Structure):
    _fields_ = [("l", ctypes.c_int32), ("k_req", ctypes.c_int32), ("k_eff", ctypes.c_int32),
                ("accepted", ctypes.c_int32), ("n_emitted", ctypes.c_int32), ("tokens", ctypes.c_int32 * 17),
                ("drafts", ctypes.c_int32 * 16), ("q_action", ctypes.c_int32), ("q_max", ctypes.c_float),
                ("reward", ctypes.c_float), ("seq_len", ctypes.c_int32), ("pending", ctypes.c_int32)]


EXPORTED = ["lede_region_bytes", "lede_create", "lede_destroy", "lede_last_error", "lede_load_tensor",
            "lede_set_free_list", "lede_set_options", "lede_prefill", "lede_set_pending", "lede_truncate",
            "lede_draft", "lede_verify", "lede_step", "lede_get_kv_state", "lede_debug_read",
            "lede_prof_enable", "lede_prof_read", "lede_op_tiled_bytes", "lede_op_repack", "lede_op_linear",
            "lede_op_read_probe", "lede_op_read_groups", "lede_step_sampled", "lede_op_sample", "lede_step_policy", "lede_set_trace",
            "lede_get_trace", "lede_set_verify_reuse", "lede_dqn_region_bytes", "lede_dqn_create", "lede_dqn_destroy",
            "lede_dqn_last_error", "lede_dqn_init", "lede_dqn_push", "lede_dqn_record", "lede_dqn_end_episode",
            "lede_dqn_update", "lede_dqn_sync_target", "lede_dqn_act", "lede_dqn_read", "lede_step_submit",
            "lede_step_collect", "lede_load_weights", "lede_debug_logits", "lede_debug_inject_failure", "lede_op_sample_noalloc"]
MAX_IN_FLIGHT = 2
SAMPLE_SLOTS = 16
SAMPLE_STRIDE = 33

_lib = None


def load(path: str = LIB_PATH):
    """Load liblede.so and declare its signatures.  Raises if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError("liblede.so not built (run __graft_entry__.build()): %s" % path)
    L = ctypes.CDLL(path)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    P = ctypes.POINTER
    L.lede_region_bytes.argtypes = [P(LedeConfig), P(sz), P(sz), P(sz)]
    L.lede_create.argtypes = [P(LedeConfig), vp, sz, vp, sz, vp, sz, P(vp)]
    L.lede_destroy.argtypes = [vp]
    L.lede_destroy.restype = None
    L.lede_last_error.argtypes = [vp]
    L.lede_last_error.restype = ctypes.c_char_p
    L.lede_load_tensor.argtypes = [vp, i32, i32, vp, vp]
    L.lede_load_weights.argtypes = [vp, P(LedeWeights), vp]
    L.lede_debug_logits.argtypes = [vp, i32, P(ctypes.c_float), sz, P(i32), vp]
    L.lede_debug_inject_failure.argtypes = [vp, i32]
    L.lede_set_free_list.argtypes = [vp, P(i32), i32]
    L.lede_set_options.argtypes = [vp, i32, i32]
    L.lede_set_verify_reuse.argtypes = [vp, i32]
    L.lede_prefill.argtypes = [vp, P(i32), i32, vp, P(i32)]
    L.lede_set_pending.argtypes = [vp, i32, vp]
    L.lede_truncate.argtypes = [vp, i32, vp]
    L.lede_draft.argtypes = [vp, i32, i32, vp, P(i32)]
    L.lede_verify.argtypes = [vp, vp, P(i32), P(i32), P(i32), P(i32)]
    L.lede_step.argtypes = [vp, P(LedeAction), i32, i32, vp, P(LedeStepRecord)]
    L.lede_step_submit.argtypes = [vp, P(LedeAction), i32, i32, vp]
    L.lede_step_collect.argtypes = [vp, vp, P(LedeStepRecord)]
    L.lede_get_kv_state.argtypes = [vp, P(i32), P(i32), P(i32), i32, P(i32)]
    L.lede_debug_read.argtypes = [vp, i32, P(ctypes.c_float), sz, P(i32), vp]
    L.lede_prof_enable.argtypes = [vp, i32]
    L.lede_prof_read.argtypes = [vp, P(LedeProfEntry), i32]
    L.lede_op_tiled_bytes.argtypes = [i32, i32, i32]
    L.lede_op_tiled_bytes.restype = sz
    L.lede_op_repack.argtypes = [i32, vp, i32, i32, vp, vp]
    L.lede_op_linear.argtypes = [i32, vp, i32, i32, vp, i32, i32, vp, i32, vp]
    L.lede_op_read_probe.argtypes = [vp, sz, vp, i32, vp, P(ctypes.c_float)]
    L.lede_op_read_groups.argtypes = [vp, i32, i32, vp, vp, P(ctypes.c_float)]
    L.lede_step_sampled.argtypes = [vp, P(LedeAction), i32, i32, ctypes.c_float, P(ctypes.c_float), vp,
                                    P(LedeStepRecord)]
    L.lede_op_sample.argtypes = [vp, i32, ctypes.c_float, ctypes.c_float, P(i32), vp]
    L.lede_op_sample_noalloc.argtypes = [vp, i32, i32, i32, ctypes.c_float, P(ctypes.c_float), P(i32), vp]
    L.lede_step_policy.argtypes = [vp, i32, vp, P(LedeStepRecord)]
    L.lede_set_trace.argtypes = [vp, P(ctypes.c_float), i32, vp]
    L.lede_get_trace.argtypes = [vp, P(ctypes.c_float), P(i32), vp]
    fp = P(ctypes.c_float)
    L.lede_dqn_region_bytes.argtypes = [P(LedeDqnConfig)]
    L.lede_dqn_region_bytes.restype = sz
    L.lede_dqn_create.argtypes = [P(LedeDqnConfig), vp, sz, P(vp)]
    L.lede_dqn_destroy.argtypes = [vp]
    L.lede_dqn_destroy.restype = None
    L.lede_dqn_last_error.argtypes = [vp]
    L.lede_dqn_last_error.restype = ctypes.c_char_p
    L.lede_dqn_init.argtypes = [vp, vp, vp]
    L.lede_dqn_push.argtypes = [vp, vp, i32, vp]
    L.lede_dqn_record.argtypes = [vp, vp, i32, vp]
    L.lede_dqn_end_episode.argtypes = [vp, vp]
    L.lede_dqn_update.argtypes = [vp, vp, vp, vp, fp]
    L.lede_dqn_sync_target.argtypes = [vp, vp]
    L.lede_dqn_act.argtypes = [vp, vp, vp, vp]
    L.lede_dqn_read.argtypes = [vp, i32, fp, sz, P(i32), vp]
    for name in EXPORTED:
        if name not in ("lede_destroy", "lede_last_error", "lede_op_tiled_bytes", "lede_dqn_region_bytes",
                        "lede_dqn_destroy", "lede_dqn_last_error"):
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


class LedeDqnConfig(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("capacity", ctypes.c_int32), ("batch", ctypes.c_int32),
                ("n_step", ctypes.c_int32), ("gamma", ctypes.c_float), ("lr", ctypes.c_float),
                ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("adam_eps", ctypes.c_float),
                ("sigma0", ctypes.c_float)]


class LedeError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__("%s (%d): %s" % (STATUS.get(code, "?"), code, msg))
        self.code = code


def make_config(model, max_ctx: int, n_pages: Optional[int] = None, k_max: int = 15,
                exit_hidden: int = 0) -> LedeConfig:
    """lede_config from a model shape (any object with the ModelConfig fields);
    exit_hidden > 0 adds the paper's exit policy (its candidate layers are the
    model's exits)."""
    c = LedeConfig()
    c.n_layers, c.d_model, c.n_heads = model.n_layers, model.d_model, model.n_heads
    c.n_kv_heads, c.head_dim, c.ffn_dim, c.vocab = model.n_kv_heads, model.head_dim, model.ffn_dim, model.vocab
    c.rms_eps, c.rope_base = model.rms_eps, model.rope_base
    c.dtype = 1 if model.dtype == "bf16" else 0
    c.max_ctx, c.page_size = max_ctx, 64
    c.n_pages = n_pages if n_pages is not None else -(-max_ctx // 64)
    c.qnet_hidden = model.qnet_hidden
    c.n_exits, c.n_lengths = len(model.exits), len(model.lengths)
    for i, e in enumerate(model.exits):
        c.exits[i] = e
    for i, k in enumerate(model.lengths):
        c.lengths[i] = k
    c.k_max = k_max
    c.exit_qnet_hidden = exit_hidden
    return c


def _i32p(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


@dataclass
class StepRecord:
    l: int
    k_req: int
    k_eff: int
    accepted: int
    emitted: List[int]
    drafts: List[int]
    q_action: int
    q_max: float
    reward: float
    seq_len: int
    pending: int


class Engine:
    """A liblede context over torch-allocated device regions."""

    def __init__(self, model, max_ctx: int, n_pages: Optional[int] = None, k_max: int = 15, device: int = 0,
                 exit_hidden: int = 0):
        import torch
        self.torch = torch
        self.L = load()
        self.model = model
        self.cfg = make_config(model, max_ctx, n_pages, k_max, exit_hidden)
        wb, kvb, wsb = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
        self._check(self.L.lede_region_bytes(ctypes.byref(self.cfg), ctypes.byref(wb), ctypes.byref(kvb),
                                             ctypes.byref(wsb)), None)
        self.region_bytes = (wb.value, kvb.value, wsb.value)
        dev = torch.device("cuda", device)
        self.device = dev
        self.weights = torch.empty(wb.value, dtype=torch.uint8, device=dev)
        self.kv = torch.empty(kvb.value, dtype=torch.uint8, device=dev)
        self.ws = torch.empty(wsb.value, dtype=torch.uint8, device=dev)
        h = ctypes.c_void_p()
        self._check(self.L.lede_create(ctypes.byref(self.cfg), self.weights.data_ptr(), wb.value,
                                       self.kv.data_ptr(), kvb.value, self.ws.data_ptr(), wsb.value,
                                       ctypes.byref(h)), None)
        self.ctx = h

    # -- plumbing ----------------------------------------------------------
    @property
    def stream(self):
        return ctypes.c_void_p(self.torch.cuda.current_stream(self.device).cuda_stream)

    def _check(self, rc: int, ctx):
        if rc != LEDE_OK:
            msg = self.L.lede_last_error(ctx).decode() if ctx is not None else ""
            raise LedeError(rc, msg)

    def close(self):
        if getattr(self, "ctx", None):
            self.L.lede_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- weights -------------------------------------------------------------
    def load_tensor(self, kind: int, layer: int, host: np.ndarray):
        t = self.torch
        a = np.ascontiguousarray(host)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        dev = t.from_numpy(a).to(self.device)
        self._check(self.L.lede_load_tensor(self.ctx, kind, layer, dev.data_ptr(), self.stream), self.ctx)
        t.cuda.current_stream(self.device).synchronize()

    def _dev(self, host: np.ndarray):
        a = np.ascontiguousarray(host)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        return self.torch.from_numpy(a).to(self.device)

    def lede_load_weights(self, weights: Optional[dict] = None, qnet: Optional[dict] = None,
                          exit_qnet: Optional[dict] = None, first_layer: int = 0, n_layers: int = 0):
        """One lede_load_weights call: the tensors given (host arrays in the
        lede_inputs.weights() layout) are staged on the device and repacked;
        absent ones are left as they are.  Layers [first_layer, first_layer +
        n_layers) come from weights["layers"]."""
        keep = []

        def ptr(host):
            if host is None:
                return None
            if isinstance(host, self.torch.Tensor) and host.device == self.device:
                keep.append(host)  # already staged on the device
                return host.data_ptr()
            d = self._dev(host)
            keep.append(d)
            return d.data_ptr()

        w = LedeWeights()
        weights = weights or {}
        w.embed, w.final_norm, w.head = (ptr(weights.get(n)) for n in ("embed", "final_norm", "head"))
        w.first_layer, w.n_layers = first_layer, n_layers
        table = (ctypes.c_void_p * max(1, n_layers * LAYER_TENSORS))()
        layers = weights.get("layers", [])
        for j in range(n_layers):
            if first_layer + j >= len(layers):
                break  # the library checks the range against the model
            for t, name in enumerate(LAYER_ORDER):
                table[j * LAYER_TENSORS + t] = ptr(layers[first_layer + j][name])
        w.layer = ctypes.cast(table, ctypes.POINTER(ctypes.c_void_p))
        f32 = lambda a: None if a is None else ptr(np.ascontiguousarray(a, dtype=np.float32))  # noqa: E731
        if qnet is not None:
            w.qnet_w1, w.qnet_b1, w.qnet_w2, w.qnet_b2 = (f32(qnet[n]) for n in ("w1", "b1", "w2", "b2"))
        if exit_qnet is not None:
            w.exit_w1, w.exit_b1, w.exit_w2, w.exit_b2 = (f32(exit_qnet[n]) for n in ("w1", "b1", "w2", "b2"))
        self._check(self.L.lede_load_weights(self.ctx, ctypes.byref(w), self.stream), self.ctx)
        self.torch.cuda.current_stream(self.device).synchronize()
        del keep

    def load_weights(self, weights: dict, qnet: Optional[dict] = None, staging_bytes: int = 16 << 30):
        """weights: lede_inputs.weights() layout; qnet: lede_inputs.qnet_weights().
        Through lede_load_weights: the embedding, head and Q-network in one
        call, then the layers in groups whose staging copies take at most
        staging_bytes of device memory."""
        self.lede_load_weights({n: weights[n] for n in ("embed", "final_norm", "head")}, qnet)
        layers = weights["layers"]
        per_layer = max(1, sum(np.asarray(a).nbytes for a in layers[0].values())) if layers else 1
        group = max(1, staging_bytes // per_layer)
        for j0 in range(0, len(layers), group):
            n = min(group, len(layers) - j0)
            self.lede_load_weights({"layers": layers}, first_layer=j0, n_layers=n)

    # -- C-ABI calls (same names) --------------------------------------------------
    def lede_set_options(self, use_graphs: int = 0, debug: int = 0):
        self._check(self.L.lede_set_options(self.ctx, use_graphs, debug), self.ctx)

    def lede_set_verify_reuse(self, enable: bool = True):
        self._check(self.L.lede_set_verify_reuse(self.ctx, int(enable)), self.ctx)

    def lede_set_free_list(self, order: Sequence[int]):
        a = np.ascontiguousarray(order, dtype=np.int32)
        self._check(self.L.lede_set_free_list(self.ctx, _i32p(a), len(a)), self.ctx)

    def lede_prefill(self, tokens: Sequence[int]) -> int:
        a = np.ascontiguousarray(tokens, dtype=np.int32)
        nxt = ctypes.c_int32()
        self._check(self.L.lede_prefill(self.ctx, _i32p(a), len(a), self.stream, ctypes.byref(nxt)), self.ctx)
        return nxt.value

    def lede_set_pending(self, token: int):
        self._check(self.L.lede_set_pending(self.ctx, token, self.stream), self.ctx)

    def lede_truncate(self, new_len: int):
        self._check(self.L.lede_truncate(self.ctx, new_len, self.stream), self.ctx)

    def lede_draft(self, l: int, k: int, read: bool = True) -> Optional[List[int]]:
        out = np.zeros(max(k, 1), dtype=np.int32)
        self._check(self.L.lede_draft(self.ctx, l, k, self.stream, _i32p(out) if read else None), self.ctx)
        return [int(x) for x in out[:k]] if read else None

    def lede_verify(self):
        """Returns (accepted, emitted tokens, verify argmax of every row)."""
        acc, ne = ctypes.c_int32(), ctypes.c_int32()
        toks = np.zeros(17, dtype=np.int32)
        ver = np.zeros(17, dtype=np.int32)
        self._check(self.L.lede_verify(self.ctx, self.stream, ctypes.byref(acc), _i32p(toks), ctypes.byref(ne),
                                       _i32p(ver)), self.ctx)
        return acc.value, [int(x) for x in toks[:ne.value]], ver

    @staticmethod
    def _record(rec) -> StepRecord:
        return StepRecord(l=rec.l, k_req=rec.k_req, k_eff=rec.k_eff, accepted=rec.accepted,
                          emitted=[rec.tokens[i] for i in range(rec.n_emitted)],
                          drafts=[rec.drafts[i] for i in range(rec.k_eff)], q_action=rec.q_action,
                          q_max=rec.q_max, reward=rec.reward, seq_len=rec.seq_len, pending=rec.pending)

    def lede_step(self, action=None, n_remaining: int = 1 << 30, log_qnet: bool = True) -> StepRecord:
        rec = LedeStepRecord()
        act = LedeAction(int(action[0]), int(action[1])) if action is not None else None
        self._check(self.L.lede_step(self.ctx, ctypes.byref(act) if act is not None else None, int(log_qnet),
                                     int(n_remaining), self.stream, ctypes.byref(rec)), self.ctx)
        return self._record(rec)

    def lede_step_submit(self, action, n_remaining: int = 1 << 30, log_qnet: bool = True) -> None:
        """Queue a forced greedy step; at most MAX_IN_FLIGHT wait for lede_step_collect."""
        act = LedeAction(int(action[0]), int(action[1]))
        self._check(self.L.lede_step_submit(self.ctx, ctypes.byref(act), int(log_qnet), int(n_remaining),
                                            self.stream), self.ctx)

    def lede_step_collect(self) -> StepRecord:
        """The record of the oldest submitted step (waits for it)."""
        rec = LedeStepRecord()
        self._check(self.L.lede_step_collect(self.ctx, self.stream, ctypes.byref(rec)), self.ctx)
        return self._record(rec)

    def lede_step_sampled(self, action, temperature: float, uniforms, n_remaining: int = 1 << 30,
                          log_qnet: bool = True) -> StepRecord:
        """A speculative-sampling step; uniforms: SAMPLE_STRIDE floats in [0, 1)."""
        rec = LedeStepRecord()
        act = LedeAction(int(action[0]), int(action[1])) if action is not None else None
        u = np.ascontiguousarray(uniforms, dtype=np.float32)
        if u.size != SAMPLE_STRIDE:
            raise ValueError("need %d uniforms" % SAMPLE_STRIDE)
        self._check(self.L.lede_step_sampled(self.ctx, ctypes.byref(act) if act is not None else None,
                                             int(log_qnet), int(n_remaining), float(temperature),
                                             u.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), self.stream,
                                             ctypes.byref(rec)), self.ctx)
        return self._record(rec)

    def load_exit_qnet(self, w: dict):
        """The exit policy's Q-network: lede_inputs.exit_qnet_weights() layout."""
        self.lede_load_weights(exit_qnet=w)

    def lede_step_policy(self, n_remaining: int = 1 << 30) -> StepRecord:
        rec = LedeStepRecord()
        self._check(self.L.lede_step_policy(self.ctx, int(n_remaining), self.stream, ctypes.byref(rec)), self.ctx)
        return self._record(rec)

    def policy_log(self) -> np.ndarray:
        """Decisions of the last lede_step_policy: rows of (kind, layer / draft,
        C_5, H, C_trace, Q(continue), Q(exit), action)."""
        out, rows = self.lede_debug_read(4, (64 + 12) * 8)
        return out[:rows * 8].reshape(rows, 8)

    def lede_set_trace(self, values):
        v = np.ascontiguousarray(values, dtype=np.float32)
        self._check(self.L.lede_set_trace(self.ctx, v.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), len(v),
                                          self.stream), self.ctx)

    def lede_get_trace(self) -> np.ndarray:
        v = np.zeros(20, dtype=np.float32)
        n = ctypes.c_int32()
        self._check(self.L.lede_get_trace(self.ctx, v.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                          ctypes.byref(n), self.stream), self.ctx)
        return v[:n.value]

    def lede_get_kv_state(self):
        """(seq_len, pending, block table)."""
        sl, pend, n = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        cap = self.cfg.max_ctx // 64 + 2
        bt = np.zeros(cap, dtype=np.int32)
        self._check(self.L.lede_get_kv_state(self.ctx, ctypes.byref(sl), ctypes.byref(pend), _i32p(bt), cap,
                                             ctypes.byref(n)), self.ctx)
        return sl.value, pend.value, [int(x) for x in bt[:n.value]]

    def lede_debug_read(self, which: int, n_floats: int) -> np.ndarray:
        out = np.zeros(n_floats, dtype=np.float32)
        rows = ctypes.c_int32()
        self._check(self.L.lede_debug_read(self.ctx, which, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                           n_floats, ctypes.byref(rows), self.stream), self.ctx)
        return out, rows.value

    def lede_debug_logits(self, which: int = LOGITS_VERIFY) -> np.ndarray:
        """Logits of the last verify / prefill head (LOGITS_VERIFY) or of the
        last step's draft heads (LOGITS_DRAFT), [rows][vocab]."""
        V = self.model.vocab
        out = np.zeros(16 * V, dtype=np.float32)
        rows = ctypes.c_int32()
        self._check(self.L.lede_debug_logits(self.ctx, int(which), out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                             out.size, ctypes.byref(rows), self.stream), self.ctx)
        return out[:rows.value * V].reshape(rows.value, V)

    def lede_debug_inject_failure(self, n_ops: int):
        """The (n_ops + 1)-th device operation of the next calls fails with
        E_HIP before it is issued (one-shot; n_ops < 0 disables)."""
        self._check(self.L.lede_debug_inject_failure(self.ctx, int(n_ops)), self.ctx)

    def lede_prof_enable(self, level: int):
        """0 off, 1 draft / verify phases only, 2 phases and every launch."""
        self._check(self.L.lede_prof_enable(self.ctx, int(level)), self.ctx)

    def lede_prof_read(self, reset: bool = True) -> dict:
        arr = (LedeProfEntry * K_NCLASS)()
        self._check(self.L.lede_prof_read(self.ctx, arr, int(reset)), self.ctx)
        return {K_NAMES[i]: {"ms": arr[i].ms, "bytes": arr[i].bytes, "launches": arr[i].launches}
                for i in range(K_NCLASS)}

    def logits(self, which: int = 0) -> np.ndarray:
        """Debug logits of the last verify/prefill head (which=0) or of the
        last draft passes (which=3), shape [rows][vocab]."""
        V = self.model.vocab
        out, rows = self.lede_debug_read(which, 16 * V)
        return out[:rows * V].reshape(rows, V)


# ---- single-op helpers (kernel-level tests) ----------------------------------------

def op_linear(W, x, use_mfma: bool):
    """y = x W^T through the library's tiled linear kernels.  W [N][K] and x
    [M][K] are torch tensors on the GPU (float32 or bfloat16)."""
    import torch
    L = load()
    dtype = 1 if W.dtype == torch.bfloat16 else 0
    N, K = W.shape
    M = x.shape[0]
    tiled = torch.empty(L.lede_op_tiled_bytes(dtype, N, K), dtype=torch.uint8, device=W.device)
    y = torch.empty(M, N, dtype=torch.float32, device=W.device)
    s = ctypes.c_void_p(torch.cuda.current_stream(W.device).cuda_stream)
    rc = L.lede_op_repack(dtype, W.data_ptr(), N, K, tiled.data_ptr(), s)
    if rc:
        raise LedeError(rc, "op_repack")
    # rows padded with zeros to the tile width, which the kernels read whole
    tk = 32 if dtype == 1 else 16
    ldx = -(-K // tk) * tk
    xp = torch.zeros(M, ldx, dtype=x.dtype, device=x.device)
    xp[:, :K] = x
    rc = L.lede_op_linear(dtype, tiled.data_ptr(), N, K, xp.data_ptr(), ldx, M, y.data_ptr(), int(use_mfma), s)
    if rc:
        raise LedeError(rc, "op_linear")
    return y


def op_read_probe(buf, grid: int = 0) -> float:
    """Kernel milliseconds for one read of the whole GPU tensor buf (its byte
    size a multiple of 16) with the weight-streaming loads."""
    import torch
    L = load()
    nbytes = buf.numel() * buf.element_size()
    grid = grid or 256 * 16
    sink = torch.empty(grid, dtype=torch.int32, device=buf.device)
    ms = ctypes.c_float()
    s = ctypes.c_void_p(torch.cuda.current_stream(buf.device).cuda_stream)
    rc = L.lede_op_read_probe(buf.data_ptr(), nbytes, sink.data_ptr(), int(grid), s, ctypes.byref(ms))
    if rc:
        raise LedeError(rc, "op_read_probe")
    return ms.value


def op_read_groups(buf, n_groups: int, tiles: int) -> float:
    """Kernel milliseconds for reading n_groups x tiles 1 KiB tiles at the start
    of the GPU tensor buf with the one-row linear kernel's load structure."""
    import torch
    L = load()
    if n_groups * tiles * 1024 > buf.numel() * buf.element_size():
        raise LedeError(LEDE_E_ARG, "buffer smaller than n_groups x tiles KiB")
    sink = torch.empty(n_groups, dtype=torch.int32, device=buf.device)
    ms = ctypes.c_float()
    s = ctypes.c_void_p(torch.cuda.current_stream(buf.device).cuda_stream)
    rc = L.lede_op_read_groups(buf.data_ptr(), int(n_groups), int(tiles), sink.data_ptr(), s, ctypes.byref(ms))
    if rc:
        raise LedeError(rc, "op_read_groups")
    return ms.value


def op_sample(logits, temperature: float, u: float) -> int:
    """One inverse-CDF draw from softmax(logits / temperature) by the
    library's sampling kernel; logits is a float32 GPU tensor of one row."""
    import torch
    L = load()
    tok = ctypes.c_int32()
    s = ctypes.c_void_p(torch.cuda.current_stream(logits.device).cuda_stream)
    x = logits.contiguous()
    rc = L.lede_op_sample(x.data_ptr(), x.numel(), float(temperature), float(u), ctypes.byref(tok), s)
    if rc:
        raise LedeError(rc, "op_sample")
    return tok.value


def op_sample_noalloc(logits, temperature: float, u) -> List[int]:
    """One inverse-CDF draw per row of the float32 GPU tensor logits [rows][V]
    (rows <= 32) with the uniforms u [rows], through the entry point that
    allocates nothing."""
    import torch
    L = load()
    x = logits.contiguous()
    rows, V = x.shape
    uu = np.ascontiguousarray(u, dtype=np.float32)
    out = np.zeros(max(rows, 1), dtype=np.int32)
    s = ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream)
    rc = L.lede_op_sample_noalloc(x.data_ptr(), rows, V, V, float(temperature),
                                  uu.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), _i32p(out), s)
    if rc:
        raise LedeError(rc, "op_sample_noalloc")
    return [int(t) for t in out[:rows]]


def dqn_noise_count(hidden: int) -> int:
    """Standard normals one network draw takes: eps_in, eps_out of both layers."""
    return 2 * hidden + 5


def dqn_param_count(hidden: int) -> int:
    """Entries of [mu, sigma] of the 3 -> H -> 2 network."""
    return 2 * (6 * hidden + 2)


class Dqn:
    """A liblede policy trainer (lede_dqn_*) over a torch-allocated region."""

    def __init__(self, hidden: int = 16, capacity: int = 1 << 16, batch: int = 32, n_step: int = 3,
                 gamma: float = 0.99, lr: float = 6.25e-5, beta1: float = 0.9, beta2: float = 0.999,
                 adam_eps: float = 1.5e-4, sigma0: float = 0.1, device: int = 0):
        import torch
        self.torch = torch
        self.L = load()
        self.cfg = LedeDqnConfig(hidden, capacity, batch, n_step, gamma, lr, beta1, beta2, adam_eps, sigma0)
        nbytes = self.L.lede_dqn_region_bytes(ctypes.byref(self.cfg))
        if nbytes == 0:
            raise LedeError(LEDE_E_ARG, "invalid trainer configuration")
        self.device = torch.device("cuda", device)
        self.region = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        rc = self.L.lede_dqn_create(ctypes.byref(self.cfg), self.region.data_ptr(), nbytes, ctypes.byref(h))
        if rc != LEDE_OK:
            raise LedeError(rc, "lede_dqn_create")
        self.q = h

    @property
    def stream(self):
        return ctypes.c_void_p(self.torch.cuda.current_stream(self.device).cuda_stream)

    def _check(self, rc: int):
        if rc != LEDE_OK:
            raise LedeError(rc, self.L.lede_dqn_last_error(self.q).decode())

    def _dev(self, a):
        """A device fp32 copy of a host array (kept alive by the caller)."""
        return self.torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(self.device)

    def close(self):
        if getattr(self, "q", None):
            self.L.lede_dqn_destroy(self.q)
            self.q = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def lede_dqn_init(self, u):
        d = self._dev(u)
        self._check(self.L.lede_dqn_init(self.q, d.data_ptr(), self.stream))
        self.torch.cuda.current_stream(self.device).synchronize()

    def lede_dqn_push(self, transitions):
        t = np.ascontiguousarray(transitions, dtype=np.float32).reshape(-1, 6)
        d = self._dev(t)
        self._check(self.L.lede_dqn_push(self.q, d.data_ptr(), len(t), self.stream))
        self.torch.cuda.current_stream(self.device).synchronize()

    def lede_dqn_record(self, engine, episode_end: bool = False):
        self._check(self.L.lede_dqn_record(self.q, engine.ctx, int(episode_end), self.stream))

    def lede_dqn_end_episode(self):
        self._check(self.L.lede_dqn_end_episode(self.q, self.stream))

    def lede_dqn_update(self, u, noise, want_loss: bool = True):
        """u: [batch] uniforms m / 2^24, noise: [2][2H + 5] normals, host
        arrays or device tensors; returns the loss (or None)."""
        t = self.torch
        ud = u if isinstance(u, t.Tensor) else self._dev(u)
        nd = noise if isinstance(noise, t.Tensor) else self._dev(noise)
        loss = ctypes.c_float()
        self._check(self.L.lede_dqn_update(self.q, ud.data_ptr(), nd.data_ptr(), self.stream,
                                           ctypes.byref(loss) if want_loss else None))
        return loss.value if want_loss else None

    def lede_dqn_sync_target(self):
        self._check(self.L.lede_dqn_sync_target(self.q, self.stream))

    def lede_dqn_act(self, engine, noise=None):
        nd = None if noise is None else self._dev(noise)
        self._check(self.L.lede_dqn_act(self.q, engine.ctx, None if nd is None else nd.data_ptr(), self.stream))
        self.torch.cuda.current_stream(self.device).synchronize()

    def lede_dqn_read(self, which: int) -> np.ndarray:
        """0 online [mu, sigma], 1 target, 2 Adam m, 3 Adam v; 4 transitions [count][6]."""
        cap = dqn_param_count(self.cfg.hidden) if which < 4 else self.cfg.capacity * 6
        out = np.zeros(cap, dtype=np.float32)
        n = ctypes.c_int32()
        self._check(self.L.lede_dqn_read(self.q, which, out.ctypes.data_as(ctypes.POINTER(ctypes.c_float)), cap,
                                         ctypes.byref(n), self.stream))
        return out[:n.value] if which < 4 else out[:n.value * 6].reshape(n.value, 6)
