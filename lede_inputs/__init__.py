"""Seeded synthetic inputs shared by the CPU oracle and the GPU path.

This package holds no part of the decoding method's arithmetic.  It builds a
small C library (``gen.c``: Philox4x32-10 counters + Box-Muller) and exposes:

* ``weights(model)`` -- the decoder's weights as host numpy arrays in the
  logical row-major ``[out][in]`` layout (bf16 as uint16 bit patterns);
* ``weight_tensor(model, name, layer)`` -- one tensor, regenerable alone;
* ``weight_rows(model, name, layer, rows)`` -- selected rows only;
* ``qnet_weights(model)``, ``prompt(workload)``, ``schedule(workload)``;
* ``step_uniforms(step)`` -- the uniforms a speculative-sampling step draws.

Every value is a pure function of (seed, stream, index), so the oracle and
the GPU upload see identical bytes.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

from .configs import (PAGE_SIZE, SAMPLE_SLOTS, SAMPLE_STRIDE, SEED_DQN, SEED_PROMPT, SEED_QNET, SEED_SAMPLE,
                      SEED_SCHEDULE, SEED_WEIGHTS, WEIGHT_STD, WORKLOADS, ModelConfig, Workload, shrink)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liblede_inputs.so")
_lock = threading.Lock()
_lib = None

# Stream ids of the generated tensors.  Per-layer tensors use
# LAYER_BASE + LAYER_STRIDE * layer + offset.
STREAM_EMBED = 1
STREAM_HEAD = 2
STREAM_QNET_W1 = 10
STREAM_QNET_W2 = 11
STREAM_PROMPT = 20
STREAM_SCHED_L = 30
STREAM_SCHED_K = 31
STREAM_SAMPLE = 40
STREAM_EXIT_QNET = 12
STREAM_DQN_STATE = 50
STREAM_DQN_ACTION = 51
STREAM_DQN_REWARD = 52
STREAM_DQN_DONE = 53
STREAM_DQN_BATCH = 54
STREAM_DQN_NOISE = 55
STREAM_DQN_INIT = 56
LAYER_BASE = 1000
LAYER_STRIDE = 16
LAYER_TENSORS = {"wq": 1, "wk": 2, "wv": 3, "wo": 4, "wg": 6, "wu": 7, "wd": 8}
NORM_TENSORS = ("attn_norm", "ffn_norm")


def build(force: bool = False) -> str:
    """Compile gen.c into liblede_inputs.so (gcc, OpenMP)."""
    src = os.path.join(_HERE, "gen.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, src, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def _load():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_SO):
                build()
            lib = ctypes.CDLL(_SO)
            u32, u64, dbl, i32 = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_double, ctypes.c_int32
            vp = ctypes.c_void_p
            lib.lede_gen_normal_f32.argtypes = [u32, u32, u64, u64, dbl, vp]
            lib.lede_gen_normal_bf16.argtypes = [u32, u32, u64, u64, dbl, vp]
            lib.lede_gen_uniform_int.argtypes = [u32, u32, u64, u64, i32, i32, vp]
            lib.lede_gen_philox_block.argtypes = [u32] * 6 + [vp]
            lib.lede_gen_uniform01.argtypes = [u32, u32, u64, u64, vp]
            _lib = lib
    return _lib


def philox_block(ctr, key):
    out = np.zeros(4, dtype=np.uint32)
    _load().lede_gen_philox_block(*[int(c) for c in ctr], *[int(k) for k in key],
                                  out.ctypes.data)
    return out


def normal(seed: int, stream: int, n: int, std: float, dtype: str, offset: int = 0) -> np.ndarray:
    lib = _load()
    if dtype == "bf16":
        out = np.empty(n, dtype=np.uint16)
        lib.lede_gen_normal_bf16(seed, stream, offset, n, std, out.ctypes.data)
    elif dtype == "f32":
        out = np.empty(n, dtype=np.float32)
        lib.lede_gen_normal_f32(seed, stream, offset, n, std, out.ctypes.data)
    else:
        raise ValueError(dtype)
    return out


def uniform_int(seed: int, stream: int, n: int, lo: int, hi: int, offset: int = 0) -> np.ndarray:
    out = np.empty(n, dtype=np.int32)
    _load().lede_gen_uniform_int(seed, stream, offset, n, lo, hi, out.ctypes.data)
    return out


def uniform01(seed: int, stream: int, n: int, offset: int = 0) -> np.ndarray:
    """Exact float32 uniforms in [0, 1) (24 random bits each)."""
    out = np.empty(n, dtype=np.float32)
    _load().lede_gen_uniform01(seed, stream, offset, n, out.ctypes.data)
    return out


def step_uniforms(step: int, seed: int = SEED_SAMPLE) -> np.ndarray:
    """The SAMPLE_STRIDE uniforms of one speculative-sampling step: draft
    samples [0, SAMPLE_SLOTS), acceptance tests [SAMPLE_SLOTS, 2 SAMPLE_SLOTS),
    the residual / bonus sample last."""
    return uniform01(seed, STREAM_SAMPLE, SAMPLE_STRIDE, offset=SAMPLE_STRIDE * step)


def tensor_shape(m: ModelConfig, name: str):
    d, f = m.d_model, m.ffn_dim
    return {
        "embed": (m.vocab, d), "head": (m.vocab, d), "final_norm": (d,),
        "attn_norm": (d,), "ffn_norm": (d,),
        "wq": (m.q_dim, d), "wk": (m.kv_dim, d), "wv": (m.kv_dim, d), "wo": (d, m.q_dim),
        "wg": (f, d), "wu": (f, d), "wd": (d, f),
    }[name]


def _stream(name: str, layer: int) -> int:
    if name == "embed":
        return STREAM_EMBED
    if name == "head":
        return STREAM_HEAD
    return LAYER_BASE + LAYER_STRIDE * layer + LAYER_TENSORS[name]


def _ones(m: ModelConfig, n: int) -> np.ndarray:
    if m.dtype == "bf16":
        return np.full(n, 0x3F80, dtype=np.uint16)  # bf16 bit pattern of 1.0
    return np.ones(n, dtype=np.float32)


def weight_tensor(m: ModelConfig, name: str, layer: int = 0, seed: int = SEED_WEIGHTS) -> np.ndarray:
    """One weight tensor in logical row-major layout.  RMSNorm gains are 1."""
    shape = tensor_shape(m, name)
    if name in ("final_norm",) + NORM_TENSORS:
        return _ones(m, shape[0])
    n = int(np.prod(shape))
    return normal(seed, _stream(name, layer), n, WEIGHT_STD, m.dtype).reshape(shape)


def weight_rows(m: ModelConfig, name: str, layer: int, rows, seed: int = SEED_WEIGHTS) -> np.ndarray:
    """Selected rows of a 2-D weight tensor, regenerated without the rest."""
    n_out, n_in = tensor_shape(m, name)
    rows = np.asarray(rows, dtype=np.int64)
    out = np.empty((len(rows), n_in), dtype=np.uint16 if m.dtype == "bf16" else np.float32)
    for i, r in enumerate(rows):
        out[i] = normal(seed, _stream(name, layer), n_in, WEIGHT_STD, m.dtype, offset=int(r) * n_in)
    return out


def weights(m: ModelConfig, seed: int = SEED_WEIGHTS) -> dict:
    """All decoder weights: {'embed','head','final_norm', 'layers': [dict per layer]}."""
    out = {"embed": weight_tensor(m, "embed", seed=seed),
           "head": weight_tensor(m, "head", seed=seed),
           "final_norm": weight_tensor(m, "final_norm")}
    layers = []
    for j in range(m.n_layers):
        layers.append({name: weight_tensor(m, name, j, seed) for name in
                       ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd")})
    out["layers"] = layers
    return out


def qnet_weights(m: ModelConfig, seed: int = SEED_QNET) -> dict:
    """fp32 Q-network: W1 [H][d], b1 [H] = 0, W2 [E*K][H], b2 [E*K] = 0."""
    h, a = m.qnet_hidden, m.n_actions
    return {
        "w1": normal(seed, STREAM_QNET_W1, h * m.d_model, WEIGHT_STD, "f32").reshape(h, m.d_model),
        "b1": np.zeros(h, dtype=np.float32),
        "w2": normal(seed, STREAM_QNET_W2, a * h, WEIGHT_STD, "f32").reshape(a, h),
        "b2": np.zeros(a, dtype=np.float32),
    }


def exit_qnet_weights(hidden: int = 16, seed: int = SEED_QNET, std: float = 0.5) -> dict:
    """fp32 2-action exit Q-network of the paper's policy: W1 [H][3], b1 [H],
    W2 [2][H], b2 [2] = 0 (rows of W2: continue, exit)."""
    return {
        "w1": normal(seed, STREAM_EXIT_QNET, hidden * 3, std, "f32").reshape(hidden, 3),
        "b1": normal(seed, STREAM_EXIT_QNET + 1, hidden, std, "f32"),
        "w2": normal(seed, STREAM_EXIT_QNET + 2, 2 * hidden, std, "f32").reshape(2, hidden),
        "b2": np.zeros(2, dtype=np.float32),
    }


def dqn_transitions(n: int, seed: int = SEED_DQN, p_done: float = 0.15, offset: int = 0) -> np.ndarray:
    """[n][6] float32 synthetic transitions: state (3, N(0, 2^2)), action
    0 / 1, reward N(0, 1), terminal with probability p_done."""
    t = np.zeros((n, 6), dtype=np.float32)
    t[:, :3] = normal(seed, STREAM_DQN_STATE, 3 * n, 2.0, "f32", offset=3 * offset).reshape(n, 3)
    t[:, 3] = uniform_int(seed, STREAM_DQN_ACTION, n, 0, 1, offset=offset)
    t[:, 4] = normal(seed, STREAM_DQN_REWARD, n, 1.0, "f32", offset=offset)
    t[:, 5] = uniform01(seed, STREAM_DQN_DONE, n, offset=offset) < p_done
    return t


def dqn_init_uniforms(hidden: int, seed: int = SEED_DQN) -> np.ndarray:
    """Uniforms of one parameter set of the 3 -> H -> 2 network (6H + 2)."""
    return uniform01(seed, STREAM_DQN_INIT, 6 * hidden + 2)


def dqn_update_inputs(i: int, hidden: int, batch: int, seed: int = SEED_DQN):
    """Inputs of learning update i: batch uniforms and the standard normals of
    the online and the target network's noise ([2][2H + 5])."""
    nc = 2 * hidden + 5
    u = uniform01(seed, STREAM_DQN_BATCH, batch, offset=i * batch)
    noise = normal(seed, STREAM_DQN_NOISE, 2 * nc, 1.0, "f32", offset=i * 2 * nc).reshape(2, nc)
    return u, noise


def prompt(w: Workload, seed: int = SEED_PROMPT, length: int | None = None) -> np.ndarray:
    n = w.prompt_len if length is None else length
    return uniform_int(seed, STREAM_PROMPT, n, 0, w.model.vocab - 1)


def schedule(w: Workload, n_steps: int | None = None, seed: int = SEED_SCHEDULE) -> np.ndarray:
    """Seeded per-step (l, k) pairs, shape [n_steps, 2]."""
    n = w.n_gen if n_steps is None else n_steps
    if w.policy == "fixed":
        return np.tile(np.array(w.fixed, dtype=np.int32), (n, 1))
    ls = uniform_int(seed, STREAM_SCHED_L, n, w.sched_l[0], w.sched_l[1])
    ks = uniform_int(seed, STREAM_SCHED_K, n, w.sched_k[0], w.sched_k[1])
    return np.stack([ls, ks], axis=1)


def bf16_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


__all__ = ["PAGE_SIZE", "WORKLOADS", "ModelConfig", "Workload", "shrink", "build", "weights",
           "weight_tensor", "weight_rows", "qnet_weights", "prompt", "schedule", "normal",
           "uniform_int", "philox_block", "bf16_to_f32", "tensor_shape"]
