"""Decode throughput of batch-1 self-speculative decoding on one MI355X.

Workload (default): the Llama-2-7B-shaped random-init bf16 decoder, a
512-token uniform-random prompt, 256 generated tokens, static exit layer
l = 8 and draft length k = 4 (the Q-network is evaluated and logged every
step).  A step is one pass of the whole hot path: Q-network, k draft passes
through layers 1..l with the shared final norm + LM head + argmax, one
(k+1)-row verify pass through all L layers, greedy acceptance, KV
truncation.  Inputs are synthetic and already resident in HBM when timing
starts.

Prints one JSON line: tokens/s over the timed steps, the HBM roofline of the
dominant kernel (algorithmic bytes / HIP-event duration, from an instrumented
replay of the same steps), per-pass rates (draft and verify phases timed in a
replay with no other events), plain autoregressive decoding on the same path
(verify with no drafts), the achievable read bandwidth of the weight arena
(a read-once probe kernel), and the CPU oracle timed on a bounded sample of
the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def pass_bytes(m, l, c):
    """Algorithmic bytes of one draft pass through l layers at KV length c."""
    kv = m.kv_bytes_per_token_layer()
    return l * m.layer_weight_bytes() + m.head_weight_bytes() + l * (c + 1) * kv


def verify_bytes(m, k, c, from_layer=0):
    """Algorithmic bytes of the verify pass of k drafts at KV length c, from
    layer from_layer (verify reuse) or from the embedding."""
    kv = m.kv_bytes_per_token_layer()
    n = m.n_layers - from_layer
    return n * m.layer_weight_bytes() + m.head_weight_bytes() + n * (c + k + 1) * kv


def policy_draft_bytes(m, l_star, c, n_cand, n_draft):
    """Algorithmic bytes of the draft passes of one exit-policy step at KV
    length c: the pending token up to l* with the shared head read at each of
    the n_cand candidate layers visited, then n_draft further passes through
    l* layers and the head (the last one ended by 'continue')."""
    kv = m.kv_bytes_per_token_layer()
    b = l_star * m.layer_weight_bytes() + n_cand * m.head_weight_bytes() + l_star * (c + 1) * kv
    for i in range(1, n_draft + 1):
        b += pass_bytes(m, l_star, c + i)
    return b


def extend_bytes(m, l, c, k):
    """Verify reuse: the last draft's pass through layers 1..l (no head)."""
    return l * m.layer_weight_bytes() + l * (c + k + 1) * m.kv_bytes_per_token_layer()


def _span(xs):
    xs = list(xs)
    step = xs[1] - xs[0] if len(xs) > 1 else 1
    if len(xs) > 2 and all(b - a == step for a, b in zip(xs, xs[1:])):
        return "{%d, %d, ..., %d}" % (xs[0], xs[1], xs[-1])
    return "{%s}" % ", ".join(map(str, xs))


def kernel_source_sha():
    """Hash of the sources the weight-streaming linear kernels are built from."""
    h = hashlib.sha256()
    for f in ("linear.hip", "linear.h", "device.h"):
        h.update(open(os.path.join(ROOT, "paper_2606_03113_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profile(kclass, workload, launches):
    """HBM bytes per launch of the dominant kernel from the committed
    rocprofv3 FETCH_SIZE / WRITE_SIZE runs (profiles/traffic_*.txt), if they
    were taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "traffic_%s_%s.txt" % (kclass, workload))
    if not os.path.exists(path):
        return None
    for line in open(path):
        if line.startswith("traffic_json:"):
            d = json.loads(line.split(":", 1)[1])
            if d.get("kernel_src_sha") == kernel_source_sha():
                return d.get("hbm_bytes_per_launch")
    return None


def cpu_baseline(wl, weights, qnet, prompt_next, policy, actions, budget_s=15.0, max_steps=8):
    """The CPU oracle on a bounded sample: SSD steps under the bench's policy
    (fixed action, seeded schedule, or the Q-network's choice) from KV length
    = prompt length, with the prompt's KV cache filled with synthetic bf16
    values instead of an oracle prefill."""
    from oracle.model import OracleDecoder, SSDState
    m = wl.model
    P = wl.prompt_len
    max_ctx = P + 64
    dec = OracleDecoder(m, weights, max_ctx, qnet)
    rng = np.random.default_rng(0)
    for cache in (dec.kcache, dec.vcache):
        vals = rng.standard_normal((m.n_layers, P, m.kv_dim)).astype(np.float32)
        cache[:, :P, :] = (vals.view(np.uint32) & 0xFFFF0000).view(np.float32)
    st = SSDState(dec, -(-max_ctx // 64), 64)
    st.pager.ensure(P)
    st.c, st.pending, st.out = P, prompt_next, [prompt_next]
    t0 = time.time()
    toks = steps = 0
    while steps < max_steps and (steps < 2 or time.time() - t0 < budget_s):
        l, k = actions[steps % len(actions)]
        rec = st.step(int(l), int(k), wl.n_gen, qnet=m.qnet_hidden > 0, use_qnet_action=policy == "qnet")
        toks += len(rec.emitted)
        steps += 1
    el = time.time() - t0
    # plain autoregressive steps of the oracle on the same state (k = 0)
    t1 = time.time()
    ar_toks = 0
    while ar_toks < 2 or (ar_toks < max_steps and time.time() - t1 < budget_s / 3):
        ar_toks += len(st.step(1, 0, wl.n_gen).emitted)
    ar_el = time.time() - t1
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": toks / el, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "ar_value": ar_toks / ar_el, "ar_sample": "%d autoregressive steps after the SSD sample; %.1f s" % (
                ar_toks, ar_el),
            "sample": "%d SSD steps (%s) of %s from KV length %d (prompt KV filled with synthetic "
                      "bf16 values, no oracle prefill); %.1f s" % (
                          steps, "Q-network's actions" if policy == "qnet" else
                          "seeded schedule" if policy == "schedule" else "l=%d, k=%d" % tuple(actions[0]),
                          wl.name, P, el),
            "host": "%s; %d logical CPUs visible; OMP_NUM_THREADS=%s" % (
                host_cpu_model(), os.cpu_count() or 0, os.environ.get("OMP_NUM_THREADS", "unset"))}


REPEAT_LAYERS = 4  # distinct generated layers of a model too large to generate whole


class RepeatedLayers:
    """The layer weights of a model too large to generate on the host in a
    bench run (the 70B shape: 138 GB, about a quarter of an hour of host
    generation): layers 0..REPEAT_LAYERS-1 are generated from the seeded
    generator and staged on the device once, and layer j is loaded from
    layer j mod REPEAT_LAYERS.  Every layer still has its own weights in the
    arena, so a pass streams the same bytes."""

    def __init__(self, m, torch):
        import lede_inputs as li
        self.m = m
        self.dev = []
        for j in range(min(REPEAT_LAYERS, m.n_layers)):
            lw = {}
            for n in ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "wg", "wu", "wd"):
                a = np.ascontiguousarray(li.weight_tensor(m, n, j))
                lw[n] = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).cuda()
            self.dev.append(lw)

    def __len__(self):
        return self.m.n_layers

    def __getitem__(self, j):
        if not 0 <= j < self.m.n_layers:
            raise IndexError(j)
        return self.dev[j % len(self.dev)]


def host_cpu_model():
    """The host CPU's model name (Linux /proc/cpuinfo), or 'unknown'."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def dqn_leg(torch, li, n_updates=2000, H=16, B=32):
    """Learning updates of the exit policy's trainer with the paper's
    hyperparameters (mini-batch 32, n = 3, gamma = 0.99, Adam 6.25e-5, noisy
    layers sigma0 = 0.1, a target copy every 512 updates) on a ring of 8192
    synthetic transitions; inputs resident on the device."""
    from paper_2606_03113_amd import Dqn
    q = Dqn(hidden=H, capacity=1 << 16, batch=B)
    q.lede_dqn_init(li.dqn_init_uniforms(H))
    q.lede_dqn_push(li.dqn_transitions(8192))
    ins = [li.dqn_update_inputs(i, H, B) for i in range(n_updates)]
    u = torch.from_numpy(np.stack([a for a, _ in ins])).cuda()
    nz = torch.from_numpy(np.stack([b for _, b in ins])).cuda()
    for i in range(20):
        q.lede_dqn_update(u[i], nz[i], want_loss=False)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(n_updates):
        q.lede_dqn_update(u[i], nz[i], want_loss=False)
        if i % 512 == 511:
            q.lede_dqn_sync_target()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    loss = q.lede_dqn_update(u[0], nz[0])
    q.close()
    return {"updates_per_s": round(n_updates / (ms / 1e3), 1), "us_per_update": round(1e3 * ms / n_updates, 2),
            "hidden": H, "batch": B, "n_step": 3, "replay": 8192, "last_loss": round(loss, 5),
            "bound": "latency (one block per update; host launch included)"}


def dqn_oracle_rate(li, budget_s=3.0, H=16, B=32):
    """The oracle trainer's learning updates per second on the same inputs."""
    from oracle import dqn as od
    tr = od.Trainer(od.Hyper(hidden=H, batch=B), 1 << 16, li.dqn_init_uniforms(H).astype(np.float64))
    for row in li.dqn_transitions(8192).astype(np.float64):
        tr.replay.push(row[:3], int(row[3]), row[4], bool(row[5]))
    t0 = time.time()
    n = 0
    while n < 5 or time.time() - t0 < budget_s:
        u, nz = li.dqn_update_inputs(n, H, B)
        tr.update(u.astype(np.float64), nz[0].astype(np.float64), nz[1].astype(np.float64))
        n += 1
    return round(n / (time.time() - t0), 1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama2-7b")
    ap.add_argument("--l", type=int, default=None)
    ap.add_argument("--k", type=int, default=None)
    ap.add_argument("--prof-steps", type=int, default=30)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dqn", action="store_true", help="skip the policy-trainer update timing")
    ap.add_argument("--sweep", action="store_true",
                    help="also time the exit layer x draft length grid {4,8,12,16} x {2,4,6,8} (llama2-7b)")
    ap.add_argument("--verify-reuse", action="store_true",
                    help="verify from the exit layer on the draft passes' hidden states and KV")
    ap.add_argument("--graphs", type=int, default=0)
    ap.add_argument("--in-flight", type=int, default=1,
                    help="forced greedy eager steps: how many are queued on the stream before the oldest "
                         "record is read back (1: one synchronous lede_step at a time)")
    ap.add_argument("--policy", choices=["fixed", "qnet", "schedule", "paper"], default=None,
                    help="how (l*, k) is chosen per step (default: the workload's own): fixed -- the workload's "
                         "static action (or --l / --k); qnet -- the argmax of the seeded (exit, length) "
                         "Q-network; schedule -- the workload's seeded uniform schedule; paper -- the paper's exit "
                         "policy (seeded random exit Q-network)")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="> 0: speculative sampling at this temperature (uniforms from the seeded generator)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before timing, copy this many MiB device-to-device three times (a kernel of "
                         "known traffic for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the decode path runs on a single device and has no "
              "multi-GPU mode; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import lede_inputs as li
    from lede_inputs.configs import WORKLOADS
    from paper_2606_03113_amd import Engine

    if args.graphs:
        # captured graphs need a stream other than the legacy default one
        torch.cuda.set_stream(torch.cuda.Stream())
    wl = WORKLOADS[args.workload]
    m = wl.model
    l, k = wl.fixed
    if args.l is not None or args.k is not None:
        from dataclasses import replace
        l = args.l if args.l is not None else l
        k = args.k if args.k is not None else k
        wl = replace(wl, fixed=(l, k))
    policy = args.policy or wl.policy
    if args.l is not None or args.k is not None:
        policy = "fixed"
    t0 = time.time()
    # models too large to generate whole in a bench run repeat a few
    # generated layers (the oracle's CPU baseline then is not run)
    lazy = m.n_layers * m.layer_weight_bytes() > (60 << 30)
    log("generating %s weights%s ..." % (m.name, " (%d distinct layers, repeated)" % REPEAT_LAYERS if lazy else ""))
    if lazy:
        weights = {n: li.weight_tensor(m, n) for n in ("embed", "head", "final_norm")}
        weights["layers"] = RepeatedLayers(m, torch)
    else:
        weights = li.weights(m)
    qnet = li.qnet_weights(m) if m.qnet_hidden else None
    prompt = li.prompt(wl)
    log("  %.1f s" % (time.time() - t0))
    paper = policy == "paper"
    sched = li.schedule(wl, wl.n_gen) if policy == "schedule" else None
    if paper and (args.temperature > 0 or args.graphs):
        sys.exit("the exit policy runs greedy, eager steps")
    eng = Engine(m, max_ctx=wl.max_ctx + (16 if paper else 0), k_max=max(12 if paper else 8, k),
                 exit_hidden=16 if paper else 0)
    if lazy:
        eng.lede_load_weights({n: weights[n] for n in ("embed", "final_norm", "head")}, qnet)
        for j0 in range(0, m.n_layers, 8):
            eng.lede_load_weights(weights, first_layer=j0, n_layers=min(8, m.n_layers - j0))
        log("  %d layers loaded  %.1f s" % (m.n_layers, time.time() - t0))
    else:
        eng.load_weights(weights, qnet)
    if paper:
        eng.load_exit_qnet(li.exit_qnet_weights(16))
    eng.lede_set_options(args.graphs, 0)
    if args.verify_reuse:
        if args.graphs:
            sys.exit("steps with verify reuse run eagerly")
        eng.lede_set_verify_reuse(True)
    log("weights resident (%.1f GB arena)  %.1f s" % (eng.region_bytes[0] / 1e9, time.time() - t0))
    first = eng.lede_prefill(prompt)
    log("prefill %d tokens done  %.1f s" % (wl.prompt_len, time.time() - t0))

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copies of %d MiB done" % args.calib_copy_mib)

    produced = [first]
    log_q = m.qnet_hidden > 0

    n_steps = [0]

    def action():
        if policy == "schedule":
            return tuple(int(x) for x in sched[n_steps[0] % len(sched)])
        return (l, k)

    def step():
        if paper:
            rec = eng.lede_step_policy(n_remaining=wl.n_gen - len(produced))
            kinds = eng.policy_log()[:, 0]
            rec.n_cand, rec.n_draft = int((kinds == 0).sum()), int((kinds == 1).sum())
        elif policy == "qnet":
            rec = eng.lede_step(None, n_remaining=wl.n_gen - len(produced), log_qnet=False)
        elif args.temperature > 0:
            rec = eng.lede_step_sampled(action(), args.temperature, li.step_uniforms(n_steps[0]),
                                        n_remaining=wl.n_gen - len(produced), log_qnet=log_q)
        else:
            rec = eng.lede_step(action(), n_remaining=wl.n_gen - len(produced), log_qnet=log_q)
        n_steps[0] += 1
        produced.extend(rec.emitted)
        return rec

    from paper_2606_03113_amd.lede import MAX_IN_FLIGHT
    if not 1 <= args.in_flight <= MAX_IN_FLIGHT:
        sys.exit("--in-flight must be in 1..%d" % MAX_IN_FLIGHT)
    pipelined = (args.in_flight > 1 and policy == "fixed" and args.temperature == 0 and not args.graphs
                 and not args.verify_reuse)

    def run_steps(n):
        """n steps; pipelined, each step is queued while up to in_flight - 1 earlier
        ones still run, and n_remaining is the fewest tokens that can be left."""
        if not pipelined:
            return [step() for _ in range(n)]
        rs, queued = [], []  # queued: the k_eff bound of each step in flight

        def collect():
            r = eng.lede_step_collect()
            queued.pop(0)
            produced.extend(r.emitted)
            rs.append(r)

        for _ in range(n):
            if len(queued) == args.in_flight:
                collect()
            left = max(1, wl.n_gen - len(produced) - sum(q + 1 for q in queued))
            eng.lede_step_submit((l, k), n_remaining=left, log_qnet=log_q)
            queued.append(min(k, left - 1))
            n_steps[0] += 1
        while queued:
            collect()
        return rs

    if args.graphs and args.temperature > 0:
        sys.exit("sampled steps are not captured in graphs")
    if args.warmup + args.steps >= wl.n_gen - 1:
        sys.exit("warmup + steps must stay below the %d generated tokens" % wl.n_gen)
    run_steps(args.warmup)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    n0 = len(produced)
    recs = []
    w0 = time.perf_counter()
    e0.record(stream)
    recs = run_steps(args.steps)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = e0.elapsed_time(e1)
    toks = len(produced) - n0
    log("timed %d steps: %.3f ms/step (wall %.3f ms/step), %d tokens" % (args.steps, ms / args.steps,
                                                                        1e3 * wall / args.steps, toks))

    def replay(level, n):
        """The same steps again from the prompt state, timed at a level."""
        eng.lede_truncate(wl.prompt_len)
        eng.lede_set_pending(first)
        del produced[1:]
        n_steps[0] = 0
        for _ in range(min(args.warmup, 3)):
            step()
        eng.lede_prof_enable(level)
        eng.lede_prof_read(reset=True)
        rs = [step() for _ in range(n)]
        pr = eng.lede_prof_read(reset=True)
        eng.lede_prof_enable(0)
        return rs, pr

    # draft / verify phase times with nothing else recorded, then every launch
    phase_recs, phases = replay(1, args.prof_steps)
    prof_recs, prof = replay(2, args.prof_steps)

    # plain autoregressive decoding on the same path (verify with no drafts)
    eng.lede_truncate(wl.prompt_len)
    eng.lede_set_pending(first)
    del produced[1:]
    n_ar = min(args.steps, wl.n_gen - 2)
    def ar_step(i):
        if args.temperature > 0:
            return eng.lede_step_sampled((l, 0), args.temperature, li.step_uniforms(i), log_qnet=False)
        return eng.lede_step((l, 0), log_qnet=False)

    for i in range(min(args.warmup, 3)):
        ar_step(i)
    torch.cuda.synchronize()
    e0.record(stream)
    ar_recs = [ar_step(i) for i in range(n_ar)]
    e1.record(stream)
    torch.cuda.synchronize()
    ar_ms = e0.elapsed_time(e1)
    ar_bytes = sum(verify_bytes(m, 0, r.seq_len - 1) for r in ar_recs)

    sweep = None
    if args.sweep:
        # the workload's (exit layer x draft length) grid from the prompt state:
        # 20 timed steps per point, then 10 with the draft / verify phases timed
        sweep = []
        for ls in (4, 8, 12, 16):
            for ks in (2, 4, 6, 8):
                gen = [1]

                def fixed_step():
                    r = eng.lede_step((ls, ks), n_remaining=max(1, wl.n_gen - gen[0]), log_qnet=log_q)
                    gen[0] += len(r.emitted)
                    return r
                eng.lede_truncate(wl.prompt_len)
                eng.lede_set_pending(first)
                for _ in range(2):
                    fixed_step()
                torch.cuda.synchronize()
                e0.record(stream)
                rs = [fixed_step() for _ in range(20)]
                e1.record(stream)
                torch.cuda.synchronize()
                sw_ms = e0.elapsed_time(e1)
                eng.lede_prof_enable(1)
                eng.lede_prof_read(reset=True)
                prs = [fixed_step() for _ in range(10)]
                pr = eng.lede_prof_read(reset=True)
                eng.lede_prof_enable(0)
                sdb = svb = 0.0
                for r in prs:
                    c = r.seq_len - r.accepted - 1
                    sdb += sum(pass_bytes(m, r.l, c + i) for i in range(r.k_eff)) + (m.qnet_bytes() if log_q else 0)
                    svb += verify_bytes(m, r.k_eff, c)
                dpm, vpm = pr["draft_phase"]["ms"], pr["verify_phase"]["ms"]
                sweep.append({"l": ls, "k": ks, "ms_per_step": round(sw_ms / 20, 4),
                              "tokens_per_s": round(sum(len(r.emitted) for r in rs) / (sw_ms / 1e3), 2),
                              "draft_frac": round(sdb / (dpm * 1e6) / HBM_PEAK_GBPS, 4) if dpm else None,
                              "verify_frac": round(svb / (vpm * 1e6) / HBM_PEAK_GBPS, 4) if vpm else None})
                log("sweep l=%d k=%d: %.3f ms/step" % (ls, ks, sw_ms / 20))

    # achievable read bandwidth: the weight arena read once by the probe kernel
    from paper_2606_03113_amd import op_read_probe
    probe_bytes = min(eng.weights.numel(), 16 << 30) // 16 * 16  # at most 16 GiB of the arena
    probe = {}
    for grid in (1024, 4096, 16384):
        op_read_probe(eng.weights[:probe_bytes], grid)
        probe[grid] = probe_bytes / (min(op_read_probe(eng.weights[:probe_bytes], grid) for _ in range(3)) * 1e6)
    # the same read with the one-row linear kernel's load structure and no
    # arithmetic, per matrix shape of a draft pass, from arena regions not read
    # for at least 600 MB (beyond the 256 MB memory-side cache)
    from paper_2606_03113_amd import op_read_groups
    kt = lambda K: -(-K // (32 if m.dtype == "bf16" else 16))  # noqa: E731
    qkv_rows = m.n_heads * m.head_dim + 2 * m.n_kv_heads * m.head_dim
    shapes = {"qkv": (qkv_rows // 16, kt(m.d_model)), "o": (m.d_model // 16, kt(m.n_heads * m.head_dim)),
              "gate_up": (2 * m.ffn_dim // 16, kt(m.d_model)), "down": (m.d_model // 16, kt(m.ffn_dim)),
              "head": (m.vocab // 16, kt(m.d_model))}
    arena = eng.weights.numel()
    ceiling = {}
    rot = 0
    for name, (ng, nt) in shapes.items():
        size = ng * nt * 1024
        ts = []
        for _ in range(4):
            off = (rot * (600 << 20)) % (arena - size) // 256 * 256
            rot += 1
            ts.append(op_read_groups(eng.weights[off:off + size], ng, nt))
        t = min(ts[1:])
        ceiling[name] = {"groups": ng, "MB": round(size / 1e6, 1), "us": round(1e3 * t, 2),
                         "GBps": round(size / (t * 1e6), 1)}
    # one draft pass at the workload's exit layer, weights only
    pass_w = l * sum(ceiling[n]["MB"] for n in ("qkv", "o", "gate_up", "down")) + ceiling["head"]["MB"]
    pass_t = l * sum(ceiling[n]["us"] for n in ("qkv", "o", "gate_up", "down")) + ceiling["head"]["us"]
    vec_ceiling = 1e3 * pass_w / pass_t  # GB/s
    from paper_2606_03113_amd.lede import K_SYMBOLS
    lin = {n: prof[n] for n in K_SYMBOLS}
    # the linear class that moves the most algorithmic bytes per step (a choice by
    # time would flip under a profiler, which stretches the two classes unequally)
    dom = max(lin, key=lambda n: lin[n]["bytes"])
    d = lin[dom]
    achieved = d["bytes"] / (d["ms"] * 1e6)  # GB/s
    kname = K_SYMBOLS[dom] if m.dtype == "bf16" else K_SYMBOLS[dom].replace("<1,", "<0,")
    traffic = traffic_from_profile(dom, wl.name, d["launches"])
    dp, vp = phases["draft_phase"], phases["verify_phase"]
    # algorithmic bytes of the phase-timed steps' passes
    db = vb = 0.0
    for r in phase_recs:
        c = r.seq_len - r.accepted - 1  # KV length when the step started
        if paper:
            db += policy_draft_bytes(m, r.l, c, r.n_cand, r.n_draft) if r.k_eff else 0
        else:
            db += sum(pass_bytes(m, r.l, c + i) for i in range(r.k_eff))
        db += m.qnet_bytes() if (log_q or policy == "qnet") and r.k_eff else 0
        if args.verify_reuse and r.k_eff:
            db += extend_bytes(m, r.l, c, r.k_eff)
            vb += verify_bytes(m, r.k_eff, c, r.l)
        else:
            vb += verify_bytes(m, r.k_eff, c)
    acc_tokens = sum(len(r.emitted) for r in recs)
    policy_text = {
        "fixed": "static exit l=%d, draft k=%d%s" % (l, k, ", Q-network logged" if log_q else ""),
        "qnet": "exit layer and draft length per step from the Q-network (%d->%d->%dx%d) over exits %s x lengths %s"
                % (m.d_model, m.qnet_hidden, len(m.exits), len(m.lengths), _span(m.exits), _span(m.lengths)),
        "schedule": "seeded uniform schedule l in %d..%d, k in %d..%d" % (wl.sched_l + wl.sched_k),
        "paper": "exit layer and draft length per step from the exit policy over exits %s" % (list(m.exits),),
    }[policy]
    kv_from = recs[0].seq_len - recs[0].accepted - 1
    kv_to = recs[-1].seq_len
    accepted = sum(r.accepted for r in recs)
    drafted = sum(r.k_eff for r in recs)
    out = {
        "metric": ("decode tokens/s (batch 1, SSD) + % of HBM peak, Llama-2-7B-shaped bf16"
                   if wl.name == "llama2-7b" else "decode tokens/s (batch 1, SSD), %s" % wl.name)
        + (", speculative sampling T=%g" % args.temperature if args.temperature > 0 else ""),
        "value": round(acc_tokens / (ms / 1e3), 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms / args.steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": m.dtype,
        "data": "synthetic (random-init N(0,0.02) weights, uniform-random prompt%s)" % (
            "; the %d layers repeat %d generated ones" % (m.n_layers, REPEAT_LAYERS) if lazy else ""),
        "config": {"workload": "%s: L=%d d=%d heads=%d/%d ffn=%d vocab=%d, prompt %d; %s; timed: %d steps "
                               "from KV length %d to %d (%d tokens) after %d warm-up steps" %
                               (m.name, m.n_layers, m.d_model, m.n_heads, m.n_kv_heads, m.ffn_dim, m.vocab,
                                wl.prompt_len, policy_text, args.steps, kv_from, kv_to, acc_tokens, args.warmup),
                   "batch": 1, "prompt_len": wl.prompt_len, "exit_layer": l, "draft_len": k,
                   "graphs": bool(args.graphs), "verify_reuse": bool(args.verify_reuse),
                   "steps_in_flight": args.in_flight if pipelined else 1,
                   "acceptance": ("speculative sampling, T=%g" % args.temperature if args.temperature > 0
                                  else "greedy"),
                   "policy": policy},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic, "kernel": kname,
                     "avg_launch_us": round(1e3 * d["ms"] / max(d["launches"], 1), 3),
                     "launches": d["launches"]},
        "passes": {
            "draft_GBps": round(db / (dp["ms"] * 1e6), 1) if dp["ms"] else None,
            "verify_GBps": round(vb / (vp["ms"] * 1e6), 1) if vp["ms"] else None,
            "draft_frac": round(db / (dp["ms"] * 1e6) / HBM_PEAK_GBPS, 4) if dp["ms"] else None,
            "verify_frac": round(vb / (vp["ms"] * 1e6) / HBM_PEAK_GBPS, 4) if vp["ms"] else None,
            "kernel_ms": {n: round(v["ms"] / args.prof_steps, 4) for n, v in prof.items()
                          if not n.endswith("_phase")},
            "kernel_ms_source": "per step, from an instrumented replay of the same steps with every launch "
                                "bracketed by its own HIP events (slower than the timed region); phases from a "
                                "replay with only the draft / verify phases timed",
        },
        "acceptance": {"accepted": accepted, "drafted": drafted,
                       "acc_rate": round(accepted / drafted, 4) if drafted else None,
                       # Section 4.1: E = mean exit layer and d = mean draft length of the drafting steps
                       "E": round(float(np.mean([r.l for r in recs if r.k_eff])), 3) if drafted else None,
                       "d": round(float(np.mean([r.k_eff for r in recs if r.k_eff])), 3) if drafted else None},
        "ar": {"tokens_per_s": round(n_ar / (ar_ms / 1e3), 3), "ms_per_token": round(ar_ms / n_ar, 4),
               "GBps": round(ar_bytes / (ar_ms * 1e6), 1), "frac": round(ar_bytes / (ar_ms * 1e6) / HBM_PEAK_GBPS, 4),
               "ssd_speedup": round((acc_tokens / (ms / 1e3)) / (n_ar / (ar_ms / 1e3)), 4)},
        "load_structure_ceiling": {"shapes": ceiling, "draft_pass_GBps": round(vec_ceiling, 1),
                                   "roofline_kernel_vs_ceiling": round(achieved / vec_ceiling, 4)},
        "hbm_read_probe": {"GBps": round(max(probe.values()), 1),
                           "frac": round(max(probe.values()) / HBM_PEAK_GBPS, 4),
                           "bytes": probe_bytes, "by_grid": {str(g): round(v, 1) for g, v in probe.items()}},
    }
    if sweep is not None:
        out["sweep"] = sweep
    if paper:
        nd = [r.n_cand + r.n_draft for r in phase_recs]
        out["exit_policy"] = {
            "decisions_per_step": round(float(np.mean(nd)), 3),
            "candidates_per_step": round(float(np.mean([r.n_cand for r in phase_recs])), 3),
            "draft_phase_ms_per_step": round(dp["ms"] / len(phase_recs), 4),
            "note": "each decision is one exit-policy kernel and a read-back the host waits for; the draft "
                    "phase (and draft_frac) includes those waits"}
    if not args.no_dqn:
        log("policy trainer updates ...")
        out["dqn"] = dqn_leg(torch, li)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) ...")
        if lazy:
            log("  not run: the model's layers repeat a few generated ones")
        else:
            acts = sched if policy == "schedule" else [(l, k)]
            out["cpu_baseline"] = cpu_baseline(wl, weights, qnet, first, policy, acts)
        if "dqn" in out:
            out["dqn"]["oracle_updates_per_s"] = dqn_oracle_rate(li)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
