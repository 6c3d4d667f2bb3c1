#!/usr/bin/env python3
"""Decode-step attention benchmark: the full layer stack vs the DELTA layer stack on one GPU.

One step = one decoding step of every layer's attention over a full-resident paged bf16 KV
cache (inputs already in HBM): all-full roles for the full stack; full, Delta (attention +
page scoring + page selection) and sparse layers for the DELTA stack (App. A, Alg. 1).
Each step is one call of delta_decode_step, captured in a HIP graph and replayed; when a step
touches less than ~1 GiB, several copies of the inputs are rotated so that the 256 MB
Infinity Cache cannot serve a step from the previous one.

Printed JSON line (rank 0, N = 1): value = DELTA-stack microseconds per step (lower is
better), with the full stack, tokens/s, algorithmic HBM GB/s, per-role layer times, the
Delta-select overhead, the roofline of the dominant kernel (per-launch time from HIP events
around graph-captured launches of that role on the launch stream) and the CPU oracle timed on
this host.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2510_09883_amd import configs, synth  # noqa: E402

METRIC = "decode attention µs/step + achieved HBM GB/s (% peak), full vs DELTA stack"
HBM_PEAK_GBPS = 8000.0
ROLE_NAME = {configs.ROLE_FULL: "full", configs.ROLE_DELTA: "delta", configs.ROLE_SPARSE: "sparse"}


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


# ------------------------------------------------------------------------------------------
# algorithmic bytes (what the method itself must move; logits/partials are overhead)
# ------------------------------------------------------------------------------------------
def full_layer_bytes(w, lens):
    kv = sum(4 * w.n_kv_heads * w.head_dim * s for s in lens)
    qo = 4 * w.n_q_heads * w.head_dim * w.batch
    pt = sum(4 * ((s + 15) // 16) for s in lens)
    return kv + qo + pt


def sparse_layer_bytes(w, lens, sel_idx, sel_cnt):
    """sel_idx [B, K_u], sel_cnt [B] (host): tokens of the selected units, clipped at s_b."""
    U = w.unit_tokens
    toks = 0
    for b, s in enumerate(lens):
        for u in sel_idx[b, :sel_cnt[b]].tolist():
            toks += min(U, s - u * U)
    kv = 4 * w.n_kv_heads * w.head_dim * toks
    qo = 4 * w.n_q_heads * w.head_dim * w.batch
    idx = 4 * w.budget_units * w.batch
    return kv + qo + idx


# ------------------------------------------------------------------------------------------
def build_sets(w, n_sets):
    log(f"generating inputs: {w.describe()}, {n_sets} rotating copies")
    base = synth.make_inputs(w, "cuda", poison_tail=False)
    sets = [base]
    for _ in range(1, n_sets):
        sets.append(synth.DecodeInputs(
            w, [k.clone() for k in base.k_cache], [v.clone() for v in base.v_cache],
            [q.clone() for q in base.q], base.page_table, base.seq_lens, base.seq_lens_host,
            base.max_pages_per_seq, base.n_phys_pages))
    torch.cuda.synchronize()
    return sets


class Stack:
    """Per-input-set step arguments and a captured graph for one role list."""

    def __init__(self, D, w, sets, roles, shape, sel, ws):
        self.D, self.roles, self.sets = D, roles, sets
        n_delta = max(1, sum(r == configs.ROLE_DELTA for r in roles))
        self.sel_idx = torch.zeros((n_delta, w.batch, w.budget_units), dtype=torch.int32, device="cuda")
        self.sel_cnt = torch.zeros((n_delta, w.batch), dtype=torch.int32, device="cuda")
        self.sel_phys = torch.zeros((n_delta, w.batch, w.budget_units), dtype=torch.int32, device="cuda")
        self.outs, self.args = [], []
        for inp in sets:
            outs = [torch.empty_like(q) for q in inp.q]
            kvs = [D.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens)
                   for i in range(len(roles))]
            self.outs.append(outs)
            self.args.append(D.StepArgs(shape, roles, kvs, inp.q, outs, sel, self.sel_idx,
                                        self.sel_cnt, ws))
        self.graphs = []

    def eager(self, k):
        self.D.delta_decode_step(self.args[k % len(self.args)])

    def capture(self):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for a in self.args:
                self.D.delta_decode_step(a)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        for a in self.args:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self.D.delta_decode_step(a)
            self.graphs.append(g)
        torch.cuda.synchronize()

    def replay(self, k):
        self.graphs[k % len(self.graphs)].replay()


def time_steps(stack, steps, warmup):
    for k in range(warmup):
        stack.replay(k)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for k in range(steps):
        stack.replay(k)
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps   # ms per step


def time_layers(D, w, sets, stack, shape, sel, ws, steps):
    """Average duration of one launch of each role's entry point.  For each role, every layer
    of the stack runs that role (its own K/V cache and query), the n launches of one step are
    captured in a HIP graph (one graph per rotating input set), and the graphs are replayed
    `steps` times between two HIP events on the launch stream; per-launch time = elapsed time
    over the number of launches.  Host launch latency and per-call event overhead are excluded;
    the gap between kernels inside a graph is included.  Sparse launches use the selection of
    the Delta layer that precedes them in the schedule (the first Delta layer's for layers
    before it), with its physical pages, as delta_decode_step does.  Also returns how many
    layers of the step run each role."""
    roles = stack.roles
    slots, cur = [], -1
    for r in roles:
        if r == configs.ROLE_DELTA:
            cur += 1
        slots.append(cur)

    def step_role(i):
        r = roles[i]
        return "full" if (r == configs.ROLE_FULL or slots[i] < 0) else ROLE_NAME[r]

    counts = {}
    for i in range(len(roles)):
        counts[step_role(i)] = counts.get(step_role(i), 0) + 1
    # every selection slot holds this step's selection and its physical pages
    for i, r in enumerate(roles):
        if r == configs.ROLE_DELTA:
            inp = sets[0]
            kv = D.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens)
            D.delta_delta_attn_select(shape, kv, inp.q[i], stack.outs[0][i], sel, stack.sel_idx[slots[i]],
                                      stack.sel_cnt[slots[i]], None, ws, sel_phys=stack.sel_phys[slots[i]])
    torch.cuda.synchronize()
    scratch_idx = torch.empty_like(stack.sel_idx[0])
    scratch_cnt = torch.empty_like(stack.sel_cnt[0])
    scratch_phys = torch.empty_like(stack.sel_phys[0])

    def call(name, si, i):
        inp = sets[si]
        out = stack.outs[si][i]
        kv = D.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens)
        if name == "full":
            D.delta_full_attn(shape, kv, inp.q[i], out, ws)
        elif name == "delta":
            D.delta_delta_attn_select(shape, kv, inp.q[i], out, sel, scratch_idx, scratch_cnt, None,
                                      ws, sel_phys=scratch_phys)
        else:
            sd = max(slots[i], 0)
            D.delta_sparse_attn(shape, kv, inp.q[i], out, sel, stack.sel_idx[sd], stack.sel_cnt[sd],
                                ws, sel_phys=stack.sel_phys[sd])

    per_role = {}
    for name in ("full", "delta", "sparse"):
        if name not in counts:
            continue
        graphs = []
        for si in range(len(sets)):
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                for i in range(len(roles)):
                    call(name, si, i)
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for i in range(len(roles)):
                    call(name, si, i)
            graphs.append(g)
        for r in range(2):
            graphs[r % len(graphs)].replay()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for r in range(steps):
            graphs[r % len(graphs)].replay()
        e1.record()
        torch.cuda.synchronize()
        per_role[name] = e0.elapsed_time(e1) * 1e3 / (steps * len(roles))
    return per_role, counts


# ------------------------------------------------------------------------------------------
def cpu_baseline(w, inp, roles, budget_s):
    """The oracle as it stands, on this host: gather + every layer of the DELTA-stack step for
    whole sequences, until `budget_s` seconds are spent; scaled to microseconds per step."""
    import numpy as np
    from oracle import delta_oracle as O
    try:
        import threadpoolctl
        threads = max([p.get("num_threads", 1) for p in threadpoolctl.threadpool_info()] or [1])
    except Exception:   # pragma: no cover
        threads = 1
    scale = O.default_scale(w.head_dim)
    done, spent = 0, 0.0
    for b in range(w.batch):
        host = [synth.sequence_pages(inp, i, b) for i in range(len(roles))]
        qs = [O.bf16_bits_to_f64(synth.bits(inp.q[i][b])) for i in range(len(roles))]
        s_b = inp.seq_lens_host[b]
        t = time.perf_counter()
        ident = np.arange(host[0][0].shape[0])
        Ks = [O.gather_tokens(kb, ident, s_b) for kb, _ in host]
        Vs = [O.gather_tokens(vb, ident, s_b) for _, vb in host]
        O.decode_step_sequence(roles, qs, Ks, Vs, scale, w.unit_tokens, w.budget_units,
                               w.recent_units)
        spent += time.perf_counter() - t
        done += 1
        del host, Ks, Vs
        if spent >= budget_s:
            break
    us_per_step = spent / done * w.batch * 1e6
    sample = (f"oracle DELTA-stack step (gather + {len(roles)} layers) of {done} of {w.batch} "
              f"sequence(s), {spent:.1f} s; per-step value scaled by {w.batch}/{done}")
    return {"value": us_per_step, "unit": "us/step", "cores": threads, "kind": "oracle",
            "sample": sample, "host_cpus": len(os.sched_getaffinity(0))}


def measured_traffic(role, w, kernel_tag):
    """HBM bytes per launch of the dominant kernel from the committed rocprofv3 counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by a known-size copy), or None when there is none for this
    kernel and workload or the kernel source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"attn_{role}_{w.name}.md")
    src = os.path.join(ROOT, "paper_2510_09883_amd", "csrc", "attn_kernel.hip")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line:
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel") != kernel_tag:
        return None
    if kv.get("source_sha256") != hashlib.sha256(open(src, "rb").read()).hexdigest():
        return None
    return int(kv["traffic_bytes_per_launch"])


def copy_calibration():
    """A plain device copy of known size (64 MiB read + 64 MiB written), for scaling the
    FETCH_SIZE / WRITE_SIZE counters of the profiled kernels."""
    a = torch.empty(64 << 20, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    # default: the Llama-8B shape at 32K context, batch 16 -- the bandwidth-bound case the
    # targets are stated for (the B = 1, 8K workload is launch-latency bound)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--unit-tokens", type=int, default=16, choices=[16, 1])
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: this build has no multi-GPU path "
              "(--gpus must be 1).", file=sys.stderr)
        sys.exit(2)
    from paper_2510_09883_amd import delta as D

    w = configs.get(args.config, args.unit_tokens)
    lens = synth.seq_lens_for(w)
    fb = full_layer_bytes(w, lens)
    n_delta = sum(r == configs.ROLE_DELTA for r in w.roles)
    n_sets = 1
    approx_delta_step = (len(w.roles) - n_delta) * fb * min(1.0, w.budget_tokens / max(lens)) + n_delta * fb
    if approx_delta_step < (1 << 30):
        n_sets = min(8, 1 + math.ceil((1 << 30) / approx_delta_step))
    sets = build_sets(w, n_sets)
    inp = sets[0]
    shape = D.make_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, inp.max_pages_per_seq,
                         inp.max_seq_len)
    sel = D.make_select(w.budget_tokens, w.recent_tokens, w.unit_tokens, D.DELTA_AGG_MAX)
    ws = D.alloc_workspace(shape, sel)

    delta_stack = Stack(D, w, sets, w.roles, shape, sel, ws)
    full_stack = Stack(D, w, sets, [configs.ROLE_FULL] * len(w.roles), shape, sel, ws)
    delta_stack.capture()
    full_stack.capture()
    log("graphs captured")

    ms_full = time_steps(full_stack, args.steps, args.warmup)
    ms_delta = time_steps(delta_stack, args.steps, args.warmup)
    log(f"full stack {ms_full * 1e3:.1f} us/step, DELTA stack {ms_delta * 1e3:.1f} us/step")

    # algorithmic bytes of one DELTA step from the selections it made
    idx = delta_stack.sel_idx.cpu().numpy()
    cnt = delta_stack.sel_cnt.cpu().numpy()
    slot = -1
    delta_bytes = 0
    sparse_bytes = []
    for r in w.roles:
        if r == configs.ROLE_DELTA:
            slot += 1
        if r == configs.ROLE_SPARSE and slot >= 0:
            sb = sparse_layer_bytes(w, lens, idx[slot], cnt[slot])
            sparse_bytes.append(sb)
            delta_bytes += sb
        else:
            delta_bytes += fb
    full_bytes = fb * len(w.roles)

    layer_us, per_step = time_layers(D, w, sets, delta_stack, shape, sel, ws, args.steps)
    log(f"per-launch us: {layer_us}")
    sb_avg = sum(sparse_bytes) / len(sparse_bytes) if sparse_bytes else 0
    role_bytes = {"full": fb, "delta": fb, "sparse": sb_avg}
    dominant = max(layer_us, key=lambda r: layer_us[r] * per_step[r])
    kernel_name = {"full": "attn_kernel (dense rows)", "delta": "attn_kernel + score + select",
                   "sparse": "attn_kernel (selected pages)"}[dominant]
    mode = {"full": 0, "delta": 0, "sparse": 1 if w.unit_tokens == 16 else 2}[dominant]
    logits = "true" if dominant == "delta" else "false"
    kernel_tag = f"attn_kernel<{w.head_dim}, {w.group}, {mode}, {logits}>"
    traffic = measured_traffic(dominant, w, kernel_tag)
    achieved = role_bytes[dominant] / (layer_us[dominant] * 1e-6) / 1e9
    overhead = (layer_us["delta"] - layer_us["full"]) / layer_us["full"] if "delta" in layer_us and "full" in layer_us else None

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU oracle")
        cpu = cpu_baseline(w, inp, w.roles, args.cpu_seconds)

    copy_calibration()

    us_delta = ms_delta * 1e3
    rec = {
        "metric": METRIC,
        "value": round(us_delta, 2),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_delta, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "accum": "fp32",
        "data": "synthetic",
        "config": {
            "workload": w.describe(),
            "batch": w.batch, "seq_len": w.max_seq_len, "layers": len(w.roles),
            "budget_tokens": w.budget_tokens, "recent_tokens": w.recent_tokens,
            "unit_tokens": w.unit_tokens,
            "delta_layers": [i for i, r in enumerate(w.roles) if r == configs.ROLE_DELTA],
            "input_copies_rotated": n_sets, "graph": True,
        },
        "full_stack_us_per_step": round(ms_full * 1e3, 2),
        "delta_speedup_vs_full": round(ms_full / ms_delta, 3),
        "tokens_per_s": {"delta": round(w.batch / (ms_delta * 1e-3), 1),
                         "full": round(w.batch / (ms_full * 1e-3), 1)},
        "hbm_gbps_algorithmic": {"delta_stack": round(delta_bytes / (ms_delta * 1e-3) / 1e9, 1),
                                 "full_stack": round(full_bytes / (ms_full * 1e-3) / 1e9, 1)},
        "frac_of_peak": {"delta_stack": round(delta_bytes / (ms_delta * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                         "full_stack": round(full_bytes / (ms_full * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)},
        "layer_us": {k: round(v, 2) for k, v in layer_us.items()},
        "layer_gbps": {k: round(role_bytes[k] / (layer_us[k] * 1e-6) / 1e9, 1) for k in layer_us},
        "delta_select_overhead": None if overhead is None else round(overhead, 4),
        "roofline": {"bound": "hbm", "kernel": kernel_name, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic, "bytes_per_launch": int(role_bytes[dominant]),
                     "avg_launch_us": round(layer_us[dominant], 3)},
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
