"""Helpers for the GPU parity tests: run the HIP path through the C ABI and compare it with
the oracle, sequence by sequence and layer by layer."""
from __future__ import annotations

import sys
import time

import numpy as np
import torch

from oracle import accept as A
from oracle import delta_oracle as O
from paper_2510_09883_amd import configs, synth

ROLE_FULL, ROLE_DELTA, ROLE_SPARSE = configs.ROLE_FULL, configs.ROLE_DELTA, configs.ROLE_SPARSE


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def D():
    from paper_2510_09883_amd import delta
    return delta


def shape_of(inp, sm_scale=0.0):
    w = inp.workload
    return D().make_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim, inp.max_pages_per_seq,
                          inp.max_seq_len, sm_scale)


def select_of(w, agg=0, budget=None, recent=None, path=0):
    return D().make_select(w.budget_tokens if budget is None else budget,
                           w.recent_tokens if recent is None else recent, w.unit_tokens, agg,
                           path)


class StepResult:
    def __init__(self, outs, sel_idx, sel_cnt):
        self.outs, self.sel_idx, self.sel_cnt = outs, sel_idx, sel_cnt


def run_step(inp, roles=None, agg=0, budget=None, recent=None, ws=None, path=0):
    """One decoding step of the whole stack through delta_decode_step (path: the Delta-layer
    path, DELTA_PATH_AUTO by default)."""
    d = D()
    w = inp.workload
    roles = w.roles if roles is None else roles
    shape = shape_of(inp)
    sel = select_of(w, agg, budget, recent, path)
    if ws is None:
        ws = d.alloc_workspace(shape, sel)
    outs = [torch.full_like(inp.q[i], float("nan")) for i in range(len(roles))]
    n_delta = max(1, sum(r == ROLE_DELTA for r in roles))
    K = sel.budget_tokens // sel.unit_tokens
    sel_idx = torch.full((n_delta, w.batch, K), -7, dtype=torch.int32, device="cuda")
    sel_cnt = torch.full((n_delta, w.batch), -7, dtype=torch.int32, device="cuda")
    kvs = [d.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens)
           for i in range(len(roles))]
    args = d.StepArgs(shape, roles, kvs, inp.q[:len(roles)], outs, sel, sel_idx, sel_cnt, ws)
    d.delta_decode_step(args)
    torch.cuda.synchronize()
    return StepResult(outs, sel_idx, sel_cnt)


def oracle_kv(inp, layer, b, host_cache=None):
    """float64 K, V [s, Hkv, d] and q [Hq, d] of sequence b at `layer`, decoded by the oracle
    from bf16 bits.  With host_cache = (k_bits, v_bits, pt) the oracle gathers through the real
    page table; otherwise only the sequence's pages are copied (in logical order)."""
    s_b = inp.seq_lens_host[b]
    if host_cache is not None:
        kb, vb, pt = host_cache
        row = pt[b]
    else:
        kb, vb = synth.sequence_pages(inp, layer, b)
        row = np.arange(kb.shape[0])
    K = O.gather_tokens(kb, row, s_b)
    V = O.gather_tokens(vb, row, s_b)
    q = O.bf16_bits_to_f64(synth.bits(inp.q[layer][b]))
    return q, K, V


def host_cache_of(inp, layer):
    return (synth.bits(inp.k_cache[layer]), synth.bits(inp.v_cache[layer]),
            inp.page_table.cpu().numpy())


def out_of(res, layer, b):
    return res.outs[layer][b].float().cpu().numpy().astype(np.float64)


class Report:
    def __init__(self):
        self.max_err = 0.0
        self.band_resolved = 0
        self.checked = 0
        self.failures = []

    def out(self, tag, o_dev, o_orc):
        ok, err, nbad = A.check_output(o_dev, o_orc)
        self.max_err = max(self.max_err, err)
        self.checked += 1
        if not ok:
            self.failures.append(f"{tag}: {nbad} outputs out of tolerance, max err {err:.3g}")

    def sel(self, tag, v):
        self.band_resolved += v.band_resolved
        if not v.ok:
            self.failures.append(f"{tag}: selection rejected: {v.reasons}")

    def assert_ok(self):
        log(f"checked {self.checked} layer outputs, max abs err {self.max_err:.3g}, "
            f"band-resolved units {self.band_resolved}")
        assert not self.failures, "\n".join(self.failures[:20])


def check_step(inp, res, seqs=None, layers=None, roles=None, agg=0, budget=None, recent=None,
               use_page_table=None, report=None):
    """Compare a delta_decode_step result with the oracle for sequences `seqs` and layers
    `layers` (default all).  Delta layers: full-attention output plus the selection, judged by
    the band rule against the oracle's scores.  Sparse layers: the oracle's sparse attention on
    the DEVICE's (accepted) selection of the most recent Delta layer."""
    w = inp.workload
    roles = w.roles if roles is None else roles
    U = w.unit_tokens
    K_u = (w.budget_tokens if budget is None else budget) // U
    L_u = O.recent_units_of(w.recent_tokens if recent is None else recent, U)
    seqs = range(w.batch) if seqs is None else seqs
    layers = range(len(roles)) if layers is None else sorted(layers)
    rep = report or Report()
    scale = O.default_scale(w.head_dim)
    if use_page_table is None:
        use_page_table = inp.k_cache[0 if inp.k_cache[0] is not None else layers[0]].numel() * 2 < (256 << 20)
    delta_slot = {}
    slot = -1
    for i, r in enumerate(roles):
        if r == ROLE_DELTA:
            slot += 1
        delta_slot[i] = slot
    for i in layers:
        hc = host_cache_of(inp, i) if use_page_table else None
        for b in seqs:
            q, K, V = oracle_kv(inp, i, b, hc)
            tag = f"layer {i} seq {b} role {roles[i]}"
            od = out_of(res, i, b)
            if roles[i] == ROLE_FULL or (roles[i] == ROLE_SPARSE and delta_slot[i] < 0):
                o, _ = O.full_attention(q, K, V, scale)
                rep.out(tag, od, o)
            elif roles[i] == ROLE_DELTA:
                o, alpha = O.full_attention(q, K, V, scale)
                rep.out(tag, od, o)
                rho, S = O.refresh_units(alpha, U, K_u, L_u, agg)
                cnt = int(res.sel_cnt[delta_slot[i], b])
                dev = res.sel_idx[delta_slot[i], b].cpu().numpy()
                if cnt != min(K_u, len(S)) or np.any(dev[cnt:] != -1):
                    rep.failures.append(f"{tag}: count {cnt} / padding wrong")
                rep.sel(tag, A.check_selection(S, K_u, L_u, dev[:cnt], rho))
            else:
                sd = delta_slot[i]
                cnt = int(res.sel_cnt[sd, b])
                rho = res.sel_idx[sd, b, :cnt].cpu().numpy().astype(np.int64)
                o = O.sparse_attention(q, K, V, rho, U, scale)
                rep.out(tag, od, o)
    return rep
