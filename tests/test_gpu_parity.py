"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Every input comes from the seeded generator; every expected value from the oracle.  Outputs
must satisfy |o - o_oracle| <= 2e-2 + 1e-2 |o_oracle|; selected units must equal the oracle's
except where the oracle's own scores at the k-th boundary are within 1e-5 relative (the band
rule of oracle.accept).
"""
import numpy as np
import pytest
import torch

from gpu_helpers import (ROLE_DELTA, ROLE_FULL, ROLE_SPARSE, D, check_step, log, oracle_kv,
                         host_cache_of, run_step, select_of, shape_of)
from oracle import accept as A
from oracle import delta_oracle as O
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu


def _inputs(cfg, unit_tokens=16, **kw):
    w = configs.get(cfg, unit_tokens)
    for k in [k for k in kw if hasattr(w, k)]:
        setattr(w, k, kw.pop(k))
    log(f"generating {w.describe()}")
    inp = synth.make_inputs(w, "cuda", **kw)
    torch.cuda.synchronize()
    return inp


# ------------------------------------------------------------------------------------------
# Config 1 (tiny): every layer, both aggregations, both unit sizes
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("agg", [0, 1])
@pytest.mark.parametrize("U", [16, 1])
def test_config1_step(agg, U):
    inp = _inputs(1, U)
    res = run_step(inp, agg=agg)
    check_step(inp, res, agg=agg).assert_ok()


def test_config1_standalone_entry_points_and_scores():
    d = D()
    inp = _inputs(1)
    w = inp.workload
    shape, sel = shape_of(inp), select_of(w)
    ws = d.alloc_workspace(shape, sel)
    kv = d.make_kv(inp.k_cache[1], inp.v_cache[1], inp.page_table, inp.seq_lens)
    out_f = torch.empty_like(inp.q[1])
    out_d = torch.empty_like(inp.q[1])
    K = w.budget_units
    sel_idx = torch.empty((w.batch, K), dtype=torch.int32, device="cuda")
    sel_cnt = torch.empty((w.batch,), dtype=torch.int32, device="cuda")
    n_u = (inp.max_seq_len + 15) // 16
    us = torch.full((w.batch, n_u), -1.0, device="cuda")
    d.delta_full_attn(shape, kv, inp.q[1], out_f, ws)
    d.delta_delta_attn_select(shape, kv, inp.q[1], out_d, sel, sel_idx, sel_cnt, us, ws)
    torch.cuda.synchronize()
    # Delta-layer attention is the full attention, bit for bit (App. A, Alg. 1)
    assert torch.equal(out_f.view(torch.int16), out_d.view(torch.int16))
    q, Kt, V = oracle_kv(inp, 1, 0, host_cache_of(inp, 1))
    o, alpha = O.full_attention(q, Kt, V, O.default_scale(w.head_dim))
    rho, S = O.refresh_units(alpha, 16, K, w.recent_units)
    dev_S = us[0].cpu().numpy().astype(np.float64)
    rel = np.abs(dev_S - S) / S
    log(f"unit scores max rel err {rel.max():.3g}")
    assert rel.max() <= 1e-5
    v = A.check_selection(S, K, w.recent_units, sel_idx[0, :int(sel_cnt[0])].cpu().numpy(), rho)
    assert v.ok, v.reasons
    # sparse attention over the device's selection
    out_s = torch.empty_like(inp.q[2])
    kv2 = d.make_kv(inp.k_cache[2], inp.v_cache[2], inp.page_table, inp.seq_lens)
    d.delta_sparse_attn(shape, kv2, inp.q[2], out_s, sel, sel_idx, sel_cnt, ws)
    torch.cuda.synchronize()
    q2, K2, V2 = oracle_kv(inp, 2, 0, host_cache_of(inp, 2))
    o2 = O.sparse_attention(q2, K2, V2, sel_idx[0, :int(sel_cnt[0])].cpu().numpy(), 16,
                            O.default_scale(w.head_dim))
    ok, err, _ = A.check_output(out_s[0].float().cpu().numpy(), o2)
    assert ok, err


@pytest.mark.parametrize("U", [16, 1])
def test_physical_selection_matches_page_table(U):
    """sel_phys is sel_idx read through the page table (exactly, -1 padding included), and a
    sparse layer given sel_phys computes bit for bit what it computes through the page table.
    Lengths mix sequences that fit the budget (every unit kept) with ones that select."""
    d = D()
    w = configs.get(1, U)
    lens = [1024, 100, 129, 1000]
    w.batch = len(lens)
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    shape, sel = shape_of(inp), select_of(w)
    ws = d.alloc_workspace(shape, sel)
    kv = d.make_kv(inp.k_cache[1], inp.v_cache[1], inp.page_table, inp.seq_lens)
    K = w.budget_tokens // U
    sel_idx = torch.empty((w.batch, K), dtype=torch.int32, device="cuda")
    sel_cnt = torch.empty((w.batch,), dtype=torch.int32, device="cuda")
    sel_phys = torch.full((w.batch, K), -7, dtype=torch.int32, device="cuda")
    out_d = torch.empty_like(inp.q[1])
    d.delta_delta_attn_select(shape, kv, inp.q[1], out_d, sel, sel_idx, sel_cnt, None, ws,
                              sel_phys=sel_phys)
    torch.cuda.synchronize()
    idx, ph, pt = sel_idx.cpu().numpy(), sel_phys.cpu().numpy(), inp.page_table.cpu().numpy()
    for b in range(w.batch):
        valid = idx[b] >= 0
        assert valid.sum() == int(sel_cnt[b])
        u = idx[b][valid]
        want = pt[b][u] if U == 16 else pt[b][u // 16] * 16 + u % 16
        np.testing.assert_array_equal(ph[b][valid], want)
        assert np.all(ph[b][~valid] == -1)
    kv2 = d.make_kv(inp.k_cache[2], inp.v_cache[2], inp.page_table, inp.seq_lens)
    out_a, out_b = torch.empty_like(inp.q[2]), torch.empty_like(inp.q[2])
    d.delta_sparse_attn(shape, kv2, inp.q[2], out_a, sel, sel_idx, sel_cnt, ws)
    d.delta_sparse_attn(shape, kv2, inp.q[2], out_b, sel, sel_idx, sel_cnt, ws, sel_phys=sel_phys)
    torch.cuda.synchronize()
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))


# ------------------------------------------------------------------------------------------
# Config 2 (Llama-8B shape, B=1, 8k): every layer of the step
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("agg", [0, 1])
@pytest.mark.parametrize("U", [16, 1])
def test_config2_step(U, agg):
    """32 query heads: the scoring kernel's eight-head load batches, for the paper's maximum
    over heads and for the sum (Sec. 4 "Selection mechanism"; App. A, Alg. 2)."""
    inp = _inputs(2, U)
    res = run_step(inp, agg=agg)
    check_step(inp, res, agg=agg).assert_ok()


# ------------------------------------------------------------------------------------------
# Edge cases
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("lens", [[1], [15], [16], [17], [100], [129], [1000], [1024], [5, 1024, 333, 48]])
def test_ragged_and_short_lengths(lens):
    """s = 1, s < budget, s mod 16 != 0, mixed lengths in one batch (poisoned page tails)."""
    w = configs.get(1)
    w.batch = len(lens)
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    res = run_step(inp)
    check_step(inp, res).assert_ok()


@pytest.mark.parametrize("recent", [0, 16, 112, 8, 17, 100])
def test_recency_window_sizes(recent):
    """Windows of whole pages and of token counts that round up to the next page (App. A,
    Alg. 1: ceil(L / P) pages)."""
    inp = _inputs(1)
    res = run_step(inp, recent=recent)
    check_step(inp, res, recent=recent).assert_ok()


@pytest.mark.parametrize("hq,hkv,d", [(8, 8, 64), (7, 1, 128), (16, 2, 128), (12, 4, 64), (6, 2, 128)])
def test_group_sizes_and_head_dims(hq, hkv, d):
    w = configs.get(1)
    w.n_q_heads, w.n_kv_heads, w.head_dim, w.batch = hq, hkv, d, 2
    inp = synth.make_inputs(w, "cuda", seq_lens=[700, 1024])
    res = run_step(inp)
    check_step(inp, res).assert_ok()


def test_shuffled_page_table_is_bitwise_identical():
    w = configs.get(1)
    w.batch = 3
    a = synth.make_inputs(w, "cuda", seq_lens=[1024, 999, 640])
    w2 = configs.get(1)
    w2.batch, w2.shuffled_pages = 3, True
    b = synth.make_inputs(w2, "cuda", seq_lens=[1024, 999, 640])
    assert not torch.equal(a.page_table, b.page_table)
    ra, rb = run_step(a), run_step(b)
    for i in range(3):
        assert torch.equal(ra.outs[i].view(torch.int16), rb.outs[i].view(torch.int16))
    assert torch.equal(ra.sel_idx, rb.sel_idx)
    check_step(b, rb).assert_ok()


def test_duplicated_pages_force_exact_ties():
    """Many logical pages share one physical page: their scores are exactly equal, and the
    lower indices must be taken (exact equality with the oracle, no band)."""
    inp = _inputs(1)
    w = inp.workload
    scale = O.default_scale(w.head_dim)
    q, K, V = oracle_kv(inp, 1, 0, host_cache_of(inp, 1))
    _, alpha = O.full_attention(q, K, V, scale)
    _, S0 = O.refresh_units(alpha, 16, w.budget_units, w.recent_units)
    top = int(np.argmax(S0[:-w.recent_units]))
    pt = inp.page_table.clone()
    dups = [u for u in range(1, 60) if u != top][:48]
    pt[0, dups] = int(pt[0, top])   # 48 exact copies of the best page among the candidates
    inp.page_table = pt
    res = run_step(inp)
    q, K, V = oracle_kv(inp, 1, 0, host_cache_of(inp, 1))
    _, alpha = O.full_attention(q, K, V, scale)
    rho, S = O.refresh_units(alpha, 16, w.budget_units, w.recent_units)
    dev = res.sel_idx[0, 0, :int(res.sel_cnt[0, 0])].cpu().numpy()
    tied = int(np.sum(S[:-w.recent_units] == S[top]))
    log(f"{tied} exactly tied pages; oracle {rho.tolist()} device {dev.tolist()}")
    assert dev.tolist() == rho.tolist()
    check_step(inp, res).assert_ok()


def test_all_full_roles_and_sparse_before_delta():
    inp = _inputs(1)
    r_full = run_step(inp, roles=[ROLE_FULL] * 3)
    r_sp = run_step(inp, roles=[ROLE_SPARSE, ROLE_DELTA, ROLE_SPARSE])
    # a sparse layer before any Delta layer attends to every unit: identical to full
    assert torch.equal(r_full.outs[0].view(torch.int16), r_sp.outs[0].view(torch.int16))
    assert torch.equal(r_full.outs[1].view(torch.int16), r_sp.outs[1].view(torch.int16))
    check_step(inp, r_sp, roles=[ROLE_SPARSE, ROLE_DELTA, ROLE_SPARSE]).assert_ok()


def test_repeat_is_bitwise_deterministic():
    inp = _inputs(2)
    a = run_step(inp)
    b = run_step(inp)
    for x, y in zip(a.outs, b.outs):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert torch.equal(a.sel_idx, b.sel_idx) and torch.equal(a.sel_cnt, b.sel_cnt)


def test_graph_replay_matches_eager():
    """The step captured in a HIP graph (as the benchmark runs it) gives the eager results on
    every replay, with eager work and synchronisations between replays."""
    d = D()
    inp = _inputs(1)
    w = inp.workload
    shape, sel = shape_of(inp), select_of(w)
    ws = d.alloc_workspace(shape, sel)
    eager = run_step(inp, ws=ws)
    outs = [torch.empty_like(q) for q in inp.q]
    sel_idx = torch.empty((2, 1, w.budget_units), dtype=torch.int32, device="cuda")
    sel_cnt = torch.empty((2, 1), dtype=torch.int32, device="cuda")
    kvs = [d.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens) for i in range(3)]
    args = d.StepArgs(shape, w.roles, kvs, inp.q, outs, sel, sel_idx, sel_cnt, ws)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        d.delta_decode_step(args)        # warm-up outside capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        d.delta_decode_step(args)
    for rep in range(4):
        for o in outs:
            o.fill_(0)
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip(eager.outs, outs):
            assert torch.equal(x.view(torch.int16), y.view(torch.int16)), f"replay {rep}"
        assert torch.equal(sel_idx[0], eager.sel_idx[0])
        run_step(inp, ws=ws)             # eager work on the same workspace between replays


# ------------------------------------------------------------------------------------------
# Full-size workloads 3-8: the launch configuration the benchmark and its sweeps time,
# sampled sequences (6-8: the Qwen-1.5B, Qwen-7B-rank and Qwen-14B-rank runtime settings at
# batch 64 / 64 / 32 and 16-19K tokens, with the paper's Delta-layer sets)
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("cfg,seqs", [(3, [0, 9]), (4, [0, 5]), (5, [0, 17, 31]), (6, [0, 63]),
                                      (7, [1, 40]), (8, [0, 31])])
def test_full_size_sampled(cfg, seqs, agg=0):
    inp = _inputs(cfg)
    w = inp.workload
    res = run_step(inp, agg=agg)
    log("device step done; checking sampled sequences")
    first_sparse = [i for i, r in enumerate(w.roles) if r == ROLE_SPARSE]
    deltas = [i for i, r in enumerate(w.roles) if r == ROLE_DELTA]
    layers = sorted({0, 1, *deltas, first_sparse[0], first_sparse[-1]})
    rep = check_step(inp, res, seqs=seqs, layers=layers, use_page_table=False, agg=agg)
    rep.assert_ok()
    # every sequence's selection is structurally valid (size, order, recency units)
    cnt = res.sel_cnt.cpu().numpy()
    idx = res.sel_idx.cpu().numpy()
    for sd in range(len(deltas)):
        for b in range(w.batch):
            n_u = (inp.seq_lens_host[b] + 15) // 16
            c = cnt[sd, b]
            assert c == min(w.budget_units, n_u)
            r = idx[sd, b, :c]
            assert np.all(np.diff(r) > 0) and r[0] >= 0 and r[-1] == n_u - 1
            assert set(range(n_u - w.recent_units, n_u)) <= set(r.tolist())
    del inp, res
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cfg,seqs", [(4, [0, 7]), (5, [0, 31])])
def test_full_size_sampled_sum_aggregation(cfg, seqs):
    """The sum over heads at the full-size head counts: 28 query heads (the last load batch of
    every scoring wave is part masked) and 32 (Sec. 4 "Selection mechanism" reading)."""
    test_full_size_sampled(cfg, seqs, agg=1)


def test_shared_workspace_alternating_inputs():
    """Calls on one workspace with different inputs: every call must see only its own split
    partials (no stale data from the previous call), on every layer."""
    d = D()
    w = configs.get(2)
    w.batch = 2
    a = synth.make_inputs(w, "cuda", seq_lens=[8192, 5000], layers=range(4))
    w2 = configs.get(2)
    w2.batch, w2.cfg_id = 2, 7
    b = synth.make_inputs(w2, "cuda", seq_lens=[8192, 5000], layers=range(4))
    roles = [ROLE_FULL, ROLE_DELTA, ROLE_SPARSE, ROLE_SPARSE]
    shape, sel = shape_of(a), select_of(w)
    ws = d.alloc_workspace(shape, sel)
    for rep in range(2):
        for inp in (a, b):
            res = run_step(inp, roles=roles, ws=ws)
            check_step(inp, res, roles=roles).assert_ok()
