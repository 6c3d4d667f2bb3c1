"""GPU parity of the balanced decomposition of dense (full and Delta) launches: a ragged
batch's 16-row groups, in (sequence, KV head, page) order, are cut into equal runs, one per
workgroup, and a run may hold the end of one (sequence, KV head) pair and the start of the next.
The cut is taken only where it shortens the longest run by a tenth against the static pieces;
equal lengths keep the static split (the CPU model of the cut, tests/test_balanced_cut.py,
says which cases take it).

Llama-8B attention shape, six sequences of 1.8K-4K tokens: the launch has 288 workgroups
(6 splits of 43 groups over 48 pairs), the batch 8920 groups, so every run is 31 groups and the
pairs (113 to 256 groups) are each combined from 5 to 10 pieces cut at places that do not
depend on the pair.  Qwen-7B shape with twelve sequences of 65-1455 tokens: runs of 8 groups
(against static pieces of 16), so some runs hold a whole short pair (written directly, no
combine) and parts of its neighbours, three pairs in one run.  Eight seeded random shapes
(group sizes 1-8, head dims 64 and 128, 2-8 KV heads, 6-24 sequences of lengths in [L/4, L],
shuffled page tables on odd seeds) cover the other kernel instantiations.  Outputs and
selections are checked against the oracle, and the Delta layer's output against the full
layer's, bit for bit (App. A, Alg. 1: the Delta layer's attention is the full attention).
"""
import pytest
import torch

import balanced_cases as BC
from gpu_helpers import D, check_step, log, run_step, select_of, shape_of
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu


def _ragged(cid, lens):
    w = configs.get(cid)
    w.batch = len(lens)
    w.n_layers = 3
    w.set_delta_layers([1])
    log(f"generating {w.describe()} lens {lens}")
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    return w, inp


def _delta_equals_full(w, inp, layer=1):
    d = D()
    shape, sel = shape_of(inp), select_of(w)
    ws = d.alloc_workspace(shape, sel)
    kv = d.make_kv(inp.k_cache[layer], inp.v_cache[layer], inp.page_table, inp.seq_lens)
    out_f = torch.full_like(inp.q[layer], float("nan"))
    out_d = torch.full_like(inp.q[layer], float("nan"))
    K = w.budget_units
    sel_idx = torch.empty((w.batch, K), dtype=torch.int32, device="cuda")
    sel_cnt = torch.empty((w.batch,), dtype=torch.int32, device="cuda")
    d.delta_full_attn(shape, kv, inp.q[layer], out_f, ws)
    d.delta_delta_attn_select(shape, kv, inp.q[layer], out_d, sel, sel_idx, sel_cnt, None, ws)
    torch.cuda.synchronize()
    assert not torch.isnan(out_f.float()).any()
    assert torch.equal(out_f.view(torch.int16), out_d.view(torch.int16))


@pytest.mark.parametrize("cid,lens", [(c, lens) for c, _, lens in BC.RAGGED])
def test_balanced_runs_match_oracle(cid, lens):
    w, inp = _ragged(cid, lens)
    d = D()
    ws = d.alloc_workspace(shape_of(inp), select_of(w))
    res = run_step(inp, ws=ws)
    check_step(inp, res).assert_ok()
    _delta_equals_full(w, inp)
    # repeated launches on one workspace give the same bits (the counters re-arm)
    res2 = run_step(inp, ws=ws)
    for a, b in zip(res.outs, res2.outs):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    log(f"{w.name}: balanced runs ok")


def _random_case(seed, G):
    """A seeded random shape with group size G (tests/balanced_cases.py; shuffled page tables
    on odd seeds).  The seeds are ones whose batch takes the balanced cut, which
    tests/test_balanced_cut.py checks on the CPU model of the cut."""
    hkv, d, lens = BC.random_case(seed)
    w = configs.Workload(90 + seed, f"random{seed}", 3, G * hkv, hkv, d, len(lens), max(lens), 256,
                         hh_frac=0.02, shuffled_pages=bool(seed % 2),
                         roles=[configs.ROLE_FULL, configs.ROLE_DELTA, configs.ROLE_SPARSE])
    return w, lens


@pytest.mark.parametrize("G,seed", BC.RANDOM)
def test_balanced_random_shapes(G, seed):
    w, lens = _random_case(seed, G)
    log(f"random case {seed}: Hq {w.n_q_heads} Hkv {w.n_kv_heads} d {w.head_dim} lens {lens}")
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    res = run_step(inp)
    check_step(inp, res, seqs=sorted({0, len(lens) // 2, len(lens) - 1})).assert_ok()
    _delta_equals_full(w, inp)


@pytest.mark.parametrize("B", BC.BATCH_LIMIT)
def test_balanced_batch_limit(B):
    """64 sequences fill the lanes of the balanced cut; at 65 the host keeps the static split.
    Qwen-1.5B attention shape (12/2/128) with lengths in [400, 800]."""
    lens = BC.batch_limit_lens(B)
    w = configs.get(6)
    w.batch = B
    w.n_layers = 3
    w.set_delta_layers([1])
    log(f"generating {w.describe()} B={B}")
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    res = run_step(inp)
    check_step(inp, res, seqs=[0, 31, B - 2, B - 1]).assert_ok()
    _delta_equals_full(w, inp)


def test_balanced_launch_in_graph_replays():
    """A balanced full launch captured in a HIP graph and replayed three times, with eager
    launches of the same call between the replays, gives the eager output bit for bit each
    time (the arrival counters re-arm inside the captured kernel)."""
    cid, _, lens = BC.RAGGED[0]
    w, inp = _ragged(cid, lens)
    d = D()
    shape = shape_of(inp)
    ws = d.alloc_workspace(shape)
    kv = d.make_kv(inp.k_cache[0], inp.v_cache[0], inp.page_table, inp.seq_lens)
    eager = torch.empty_like(inp.q[0])
    d.delta_full_attn(shape, kv, inp.q[0], eager, ws)
    torch.cuda.synchronize()
    out = torch.full_like(inp.q[0], float("nan"))
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        d.delta_full_attn(shape, kv, inp.q[0], out, ws)
    for rep in range(3):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), rep
        again = torch.empty_like(eager)
        d.delta_full_attn(shape, kv, inp.q[0], again, ws)
        torch.cuda.synchronize()
        assert torch.equal(again.view(torch.int16), eager.view(torch.int16)), rep
