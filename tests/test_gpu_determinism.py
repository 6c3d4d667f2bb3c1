"""Long determinism runs of the cross-workgroup protocols: the split combine (partials published
with device-coherent stores, counted in with a device-scope atomic, merged by the last
workgroup), the balanced cut of a ragged batch, and the fused Delta kernel's sequence barrier.

A decoding step [full, Delta, sparse] is captured in a HIP graph and replayed 200 times, with a
synchronisation and a comparison after every replay; every replay must give the first run's
bits (outputs of the three layers, selected units and counts), and the run stops at the first
mismatch.  App. A, Alg. 1 makes the Delta layer's attention the full attention, and its
selection feeds the sparse layer, so a protocol that let a stale or missing partial through
would show up in all three.  Two shapes: 32 ragged sequences of 16K-32K tokens on a shuffled
page table (Llama-8B attention shape; balanced dense launches, split Delta path), and 8
sequences of 32K tokens with 28/4 heads (the fused Delta kernel, which the automatic path
takes there).
"""
import pytest
import torch

from gpu_helpers import ROLE_DELTA, ROLE_FULL, ROLE_SPARSE, D, log, select_of, shape_of
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu

ROLES = [ROLE_FULL, ROLE_DELTA, ROLE_SPARSE]
REPLAYS = 200


@pytest.mark.parametrize("cfg", [5, 4])
def test_graph_replays_are_bitwise_stable(cfg):
    d = D()
    w = configs.get(cfg)
    w.n_layers = len(ROLES)
    w.roles = list(ROLES)
    log(f"generating {w.describe()}")
    inp = synth.make_inputs(w, "cuda", poison_tail=False)
    shape, sel = shape_of(inp), select_of(w)
    log(f"Delta path: {'fused' if d.delta_delta_path(shape, sel) else 'split'}")
    ws = d.alloc_workspace(shape, sel)
    outs = [torch.empty_like(q) for q in inp.q]
    sel_idx = torch.full((1, w.batch, w.budget_units), -7, dtype=torch.int32, device="cuda")
    sel_cnt = torch.full((1, w.batch), -7, dtype=torch.int32, device="cuda")
    kvs = [d.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens)
           for i in range(len(ROLES))]
    args = d.StepArgs(shape, ROLES, kvs, inp.q, outs, sel, sel_idx, sel_cnt, ws)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        d.delta_decode_step(args)          # the reference run, eager
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs] + [sel_idx.clone(), sel_cnt.clone()]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        d.delta_decode_step(args)
    for rep in range(REPLAYS):
        for o in outs:
            o.fill_(0)
        sel_idx.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        got = list(outs) + [sel_idx, sel_cnt]
        for k, (a, b) in enumerate(zip(got, ref)):
            same = torch.equal(a.view(torch.int16), b.view(torch.int16)) if a.dtype == torch.bfloat16 \
                else torch.equal(a, b)
            assert same, f"replay {rep}: {'layer %d output' % k if k < 3 else 'selection'} differs"
    log(f"{REPLAYS} replays bitwise identical")
