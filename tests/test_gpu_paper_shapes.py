"""GPU parity on the runtime settings of the paper's throughput and Delta-layer experiments:
the Qwen-1.5B, Qwen-7B (one tensor-parallel rank of two) and Qwen-14B (one rank of four)
attention shapes (group sizes 6, 7 and 5 over two KV heads), a 1k-token budget with an
8-page recency window, and the paper's Delta-layer sets on a shortened stack.

Also checks the inputs the runtime sweeps build for short contexts (a page-table slice of a
longer cache) against the oracle, so that a sweep point reads what it claims to read.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import check_step, log, run_step
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu


def _shortened(cid, lens, n_layers, delta_layers):
    w = configs.get(cid)
    w.batch = len(lens)
    w.n_layers = n_layers
    w.set_delta_layers(delta_layers)
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    return w, inp


@pytest.mark.parametrize("cid", [6, 7, 8])
def test_runtime_shapes_step_matches_oracle(cid):
    # 2500 tokens select 64 of 157 pages; 1100 tokens select 64 of 69; 1000 fit the budget;
    # 17 is one partial page
    lens = [2500, 1100, 1000, 17]
    w, inp = _shortened(cid, lens, 6, [2, 4])
    res = run_step(inp)
    rep = check_step(inp, res)
    rep.assert_ok()
    cnt = res.sel_cnt.cpu().numpy()
    assert cnt[:, 0].tolist() == [64, 64] and cnt[:, 2].tolist() == [63, 63]
    log(f"{w.name}: step ok")


def test_page_table_slice_inputs_match_oracle():
    """A context-s view of a longer cache that reads logical pages [k*n, (k+1)*n) of every
    sequence (the rotation the runtime sweeps use below 1 GiB per step)."""
    w, base = _shortened(6, [4096, 4096], 4, [2])
    s, n, k = 1500, 94, 2
    assert (k + 1) * n <= base.max_pages_per_seq
    pt = torch.zeros_like(base.page_table)
    pt[:, :n] = base.page_table[:, k * n:(k + 1) * n]
    lens = torch.full((w.batch,), s, dtype=torch.int32, device="cuda")
    view = synth.DecodeInputs(w, base.k_cache, base.v_cache, base.q, pt, lens, [s] * w.batch,
                              base.max_pages_per_seq, base.n_phys_pages)
    res = run_step(view)
    check_step(view, res, use_page_table=True).assert_ok()
    # the view really reads the slice: its full-layer output differs from the first s tokens'
    res0 = run_step(synth.DecodeInputs(w, base.k_cache, base.v_cache, base.q, base.page_table,
                                       lens, [s] * w.batch, base.max_pages_per_seq,
                                       base.n_phys_pages))
    assert not np.array_equal(res.outs[0].float().cpu().numpy(), res0.outs[0].float().cpu().numpy())
