"""The debug build of the library (python -m paper_2510_09883_amd.build --debug, -DDELTA_DEBUG=1):
its kernels check the device-side preconditions that release builds only document and record a
failure as a bit of the workspace's status word (byte 0) instead of reading out of bounds.

Every bad input here still keeps every access inside the caller's buffers (the "out of range"
page lies inside a larger allocation than the descriptor states, the long sequence is clamped
by release builds too, the selected unit is past the sequence but inside its page-table row), so
a missing check would show up as a missing status bit, never as a stray access.
"""
import ctypes
import os

import pytest
import torch

from gpu_helpers import D, check_step, log, run_step, select_of, shape_of
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu

DBG = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "paper_2510_09883_amd", "libdelta_attn_debug.so")


@pytest.fixture
def dbg(monkeypatch):
    if not os.path.exists(DBG):
        pytest.skip("the debug library is not built (python -m paper_2510_09883_amd.build --debug)")
    d = D()
    lib = d._bind(ctypes.CDLL(DBG))
    assert lib.delta_build_flags() == d.DELTA_BUILD_DEBUG
    monkeypatch.setattr(d, "_lib", lib)
    return d


def _status(ws):
    torch.cuda.synchronize()
    return int(ws[:4].view(torch.int32)[0].item())


def _tiny(lens):
    w = configs.get(1)
    w.batch = len(lens)
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    return w, inp


def test_debug_build_changes_no_result(dbg):
    """A valid step gives the release library's bits and leaves the status word at 0."""
    w, inp = _tiny([1024, 700])
    ws = dbg.alloc_workspace(shape_of(inp), select_of(w))
    res_dbg = run_step(inp, ws=ws)
    assert _status(ws) == 0
    check_step(inp, res_dbg).assert_ok()
    rel = dbg._bind(ctypes.CDLL(os.path.join(os.path.dirname(DBG), "libdelta_attn.so")))
    lib_dbg, dbg._lib = dbg._lib, rel
    try:
        res_rel = run_step(inp)
    finally:
        dbg._lib = lib_dbg
    for a, b in zip(res_dbg.outs, res_rel.outs):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(res_dbg.sel_idx, res_rel.sel_idx)


def test_page_table_entry_past_the_cache_is_flagged(dbg):
    w, inp = _tiny([1024])
    n = inp.n_phys_pages
    # 8 more pages than the descriptor states, so that the bad entry stays inside the buffer
    k = torch.cat([inp.k_cache[0], inp.k_cache[0][:8]])
    v = torch.cat([inp.v_cache[0], inp.v_cache[0][:8]])
    pt = inp.page_table.clone()
    pt[0, 5] = n + 3
    kv = dbg.delta_kv_t(k.data_ptr(), v.data_ptr(), pt.data_ptr(), inp.seq_lens.data_ptr(), n)
    shape = shape_of(inp)
    ws = dbg.alloc_workspace(shape)
    out = torch.empty_like(inp.q[0])
    dbg.delta_full_attn(shape, kv, inp.q[0], out, ws)
    st = _status(ws)
    log(f"status {st:#x}")
    assert st & dbg.DELTA_DEBUG_PAGE
    assert torch.isfinite(out.float()).all()


def test_sequence_longer_than_the_bound_is_flagged(dbg):
    w, inp = _tiny([1024])
    shape = shape_of(inp)
    seq = torch.tensor([1030], dtype=torch.int32, device="cuda")   # max_seq_len is 1024
    kv = dbg.make_kv(inp.k_cache[0], inp.v_cache[0], inp.page_table, seq)
    ws = dbg.alloc_workspace(shape)
    out = torch.empty_like(inp.q[0])
    dbg.delta_full_attn(shape, kv, inp.q[0], out, ws)
    assert _status(ws) & dbg.DELTA_DEBUG_SEQ_LEN


def test_selected_unit_past_the_sequence_is_flagged(dbg):
    w, inp = _tiny([700])                       # 44 pages in a 64-page page-table row
    shape, sel = shape_of(inp), select_of(w)
    ws = dbg.alloc_workspace(shape, sel)
    kv = dbg.make_kv(inp.k_cache[2], inp.v_cache[2], inp.page_table, inp.seq_lens)
    idx = torch.tensor([[0, 5, 10, 20, 30, 43, 50, 40]], dtype=torch.int32, device="cuda")
    cnt = torch.tensor([8], dtype=torch.int32, device="cuda")
    out = torch.empty_like(inp.q[2])
    dbg.delta_sparse_attn(shape, kv, inp.q[2], out, sel, idx, cnt, ws)
    assert _status(ws) & dbg.DELTA_DEBUG_SELECTION
    # a valid selection leaves the word alone
    dbg.delta_workspace_init(ws)
    idx[0, 6] = 41
    dbg.delta_sparse_attn(shape, kv, inp.q[2], out, sel, idx, cnt, ws)
    assert _status(ws) == 0
