"""The allocation-free decode step (delta_decode_step_noalloc) against delta_decode_step with a
caller-owned workspace: the same kernels on the library's scratch array, so every output,
selected index and count must be the same bits.  Two calls in a row share the scratch, the
second with a smaller input (fewer sequences, shorter contexts, another layout of the scratch),
then the first shape again."""
import pytest
import torch

from gpu_helpers import (ROLE_DELTA, ROLE_FULL, ROLE_SPARSE, D, StepResult, check_step, log,
                         select_of, shape_of)
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu

ROLES = [ROLE_FULL, ROLE_DELTA, ROLE_SPARSE, ROLE_SPARSE]


def _inputs(lens, cfg_id):
    w = configs.get(2)
    w.batch, w.cfg_id, w.n_layers = len(lens), cfg_id, len(ROLES)
    w.roles = list(ROLES)
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    return w, inp


def _args(d, w, inp, ws):
    outs = [torch.full_like(inp.q[i], float("nan")) for i in range(len(ROLES))]
    sel_idx = torch.full((1, w.batch, w.budget_units), -7, dtype=torch.int32, device="cuda")
    sel_cnt = torch.full((1, w.batch), -7, dtype=torch.int32, device="cuda")
    kvs = [d.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens)
           for i in range(len(ROLES))]
    return d.StepArgs(shape_of(inp), ROLES, kvs, inp.q, outs, select_of(w), sel_idx, sel_cnt, ws)


def _result(args):
    return StepResult(args._keep[1], args.sel_idx, args.sel_cnt)


def _same(a, b):
    for x, y in zip(a.outs, b.outs):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert torch.equal(a.sel_idx, b.sel_idx) and torch.equal(a.sel_cnt, b.sel_cnt)


def test_noalloc_step_matches_workspace_step():
    d = D()
    big = _inputs([8192, 5000, 7777], 21)
    small = _inputs([3001], 22)
    log("allocation-free steps: 3 x (8192, 5000, 7777) tokens, then 1 x 3001, then the first again")
    runs = []
    for w, inp in (big, small, big):
        runs.append((w, inp, _args(d, w, inp, None)))
    for _, _, a in runs[:2]:
        d.delta_decode_step_noalloc(a)          # two calls in a row, no synchronisation between
    torch.cuda.synchronize()
    d.delta_decode_step_noalloc(runs[2][2])
    torch.cuda.synchronize()
    for w, inp, a in runs:
        ref = _args(d, w, inp, d.alloc_workspace(shape_of(inp), select_of(w)))
        d.delta_decode_step(ref)
        torch.cuda.synchronize()
        _same(_result(a), _result(ref))
        # and the step is the method's: the oracle's outputs and selections
        check_step(inp, _result(a), roles=ROLES).assert_ok()
    log("allocation-free steps match the workspace steps bit for bit")


def test_noalloc_rejects_oversize_before_launch():
    d = D()
    shape = d.make_shape(64, 32, 8, 128, 2048, 32768)
    sel = d.make_select(2048, 128)
    assert d.delta_workspace_bytes(shape, sel) > d.DELTA_NOALLOC_SCRATCH_BYTES
    import ctypes
    roles = (ctypes.c_int32 * 1)(1)
    kv = d.delta_kv_t(1, 2, 3, 4)
    kvs = (d.delta_kv_t * 1)(kv)
    ptrs = (ctypes.c_void_p * 1)(0x1000)
    fake = ctypes.c_void_p(0x1000)
    rc = d._lib.delta_decode_step_noalloc(ctypes.byref(shape), 1, roles, kvs, ptrs, ptrs,
                                          ctypes.byref(sel), fake, fake, None)
    assert rc == d.DELTA_ERR_WORKSPACE
