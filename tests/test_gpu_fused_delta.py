"""GPU parity of the fused Delta-layer kernel (attention, scoring and selection in one
launch, logits kept in LDS) against the CPU oracle.

The fused kernel runs wherever it fits with DELTA_PATH_FUSED (DELTA_PATH_AUTO takes it only
where its grid fills the device, e.g. 8 sequences of 32K tokens).  Here it runs on
short, ragged and multi-chunk sequences of the Qwen-7B shape, with both aggregations and both
unit sizes, and is compared with the oracle and with the split path.  Its fallback (a
workgroup whose sequence barrier times out leaves its chunk to the sequence's last workgroup)
is forced from the host with a zero wait and must give the same bits.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import ROLE_DELTA, D, Report, check_step, log, oracle_kv, run_step, select_of, shape_of
from oracle import accept as A
from oracle import delta_oracle as O
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu

LAYER = 2   # the first Delta layer of the Qwen-7B schedule


def _qwen(U, lens, layers=(LAYER,)):
    w = configs.get(4, U)
    w.batch = len(lens)
    inp = synth.make_inputs(w, "cuda", seq_lens=lens, layers=list(layers))
    torch.cuda.synchronize()
    return inp


FUSED, SPLIT = 2, 1   # DELTA_PATH_FUSED, DELTA_PATH_SPLIT


def _delta_call(inp, agg, layer=LAYER, ws=None, scores=None, path=FUSED):
    d = D()
    w = inp.workload
    shape, sel = shape_of(inp), select_of(w, agg, path=path)
    assert d.delta_delta_path(shape, sel) == (path == FUSED)
    ws = d.alloc_workspace(shape, sel) if ws is None else ws
    kv = d.make_kv(inp.k_cache[layer], inp.v_cache[layer], inp.page_table, inp.seq_lens)
    out = torch.full_like(inp.q[layer], float("nan"))
    K = w.budget_units
    sel_idx = torch.full((w.batch, K), -7, dtype=torch.int32, device="cuda")
    sel_cnt = torch.full((w.batch,), -7, dtype=torch.int32, device="cuda")
    phys = torch.full((w.batch, K), -7, dtype=torch.int32, device="cuda")
    d.delta_delta_attn_select(shape, kv, inp.q[layer], out, sel, sel_idx, sel_cnt, scores, ws,
                              sel_phys=phys)
    torch.cuda.synchronize()
    return out, sel_idx, sel_cnt, phys, ws


def _check(inp, agg, out, sel_idx, sel_cnt, phys, layer=LAYER):
    w = inp.workload
    U = w.unit_tokens
    rep = Report()
    scale = O.default_scale(w.head_dim)
    pt = inp.page_table.cpu().numpy()
    for b in range(w.batch):
        q, K, V = oracle_kv(inp, layer, b)
        o, alpha = O.full_attention(q, K, V, scale)
        rep.out(f"seq {b}", out[b].float().cpu().numpy().astype(np.float64), o)
        rho, S = O.refresh_units(alpha, U, w.budget_units, w.recent_units, agg)
        cnt = int(sel_cnt[b])
        dev = sel_idx[b].cpu().numpy()
        assert cnt == min(w.budget_units, len(S)) and np.all(dev[cnt:] == -1), f"seq {b}: count"
        rep.sel(f"seq {b}", A.check_selection(S, w.budget_units, w.recent_units, dev[:cnt], rho))
        # physical locations through the page table
        ph = phys[b].cpu().numpy()
        want = pt[b, dev[:cnt]] if U == 16 else pt[b, dev[:cnt] // 16] * 16 + dev[:cnt] % 16
        np.testing.assert_array_equal(ph[:cnt], want)
        assert np.all(ph[cnt:] == -1)
    rep.assert_ok()


@pytest.mark.parametrize("agg", [0, 1])
@pytest.mark.parametrize("U", [16, 1])
def test_fused_delta_layer_matches_oracle(U, agg):
    # 3 chunks of 64 pages, 1 chunk, and a one-page sequence; with single tokens as units the
    # candidates stay within the fused kernel's 2048
    lens = [2100, 1000, 17] if U == 1 else [3000, 1000, 17]
    inp = _qwen(U, lens)
    n_u = (max(lens) + U - 1) // U
    sc_f = torch.full((len(lens), n_u), -1.0, device="cuda")
    sc_s = torch.full((len(lens), n_u), -1.0, device="cuda")
    out, idx, cnt, phys, _ = _delta_call(inp, agg, scores=sc_f)
    _check(inp, agg, out, idx, cnt, phys)
    out_s, idx_s, cnt_s, phys_s, _ = _delta_call(inp, agg, scores=sc_s, path=SPLIT)
    _check(inp, agg, out_s, idx_s, cnt_s, phys_s)
    # both paths give the same scores up to the rounding of their different summation orders,
    # and the fused kernel did run (its scores and outputs are not the split path's bits)
    for b, s_b in enumerate(lens):
        m = (s_b + U - 1) // U
        np.testing.assert_allclose(sc_f[b, :m].cpu().numpy(), sc_s[b, :m].cpu().numpy(), rtol=1e-5)
    assert not (torch.equal(sc_f, sc_s) and torch.equal(out.view(torch.int16), out_s.view(torch.int16)))


def test_fused_delta_repeat_rearm_and_determinism():
    """Consecutive fused calls on one workspace (the in-kernel counters re-arm themselves) with
    different inputs each match the oracle; repeating a call gives identical bits."""
    inp = _qwen(16, [4096, 2048, 700], layers=(2, 14))
    r2 = _delta_call(inp, 0, layer=2)
    r14 = _delta_call(inp, 0, layer=14, ws=r2[4])
    r2b = _delta_call(inp, 0, layer=2, ws=r2[4])
    _check(inp, 0, *r2[:4], layer=2)
    _check(inp, 0, *r14[:4], layer=14)
    assert torch.equal(r2[0].view(torch.int16), r2b[0].view(torch.int16))
    assert torch.equal(r2[1], r2b[1]) and torch.equal(r2[2], r2b[2])


def test_fused_delta_in_decode_step():
    """A step [full, Delta, sparse, sparse] through delta_decode_step with the fused Delta
    kernel: the sparse layers read its selection and physical pages."""
    lens = [2500, 1200]
    w = configs.get(4)
    w.batch = len(lens)
    roles = [configs.ROLE_FULL, ROLE_DELTA, configs.ROLE_SPARSE, configs.ROLE_SPARSE]
    inp = synth.make_inputs(w, "cuda", seq_lens=lens, layers=[0, 1, 2, 3])
    res = run_step(inp, roles=roles, path=FUSED)
    check_step(inp, res, roles=roles, layers=[0, 1, 2, 3]).assert_ok()
    log("fused Delta step ok")


@pytest.mark.parametrize("U", [16, 1])
def test_fused_barrier_fallback_gives_the_same_bits(monkeypatch, U):
    """With no wait at the sequence barrier every workgroup but the last to arrive leaves its
    chunk (logits to the workspace); the last one merges, scores and selects for all of them.
    Outputs, scores and selections equal the normal fused run bit for bit, and the oracle."""
    lens = [2100, 1000, 17] if U == 1 else [4000, 1000, 17]
    inp = _qwen(U, lens)
    n_u = (max(lens) + U - 1) // U
    sc_a = torch.full((len(lens), n_u), -1.0, device="cuda")
    out_a, idx_a, cnt_a, phys_a, ws = _delta_call(inp, 0, scores=sc_a)
    monkeypatch.setenv("DELTA_FUSED_SPIN_TICKS", "0")
    sc_b = torch.full((len(lens), n_u), -1.0, device="cuda")
    out_b, idx_b, cnt_b, phys_b, _ = _delta_call(inp, 0, scores=sc_b, ws=ws)
    _check(inp, 0, out_b, idx_b, cnt_b, phys_b)
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    assert torch.equal(sc_a, sc_b)
    assert torch.equal(idx_a, idx_b) and torch.equal(cnt_a, cnt_b) and torch.equal(phys_a, phys_b)
    # the workspace is re-armed: a normal call after the fallback gives the same bits again
    monkeypatch.delenv("DELTA_FUSED_SPIN_TICKS")
    sc_c = torch.full((len(lens), n_u), -1.0, device="cuda")
    out_c, idx_c, _, _, _ = _delta_call(inp, 0, scores=sc_c, ws=ws)
    assert torch.equal(out_a.view(torch.int16), out_c.view(torch.int16)) and torch.equal(sc_a, sc_c)
    assert torch.equal(idx_a, idx_c)


@pytest.mark.parametrize("cfg,fused", [(4, True), (2, False), (3, False), (5, False), (1, False)])
def test_auto_path_takes_the_fused_kernel_where_its_grid_fills_the_device(cfg, fused):
    """DELTA_PATH_AUTO: 8 sequences of 32K tokens with 28/4 heads give 8 x 32 = 256 fused
    workgroups, one per CU, resident at once: fused.  One 8K sequence (8 workgroups) would leave
    the device idle, and 16 or 32 sequences of 32K (512, 1024 workgroups) do not fit at once:
    split."""
    d = D()
    w = configs.get(cfg)
    shape = d.make_shape(w.batch, w.n_q_heads, w.n_kv_heads, w.head_dim,
                         (w.max_seq_len + 15) // 16, w.max_seq_len)
    assert d.delta_delta_path(shape, select_of(w)) is fused
    assert d.delta_delta_path(shape, select_of(w, path=SPLIT)) is False
