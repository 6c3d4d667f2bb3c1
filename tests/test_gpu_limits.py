"""GPU parity at the limits of the path: the longest contexts the selection supports (8192
candidate units per sequence, with pages and with single tokens), every selection width the
selection kernel is built for, and the group sizes not covered by the workload shapes."""
import pytest
import torch

from gpu_helpers import check_step, log, run_step
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu


def _tiny(lens, U=16, budget=None, recent_pages=None, **shape):
    w = configs.get(1, U)
    w.batch = len(lens)
    for k, v in shape.items():
        setattr(w, k, v)
    if budget is not None:
        w.budget_tokens = budget
    if recent_pages is not None:
        w.recent_pages = recent_pages
    w.seq_len = max(lens)
    log(f"generating {w.describe()} lens {lens}")
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    return w, inp


def test_longest_page_contexts():
    """131072 tokens = 8192 pages, 8184 candidates (32 keys per selecting thread), beside a
    sequence one token into its last page and one with 16 keys per thread."""
    w, inp = _tiny([131072, 65537, 50000], budget=2048, recent_pages=8)
    res = run_step(inp)
    rep = check_step(inp, res, use_page_table=False)
    rep.assert_ok()
    assert res.sel_cnt[0].tolist() == [128, 128, 128]


def test_longest_token_context():
    """Single-token units: 8192 candidates older than the window (the most one workgroup holds)."""
    w, inp = _tiny([8208, 3000], U=1, budget=256, recent_pages=1)
    assert w.recent_units == 16
    res = run_step(inp)
    check_step(inp, res, use_page_table=False).assert_ok()


@pytest.mark.parametrize("hq,hkv,d", [(4, 2, 64), (10, 2, 128), (5, 1, 64), (12, 2, 64), (24, 4, 128)])
def test_remaining_group_sizes(hq, hkv, d):
    w, inp = _tiny([900, 2000], n_q_heads=hq, n_kv_heads=hkv, head_dim=d)
    res = run_step(inp)
    check_step(inp, res).assert_ok()


def test_workspace_moves_between_shapes_after_init():
    """One workspace, sized for the larger call, serves calls of two different shapes (batch,
    context and budget) after delta_workspace_init, as the runtime sweeps use it."""
    from gpu_helpers import D, shape_of, select_of
    d = D()
    w1, inp1 = _tiny([3000, 900, 17])
    w2, inp2 = _tiny([5000, 2000], budget=256, recent_pages=2, n_q_heads=16, n_kv_heads=4,
                     head_dim=128)
    big = max(d.delta_workspace_bytes(shape_of(i), select_of(w)) for i, w in ((inp1, w1), (inp2, w2)))
    ws = torch.zeros(big, dtype=torch.uint8, device="cuda")
    for rnd in range(2):
        for w, inp in ((w1, inp1), (w2, inp2)):
            d.delta_workspace_init(ws)
            res = run_step(inp, ws=ws, budget=w.budget_tokens, recent=w.recent_tokens)
            check_step(inp, res, budget=w.budget_tokens, recent=w.recent_tokens).assert_ok()
    log("workspace reuse across shapes ok")


def test_large_batch_of_short_ragged_sequences():
    """512 sequences of 1..600 tokens (one to 38 pages, most shorter than the 8-page budget
    or just above it): many small (sequence, KV head) pairs and selection workgroups."""
    g = torch.Generator().manual_seed(512)
    lens = torch.randint(1, 601, (512,), generator=g).tolist()
    w, inp = _tiny(lens)
    res = run_step(inp)
    check_step(inp, res, seqs=list(range(0, 512, 7)) + [511]).assert_ok()
    cnt = res.sel_cnt[0].cpu().tolist()
    assert cnt == [min(w.budget_units, (s + 15) // 16) for s in lens]
