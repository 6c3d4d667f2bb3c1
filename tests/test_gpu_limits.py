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
