"""GPU tests of the decode-step integration: the KV append (Eq. kv_update) against the oracle's
append, bit for bit, and a whole step through delta_decode_step_hooked whose per-layer hooks
produce the layer's query and append its key and value before the attention reads them,
eagerly and captured in a HIP graph that is replayed on new inputs.
"""
import numpy as np
import pytest
import torch

from gpu_helpers import D, check_step, log, shape_of, select_of
from oracle import delta_oracle as O
from paper_2510_09883_amd import configs, synth

pytestmark = pytest.mark.gpu


def _inputs(lens, n_layers=1, shuffled=True, roles=None):
    w = configs.get(4)
    w.batch = len(lens)
    w.n_layers = n_layers
    w.shuffled_pages = shuffled
    if roles is not None:
        w.roles = roles
    inp = synth.make_inputs(w, "cuda", seq_lens=lens)
    torch.cuda.synchronize()
    return w, inp


def _rand_bf16(shape, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randn(shape, generator=g, device="cuda").to(torch.bfloat16)


def _oracle_append(cache_bits, pt, lens, new_bits):
    out = cache_bits
    for b, s in enumerate(lens):
        if 1 <= s <= 16 * pt.shape[1]:
            out = O.append_token(out, pt[b], s, new_bits[b])
    return out


def test_kv_append_bit_exact():
    lens = [1, 16, 17, 1000, 4096]
    w, inp = _inputs(lens)
    d = D()
    shape = shape_of(inp)
    k_new = _rand_bf16((w.batch, w.n_kv_heads, w.head_dim), 11)
    v_new = _rand_bf16((w.batch, w.n_kv_heads, w.head_dim), 12)
    pt = inp.page_table.cpu().numpy()
    k0, v0 = synth.bits(inp.k_cache[0]), synth.bits(inp.v_cache[0])
    d.delta_kv_append(shape, inp.k_cache[0], inp.v_cache[0], inp.page_table, inp.seq_lens, k_new, v_new)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(synth.bits(inp.k_cache[0]), _oracle_append(k0, pt, lens, synth.bits(k_new)))
    np.testing.assert_array_equal(synth.bits(inp.v_cache[0]), _oracle_append(v0, pt, lens, synth.bits(v_new)))
    # sequences without a slot for the token (length 0, or past the page table) are skipped
    lens_bad = torch.tensor([0, 16 * inp.max_pages_per_seq + 1, 17, 0, 5], dtype=torch.int32, device="cuda")
    k1, v1 = synth.bits(inp.k_cache[0]), synth.bits(inp.v_cache[0])
    d.delta_kv_append(shape, inp.k_cache[0], inp.v_cache[0], inp.page_table, lens_bad, v_new, k_new)
    torch.cuda.synchronize()
    want_lens = lens_bad.cpu().tolist()
    np.testing.assert_array_equal(synth.bits(inp.k_cache[0]), _oracle_append(k1, pt, want_lens, synth.bits(v_new)))
    np.testing.assert_array_equal(synth.bits(inp.v_cache[0]), _oracle_append(v1, pt, want_lens, synth.bits(k_new)))


class _Model:
    """Stand-in for the rest of the decoder layer: before each layer's attention the hook
    'projects' (copies) this step's query into the layer's q buffer and appends this step's
    key and value to the layer's cache; after it, the hook copies the attention output
    onward (so an ordering mistake shows up as a stale copy)."""

    def __init__(self, d, w, inp, shape):
        self.d, self.w, self.inp, self.shape = d, w, inp, shape
        n = w.n_layers
        self.q_src = [torch.empty_like(inp.q[i]) for i in range(n)]
        self.k_src = [torch.empty((w.batch, w.n_kv_heads, w.head_dim), dtype=torch.bfloat16, device="cuda")
                      for _ in range(n)]
        self.v_src = [torch.empty_like(k) for k in self.k_src]
        self.after = [torch.empty_like(inp.q[i]) for i in range(n)]
        self.calls = []

    def new_step(self, seed):
        for i in range(self.w.n_layers):
            self.q_src[i].copy_(_rand_bf16(self.q_src[i].shape, seed + 3 * i))
            self.k_src[i].copy_(_rand_bf16(self.k_src[i].shape, seed + 3 * i + 1))
            self.v_src[i].copy_(_rand_bf16(self.v_src[i].shape, seed + 3 * i + 2))

    def poison_new_rows(self):
        """The token's row holds NaN until the append: attention before it would be NaN."""
        nan_k = torch.full_like(self.k_src[0], float("nan"))
        for i in range(self.w.n_layers):
            self.d.delta_kv_append(self.shape, self.inp.k_cache[i], self.inp.v_cache[i],
                                   self.inp.page_table, self.inp.seq_lens, nan_k, nan_k)

    def before(self, i):
        self.calls.append(("before", i))
        self.inp.q[i].copy_(self.q_src[i])
        self.d.delta_kv_append(self.shape, self.inp.k_cache[i], self.inp.v_cache[i],
                               self.inp.page_table, self.inp.seq_lens, self.k_src[i], self.v_src[i])

    def after_attn(self, outs):
        def f(i):
            self.calls.append(("after", i))
            self.after[i].copy_(outs[i])
        return f


def test_hooked_step_appends_before_attention_and_replays_in_graph():
    roles = [configs.ROLE_FULL, configs.ROLE_DELTA, configs.ROLE_SPARSE, configs.ROLE_SPARSE]
    lens = [2500, 1200, 17]
    w, inp = _inputs(lens, n_layers=4, roles=roles)
    d = D()
    shape, sel = shape_of(inp), select_of(w)
    ws = d.alloc_workspace(shape, sel)
    outs = [torch.full_like(q, float("nan")) for q in inp.q]
    K = w.budget_units
    sel_idx = torch.full((2, w.batch, K), -7, dtype=torch.int32, device="cuda")
    sel_cnt = torch.full((2, w.batch), -7, dtype=torch.int32, device="cuda")
    kvs = [d.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens) for i in range(4)]
    args = d.StepArgs(shape, roles, kvs, inp.q, outs, sel, sel_idx, sel_cnt, ws)
    m = _Model(d, w, inp, shape)
    hooks = d.LayerHooks(before=m.before, after=m.after_attn(outs))
    pt = inp.page_table.cpu().numpy()

    def verify(tag):
        torch.cuda.synchronize()
        res = type("R", (), {})()
        res.outs, res.sel_idx, res.sel_cnt = outs, sel_idx, sel_cnt
        check_step(inp, res, roles=roles, use_page_table=True).assert_ok()
        for i in range(4):
            assert torch.equal(m.after[i].view(torch.int16), outs[i].view(torch.int16)), (tag, i)
        log(f"{tag}: hooked step ok")

    def expected_caches():
        return [(_oracle_append(kb, pt, lens, synth.bits(m.k_src[i])),
                 _oracle_append(vb, pt, lens, synth.bits(m.v_src[i])))
                for i, (kb, vb) in enumerate(pre)]

    # eager
    m.new_step(100)
    m.poison_new_rows()
    torch.cuda.synchronize()
    pre = [(synth.bits(inp.k_cache[i]), synth.bits(inp.v_cache[i])) for i in range(4)]
    d.delta_decode_step_hooked(args, hooks)
    assert m.calls == [(h, i) for i in range(4) for h in ("before", "after")]
    torch.cuda.synchronize()
    for i, (kb, vb) in enumerate(expected_caches()):
        np.testing.assert_array_equal(synth.bits(inp.k_cache[i]), kb)
        np.testing.assert_array_equal(synth.bits(inp.v_cache[i]), vb)
    verify("eager")

    # captured once (the hooks run during capture), replayed on new steps' inputs
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    m.calls.clear()
    with torch.cuda.graph(g, stream=s):
        d.delta_decode_step_hooked(args, hooks)
    assert len(m.calls) == 8
    for rep in range(2):
        m.new_step(200 + 50 * rep)
        m.poison_new_rows()
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        pre = [(synth.bits(inp.k_cache[i]), synth.bits(inp.v_cache[i])) for i in range(4)]
        g.replay()
        torch.cuda.synchronize()
        for i, (kb, vb) in enumerate(expected_caches()):
            np.testing.assert_array_equal(synth.bits(inp.k_cache[i]), kb)
        verify(f"graph replay {rep}")
    assert len(m.calls) == 8   # replays run no host code


def test_hook_error_stops_step():
    roles = [configs.ROLE_FULL, configs.ROLE_FULL]
    w, inp = _inputs([300, 40], n_layers=2, roles=roles)
    d = D()
    shape = shape_of(inp)
    ws = d.alloc_workspace(shape)
    outs = [torch.full_like(q, float("nan")) for q in inp.q]
    kvs = [d.make_kv(inp.k_cache[i], inp.v_cache[i], inp.page_table, inp.seq_lens) for i in range(2)]
    args = d.StepArgs(shape, roles, kvs, inp.q, outs, None, None, None, ws)

    def before(i):
        if i == 1:
            raise ValueError("projection failed")

    with pytest.raises(ValueError, match="projection failed"):
        d.delta_decode_step_hooked(args, d.LayerHooks(before=before))
    torch.cuda.synchronize()
    assert not torch.isnan(outs[0].float()).any()       # layer 0 ran
    assert torch.isnan(outs[1].float()).all()           # layer 1 did not
