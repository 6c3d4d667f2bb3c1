"""CPU tests of the acceptance rule (with ties and near-ties made on purpose) and of the
seeded input generator."""
import numpy as np
import pytest
import torch

from oracle import accept as A
from oracle import delta_oracle as O
from paper_2510_09883_amd import configs, synth


# ------------------------------------------------------------------------------------------
# acceptance rule
# ------------------------------------------------------------------------------------------
def test_selection_exact_match_accepted():
    S = np.array([0.5, 0.1, 0.9, 0.3, 0.7, 0.2])
    rho = O.select_units(S, 4, 1)
    v = A.check_selection(S, 4, 1, rho, rho)
    assert v.ok and v.exact and v.band_resolved == 0


def test_selection_near_tie_inside_band_accepted():
    # units 1 and 2 differ by 1e-7 relative: either may be taken for the last slot
    S = np.array([0.9, 0.5, 0.5 * (1 + 1e-7), 0.1, 0.2])
    orc = O.select_units(S, 3, 1)                 # {0, 2, 4}
    alt = np.array([0, 1, 4])
    v = A.check_selection(S, 3, 1, alt, orc)
    assert orc.tolist() == [0, 2, 4]
    assert v.ok and not v.exact and v.band_resolved == 1


def test_selection_outside_band_rejected():
    S = np.array([0.9, 0.5, 0.5 * (1 + 1e-3), 0.1, 0.2])
    orc = O.select_units(S, 3, 1)
    v = A.check_selection(S, 3, 1, np.array([0, 1, 4]), orc)
    assert not v.ok


def test_selection_structural_failures():
    S = np.arange(10, dtype=np.float64)
    orc = O.select_units(S, 4, 2)
    assert not A.check_selection(S, 4, 2, orc[:-1], orc).ok              # wrong size
    assert not A.check_selection(S, 4, 2, orc[::-1], orc).ok             # not ascending
    assert not A.check_selection(S, 4, 2, np.array([5, 6, 7, 8]), orc).ok  # recency unit 9 missing
    assert not A.check_selection(S[:3], 4, 2, np.array([0, 1]), np.arange(3)).ok


def test_output_rule():
    o = np.array([1.0, -2.0, 0.0])
    assert A.check_output(o + np.array([0.02, -0.03, 0.019]), o)[0]
    assert not A.check_output(o + np.array([0.0, 0.0, 0.021]), o)[0]
    assert not A.check_output(np.array([np.nan, -2.0, 0.0]), o)[0]


# ------------------------------------------------------------------------------------------
# generator
# ------------------------------------------------------------------------------------------
def test_workload_table():
    w = configs.get(1)
    assert (w.budget_units, w.recent_units, w.group) == (8, 1, 4)
    for cid, K, L, n in ((2, 128, 8, 32), (3, 256, 8, 32), (4, 128, 8, 28), (5, 128, 8, 32)):
        w = configs.get(cid)
        assert (w.budget_units, w.recent_units, len(w.roles), w.n_layers) == (K, L, n, n)
        d = [i for i, r in enumerate(w.roles) if r == configs.ROLE_DELTA]
        assert d == ([2, 16] if cid != 4 else [2, 14])
    w = configs.get(2, unit_tokens=1)
    assert (w.budget_units, w.recent_units) == (2048, 128)
    lens = synth.seq_lens_for(configs.get(5))
    assert len(lens) == 32 and min(lens) >= 16384 and max(lens) <= 32768
    # the runtime settings: K = 64 pages, L = 8 pages, the paper's Delta-layer sets
    for cid, n, heads, d_set in ((6, 28, (12, 2), [2, 14, 23]), (7, 28, (14, 2), [2, 14, 22]),
                                 (8, 48, (10, 2), [2, 6, 42])):
        w = configs.get(cid)
        assert (w.budget_units, w.recent_units, w.n_layers, len(w.roles)) == (64, 8, n, n)
        assert (w.n_q_heads, w.n_kv_heads, w.head_dim) == (*heads, 128)
        assert w.delta_layers == d_set
        assert w.roles[:2] == [configs.ROLE_FULL] * 2
        assert all(r == configs.ROLE_SPARSE for i, r in enumerate(w.roles) if i > 2 and i not in d_set)


def test_delta_layer_schedules():
    r = configs.roles_for(8, [5, 2, 2])
    F, D_, S = configs.ROLE_FULL, configs.ROLE_DELTA, configs.ROLE_SPARSE
    assert r == [F, F, D_, S, S, D_, S, S]
    assert configs.roles_for(32, configs.PAPER_DELTA_LAYERS["ds-llama-8b"]).count(D_) == 3
    for bad in ([], [-1], [8]):
        with pytest.raises(ValueError):
            configs.roles_for(8, bad)
    # the Delta-layer count sweep: the first at layer 2, evenly spread, up to every layer
    assert configs.spread_delta_layers(28, 1) == [2]
    assert configs.spread_delta_layers(28, 2) == [2, 27]
    assert configs.spread_delta_layers(28, 26) == list(range(2, 28))
    for c in range(1, 27):
        d = configs.spread_delta_layers(28, c)
        assert len(d) == c and d[0] == 2 and d == sorted(set(d)) and d[-1] <= 27
    with pytest.raises(ValueError):
        configs.spread_delta_layers(28, 27)
    w = configs.get(3)
    w.set_delta_layers(configs.PAPER_DELTA_LAYERS["ds-llama-8b"])
    assert w.delta_layers == [2, 8, 31]


def test_generator_deterministic_and_shaped():
    w = configs.get(1)
    a = synth.make_inputs(w, "cpu")
    b = synth.make_inputs(w, "cpu")
    for i in range(w.n_layers):
        assert torch.equal(a.k_cache[i].view(torch.int16), b.k_cache[i].view(torch.int16))
        assert torch.equal(a.q[i], b.q[i])
    assert a.k_cache[0].shape == (64, 2, 16, 64) and a.q[0].shape == (1, 8, 64)
    assert a.page_table.dtype == torch.int32 and a.seq_lens.tolist() == [1024]
    # heavy hitters: position 0 plus 16 others, keys scaled by 4
    hh = synth.heavy_hitters(w, 0, 1024)
    assert hh[0] == 0 and len(hh) == 17 and len(set(hh.tolist())) == 17


def test_generator_ragged_shuffled_and_poisoned_tail():
    w = configs.get(1)
    w.shuffled_pages = True
    inp = synth.make_inputs(w, "cpu", seq_lens=[37], layers=[0])
    pt = inp.page_table[0, :3].tolist()
    assert sorted(pt) == [0, 1, 2]
    last = inp.k_cache[0][pt[2]]                      # [Hkv, 16, d]; rows 5.. are past s = 37
    assert torch.isnan(last[:, 5:].float()).all() and not torch.isnan(last[:, :5].float()).any()
