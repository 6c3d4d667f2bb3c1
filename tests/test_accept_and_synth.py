"""CPU tests of the acceptance rule (with ties and near-ties made on purpose) and of the
seeded input generator."""
import numpy as np
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
