"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names what it pins: a library routine computing the same quantity by another code
path, a closed form, an invariant the paper's definitions imply, brute force on tiny inputs,
or a hand-worked example from tests/golden (each cited to the paper).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import delta_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "selection_examples.json")


def _rng(seed):
    return np.random.default_rng(seed)


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 with torch (a library routine) and return the bits."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _paged(tokens_bits: np.ndarray, perm: np.ndarray, page=16):
    """Scatter logical tokens [s, g, d] (bits) into physical pages [n_phys, g, P, d] with
    logical page j at physical page perm[j] -- done here with plain indexing, independently of
    the oracle's gather."""
    s, g, d = tokens_bits.shape
    n_pages = (s + page - 1) // page
    n_phys = int(perm.max()) + 1
    cache = np.full((n_phys, g, page, d), 0x7FC0, dtype=np.uint16)   # NaN everywhere unused
    for t in range(s):
        cache[perm[t // page], :, t % page, :] = tokens_bits[t]
    return cache, n_pages


# ------------------------------------------------------------------------------------------
# O1: bf16 decoding
# ------------------------------------------------------------------------------------------
def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0001, 0x7F7F, 0x8000], dtype=np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 2.0 ** -133, (2 - 2.0 ** -7) * 2.0 ** 127, -0.0]
    got = O.bf16_bits_to_f64(bits)
    assert got.tolist() == want


def test_bf16_decode_matches_torch():
    x = _rng(0).standard_normal(4096) * 10
    b = _bf16_bits(x)
    ref = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.bf16_bits_to_f64(b), ref)


# ------------------------------------------------------------------------------------------
# O2: paged gather
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("s", [1, 15, 16, 17, 100])
def test_gather_inverts_independent_scatter(s):
    rng = _rng(s)
    g, d = 3, 8
    tok = _bf16_bits(rng.standard_normal((s, g, d)))
    n_pages = (s + 15) // 16
    perm = rng.permutation(n_pages + 5)[:n_pages]
    cache, _ = _paged(tok, perm)
    got = O.gather_tokens(cache, perm, s)
    assert np.array_equal(got, O.bf16_bits_to_f64(tok))


@pytest.mark.parametrize("s", [1, 16, 17, 33, 100])
def test_append_is_concatenation(s):
    """Eq. kv_update: after the append, the sequence's s tokens are its first s - 1 cached
    tokens followed by the new token, and no other cache entry changes."""
    rng = _rng(1000 + s)
    g, d = 2, 8
    tok = _bf16_bits(rng.standard_normal((s, g, d)))
    n_pages = (s + 15) // 16
    perm = rng.permutation(n_pages + 3)[:n_pages]
    cache, _ = _paged(tok, perm)
    new = _bf16_bits(rng.standard_normal((g, d)))
    got = O.append_token(cache, perm, s, new)
    full = O.gather_tokens(got, perm, s)
    assert np.array_equal(full[:s - 1], O.bf16_bits_to_f64(tok[:s - 1]))
    assert np.array_equal(full[s - 1], O.bf16_bits_to_f64(new))
    changed = np.argwhere(np.any(got != cache, axis=-1))
    t = s - 1
    assert all(tuple(c) in {(perm[t // 16], h, t % 16) for h in range(g)} for c in changed)
    assert got is not cache


# ------------------------------------------------------------------------------------------
# O3-O5: attention
# ------------------------------------------------------------------------------------------
def _sdpa(q, K, V, scale, mask=None):
    """torch scaled_dot_product_attention in float64 on CPU, KV heads expanded with
    repeat_interleave (head j reads group j // G), as a library reference."""
    m, g = q.shape[0], K.shape[1]
    G = m // g
    qt = torch.from_numpy(q)[:, None, :]                                # [m, 1, d]
    kt = torch.from_numpy(K).permute(1, 0, 2).repeat_interleave(G, 0)   # [m, s, d]
    vt = torch.from_numpy(V).permute(1, 0, 2).repeat_interleave(G, 0)
    am = None if mask is None else torch.from_numpy(mask)[None, None, :].expand(m, 1, -1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=am, scale=scale)
    return o[:, 0, :].numpy()


@pytest.mark.parametrize("m,g,d,s", [(8, 2, 64, 37), (4, 4, 16, 5), (6, 1, 32, 64), (7, 1, 8, 200)])
def test_attention_matches_torch_sdpa(m, g, d, s):
    rng = _rng(m * 1000 + s)
    q, K, V = rng.standard_normal((m, d)), rng.standard_normal((s, g, d)), rng.standard_normal((s, g, d))
    scale = O.default_scale(d)
    o, alpha = O.full_attention(q, K, V, scale)
    assert np.allclose(o, _sdpa(q, K, V, 1 / math.sqrt(d)), atol=1e-12, rtol=1e-12)
    assert np.allclose(alpha.sum(axis=1), 1.0, atol=1e-12)


def test_attention_single_token_is_value():
    rng = _rng(1)
    q, K, V = rng.standard_normal((4, 8)), rng.standard_normal((1, 2, 8)), rng.standard_normal((1, 2, 8))
    o, alpha = O.full_attention(q, K, V, 0.3)
    assert np.array_equal(alpha, np.ones((4, 1)))
    for j in range(4):
        assert np.allclose(o[j], V[0, j // 2], atol=1e-15)


def test_attention_equal_keys_is_mean_of_values():
    rng = _rng(2)
    k = rng.standard_normal(16)
    K = np.tile(k, (9, 2, 1))
    V = rng.standard_normal((9, 2, 16))
    o, _ = O.full_attention(rng.standard_normal((4, 16)), K, V, 0.25)
    for j in range(4):
        assert np.allclose(o[j], V[:, j // 2].mean(axis=0), atol=1e-13)


def test_attention_two_tokens_logistic():
    # two tokens: alpha_0 = 1 / (1 + exp(a_1 - a_0)) with a_t = q.k_t / sqrt(d)
    q = np.array([[1.0, 0.0, 2.0, -1.0]])
    K = np.array([[[0.5, 1.0, 0.0, 0.0]], [[0.0, 0.0, 1.0, 1.0]]])
    V = np.array([[[1.0, 2.0, 3.0, 4.0]], [[-1.0, 0.0, 1.0, 0.5]]])
    a0, a1 = 0.5 / 2.0, 1.0 / 2.0
    p0 = 1.0 / (1.0 + math.exp(a1 - a0))
    o, alpha = O.full_attention(q, K, V, 0.5)
    assert abs(alpha[0, 0] - p0) < 1e-15
    assert np.allclose(o[0], p0 * V[0, 0] + (1 - p0) * V[1, 0], atol=1e-15)


def test_gqa_head_to_group_map():
    # constant V per group: head j must return the constant of group floor(j / G)
    m, g, d, s = 12, 3, 4, 10
    rng = _rng(3)
    K = rng.standard_normal((s, g, d))
    V = np.zeros((s, g, d))
    for c in range(g):
        V[:, c, :] = 10.0 * (c + 1)
    o, _ = O.full_attention(rng.standard_normal((m, d)), K, V, 0.5)
    for j in range(m):
        assert np.allclose(o[j], 10.0 * (j // (m // g) + 1))


def test_attention_brute_force_loops():
    rng = _rng(4)
    m, g, d, s = 4, 2, 5, 11
    q, K, V = rng.standard_normal((m, d)), rng.standard_normal((s, g, d)), rng.standard_normal((s, g, d))
    o, _ = O.full_attention(q, K, V, 0.7)
    for j in range(m):
        c = j // 2
        a = [0.7 * sum(q[j][i] * K[t][c][i] for i in range(d)) for t in range(s)]
        w = [math.exp(x) for x in a]
        z = sum(w)
        for i in range(d):
            assert abs(o[j][i] - sum(w[t] / z * V[t][c][i] for t in range(s))) < 1e-12


# ------------------------------------------------------------------------------------------
# O6-O7: scores
# ------------------------------------------------------------------------------------------
def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


@pytest.mark.parametrize("case", _golden()["token_scores"])
def test_token_scores_golden(case):
    agg = O.AGG_MAX if case["agg"] == "max" else O.AGG_SUM
    assert np.allclose(O.token_scores(np.array(case["alpha"]), agg), case["expected"], atol=1e-15)


@pytest.mark.parametrize("case", _golden()["unit_scores"])
def test_unit_scores_golden(case):
    got = O.unit_scores(np.array(case["s_tok"], dtype=np.float64), case["unit_tokens"])
    assert np.allclose(got, case["expected"], atol=1e-15)


def test_scores_invariants():
    rng = _rng(5)
    m, s = 6, 53
    a = rng.standard_normal((m, s)) * 3
    alpha = O.softmax_per_head(a)
    # single head: token score is that head's weight
    assert np.array_equal(O.token_scores(alpha[:1], O.AGG_MAX), alpha[0])
    # sum aggregation: page scores add up to the number of heads (each head sums to 1)
    for U in (1, 4, 16):
        assert abs(O.unit_scores(O.token_scores(alpha, O.AGG_SUM), U).sum() - m) < 1e-12
        st = O.token_scores(alpha, O.AGG_MAX)
        S = O.unit_scores(st, U)
        assert abs(S.sum() - st.sum()) < 1e-12           # unit sums conserve mass
        assert 1 - 1e-12 <= S.sum() <= m + 1e-12
        assert len(S) == (s + U - 1) // U
    st = O.token_scores(alpha, O.AGG_MAX)
    assert np.array_equal(O.unit_scores(st, 1), st)
    # identical heads: max over heads equals any one head
    same = np.tile(alpha[2], (m, 1))
    assert np.array_equal(O.token_scores(same, O.AGG_MAX), alpha[2])


# ------------------------------------------------------------------------------------------
# O8: selection
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("case", _golden()["selection"])
def test_selection_golden(case):
    got = O.select_units(np.array(case["S"], dtype=np.float64), case["K"], case["L"])
    assert got.tolist() == case["expected"]


def _brute_select(S, K, L):
    n = len(S)
    if n <= K:
        return list(range(n))
    n_c = n - L
    best, best_sum = None, -1.0
    for comb in itertools.combinations(range(n_c), K - L):   # lexicographic order
        tot = sum(S[i] for i in comb)
        if tot > best_sum:
            best, best_sum = comb, tot
    return sorted(list(best) + list(range(n_c, n)))


@pytest.mark.parametrize("seed", range(40))
def test_selection_brute_force(seed):
    rng = _rng(100 + seed)
    n = int(rng.integers(1, 13))
    K = int(rng.integers(1, 9))
    L = int(rng.integers(0, K))
    # small integers force many exact ties; sums of integers are exact in float64
    S = rng.integers(0, 4, n).astype(np.float64)
    assert O.select_units(S, K, L).tolist() == _brute_select(S.tolist(), K, L)


def test_selection_invariants_and_nesting():
    rng = _rng(6)
    for _ in range(50):
        n = int(rng.integers(1, 200))
        S = np.round(rng.random(n), 2)
        L = int(rng.integers(0, 10))
        prev = None
        for K in range(L + 1, L + 40):
            r = O.select_units(S, K, L)
            assert len(r) == min(K, n)
            assert np.all(np.diff(r) > 0)
            if n > K:
                assert set(range(n - L, n)) <= set(r.tolist())
            if prev is not None:
                assert set(prev.tolist()) <= set(r.tolist())
            prev = r


def test_recency_window_in_units_brute_force():
    """Alg. 1 keeps ceil(L / P) pages for a window of L tokens.  Pinned by brute force: for a
    context of whole units, the units the window keeps are exactly the units that hold any of
    the last l tokens (a floor or a rounding would drop the unit of the window's oldest
    tokens, or keep a unit too many)."""
    for U in (1, 4, 16):
        for n_u in (1, 2, 3, 9):
            s = n_u * U
            for l in range(0, s + 1):
                touched = {t // U for t in range(s - l, s)}
                L_u = O.recent_units_of(l, U)
                assert set(range(n_u - L_u, n_u)) == touched, (U, n_u, l)
    assert O.recent_units_of(0, 16) == 0 and O.recent_units_of(8, 16) == 1
    with pytest.raises(ValueError):
        O.recent_units_of(-1, 16)


def test_token_level_topk_of_raw_logits():
    # one head, U = 1, L = 0: softmax is monotone, so rho is the top-k of the raw logits
    rng = _rng(7)
    s, d, k = 300, 16, 37
    q, K = rng.standard_normal((1, d)), rng.standard_normal((s, 1, d))
    V = rng.standard_normal((s, 1, d))
    _, alpha = O.full_attention(q, K, V, 0.25)
    rho, _ = O.refresh_units(alpha, 1, k, 0)
    raw = K[:, 0, :] @ q[0]
    assert rho.tolist() == sorted(np.argsort(-raw)[:k].tolist())


# ------------------------------------------------------------------------------------------
# O9: sparse attention
# ------------------------------------------------------------------------------------------
def test_sparse_all_units_is_full():
    rng = _rng(8)
    m, g, d, s = 8, 2, 16, 75
    q, K, V = rng.standard_normal((m, d)), rng.standard_normal((s, g, d)), rng.standard_normal((s, g, d))
    o_full, alpha = O.full_attention(q, K, V, 0.25)
    for U in (1, 16):
        allu = np.arange((s + U - 1) // U)
        assert np.allclose(O.sparse_attention(q, K, V, allu, U, 0.25), o_full, atol=1e-12)
        T = O.tokens_of_units(allu, U, s)
        assert np.array_equal(T, np.arange(s))
        assert abs(O.attention_recall(alpha[0], T) - 1.0) < 1e-12


@pytest.mark.parametrize("U", [1, 16])
def test_sparse_matches_masked_sdpa(U):
    rng = _rng(9 + U)
    m, g, d, s = 8, 2, 32, 150
    q, K, V = rng.standard_normal((m, d)), rng.standard_normal((s, g, d)), rng.standard_normal((s, g, d))
    n_u = (s + U - 1) // U
    units = np.sort(rng.permutation(n_u)[: max(1, n_u // 3)])
    units = np.union1d(units, [n_u - 1])            # include the partial last unit
    mask = np.zeros(s, dtype=bool)
    for u in units:
        mask[u * U:min(u * U + U, s)] = True
    o = O.sparse_attention(q, K, V, units, U, 1 / math.sqrt(d))
    assert np.allclose(o, _sdpa(q, K, V, 1 / math.sqrt(d), mask), atol=1e-12)


# ------------------------------------------------------------------------------------------
# O10: one decoding step over the layer stack (Alg. 1)
# ------------------------------------------------------------------------------------------
def test_decode_step_roles():
    rng = _rng(10)
    m, g, d, s, U = 8, 2, 16, 200, 16
    n_layers = 6
    qs = [rng.standard_normal((m, d)) for _ in range(n_layers)]
    Ks = [rng.standard_normal((s, g, d)) * 2 for _ in range(n_layers)]
    Vs = [rng.standard_normal((s, g, d)) for _ in range(n_layers)]
    roles = [O.ROLE_SPARSE, O.ROLE_FULL, O.ROLE_DELTA, O.ROLE_SPARSE, O.ROLE_DELTA, O.ROLE_SPARSE]
    sc = 1 / math.sqrt(d)
    outs, sels = O.decode_step_sequence(roles, qs, Ks, Vs, sc, U, 5, 1)
    full = [O.full_attention(qs[i], Ks[i], Vs[i], sc)[0] for i in range(n_layers)]
    # a sparse layer before any Delta layer attends to every page (Alg. 1 initialises rho to all)
    assert np.allclose(outs[0], full[0], atol=1e-12)
    # Delta layers compute full attention
    assert np.allclose(outs[2], full[2], atol=1e-15) and np.allclose(outs[4], full[4], atol=1e-15)
    assert [i for i, _, _ in sels] == [2, 4]
    # each sparse layer uses the most recent refresh: check against masked SDPA
    for layer, src in ((3, 0), (5, 1)):
        rho = sels[src][1]
        assert len(rho) == 5
        mask = np.zeros(s, dtype=bool)
        for u in rho:
            mask[u * U:min(u * U + U, s)] = True
        assert np.allclose(outs[layer], _sdpa(qs[layer], Ks[layer], Vs[layer], sc, mask), atol=1e-12)
    # all-full roles reproduce the full stack
    outs_f, sels_f = O.decode_step_sequence([O.ROLE_FULL] * n_layers, qs, Ks, Vs, sc, U, 5, 1)
    assert not sels_f and all(np.allclose(a, b, atol=1e-15) for a, b in zip(outs_f, full))


def test_page_table_permutation_invariance():
    rng = _rng(11)
    s, g, d, m = 90, 2, 8, 4
    tokK = _bf16_bits(rng.standard_normal((s, g, d)))
    tokV = _bf16_bits(rng.standard_normal((s, g, d)))
    q = O.bf16_bits_to_f64(_bf16_bits(rng.standard_normal((m, d))))
    n_pages = (s + 15) // 16
    res = []
    for perm in (np.arange(n_pages), rng.permutation(n_pages)):
        kc, _ = _paged(tokK, perm)
        vc, _ = _paged(tokV, perm)
        K, V = O.gather_tokens(kc, perm, s), O.gather_tokens(vc, perm, s)
        o, alpha = O.full_attention(q, K, V, 0.3)
        rho, S = O.refresh_units(alpha, 16, 3, 1)
        res.append((o, rho, S))
    assert np.array_equal(res[0][0], res[1][0])
    assert np.array_equal(res[0][1], res[1][1]) and np.array_equal(res[0][2], res[1][2])
