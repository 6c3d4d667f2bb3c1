"""CPU oracle for the DELTA decode-step attention hot path (arXiv 2510.09883).

TEST INFRASTRUCTURE. This module is the slow, plain, obviously-correct statement of what the
hot path computes, written in NumPy float64. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it. It shares no code, header, table or helper with
the HIP library, and the library never calls it.

Every function cites the passage of the paper it follows. Where the paper is silent or
ambiguous the reading taken is stated in the docstring (and in the design doc's list of readings).

Notation (paper, Sec. 2 and Sec. 4):
  m  query heads, g KV groups, G = m / g query heads per group, d head dimension,
  s  sequence length of the decoding sequence (the current token included),
  P  KV page size (16), U selection-unit size in tokens (16 = page-based DELTA, 1 = token-level),
  k / K budget (tokens / units), l / L recency window (tokens / units).

Indices are 0-based here; the paper counts from 1 (Sec. 2 "Sparse attention", Sec. 4).
"""
from __future__ import annotations

import numpy as np

AGG_MAX = 0  # token score = max over heads (Sec. 4 "Selection mechanism"; App. A, Alg. 2)
AGG_SUM = 1  # token score = sum over heads (alternative aggregation, kept as a flag)

ROLE_FULL = 0
ROLE_DELTA = 1
ROLE_SPARSE = 2


# --------------------------------------------------------------------------------------------
# Inputs
# --------------------------------------------------------------------------------------------
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """Decode bfloat16 bit patterns (uint16/int16 array) to float64, exactly.

    A bfloat16 value is the top half of an IEEE float32, so shifting the 16 bits into the high
    half of a 32-bit word and reinterpreting gives the exact float32, which widens exactly.
    """
    u = np.asarray(bits).view(np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def gather_tokens(cache_bits: np.ndarray, page_table_row: np.ndarray, seq_len: int,
                  page_size: int = 16) -> np.ndarray:
    """Gather one sequence's K (or V) rows from a paged cache, in logical token order.

    Sec. 4 "Page-based DELTA": the cache is stored in pages of P tokens and p(t) maps token t
    to its page. Logical page j of the sequence lives at physical page page_table_row[j];
    token t sits at row t mod P of physical page page_table_row[t // P].

    cache_bits: bf16 bits, [n_phys_pages, g, P, d].  Returns float64 [s, g, d].
    """
    n_pages = (seq_len + page_size - 1) // page_size
    assert n_pages <= len(page_table_row)
    out = np.empty((seq_len, cache_bits.shape[1], cache_bits.shape[3]), dtype=np.float64)
    for j in range(n_pages):
        phys = int(page_table_row[j])
        rows = min(page_size, seq_len - j * page_size)
        # physical page tile is [g, P, d]; logical rows j*P .. j*P+rows-1 are its first rows
        out[j * page_size:j * page_size + rows] = \
            bf16_bits_to_f64(cache_bits[phys, :, :rows, :]).transpose(1, 0, 2)
    return out


def append_token(cache_bits: np.ndarray, page_table_row: np.ndarray, seq_len: int,
                 new_bits: np.ndarray, page_size: int = 16) -> np.ndarray:
    """The KV update of one decoding step for one sequence (Sec. 2, Eq. kv_update): the cache
    grows by the new token's row, so that attention at this step sees s = seq_len tokens, the
    last one being the new token.  In the paged layout (Sec. 4 "Page-based DELTA") token
    s - 1 is row (s - 1) mod P of physical page page_table_row[(s - 1) // P].

    cache_bits: bf16 bits [n_phys_pages, g, P, d]; new_bits: bf16 bits [g, d].  Returns a
    new array equal to cache_bits except for that row of every KV head.
    """
    t = seq_len - 1
    out = np.array(cache_bits, copy=True)
    out[int(page_table_row[t // page_size]), :, t % page_size, :] = new_bits
    return out


# --------------------------------------------------------------------------------------------
# Attention (Sec. 2, Eq. gqa_attention)
# --------------------------------------------------------------------------------------------
def kv_group_of_head(j: int, n_q_heads: int, n_kv_heads: int) -> int:
    """phi(j): the KV group read by query head j (Sec. 2, GQA).

    The paper only says every query head is assigned one group. Reading: contiguous groups,
    phi(j) = floor(j / G) with G = m / g (MHA when g = m, MQA when g = 1).
    """
    group = n_q_heads // n_kv_heads
    return j // group


def default_scale(head_dim: int) -> float:
    """The 1/sqrt(d_head) factor of Eq. gqa_attention."""
    return 1.0 / np.sqrt(float(head_dim))


def attention_logits(q: np.ndarray, K: np.ndarray, scale: float) -> np.ndarray:
    """A_j = Q_j K_phi(j)^T / sqrt(d) for one decoding query (Eq. gqa_attention).

    q: [m, d] float64, K: [s, g, d] float64.  Returns a: [m, s] float64.
    """
    m = q.shape[0]
    g = K.shape[1]
    a = np.empty((m, K.shape[0]), dtype=np.float64)
    for j in range(m):
        kj = K[:, kv_group_of_head(j, m, g), :]          # [s, d]
        a[j] = scale * (kj @ q[j])
    return a


def softmax_per_head(a: np.ndarray) -> np.ndarray:
    """alpha_j = softmax(A_j), each head separately (Sec. 2 "Sparse attention").

    Written as exp(a - max) / sum(exp(a - max)); subtracting the row maximum does not change
    the result mathematically and keeps exp finite.
    """
    alpha = np.empty_like(a)
    for j in range(a.shape[0]):
        e = np.exp(a[j] - a[j].max())
        alpha[j] = e / e.sum()
    return alpha


def attention_output(alpha: np.ndarray, V: np.ndarray) -> np.ndarray:
    """O_j = softmax(A_j) V_phi(j) (Eq. gqa_attention).  alpha [m, s], V [s, g, d] -> [m, d]."""
    m = alpha.shape[0]
    g = V.shape[1]
    o = np.empty((m, V.shape[2]), dtype=np.float64)
    for j in range(m):
        o[j] = alpha[j] @ V[:, kv_group_of_head(j, m, g), :]
    return o


def full_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float):
    """Full decode attention over all s cached tokens (Eq. gqa_attention; App. A, Alg. 1).

    The decoding query sees every cached token, the current one included (Sec. 2, Eq.
    kv_update appends before attending), so no mask is applied.
    Returns (o [m, d], alpha [m, s]).
    """
    a = attention_logits(q, K, scale)
    alpha = softmax_per_head(a)
    return attention_output(alpha, V), alpha


# --------------------------------------------------------------------------------------------
# Scoring and selection (Sec. 4; App. A, Alg. 2)
# --------------------------------------------------------------------------------------------
def token_scores(alpha: np.ndarray, agg: int = AGG_MAX) -> np.ndarray:
    """s_t = max over all m query heads of alpha_j(t) (Sec. 4 "Selection mechanism"; Alg. 2).

    AGG_SUM replaces the max with a sum over heads (an alternative aggregation).
    """
    if agg == AGG_MAX:
        return alpha.max(axis=0)
    if agg == AGG_SUM:
        return alpha.sum(axis=0)
    raise ValueError("agg must be AGG_MAX or AGG_SUM")


def unit_scores(s_tok: np.ndarray, unit_tokens: int) -> np.ndarray:
    """S_u = sum of s_t over the tokens of unit u (Sec. 4 "Page-based DELTA"; Alg. 2).

    Units are pages of U tokens in logical order; the last unit may be partial and sums only
    the tokens that exist (reading of the paper, which is silent on a partial last page).
    U = 1 gives S_t = s_t, the token-level rule.
    """
    s = len(s_tok)
    n_units = (s + unit_tokens - 1) // unit_tokens
    S = np.zeros(n_units, dtype=np.float64)
    for u in range(n_units):
        S[u] = s_tok[u * unit_tokens:min((u + 1) * unit_tokens, s)].sum()
    return S


def recent_units_of(recent_tokens: int, unit_tokens: int) -> int:
    """The recency window in units: App. A, Alg. 1 keeps the last ceil(L / P) pages for a
    window of L tokens, so any token count is a valid window; with units of U tokens it is the
    last ceil(l / U) units."""
    if recent_tokens < 0 or unit_tokens < 1:
        raise ValueError("need l >= 0 and U >= 1")
    return -(-recent_tokens // unit_tokens)


def select_units(S: np.ndarray, budget_units: int, recent_units: int) -> np.ndarray:
    """rho = last L units  U  top-(K - L) of the older units by S (Sec. 4; Alg. 2).

    Readings where the paper is silent:
      * while the context fits the budget (n_units <= K) every unit is kept;
      * equal scores are ordered by lower unit index first (a full stable sort on
        (score descending, index ascending));
      * the result is returned as ascending, unique unit indices.
    """
    n = len(S)
    if not (0 <= recent_units < budget_units):
        raise ValueError("need 0 <= L < K")
    if n <= budget_units:
        return np.arange(n, dtype=np.int64)
    n_cand = n - recent_units
    need = budget_units - recent_units
    cand_idx = np.arange(n_cand)
    order = np.lexsort((cand_idx, -S[:n_cand]))   # last key is primary: score desc, then index
    chosen = order[:need]
    return np.sort(np.concatenate([chosen, np.arange(n_cand, n)])).astype(np.int64)


def refresh_units(alpha: np.ndarray, unit_tokens: int, budget_units: int, recent_units: int,
                  agg: int = AGG_MAX):
    """RefreshPages of App. A, Alg. 2: head aggregation -> unit sums -> recency + top-k.

    Returns (rho, S): the selected units and the unit scores they were chosen by.
    """
    s_tok = token_scores(alpha, agg)
    S = unit_scores(s_tok, unit_tokens)
    return select_units(S, budget_units, recent_units), S


def tokens_of_units(units: np.ndarray, unit_tokens: int, seq_len: int) -> np.ndarray:
    """T(rho): the token positions covered by the selected units, clipped at s (Sec. 4)."""
    toks = [t for u in units for t in range(u * unit_tokens, min((u + 1) * unit_tokens, seq_len))]
    return np.asarray(toks, dtype=np.int64)


def sparse_attention(q: np.ndarray, K: np.ndarray, V: np.ndarray, units: np.ndarray,
                     unit_tokens: int, scale: float) -> np.ndarray:
    """Sparse decode attention over the selected units only (App. A, Alg. 1, sparse branch).

    Eq. gqa_attention evaluated on the sub-cache K[T(rho)], V[T(rho)]: the softmax is
    renormalised over the selected tokens.  Returns o [m, d].
    """
    T = tokens_of_units(units, unit_tokens, K.shape[0])
    o, _ = full_attention(q, K[T], V[T], scale)
    return o


# --------------------------------------------------------------------------------------------
# One decoding step over the layer stack (App. A, Alg. 1)
# --------------------------------------------------------------------------------------------
def decode_step_sequence(roles, qs, Ks, Vs, scale: float, unit_tokens: int, budget_units: int,
                         recent_units: int, agg: int = AGG_MAX):
    """App. A, Alg. 1 for ONE sequence: rho <- all units, then per-layer role dispatch.

    roles: per-layer ROLE_FULL / ROLE_DELTA / ROLE_SPARSE.  qs[i]: [m, d]; Ks[i], Vs[i]:
    [s, g, d] float64 (already gathered).  A Delta layer runs full attention and refreshes
    rho; a sparse layer attends to the most recent rho (all units before the first refresh).

    Returns (outs, selections): outs[i] is [m, d]; selections is a list of (layer, rho, S) for
    each Delta layer in order.
    """
    s = Ks[0].shape[0]
    n_units = (s + unit_tokens - 1) // unit_tokens
    rho = np.arange(n_units, dtype=np.int64)
    outs, selections = [], []
    for i, role in enumerate(roles):
        if role == ROLE_FULL:
            o, _ = full_attention(qs[i], Ks[i], Vs[i], scale)
        elif role == ROLE_DELTA:
            o, alpha = full_attention(qs[i], Ks[i], Vs[i], scale)
            rho, S = refresh_units(alpha, unit_tokens, budget_units, recent_units, agg)
            selections.append((i, rho, S))
        elif role == ROLE_SPARSE:
            o = sparse_attention(qs[i], Ks[i], Vs[i], rho, unit_tokens, scale)
        else:
            raise ValueError(f"unknown role {role}")
        outs.append(o)
    return outs, selections


def attention_recall(alpha_j: np.ndarray, tokens: np.ndarray) -> float:
    """R_j = sum_{u in rho} alpha_j(u) / sum_u alpha_j(u) (Sec. 2, Eq. recall); diagnostic."""
    return float(alpha_j[tokens].sum() / alpha_j.sum())
