"""The five decode-step workloads measured and parity-tested for the DELTA hot path.

Shapes follow the model families the paper evaluates (Sec. 5: a 32-layer Llama-8B-class model
and a 28-layer Qwen-7B-class model; Sec. 5.1 names the layer ranges).  Budgets are given in
tokens and converted to whole pages of P = 16 tokens, the page size used in all of the
paper's experiments (Sec. 5 "Implementation details").  The recency window is
min(8, K_pages / 8) pages: the paper's L = 8 pages for the larger budgets (Sec. 5.2), scaled
down for the 8-page budget of the tiny check so that selection is not trivial.

This module holds no arithmetic of the method; it only describes inputs.
"""
from __future__ import annotations

from dataclasses import dataclass, field

ROLE_FULL = 0
ROLE_DELTA = 1
ROLE_SPARSE = 2

PAGE = 16


def llama_roles():
    """32 layers: 0-1 full, Delta-layers at 2 and 16, the rest sparse."""
    return [ROLE_FULL, ROLE_FULL, ROLE_DELTA] + [ROLE_SPARSE] * 13 + [ROLE_DELTA] + [ROLE_SPARSE] * 15


def qwen_roles():
    """28 layers: 0-1 full, Delta-layers at 2 and 14, the rest sparse."""
    return [ROLE_FULL, ROLE_FULL, ROLE_DELTA] + [ROLE_SPARSE] * 11 + [ROLE_DELTA] + [ROLE_SPARSE] * 13


@dataclass
class Workload:
    cfg_id: int
    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    batch: int
    seq_len: int                  # all sequences, unless seq_len_range is set
    budget_tokens: int
    hh_count: int = 0             # fixed number of heavy hitters (besides position 0)
    hh_frac: float = 0.0          # or a fraction of the sequence length
    hh_factor: float = 4.0        # key scaling of heavy-hitter tokens
    seq_len_range: tuple | None = None   # (lo, hi) inclusive, uniform per sequence
    shuffled_pages: bool = False
    roles: list = field(default_factory=list)
    unit_tokens: int = PAGE

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads

    @property
    def budget_units(self):
        return self.budget_tokens // self.unit_tokens

    @property
    def recent_tokens(self):
        k_pages = self.budget_tokens // PAGE
        return PAGE * min(8, k_pages // 8)

    @property
    def recent_units(self):
        return self.recent_tokens // self.unit_tokens

    @property
    def max_seq_len(self):
        return self.seq_len_range[1] if self.seq_len_range else self.seq_len

    def describe(self):
        return (f"cfg{self.cfg_id} {self.name}: {self.n_layers} layers, Hq/Hkv/d="
                f"{self.n_q_heads}/{self.n_kv_heads}/{self.head_dim}, B={self.batch}, "
                f"s={'U%s' % (self.seq_len_range,) if self.seq_len_range else self.seq_len}, "
                f"K={self.budget_tokens} tok, L={self.recent_tokens} tok, U={self.unit_tokens}")


def get(cfg_id: int, unit_tokens: int = PAGE) -> Workload:
    if cfg_id == 1:
        w = Workload(1, "tiny-check", 3, 8, 2, 64, 1, 1024, 128, hh_count=16, hh_factor=4.0,
                     roles=[ROLE_FULL, ROLE_DELTA, ROLE_SPARSE])
    elif cfg_id == 2:
        w = Workload(2, "llama8b-b1-8k", 32, 32, 8, 128, 1, 8192, 2048, hh_frac=0.02,
                     hh_factor=4.0, roles=llama_roles())
    elif cfg_id == 3:
        w = Workload(3, "llama8b-b16-32k", 32, 32, 8, 128, 16, 32768, 4096, hh_frac=0.02,
                     hh_factor=4.0, roles=llama_roles())
    elif cfg_id == 4:
        w = Workload(4, "qwen7b-b8-32k", 28, 28, 4, 128, 8, 32768, 2048, hh_frac=0.01,
                     hh_factor=6.0, roles=qwen_roles())
    elif cfg_id == 5:
        w = Workload(5, "llama8b-b32-ragged16k-32k", 32, 32, 8, 128, 32, 32768, 2048,
                     hh_frac=0.02, hh_factor=4.0, seq_len_range=(16384, 32768),
                     shuffled_pages=True, roles=llama_roles())
    else:
        raise ValueError(f"unknown workload {cfg_id}")
    w.unit_tokens = unit_tokens
    return w
