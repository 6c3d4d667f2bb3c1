"""The decode-step workloads measured and parity-tested for the DELTA hot path.

Workloads 1-5 follow the model families the paper evaluates (Sec. 5: a 32-layer
Llama-8B-class model and a 28-layer Qwen-7B-class model; Sec. 5.1 names the layer ranges).
Budgets are given in tokens and converted to whole pages of P = 16 tokens, the page size used
in all of the paper's experiments (Sec. 5 "Implementation details").  The recency window is
min(8, K_pages / 8) pages unless set explicitly: the paper's L = 8 pages for the larger
budgets (Sec. 5.2), scaled down for the 8-page budget of the tiny check so that selection is
not trivial.

Workloads 6-8 are the runtime settings of the paper's throughput and Delta-layer-count
experiments (Sec. 5.3 and Sec. 6.1): a 1k-token budget (K = 64 pages, L = 8 pages), the
model-specific Delta-layer sets of Sec. 5, and the batch and maximum decoding length quoted
for each model.  The paper runs the 7B and 14B models with tensor parallelism over 2 and 4
GPUs; those workloads hold one GPU's share of the attention heads (the KV heads split evenly
over the ranks, each with its group of query heads).  The head counts are those of the
published Qwen2.5 architectures the distilled models are built on (1.5B: 12 query / 2 KV
heads; 7B: 28 / 4; 14B: 40 / 8; head dim 128); the paper itself does not list them.

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


def roles_for(n_layers: int, delta_layers) -> list:
    """Layer roles for a set of Delta-layers (Sec. 4, Alg. 1): full attention before the first
    one, sparse attention after it except at the Delta-layers themselves."""
    d = sorted(set(int(i) for i in delta_layers))
    if not d or d[0] < 0 or d[-1] >= n_layers:
        raise ValueError(f"Delta-layers {delta_layers} outside [0, {n_layers})")
    return [ROLE_FULL if i < d[0] else ROLE_DELTA if i in d else ROLE_SPARSE
            for i in range(n_layers)]


def spread_delta_layers(n_layers: int, count: int, first: int = 2) -> list:
    """`count` Delta-layers for a sweep over their number (Sec. 6.1): the first at layer
    `first`, the others evenly spaced over the layers after it, up to every layer from
    `first` on."""
    span = n_layers - 1 - first
    if not 1 <= count <= span + 1:
        raise ValueError(f"{count} Delta-layers do not fit layers {first}..{n_layers - 1}")
    if count == 1:
        return [first]
    return sorted({first + round(i * span / (count - 1)) for i in range(count)})


# Delta-layer sets the paper uses per model (Sec. 5 "Model-specific Delta-layers")
PAPER_DELTA_LAYERS = {
    "ds-qwen-1.5b": [2, 14, 23],
    "ds-qwen-7b": [2, 14, 22],
    "ds-qwen-14b": [2, 6, 42],
    "ds-llama-8b": [2, 8, 31],
}


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
    recent_pages: int | None = None   # recency window L in pages; None: min(8, K_pages / 8)

    @property
    def group(self):
        return self.n_q_heads // self.n_kv_heads

    @property
    def budget_units(self):
        return self.budget_tokens // self.unit_tokens

    @property
    def recent_tokens(self):
        if self.recent_pages is not None:
            return PAGE * self.recent_pages
        k_pages = self.budget_tokens // PAGE
        return PAGE * min(8, k_pages // 8)

    @property
    def delta_layers(self):
        return [i for i, r in enumerate(self.roles) if r == ROLE_DELTA]

    def set_delta_layers(self, delta_layers):
        self.roles = roles_for(self.n_layers, delta_layers)

    @property
    def recent_units(self):
        return self.recent_tokens // self.unit_tokens

    @property
    def max_seq_len(self):
        return self.seq_len_range[1] if self.seq_len_range else self.seq_len

    def describe(self):
        return (f"{self.name}: {self.n_layers} layers, Hq/Hkv/d="
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
    elif cfg_id == 6:
        w = Workload(6, "qwen1.5b-b64-18k", 28, 12, 2, 128, 64, 18432, 1024, hh_frac=0.02,
                     hh_factor=4.0, recent_pages=8,
                     roles=roles_for(28, PAPER_DELTA_LAYERS["ds-qwen-1.5b"]))
    elif cfg_id == 7:
        w = Workload(7, "qwen7b-tp2share-b64-16k", 28, 14, 2, 128, 64, 16384, 1024,
                     hh_frac=0.02, hh_factor=4.0, recent_pages=8,
                     roles=roles_for(28, PAPER_DELTA_LAYERS["ds-qwen-7b"]))
    elif cfg_id == 8:
        w = Workload(8, "qwen14b-tp4share-b32-19k", 48, 10, 2, 128, 32, 19456, 1024,
                     hh_frac=0.02, hh_factor=4.0, recent_pages=8,
                     roles=roles_for(48, PAPER_DELTA_LAYERS["ds-qwen-14b"]))
    else:
        raise ValueError(f"unknown workload {cfg_id}")
    w.unit_tokens = unit_tokens
    return w
