"""Seeded synthetic decode-step inputs shaped like the paper's workloads.

Used by BOTH the HIP path (tests, benchmark) and the oracle (tests): it holds none of the
method's arithmetic, only the input recipe.

Recipe, per workload and sequence b:
  1. heavy-hitter positions H_b = {0} U a sample without replacement from [1, s_b)
     (seed 1000*cfg + b, on a CPU generator so the positions do not depend on the device);
     the paper observes that a few tokens carry most attention mass (Sec. 2 "Sparsity and query
     dependence") and that salient tokens persist across layers (Sec. 3), so H_b is shared by
     every layer and KV head of the sequence;
  2. per layer, K and V ~ N(0, 1) in float32, the K rows of H_b scaled by hh_factor, then
     rounded to bfloat16 (round-to-nearest-even);
  3. per layer, q ~ N(0, 1) [Hq, d] rounded to bfloat16;
  4. each tensor has its own seed ((cfg*1009 + layer)*1013 + b)*4 + kind, on a generator that
     lives on the target device (Philox on the GPU), so a workload is reproducible per device;
  5. pages of 16 tokens; sequence b's logical page j sits at physical page page_table[b, j]
     (contiguous per sequence, or one global random permutation with seed 7919*cfg);
  6. optionally the rows past s_b inside the last page are filled with NaN, so any read of them
     that is not masked shows up in the outputs.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from .configs import PAGE, Workload

KIND_K, KIND_V, KIND_Q = 0, 1, 2
_BF16_NAN = torch.tensor(float("nan"), dtype=torch.bfloat16)


def tensor_seed(cfg_id: int, layer: int, b: int, kind: int) -> int:
    return ((cfg_id * 1009 + layer) * 1013 + b) * 4 + kind


def seq_lens_for(w: Workload) -> list:
    if w.seq_len_range is None:
        return [w.seq_len] * w.batch
    lo, hi = w.seq_len_range
    g = torch.Generator().manual_seed(5000)
    return torch.randint(lo, hi + 1, (w.batch,), generator=g).tolist()


def heavy_hitters(w: Workload, b: int, s_b: int) -> torch.Tensor:
    n = w.hh_count if w.hh_count else int(round(w.hh_frac * s_b))
    n = min(n, s_b - 1)
    g = torch.Generator().manual_seed(1000 * w.cfg_id + b)
    rest = torch.randperm(s_b - 1, generator=g)[:n] + 1
    return torch.cat([torch.zeros(1, dtype=torch.long), rest.sort().values])


@dataclass
class DecodeInputs:
    """One decoding step's inputs, resident on `device`.

    k_cache[i], v_cache[i]: bf16 [n_phys_pages, Hkv, 16, d] for layer i
    q[i]:                  bf16 [B, Hq, d]
    page_table:            int32 [B, max_pages_per_seq]; unused entries are 0
    seq_lens:              int32 [B] (device) and seq_lens_host (python list)
    """
    workload: Workload
    k_cache: list
    v_cache: list
    q: list
    page_table: torch.Tensor
    seq_lens: torch.Tensor
    seq_lens_host: list
    max_pages_per_seq: int
    n_phys_pages: int

    @property
    def max_seq_len(self):
        return max(self.seq_lens_host)


def make_page_table(w: Workload, seq_lens: list, device) -> tuple:
    n_pages = [(s + PAGE - 1) // PAGE for s in seq_lens]
    max_pages = (w.max_seq_len + PAGE - 1) // PAGE
    total = sum(n_pages)
    if w.shuffled_pages:
        g = torch.Generator().manual_seed(7919 * w.cfg_id)
        phys = torch.randperm(total, generator=g)
    else:
        phys = torch.arange(total)
    pt = torch.zeros((w.batch, max_pages), dtype=torch.int32)
    off = 0
    for b, n in enumerate(n_pages):
        pt[b, :n] = phys[off:off + n].to(torch.int32)
        off += n
    return pt.to(device), total, max_pages


def make_inputs(w: Workload, device="cpu", layers=None, poison_tail: bool = True,
                seq_lens: list | None = None) -> DecodeInputs:
    """Build the synthetic step inputs of workload `w` on `device`.

    layers: optional subset of layer indices to materialise (others are None); seq_lens
    overrides the workload's lengths (edge-case tests).
    """
    device = torch.device(device)
    lens = list(seq_lens) if seq_lens is not None else seq_lens_for(w)
    pt, n_phys, max_pages = make_page_table(w, lens, device)
    pt_host = pt.cpu()
    layers = range(w.n_layers) if layers is None else layers
    Hkv, Hq, d = w.n_kv_heads, w.n_q_heads, w.head_dim
    hh = [heavy_hitters(w, b, s) for b, s in enumerate(lens)]
    k_cache = [None] * w.n_layers
    v_cache = [None] * w.n_layers
    qs = [None] * w.n_layers
    for i in layers:
        kc = torch.empty((n_phys, Hkv, PAGE, d), dtype=torch.bfloat16, device=device)
        vc = torch.empty_like(kc)
        q = torch.empty((w.batch, Hq, d), dtype=torch.bfloat16, device=device)
        for b, s_b in enumerate(lens):
            npg = (s_b + PAGE - 1) // PAGE
            rows = npg * PAGE
            idx = pt_host[b, :npg].to(device=device, dtype=torch.long)
            for kind, cache in ((KIND_K, kc), (KIND_V, vc)):
                g = torch.Generator(device=device).manual_seed(tensor_seed(w.cfg_id, i, b, kind))
                x = torch.randn((rows, Hkv, d), generator=g, device=device, dtype=torch.float32)
                if kind == KIND_K:
                    x[hh[b].to(device)] *= w.hh_factor
                x = x.to(torch.bfloat16)
                if poison_tail and rows > s_b:
                    x[s_b:] = _BF16_NAN.to(device)
                cache.index_copy_(0, idx, x.view(npg, PAGE, Hkv, d).permute(0, 2, 1, 3).contiguous())
            g = torch.Generator(device=device).manual_seed(tensor_seed(w.cfg_id, i, b, KIND_Q))
            q[b] = torch.randn((Hq, d), generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)
        k_cache[i], v_cache[i], qs[i] = kc, vc, q
    seq = torch.tensor(lens, dtype=torch.int32, device=device)
    return DecodeInputs(w, k_cache, v_cache, qs, pt, seq, lens, max_pages, n_phys)


def bits(t: torch.Tensor):
    """A bf16 tensor's raw bit patterns as a host numpy uint16 array (no arithmetic)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view("uint16")


def sequence_pages(inp: DecodeInputs, layer: int, b: int):
    """Host copies (bf16 bits) of sequence b's physical pages for one layer, in logical order,
    for feeding the oracle one sequence at a time without copying the whole cache."""
    npg = (inp.seq_lens_host[b] + PAGE - 1) // PAGE
    idx = inp.page_table[b, :npg].to(torch.long)
    kb = bits(inp.k_cache[layer].index_select(0, idx))
    vb = bits(inp.v_cache[layer].index_select(0, idx))
    return kb, vb
