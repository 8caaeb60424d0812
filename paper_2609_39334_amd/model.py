"""One decode step of a decoder-only transformer over a tree of candidates: the library's kernels inside
a whole model, for timing with synthetic weights.

Every candidate row (one per distinct candidate, computation deduplication Sec. 4.2) carries its
last token through L layers of pre-norm attention and a SwiGLU MLP -- the layer layout of the
paper's Qwen2.5 and Llama-3 generators (Sec. 5.1) -- and ends in next-token logits.  Per layer:

    h = RMSNorm(x);  q, k, v = h Wqkv;  q, k = RoPE(q, k, position)
    tkv_kv_append: the new token's k, v go to its pool slot          (library kernel)
    o = tree attention over the row's block table (tkv_decode)        (library kernel)
    x += o Wo;  h = RMSNorm(x);  x += (SiLU(h Wg) * (h Wu)) Wd

then logits = RMSNorm(x) W_lm, and the CD branching sampler draws each row's potential-many tokens
(tkv_cd_sample, library kernel).  One plan serves every layer: the block tables are the same in all
of them, only the pools differ.

The dense products are plain GEMMs and run in the platform BLAS (hipBLASLt through torch.mm); the
norms, RoPE and SiLU are elementwise torch ops.  Precision: the residual stream and every
elementwise step are fp32; every GEMM takes bf16 operands, accumulates in fp32 and rounds its
output to bf16 (as the attention kernel rounds o).  No biases; weights are N(0, 1/fan_in).
"""
from __future__ import annotations

from typing import List, NamedTuple

import torch

from . import Plan, tkv_cd_sample, tkv_kv_append


class DecoderShape(NamedTuple):
    layers: int
    hidden: int
    hq: int
    hkv: int
    d: int
    inter: int
    vocab: int
    rope_theta: float = 1e6
    eps: float = 1e-6


# Qwen2.5-7B-Instruct's layer layout (the paper's 7B generator): 28 layers, 28/4 heads of 128.
QWEN25_7B = DecoderShape(layers=28, hidden=3584, hq=28, hkv=4, d=128, inter=18944, vocab=152064)


class SyntheticDecoder:
    """Random weights (seeded) with the shapes of `shape`, stored as [in, out] bf16 matrices."""

    def __init__(self, shape: DecoderShape, device="cuda", seed: int = 0):
        self.shape = s = shape
        g = torch.Generator(device=device)
        g.manual_seed(seed)

        def mat(n_in, n_out):
            w = torch.empty((n_in, n_out), dtype=torch.float32, device=device)
            w.normal_(0.0, n_in ** -0.5, generator=g)
            return w.to(torch.bfloat16)

        def norm(n):
            w = torch.empty(n, dtype=torch.float32, device=device)
            return w.uniform_(0.8, 1.2, generator=g)

        self.embed = torch.empty((s.vocab, s.hidden), dtype=torch.float32, device=device).normal_(generator=g)
        self.layers = []
        for _ in range(s.layers):
            self.layers.append({"ln1": norm(s.hidden), "wqkv": mat(s.hidden, (s.hq + 2 * s.hkv) * s.d),
                                "wo": mat(s.hq * s.d, s.hidden), "ln2": norm(s.hidden),
                                "wgu": mat(s.hidden, 2 * s.inter), "wd": mat(s.inter, s.hidden)})
        self.lnf = norm(s.hidden)
        self.lm = mat(s.hidden, s.vocab)
        half = s.d // 2
        self.inv_freq = s.rope_theta ** (-torch.arange(half, dtype=torch.float32, device=device) * 2.0 / s.d)

    # ------------------------------------------------------------------ pieces
    def _rms(self, x, w):
        return (x * torch.rsqrt((x * x).mean(-1, keepdim=True) + self.shape.eps) * w).to(torch.bfloat16)

    def _rope(self, t, cos, sin):
        """Rotate-half RoPE of [rows, heads, d] bf16 at fp32, rounded back to bf16."""
        half = t.shape[-1] // 2
        x = t.float()
        x1, x2 = x[..., :half], x[..., half:]
        return torch.cat((x1 * cos - x2 * sin, x2 * cos + x1 * sin), dim=-1).to(torch.bfloat16).contiguous()

    # ------------------------------------------------------------------ one step
    def step(self, tokens: torch.Tensor, positions: torch.Tensor, dst: torch.Tensor, plan: Plan,
             k_pools: List[torch.Tensor], v_pools: List[torch.Tensor], stream=None, on_layer=None) -> torch.Tensor:
        """Logits [rows, vocab] (fp32 values of bf16) for each row's new token.

        tokens, positions: [rows] int64 (the new token and its position in the row's path); dst:
        [rows] int32 pool slots of the new tokens (tkv_bm_append); plan: a decode plan over the rows'
        block tables, which already include the new tokens; k_pools[l], v_pools[l]: layer l's pools
        [num_blocks, hkv, 16, d] bf16."""
        s = self.shape
        rows = int(tokens.numel())
        ang = positions.float()[:, None] * self.inv_freq[None, :]
        cos, sin = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
        x = self.embed[tokens]
        nq, nk = s.hq * s.d, s.hkv * s.d
        for li, w in enumerate(self.layers):
            qkv = torch.mm(self._rms(x, w["ln1"]), w["wqkv"])
            q = self._rope(qkv[:, :nq].reshape(rows, s.hq, s.d), cos, sin)
            k = self._rope(qkv[:, nq:nq + nk].reshape(rows, s.hkv, s.d), cos, sin)
            v = qkv[:, nq + nk:].reshape(rows, s.hkv, s.d).contiguous()
            tkv_kv_append(dst, k, v, k_pools[li], v_pools[li], stream)
            o = torch.empty((rows, s.hq, s.d), dtype=torch.bfloat16, device=x.device)
            plan.decode(q, k_pools[li], v_pools[li], o, None, stream)
            x = x + torch.mm(o.view(rows, nq), w["wo"]).float()
            gu = torch.mm(self._rms(x, w["ln2"]), w["wgu"]).float()
            a = (torch.nn.functional.silu(gu[:, :s.inter]) * gu[:, s.inter:]).to(torch.bfloat16)
            x = x + torch.mm(a, w["wd"]).float()
            if on_layer:
                on_layer(li)
        return torch.mm(self._rms(x, self.lnf), self.lm).float()

    def sample(self, logits, temperature, draw_off, uniform, max_potential, stream=None):
        """The CD branching step on the logits: (tokens, counts, groups per row)."""
        return tkv_cd_sample(logits.contiguous(), temperature, draw_off, uniform, max_potential, stream)
