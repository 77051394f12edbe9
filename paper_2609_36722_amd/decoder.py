"""A Qwen3-shaped decoder stack around the suffix path, chained through the
library's calls: the prefill of the suffix tokens of a batch of requests over
their assembled artifact caches, up to the greedy first token (the quantity
the paper's time-to-first-token ends with, appendix A.2; the adapted models
are Qwen3 decoder stacks, section 5.1).

Per layer l, on the residual stream h [T][H] of the T suffix tokens:
    x   = RMSNorm(h) * gamma_in                      attuner_rms_norm
    qkv = x [W_q | W_k | W_v]^T + LoRA on q          attuner_qproj_lora
    o   = attention over artifacts + causal suffix   attuner_suffix_attn (or _gather: the
                                                     launch also copies layer l + 1's pages)
    h   = h + o W_o^T                                attuner_linear (residual, in place)
    x   = RMSNorm(h) * gamma_post                    attuner_rms_norm
    g   = silu(x W_gate^T) * (x W_up^T)              attuner_gate_up_swiglu
    h   = h + g W_down^T                             attuner_linear (residual, in place)
then the last suffix token of each request: RMSNorm * gamma_final, LM head,
argmax (attuner_rms_norm on a row subset, attuner_lm_head_argmax).  Layer 0's
h is the embedding rows of the suffix tokens (attuner_embed).  Decode steps
run the same layers for one new token per request, with attuner_decode_attn
in place of the suffix attention (the generated tokens keep the adapted
query projection, section 4).

Every step runs in the library's kernels; torch only holds the device
buffers.  The weights are the caller's device tensors (bf16, row-major); the
gate and up projections are stored interleaved, gate row j at row 2j and up
row j at row 2j + 1 (see interleave_gate_up).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence, Tuple

import torch

from .api import Context


def interleave_gate_up(w_gate: torch.Tensor, w_up: torch.Tensor) -> torch.Tensor:
    """[I][H] gate and up projections -> [2I][H] with gate row j at 2j and up row j at 2j + 1
    (the layout attuner_gate_up_swiglu reads); a one-time weight-layout step."""
    assert w_gate.shape == w_up.shape
    return torch.stack([w_gate, w_up], dim=1).reshape(2 * w_gate.shape[0], w_gate.shape[1]).contiguous()


@dataclass
class LayerWeights:
    wqkv: torch.Tensor            # [(Hq + 2 Hkv) d][H]
    gamma_q: torch.Tensor         # [d]
    gamma_k: torch.Tensor         # [d]
    gamma_in: torch.Tensor        # [H]
    wo: torch.Tensor              # [H][Hq d]
    gamma_post: torch.Tensor      # [H]
    w_gu: torch.Tensor            # [2 I][H], interleaved
    w_down: torch.Tensor          # [H][I]
    a: Optional[torch.Tensor] = None   # LoRA A [rank][H]
    b: Optional[torch.Tensor] = None   # LoRA B [Hq d][rank]


@dataclass
class StackWeights:
    embed: torch.Tensor           # [vocab][H]
    gamma_final: torch.Tensor     # [H]
    w_lm: torch.Tensor            # [vocab][H]
    layers: List[LayerWeights] = field(default_factory=list)
    rank: int = 0
    scale: float = 0.0

    @property
    def intermediate(self) -> int:
        return int(self.layers[0].w_down.shape[1])

    @property
    def vocab(self) -> int:
        return int(self.w_lm.shape[0])


class DecoderStack:
    """Runs the stack for one fixed batch shape (suffix lengths, cache plan);
    the buffers are allocated once here, so a step allocates nothing."""

    def __init__(self, ctx: Context, weights: StackWeights, suffix_len: Sequence[int]):
        cfg = ctx.cfg
        if len(weights.layers) != cfg.n_layers:
            raise ValueError(f"{len(weights.layers)} layers of weights for a {cfg.n_layers}-layer context")
        if any(int(s) < 1 for s in suffix_len):
            raise ValueError("every request needs at least one suffix token to produce a first token")
        self.ctx, self.w = ctx, weights
        self.cu_q = [0]
        for s in suffix_len:
            self.cu_q.append(self.cu_q[-1] + int(s))
        self.last_rows = [self.cu_q[r + 1] - 1 for r in range(len(suffix_len))]
        T, H, dev = self.cu_q[-1], cfg.hidden, weights.embed.device
        self.nq, self.nkv = cfg.n_q_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim
        bf = dict(dtype=torch.bfloat16, device=dev)
        self.h = torch.empty(T, H, **bf)
        self.x = torch.empty(T, H, **bf)
        self.qkv = torch.empty(T, self.nq + 2 * self.nkv, **bf)
        self.o = torch.empty(T, cfg.n_q_heads, cfg.head_dim, **bf)
        self.g = torch.empty(T, weights.intermediate, **bf)
        self.x_last = torch.empty(len(suffix_len), H, **bf)
        self.ids = torch.empty(len(suffix_len), dtype=torch.int32, device=dev)
        self.max_logit = torch.empty(len(suffix_len), dtype=torch.float32, device=dev)

    def embed(self, token_ids: Sequence[int], stream=None) -> None:
        """h = the embedding rows of the suffix tokens (all requests, in order)."""
        if len(token_ids) != self.cu_q[-1]:
            raise ValueError(f"{len(token_ids)} token ids for {self.cu_q[-1]} suffix tokens")
        self.ctx.embed(token_ids, self.w.embed, self.h, stream=stream)

    STEPS = ("input_norm", "qkv_proj", "suffix_attn", "o_proj", "post_norm", "gate_up", "down_proj")

    def layers(self, cu_ctx, art_len, pos0, req_kv: torch.Tensor, cache_rows: int, stream=None,
               first: int = 0, count: Optional[int] = None,
               mark: Optional[Callable[[Optional[str]], None]] = None,
               gather: Optional[Tuple[torch.Tensor, int]] = None) -> None:
        """Decoder layers first .. first + count - 1 (default: all) over h, in
        place.  cu_ctx / art_len / pos0 as attuner_suffix_attn takes them (from
        the cache assembly).  Makes no host-to-device copy, so a caller may
        capture it into a graph.  mark, if given, is called with the name of
        each step (one of STEPS) before its call and with None after the last
        (e.g. to record timing events).  gather, if given, is (block_table,
        n_entries) of the last attuner_assemble_table call: then the cache
        need only hold layer `first`'s artifact pages, and each layer's
        attention launch copies the next layer's (attuner_suffix_attn_gather)."""
        c, w, ld = self.ctx, self.w, self.nq + 2 * self.nkv
        q, k, v = self.qkv[:, :self.nq], self.qkv[:, self.nq:self.nq + self.nkv], self.qkv[:, self.nq + self.nkv:]
        count = len(w.layers) - first if count is None else count
        m = mark if mark is not None else (lambda name: None)
        for l in range(first, first + count):
            lw = w.layers[l]
            m("input_norm")
            c.rms_norm(self.h, lw.gamma_in, self.x, stream=stream)
            m("qkv_proj")
            c.qproj_lora(self.x, lw.wqkv, lw.a, lw.b, w.rank if lw.a is not None else 0, w.scale, self.nq, self.qkv,
                         stream=stream)
            m("suffix_attn")
            if gather is not None and l + 1 < first + count:
                c.suffix_attn_gather(l, self.cu_q, cu_ctx, art_len, pos0, q, ld, k, v, ld, lw.gamma_q, lw.gamma_k,
                                     req_kv, cache_rows, self.o, gather[0], gather[1], l + 1, stream=stream)
            else:
                c.suffix_attn(l, self.cu_q, cu_ctx, art_len, pos0, q, ld, k, v, ld, lw.gamma_q, lw.gamma_k, req_kv,
                              cache_rows, self.o, stream=stream)
            m("o_proj")
            c.linear(self.o.view(-1, self.nq), lw.wo, self.h, residual=self.h, stream=stream)
            m("post_norm")
            c.rms_norm(self.h, lw.gamma_post, self.x, stream=stream)
            m("gate_up")
            c.gate_up_swiglu(self.x, lw.w_gu, self.g, stream=stream)
            m("down_proj")
            c.linear(self.g, lw.w_down, self.h, residual=self.h, stream=stream)
        m(None)

    def first_token(self, stream=None) -> torch.Tensor:
        """ids[r] = greedy first token of request r from the final h (device int32)."""
        self.ctx.rms_norm(self.h, self.w.gamma_final, self.x_last, rows=self.last_rows, stream=stream)
        self.ctx.lm_head_argmax(self.x_last, self.w.w_lm, self.ids, self.max_logit, stream=stream)
        return self.ids

    def forward(self, token_ids: Sequence[int], cu_ctx, art_len, pos0, req_kv: torch.Tensor, cache_rows: int,
                stream=None) -> torch.Tensor:
        self.embed(token_ids, stream)
        self.layers(cu_ctx, art_len, pos0, req_kv, cache_rows, stream)
        return self.first_token(stream)

    # ---- decode: one generated token per request ----------------------------------
    def _decode_buffers(self):
        if getattr(self, "hd", None) is None:
            n, cfg, dev = len(self.last_rows), self.ctx.cfg, self.w.embed.device
            bf = dict(dtype=torch.bfloat16, device=dev)
            self.hd = torch.empty(n, cfg.hidden, **bf)
            self.xd = torch.empty(n, cfg.hidden, **bf)
            self.qkvd = torch.empty(n, self.nq + 2 * self.nkv, **bf)
            self.od = torch.empty(n, cfg.n_q_heads, cfg.head_dim, **bf)
            self.gd = torch.empty(n, self.w.intermediate, **bf)

    def decode_embed(self, token_ids: Sequence[int], stream=None) -> None:
        """hd = the embedding rows of one new token per request."""
        self._decode_buffers()
        if len(token_ids) != len(self.last_rows):
            raise ValueError(f"{len(token_ids)} token ids for {len(self.last_rows)} requests")
        self.ctx.embed(token_ids, self.w.embed, self.hd, stream=stream)

    def decode_layers(self, cu_ctx, ctx_len, req_kv: torch.Tensor, cache_rows: int, stream=None) -> None:
        """Every layer for the new tokens (row r = request r, at position
        ctx_len[r], its key/value written to cache row cu_ctx[r] + ctx_len[r]),
        attending to the ctx_len[r] keys before it (attuner_decode_attn); the
        projections of a few tokens run as GEMVs.  No host-to-device copy."""
        self._decode_buffers()
        c, w, ld = self.ctx, self.w, self.nq + 2 * self.nkv
        q = self.qkvd[:, :self.nq]
        k, v = self.qkvd[:, self.nq:self.nq + self.nkv], self.qkvd[:, self.nq + self.nkv:]
        for l, lw in enumerate(w.layers):
            c.rms_norm(self.hd, lw.gamma_in, self.xd, stream=stream)
            c.qproj_lora(self.xd, lw.wqkv, lw.a, lw.b, w.rank if lw.a is not None else 0, w.scale, self.nq, self.qkvd,
                         stream=stream)
            c.decode_attn(l, cu_ctx, ctx_len, None, q, ld, k, v, ld, lw.gamma_q, lw.gamma_k, req_kv, cache_rows,
                          self.od, stream=stream)
            c.linear(self.od.view(-1, self.nq), lw.wo, self.hd, residual=self.hd, stream=stream)
            c.rms_norm(self.hd, lw.gamma_post, self.xd, stream=stream)
            c.gate_up_swiglu(self.xd, lw.w_gu, self.gd, stream=stream)
            c.linear(self.gd, lw.w_down, self.hd, residual=self.hd, stream=stream)

    def decode_token(self, stream=None) -> torch.Tensor:
        """ids[r] = greedy next token of request r from hd (device int32)."""
        self.ctx.rms_norm(self.hd, self.w.gamma_final, self.x_last, stream=stream)
        self.ctx.lm_head_argmax(self.x_last, self.w.w_lm, self.ids, self.max_logit, stream=stream)
        return self.ids

    def decode(self, token_ids: Sequence[int], cu_ctx, ctx_len, req_kv: torch.Tensor, cache_rows: int,
               stream=None) -> torch.Tensor:
        """One decode step: the next token of every request (device int32)."""
        self.decode_embed(token_ids, stream)
        self.decode_layers(cu_ctx, ctx_len, req_kv, cache_rows, stream)
        return self.decode_token(stream)
