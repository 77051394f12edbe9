"""Helpers of the GPU parity tests: run the HIP path (through the C ABI) and
the fp64 oracle on the same seeded bf16 inputs of a workload."""

from __future__ import annotations

import math
from typing import Dict, List, Sequence

import numpy as np
import torch

import oracle
import synthdata as sd
from paper_2609_36722_amd.api import Context, ModelCfg, bf16_to_device, bf16_to_host


def have_gpu() -> bool:
    return torch.cuda.is_available()


def dev_bf16(bits) -> torch.Tensor:
    return bf16_to_device(bits, "cuda")


def host_f64(t: torch.Tensor) -> np.ndarray:
    return oracle.decode_bf16(bf16_to_host(t))


class GpuWorkload:
    """A workload stored in a fresh context: its artifacts in the pool and the
    request caches assembled, for the given model layers."""

    def __init__(self, wl: sd.Workload, layers: Sequence[int] = (0,), extra_pages: int = 0, suffix_extra: int = 0,
                 host_artifacts: Sequence[int] = ()):
        self.wl = wl
        self.layers = list(layers)
        s = wl.shape
        self.cfg = ModelCfg(n_layers=len(self.layers), hidden=s.hidden, n_q_heads=s.n_q_heads,
                            n_kv_heads=s.n_kv_heads, head_dim=s.head_dim, rope_theta=s.rope_theta, rms_eps=s.rms_eps)
        used = sorted({a for r in wl.requests for a in r.artifact_ids})
        pages = sum(math.ceil(wl.artifact_lengths[a] / 16) for a in used) + extra_pages
        self.ctx = Context(self.cfg, pool_pages=max(1, pages))
        if host_artifacts:  # these artifacts go to the pinned host pool
            self.ctx.host_pool_create(sum(math.ceil(wl.artifact_lengths[a] / 16) for a in set(host_artifacts)))
        self.ids: Dict[int, int] = {}
        self.art_k: Dict[int, np.ndarray] = {}  # bits [n_layers][L][n_kv][d]
        self.art_v: Dict[int, np.ndarray] = {}
        for a in used:
            kv = [sd.artifact_kv(wl, a, l) for l in self.layers]
            k = np.stack([x[0] for x in kv])
            v = np.stack([x[1] for x in kv])
            self.art_k[a], self.art_v[a] = k, v
            kd = dev_bf16(np.ascontiguousarray(k.transpose(0, 2, 1, 3)))
            vd = dev_bf16(np.ascontiguousarray(v.transpose(0, 2, 1, 3)))
            store = self.ctx.store_artifact_host if a in host_artifacts else self.ctx.store_artifact
            self.ids[a] = store(kd, vd)
        self.requests = [[self.ids[a] for a in r.artifact_ids] for r in wl.requests]
        self.suffix_cap = [r.suffix_len + suffix_extra for r in wl.requests]
        self.n_entries, self.rows = self.ctx.assemble_plan(self.requests, self.suffix_cap)
        self.block_table = torch.zeros(max(1, self.n_entries) * 4, dtype=torch.int32, device="cuda")
        self.req_kv = torch.zeros(len(self.layers) * 2 * s.n_kv_heads * self.rows * s.head_dim,
                                  dtype=torch.bfloat16, device="cuda")
        self.cu_ctx, self.art_len = self.ctx.assemble_kv(self.requests, self.suffix_cap, self.block_table,
                                                         self.req_kv, self.rows)
        self.cu_q = [0]
        for r in wl.requests:
            self.cu_q.append(self.cu_q[-1] + r.suffix_len)
        self.pos0 = [wl.pos0(r) for r in wl.requests]

    def close(self):
        self.ctx.close()

    # ---- one layer of the suffix path -------------------------------------------
    def layer_inputs(self, li: int):
        l = self.layers[li]
        w = sd.layer_weights(self.wl, l)
        x = np.concatenate([sd.suffix_hidden(self.wl, r, l) for r in range(len(self.wl.requests))])
        return w, x

    def run_layer(self, li: int, with_lse: bool = True):
        s = self.wl.shape
        w, x = self.layer_inputs(li)
        wqkv = dev_bf16(np.concatenate([w["wq"], w["wk"], w["wv"]]))
        xd = dev_bf16(x)
        a = dev_bf16(w["a"]) if self.wl.rank else None
        b = dev_bf16(w["b"]) if self.wl.rank else None
        T = x.shape[0]
        nq, nkv = s.q_dim, s.kv_dim
        qkv = torch.empty(T, nq + 2 * nkv, dtype=torch.bfloat16, device="cuda")
        self.ctx.qproj_lora(xd, wqkv, a, b, self.wl.rank, self.wl.scale, nq, qkv)
        o = torch.empty(T, s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(T, s.n_q_heads, dtype=torch.float32, device="cuda") if with_lse else None
        self.ctx.suffix_attn(li, self.cu_q, self.cu_ctx, self.art_len, self.pos0, qkv[:, :nq], nq + 2 * nkv,
                             qkv[:, nq:nq + nkv], qkv[:, nq + nkv:], nq + 2 * nkv, dev_bf16(w["gamma_q"]),
                             dev_bf16(w["gamma_k"]), self.req_kv, self.rows, o, lse)
        torch.cuda.synchronize()
        return {"qkv": qkv, "o": o, "lse": lse}

    def cache_view(self) -> np.ndarray:
        s = self.wl.shape
        return bf16_to_host(self.req_kv).reshape(len(self.layers), 2, s.n_kv_heads, self.rows, s.head_dim)

    # ---- oracle counterparts ----------------------------------------------------------
    def oracle_layer(self, li: int, req: int, rows=None):
        s = self.wl.shape
        w, _ = self.layer_inputs(li)
        wf = {k: oracle.decode_bf16(v) for k, v in w.items()}
        r = self.wl.requests[req]
        x = oracle.decode_bf16(sd.suffix_hidden(self.wl, req, self.layers[li]))
        if r.artifact_ids:
            ka = np.concatenate([oracle.decode_bf16(self.art_k[a][li]) for a in r.artifact_ids])
            va = np.concatenate([oracle.decode_bf16(self.art_v[a][li]) for a in r.artifact_ids])
        else:
            ka = va = np.zeros((0, s.n_kv_heads, s.head_dim))
        return oracle.suffix_layer(x, wf["wq"], wf["wk"], wf["wv"], wf["a"], wf["b"], self.wl.scale, wf["gamma_q"],
                                   wf["gamma_k"], ka, va, self.wl.pos0(r), s.n_q_heads, s.n_kv_heads,
                                   s.rope_theta, s.rms_eps, rows=rows)

    def oracle_layer_blocks(self, li: int, req: int, block: int = 256, say=None):
        """Every suffix row of one request through the oracle: projections,
        norms and RoPE of all rows once (suffix_layer with no attention rows),
        then the oracle's attention over blocks of rows.  Each row's softmax
        is its own, so the blocks only bound host memory.  Also returns the
        assembled keys (for the LSE bar)."""
        s = self.wl.shape
        base = self.oracle_layer(li, req, rows=np.arange(0))
        r = self.wl.requests[req]
        if r.artifact_ids:
            ka = np.concatenate([oracle.decode_bf16(self.art_k[a][li]) for a in r.artifact_ids])
            va = np.concatenate([oracle.decode_bf16(self.art_v[a][li]) for a in r.artifact_ids])
        else:
            ka = va = np.zeros((0, s.n_kv_heads, s.head_dim))
        keys = np.concatenate([ka, base["k_hat"]])
        vals = np.concatenate([va, base["v"]])
        q_hat = base["q_hat"]
        S = q_hat.shape[0]
        o = np.empty_like(q_hat)
        lse = np.empty(q_hat.shape[:2])
        for r0 in range(0, S, block):
            rows = np.arange(r0, min(S, r0 + block))
            o[rows], lse[rows] = oracle.attention(q_hat, keys, vals, ka.shape[0], rows=rows, return_lse=True)
            if say is not None:
                say(f"oracle rows {r0}..{rows[-1]} of {S}")
        return dict(base, o=o, lse=lse, keys=keys)

