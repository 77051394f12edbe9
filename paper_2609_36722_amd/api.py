"""Python binding of the libattuner C ABI: argument marshalling only.

Each method carries the name of the C call it wraps (``attuner_<name>``),
turns torch device tensors into pointers, Python int lists into int32 host
arrays and the current torch stream into a ``hipStream_t``, and raises
:class:`AttunerError` on a non-zero status.  All arithmetic happens in the
library's HIP kernels.  bf16 tensors may be given as ``torch.bfloat16`` or as
any 2-byte integer view of the same bits.
"""

from __future__ import annotations

import ctypes as C
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from ._lib import MAX_RANK, MAX_REQUESTS, STATUS, KernelTimeC, LimitsC, ModelCfgC, lib


class AttunerError(RuntimeError):
    def __init__(self, status: int, where: str):
        msg = lib().attuner_last_error().decode(errors="replace")
        super().__init__(f"{where}: {STATUS.get(status, status)}: {msg}")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != 0:
        raise AttunerError(status, where)


def _ptr(t: Optional[torch.Tensor], elem: int = 2) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if t.element_size() != elem:
        raise ValueError(f"expected {elem}-byte elements, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _need(t: Optional[torch.Tensor], n: int, name: str) -> None:
    """Extent check the C side cannot make: t must hold at least n elements."""
    if t is not None and t.numel() < n:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {n}")


def _i32(vals: Sequence[int]):
    arr = (C.c_int32 * max(1, len(vals)))(*[int(v) for v in vals])
    return arr


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def bf16_to_device(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 bf16 bit patterns (numpy) -> torch.bfloat16 device tensor, same bits."""
    t = torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def bf16_to_host(t: torch.Tensor) -> np.ndarray:
    """torch bf16 (or 2-byte) tensor -> uint16 numpy array of its bits."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@dataclass(frozen=True)
class ModelCfg:
    n_layers: int
    hidden: int
    n_q_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    page_tokens: int = 16
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6

    def c_struct(self) -> ModelCfgC:
        return ModelCfgC(self.n_layers, self.hidden, self.n_q_heads, self.n_kv_heads, self.head_dim,
                         self.page_tokens, self.rope_theta, self.rms_eps)


class Context:
    """An ``attuner_ctx``: a paged artifact pool on one device plus workspaces."""

    def __init__(self, cfg: ModelCfg, pool_pages: int, device: int = 0):
        self.cfg = cfg
        self.device = device
        h = C.c_void_p()
        cs = cfg.c_struct()
        _check(lib().attuner_create(C.byref(cs), int(pool_pages), int(device), C.byref(h)), "attuner_create")
        self._h = h

    # ---- lifetime -------------------------------------------------------------
    def close(self) -> None:
        if getattr(self, "_h", None) is not None and self._h.value:
            lib().attuner_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def reserve(self, max_tokens: int = 0, max_position: int = 0, max_rank: int = 0, max_out: int = 0,
                max_lm_rows: int = 0, max_vocab: int = 0) -> None:
        """attuner_reserve: size the workspaces for calls within these limits
        (then they allocate nothing and can be captured into a graph)."""
        lim = LimitsC(int(max_tokens), int(max_position), int(max_rank), int(max_out), int(max_lm_rows),
                      int(max_vocab))
        _check(lib().attuner_reserve(self._h, C.byref(lim)), "attuner_reserve")

    # ---- pool -----------------------------------------------------------------
    def pool_info(self) -> Tuple[int, int, int]:
        a, b, c = C.c_int64(), C.c_int64(), C.c_int64()
        _check(lib().attuner_pool_info(self._h, C.byref(a), C.byref(b), C.byref(c)), "attuner_pool_info")
        return a.value, b.value, c.value

    def store_artifact(self, k: torch.Tensor, v: torch.Tensor, n_tokens: Optional[int] = None, stream=None) -> int:
        """k, v: [n_layers][n_kv][n_tokens][head_dim] bf16 on the device."""
        n = int(k.shape[-2]) if n_tokens is None else int(n_tokens)
        c = self.cfg
        _need(k, c.n_layers * c.n_kv_heads * n * c.head_dim, "k")
        _need(v, c.n_layers * c.n_kv_heads * n * c.head_dim, "v")
        out = C.c_int32()
        _check(lib().attuner_store_artifact(self._h, n, _ptr(k), _ptr(v), _stream(stream), C.byref(out)),
               "attuner_store_artifact")
        return out.value

    # ---- artifact caches in CPU RAM (pinned host pool) ----------------------------------
    def host_pool_create(self, host_pages: int) -> None:
        _check(lib().attuner_host_pool_create(self._h, int(host_pages)), "attuner_host_pool_create")

    def store_artifact_host(self, k: torch.Tensor, v: torch.Tensor, n_tokens: Optional[int] = None,
                            stream=None) -> int:
        """Like store_artifact, into the host pool."""
        n = int(k.shape[-2]) if n_tokens is None else int(n_tokens)
        c = self.cfg
        _need(k, c.n_layers * c.n_kv_heads * n * c.head_dim, "k")
        _need(v, c.n_layers * c.n_kv_heads * n * c.head_dim, "v")
        out = C.c_int32()
        _check(lib().attuner_store_artifact_host(self._h, n, _ptr(k), _ptr(v), _stream(stream), C.byref(out)),
               "attuner_store_artifact_host")
        return out.value

    def host_pool_info(self) -> Tuple[int, int]:
        pages, free = C.c_int64(), C.c_int64()
        _check(lib().attuner_host_pool_info(self._h, C.byref(pages), C.byref(free)), "attuner_host_pool_info")
        return pages.value, free.value

    # ---- host-pool pages moved by bulk copies into an HBM staging pool ---------------
    def stage_pool_create(self, stage_pages: int) -> None:
        _check(lib().attuner_stage_pool_create(self._h, int(stage_pages)), "attuner_stage_pool_create")

    def stage_pool_info(self) -> Tuple[int, int]:
        """(staging pages, copy runs per layer of the current staged plan)."""
        pages, runs = C.c_int64(), C.c_int64()
        _check(lib().attuner_stage_pool_info(self._h, C.byref(pages), C.byref(runs)), "attuner_stage_pool_info")
        return pages.value, runs.value

    def assemble_table_staged(self, requests: Sequence[Sequence[int]], suffix_cap: Sequence[int],
                              block_table: torch.Tensor, cache_rows: int,
                              stream=None) -> Tuple[List[int], List[int], int]:
        """Like assemble_table, with host pages remapped to staging pages;
        returns (cu_ctx, art_len, distinct host pages staged)."""
        ne, _ = self.assemble_plan(requests, suffix_cap)
        _need(block_table, 4 * ne, "block_table")
        ptr, ids = self._csr(requests)
        n = len(requests)
        cu = (C.c_int32 * (n + 1))()
        al = (C.c_int32 * max(1, n))()
        staged = C.c_int64()
        _check(lib().attuner_assemble_table_staged(self._h, n, _i32(ptr), _i32(ids), _i32(suffix_cap),
                                                   _ptr(block_table, 4) if block_table is not None else None, cu,
                                                   al, int(cache_rows), C.byref(staged), _stream(stream)),
               "attuner_assemble_table_staged")
        return list(cu), list(al)[:n], staged.value

    def stage_layers(self, layer_begin: int, n_layers: int, stream=None) -> None:
        _check(lib().attuner_stage_layers(self._h, int(layer_begin), int(n_layers), _stream(stream)),
               "attuner_stage_layers")

    def release_artifact(self, artifact_id: int) -> None:
        _check(lib().attuner_release_artifact(self._h, int(artifact_id)), "attuner_release_artifact")

    def artifact_pages(self, artifact_id: int) -> Tuple[List[int], int]:
        np_, nt = C.c_int32(), C.c_int32()
        _check(lib().attuner_artifact_pages(self._h, int(artifact_id), None, 0, C.byref(np_), C.byref(nt)),
               "attuner_artifact_pages")
        buf = (C.c_int32 * max(1, np_.value))()
        _check(lib().attuner_artifact_pages(self._h, int(artifact_id), buf, np_.value, C.byref(np_), C.byref(nt)),
               "attuner_artifact_pages")
        return list(buf)[: np_.value], nt.value

    # ---- assembly -------------------------------------------------------------
    @staticmethod
    def _csr(requests: Sequence[Sequence[int]]):
        ptr = [0]
        ids: List[int] = []
        for r in requests:
            ids.extend(int(a) for a in r)
            ptr.append(len(ids))
        return ptr, ids

    def assemble_plan(self, requests: Sequence[Sequence[int]], suffix_cap: Sequence[int]) -> Tuple[int, int]:
        ptr, ids = self._csr(requests)
        ne, rows = C.c_int64(), C.c_int64()
        _check(lib().attuner_assemble_plan(self._h, len(requests), _i32(ptr), _i32(ids), _i32(suffix_cap),
                                           C.byref(ne), C.byref(rows)), "attuner_assemble_plan")
        return ne.value, rows.value

    def assemble_kv(self, requests: Sequence[Sequence[int]], suffix_cap: Sequence[int], block_table: torch.Tensor,
                    req_kv: torch.Tensor, cache_rows: int, stream=None) -> Tuple[List[int], List[int]]:
        """Returns (cu_ctx, art_len); fills block_table (int32 device) and req_kv."""
        ne, rows = self.assemble_plan(requests, suffix_cap)
        c = self.cfg
        _need(block_table, 4 * ne, "block_table")
        _need(req_kv, c.n_layers * 2 * c.n_kv_heads * int(cache_rows) * c.head_dim, "req_kv")
        ptr, ids = self._csr(requests)
        n = len(requests)
        cu = (C.c_int32 * (n + 1))()
        al = (C.c_int32 * max(1, n))()
        _check(lib().attuner_assemble_kv(self._h, n, _i32(ptr), _i32(ids), _i32(suffix_cap),
                                         _ptr(block_table, 4) if block_table is not None else None, cu, al,
                                         _ptr(req_kv), int(cache_rows), _stream(stream)), "attuner_assemble_kv")
        return list(cu), list(al)[:n]

    # ---- prompts interleaving artifacts with online spans ------------------------------
    def assemble_segments_plan(self, segments: Sequence[Sequence[int]]) -> Tuple[int, int, int]:
        """segments[r]: request r's prompt in order, artifact ids (>= 0) and online spans (-n).
        Returns (n_entries, cache_rows, n_spans)."""
        ptr, flat = self._csr(segments)
        ne, rows, ns = C.c_int64(), C.c_int64(), C.c_int32()
        _check(lib().attuner_assemble_segments_plan(self._h, len(segments), _i32(ptr), _i32(flat), C.byref(ne),
                                                    C.byref(rows), C.byref(ns)), "attuner_assemble_segments_plan")
        return ne.value, rows.value, ns.value

    def assemble_segments(self, segments: Sequence[Sequence[int]], block_table: torch.Tensor, req_kv: torch.Tensor,
                          cache_rows: int, stream=None) -> Tuple[List[int], List[Tuple[int, int, int]]]:
        """Returns (cu_ctx, spans [(request, offset, length)]); fills block_table and req_kv."""
        ne, rows, ns = self.assemble_segments_plan(segments)
        c = self.cfg
        _need(block_table, 4 * ne, "block_table")
        _need(req_kv, c.n_layers * 2 * c.n_kv_heads * int(cache_rows) * c.head_dim, "req_kv")
        ptr, flat = self._csr(segments)
        n = len(segments)
        cu = (C.c_int32 * (n + 1))()
        sp = (C.c_int32 * max(3, 3 * ns))()
        _check(lib().attuner_assemble_segments(self._h, n, _i32(ptr), _i32(flat),
                                               _ptr(block_table, 4) if block_table is not None else None, cu, sp,
                                               _ptr(req_kv), int(cache_rows), _stream(stream)),
               "attuner_assemble_segments")
        spans = [(sp[3 * i], sp[3 * i + 1], sp[3 * i + 2]) for i in range(ns)]
        return list(cu), spans

    def assemble_table(self, requests: Sequence[Sequence[int]], suffix_cap: Sequence[int],
                       block_table: torch.Tensor, cache_rows: int, stream=None) -> Tuple[List[int], List[int]]:
        """Returns (cu_ctx, art_len); fills block_table (int32 device) only."""
        ne, _ = self.assemble_plan(requests, suffix_cap)
        _need(block_table, 4 * ne, "block_table")
        ptr, ids = self._csr(requests)
        n = len(requests)
        cu = (C.c_int32 * (n + 1))()
        al = (C.c_int32 * max(1, n))()
        _check(lib().attuner_assemble_table(self._h, n, _i32(ptr), _i32(ids), _i32(suffix_cap),
                                            _ptr(block_table, 4) if block_table is not None else None, cu, al,
                                            int(cache_rows), _stream(stream)), "attuner_assemble_table")
        return list(cu), list(al)[:n]

    def gather_layers(self, block_table: torch.Tensor, n_entries: int, layer_begin: int, n_layers: int,
                      req_kv: torch.Tensor, cache_rows: int, stream=None) -> None:
        c = self.cfg
        _need(block_table, 4 * int(n_entries), "block_table")
        _need(req_kv, c.n_layers * 2 * c.n_kv_heads * int(cache_rows) * c.head_dim, "req_kv")
        _check(lib().attuner_gather_layers(self._h, _ptr(block_table, 4) if block_table is not None else None,
                                           int(n_entries), int(layer_begin), int(n_layers), _ptr(req_kv),
                                           int(cache_rows), _stream(stream)), "attuner_gather_layers")

    # ---- projection -----------------------------------------------------------
    def qproj_lora(self, x: torch.Tensor, w: torch.Tensor, a: Optional[torch.Tensor], b: Optional[torch.Tensor],
                   rank: int, scale: float, lora_cols: int, out: torch.Tensor, stream=None) -> None:
        H, M, N = self.cfg.hidden, int(x.shape[0]), int(w.shape[0])
        _need(x, M * H, "x")
        _need(w, N * H, "w")
        _need(out, M * N, "out")
        if rank:
            _need(a, rank * H, "a")
            _need(b, lora_cols * rank, "b")
        _check(lib().attuner_qproj_lora(self._h, int(x.shape[0]), _ptr(x), _ptr(w), int(w.shape[0]), _ptr(a), _ptr(b),
                                        int(rank), float(scale), int(lora_cols), _ptr(out), _stream(stream)),
               "attuner_qproj_lora")

    def merge_lora(self, w: torch.Tensor, a: Optional[torch.Tensor], b: Optional[torch.Tensor], rank: int,
                   scale: float, lora_cols: int, w_out: torch.Tensor, stream=None) -> None:
        """w_out = w + scale * B A on rows < lora_cols (the deployment form of the adapter)."""
        N, K = int(w.shape[0]), int(w.shape[1])
        _need(w_out, N * K, "w_out")
        if rank:
            _need(a, rank * K, "a")
            _need(b, lora_cols * rank, "b")
        _check(lib().attuner_merge_lora(self._h, _ptr(w), N, K, _ptr(a), _ptr(b), int(rank), float(scale),
                                        int(lora_cols), _ptr(w_out), _stream(stream)), "attuner_merge_lora")

    # ---- the decoder layer around the path ------------------------------------------
    def embed(self, token_ids: Sequence[int], table: torch.Tensor, out: torch.Tensor, stream=None) -> None:
        """out[t] = table[token_ids[t]]: the embedding rows of the suffix tokens."""
        H = self.cfg.hidden
        V = int(table.numel()) // H
        n = len(token_ids)
        _need(out, n * H, "out")
        _check(lib().attuner_embed(self._h, n, _i32(token_ids), _ptr(table), V, _ptr(out), _stream(stream)),
               "attuner_embed")

    def rms_norm(self, x: torch.Tensor, gamma: torch.Tensor, out: torch.Tensor,
                 rows: Optional[Sequence[int]] = None, stream=None) -> None:
        """out[r] = RMSNorm(x[rows[r]]) * gamma over the hidden size (rows None: every row)."""
        H = self.cfg.hidden
        n_x = int(x.numel()) // H
        n = n_x if rows is None else len(rows)
        _need(gamma, H, "gamma")
        _need(out, n * H, "out")
        _check(lib().attuner_rms_norm(self._h, _ptr(x), n_x, H, _i32(rows) if rows is not None else None, n,
                                      _ptr(gamma), _ptr(out), _stream(stream)), "attuner_rms_norm")

    def linear(self, x: torch.Tensor, w: torch.Tensor, out: torch.Tensor, residual: Optional[torch.Tensor] = None,
               stream=None) -> None:
        """out = x w^T (+ residual); x [T][K], w [N][K], out and residual [T][N]."""
        N, K = int(w.shape[0]), int(w.shape[1])
        T = int(x.numel()) // K
        _need(x, T * K, "x")
        _need(out, T * N, "out")
        _need(residual, T * N, "residual")
        _check(lib().attuner_linear(self._h, T, _ptr(x), K, _ptr(w), N, _ptr(residual), _ptr(out), _stream(stream)),
               "attuner_linear")

    def gate_up_swiglu(self, x: torch.Tensor, w_gu: torch.Tensor, out: torch.Tensor, stream=None) -> None:
        """out = silu(x W_gate^T) * (x W_up^T); w_gu [2 I][K] with gate row j at 2j, up row j at 2j + 1."""
        I2, K = int(w_gu.shape[0]), int(w_gu.shape[1])
        T = int(x.numel()) // K
        _need(out, T * (I2 // 2), "out")
        _check(lib().attuner_gate_up_swiglu(self._h, T, _ptr(x), K, _ptr(w_gu), I2 // 2, _ptr(out), _stream(stream)),
               "attuner_gate_up_swiglu")

    def lm_head_argmax(self, x: torch.Tensor, w_lm: torch.Tensor, ids: torch.Tensor,
                       max_logit: Optional[torch.Tensor] = None, stream=None) -> None:
        """ids[r] = argmax over the vocabulary of x[r] w_lm^T (fp32 logits, smallest index on ties)."""
        V, H = int(w_lm.shape[0]), self.cfg.hidden
        n = int(x.numel()) // H
        _need(ids, n, "ids")
        _need(max_logit, n, "max_logit")
        _check(lib().attuner_lm_head_argmax(self._h, n, _ptr(x), _ptr(w_lm), V, _ptr(ids, 4),
                                            _ptr(max_logit, 4) if max_logit is not None else None,
                                            _stream(stream)), "attuner_lm_head_argmax")

    # ---- norm + rope, attention ---------------------------------------------------
    def _check_cache(self, cu_q, cu_ctx, q_hat, req_kv, cache_rows, q_raw=None, ld_q=0, k_raw=None, v_raw=None,
                     ld_kv=0) -> None:
        c = self.cfg
        T = int(cu_q[-1])
        _need(q_hat, T * c.n_q_heads * c.head_dim, "q_hat/o")
        _need(req_kv, c.n_layers * 2 * c.n_kv_heads * int(cache_rows) * c.head_dim, "req_kv")
        if T > 0 and q_raw is not None:
            for t, ld, width, name in ((q_raw, ld_q, c.n_q_heads * c.head_dim, "q_raw"),
                                       (k_raw, ld_kv, c.n_kv_heads * c.head_dim, "k_raw"),
                                       (v_raw, ld_kv, c.n_kv_heads * c.head_dim, "v_raw")):
                # the last row read ends at (T - 1) * ld + width elements past the view start
                if t.shape[0] < T or t.shape[1] < width or t.stride(0) != ld:
                    raise ValueError(f"{name}: view {tuple(t.shape)} stride {t.stride()} does not cover {T} rows "
                                     f"of {width} at row stride {ld}")

    def qk_norm_rope(self, layer: int, cu_q, cu_ctx, art_len, pos0, q_raw: torch.Tensor, ld_q: int,
                     k_raw: torch.Tensor, v_raw: torch.Tensor, ld_kv: int, gamma_q, gamma_k, q_hat, req_kv,
                     cache_rows: int, stream=None) -> None:
        n = len(art_len)
        self._check_cache(cu_q, cu_ctx, q_hat, req_kv, cache_rows, q_raw, ld_q, k_raw, v_raw, ld_kv)
        _check(lib().attuner_qk_norm_rope(self._h, int(layer), n, _i32(cu_q), _i32(cu_ctx), _i32(art_len),
                                          _i32(pos0) if pos0 is not None else None, _view_ptr(q_raw), int(ld_q),
                                          _view_ptr(k_raw), _view_ptr(v_raw), int(ld_kv), _ptr(gamma_q),
                                          _ptr(gamma_k), _ptr(q_hat), _ptr(req_kv), int(cache_rows),
                                          _stream(stream)), "attuner_qk_norm_rope")

    def attention(self, layer: int, cu_q, cu_ctx, art_len, q_hat, req_kv, cache_rows: int, o,
                  lse: Optional[torch.Tensor] = None, stream=None) -> None:
        n = len(art_len)
        self._check_cache(cu_q, cu_ctx, q_hat, req_kv, cache_rows)
        _need(o, int(cu_q[-1]) * self.cfg.n_q_heads * self.cfg.head_dim, "o")
        _need(lse, int(cu_q[-1]) * self.cfg.n_q_heads, "lse")
        _check(lib().attuner_attention(self._h, int(layer), n, _i32(cu_q), _i32(cu_ctx), _i32(art_len), _ptr(q_hat),
                                       _ptr(req_kv), int(cache_rows), _ptr(o), _ptr(lse, 4), _stream(stream)),
               "attuner_attention")

    def suffix_attn(self, layer: int, cu_q, cu_ctx, art_len, pos0, q_raw, ld_q: int, k_raw, v_raw, ld_kv: int,
                    gamma_q, gamma_k, req_kv, cache_rows: int, o, lse: Optional[torch.Tensor] = None,
                    stream=None, noalloc: bool = False) -> None:
        """attuner_suffix_attn, or with noalloc=True attuner_suffix_attn_noalloc (the key-split
        partials in the library's fixed device buffer; allocates nothing)."""
        n = len(art_len)
        self._check_cache(cu_q, cu_ctx, o, req_kv, cache_rows, q_raw, ld_q, k_raw, v_raw, ld_kv)
        _need(lse, int(cu_q[-1]) * self.cfg.n_q_heads, "lse")
        name = "attuner_suffix_attn_noalloc" if noalloc else "attuner_suffix_attn"
        _check(getattr(lib(), name)(self._h, int(layer), n, _i32(cu_q), _i32(cu_ctx), _i32(art_len),
                                    _i32(pos0) if pos0 is not None else None, _view_ptr(q_raw), int(ld_q),
                                    _view_ptr(k_raw), _view_ptr(v_raw), int(ld_kv), _ptr(gamma_q), _ptr(gamma_k),
                                    _ptr(req_kv), int(cache_rows), _ptr(o), _ptr(lse, 4), _stream(stream)),
               name)

    def suffix_attn_gather(self, layer: int, cu_q, cu_ctx, art_len, pos0, q_raw, ld_q: int, k_raw, v_raw,
                           ld_kv: int, gamma_q, gamma_k, req_kv, cache_rows: int, o, block_table: torch.Tensor,
                           n_entries: int, gather_layer: int, lse: Optional[torch.Tensor] = None,
                           stream=None) -> None:
        """attuner_suffix_attn_gather: suffix_attn for `layer` that also copies gather_layer's artifact
        pages (gather_layers(block_table, n_entries, gather_layer, 1, ...)) inside the attention launch."""
        n = len(art_len)
        self._check_cache(cu_q, cu_ctx, o, req_kv, cache_rows, q_raw, ld_q, k_raw, v_raw, ld_kv)
        _need(lse, int(cu_q[-1]) * self.cfg.n_q_heads, "lse")
        _need(block_table, 4 * int(n_entries), "block_table")
        _check(lib().attuner_suffix_attn_gather(self._h, int(layer), n, _i32(cu_q), _i32(cu_ctx), _i32(art_len),
                                                _i32(pos0) if pos0 is not None else None, _view_ptr(q_raw),
                                                int(ld_q), _view_ptr(k_raw), _view_ptr(v_raw), int(ld_kv),
                                                _ptr(gamma_q), _ptr(gamma_k), _ptr(req_kv), int(cache_rows),
                                                _ptr(o), _ptr(lse, 4),
                                                _ptr(block_table, 4) if block_table is not None else None,
                                                int(n_entries), int(gather_layer), _stream(stream)),
               "attuner_suffix_attn_gather")

    def span_attn(self, layer: int, cu_q, kv_start, offset, pos0, q_raw, ld_q: int, k_raw, v_raw, ld_kv: int,
                  gamma_q, gamma_k, req_kv, cache_rows: int, o, lse: Optional[torch.Tensor] = None,
                  stream=None) -> None:
        """Online spans at any offsets: span s = rows cu_q[s] .. cu_q[s+1]-1, its request's cache rows
        start at kv_start[s] and it sits offset[s] rows into them."""
        n = len(kv_start)
        self._check_cache(cu_q, [0] * (n + 1), o, req_kv, cache_rows, q_raw, ld_q, k_raw, v_raw, ld_kv)
        _need(lse, int(cu_q[-1]) * self.cfg.n_q_heads, "lse")
        _check(lib().attuner_span_attn(self._h, int(layer), n, _i32(cu_q), _i32(kv_start), _i32(offset),
                                       _i32(pos0) if pos0 is not None else None, _view_ptr(q_raw), int(ld_q),
                                       _view_ptr(k_raw), _view_ptr(v_raw), int(ld_kv), _ptr(gamma_q), _ptr(gamma_k),
                                       _ptr(req_kv), int(cache_rows), _ptr(o), _ptr(lse, 4), _stream(stream)),
               "attuner_span_attn")

    def decode_attn(self, layer: int, cu_ctx, ctx_len, pos, q_raw, ld_q: int, k_raw, v_raw, ld_kv: int,
                    gamma_q, gamma_k, req_kv, cache_rows: int, o, stream=None) -> None:
        """One new token per request (row r = request r) over its ctx_len[r] cached keys and its own."""
        n = len(ctx_len)
        cu_q = list(range(n + 1))
        self._check_cache(cu_q, cu_ctx, o, req_kv, cache_rows, q_raw, ld_q, k_raw, v_raw, ld_kv)
        _check(lib().attuner_decode_attn(self._h, int(layer), n, _i32(cu_ctx), _i32(ctx_len),
                                         _i32(pos) if pos is not None else None, _view_ptr(q_raw), int(ld_q),
                                         _view_ptr(k_raw), _view_ptr(v_raw), int(ld_kv), _ptr(gamma_q), _ptr(gamma_k),
                                         _ptr(req_kv), int(cache_rows), _ptr(o), _stream(stream)),
               "attuner_decode_attn")

    # ---- kernel timing ----------------------------------------------------------------
    def trace_begin(self) -> None:
        _check(lib().attuner_trace_begin(self._h), "attuner_trace_begin")

    def trace_end(self, max_kernels: int = 64) -> dict:
        """{kernel name: (launches, total_ms, max_ms)} of the launches since trace_begin."""
        buf = (KernelTimeC * max_kernels)()
        n = C.c_int32()
        _check(lib().attuner_trace_end(self._h, buf, max_kernels, C.byref(n)), "attuner_trace_end")
        return {buf[i].kernel.decode(): (buf[i].launches, buf[i].total_ms, buf[i].max_ms) for i in range(n.value)}

    def full_prefill(self, pos0: int, x, wqkv, a, b, rank: int, scale: float, gamma_q, gamma_k, o, k_out, v_out,
                     lse: Optional[torch.Tensor] = None, stream=None) -> None:
        c = self.cfg
        N, H = int(x.shape[0]), c.hidden
        _need(x, N * H, "x")
        _need(wqkv, (c.n_q_heads + 2 * c.n_kv_heads) * c.head_dim * H, "wqkv")
        _need(o, N * c.n_q_heads * c.head_dim, "o")
        _need(k_out, N * c.n_kv_heads * c.head_dim, "k_out")
        _need(v_out, N * c.n_kv_heads * c.head_dim, "v_out")
        _need(lse, N * c.n_q_heads, "lse")
        _need(gamma_q, c.head_dim, "gamma_q")
        _need(gamma_k, c.head_dim, "gamma_k")
        if rank:
            _need(a, rank * H, "a")
            _need(b, c.n_q_heads * c.head_dim * rank, "b")
        _check(lib().attuner_full_prefill(self._h, int(x.shape[0]), int(pos0), _ptr(x), _ptr(wqkv), _ptr(a), _ptr(b),
                                          int(rank), float(scale), _ptr(gamma_q), _ptr(gamma_k), _ptr(o), _ptr(k_out),
                                          _ptr(v_out), _ptr(lse, 4), _stream(stream)), "attuner_full_prefill")


def _view_ptr(t: torch.Tensor) -> int:
    """Pointer of a possibly strided row view (e.g. the k block of a fused qkv output)."""
    if not t.is_cuda or t.element_size() != 2:
        raise ValueError("expected a 2-byte device tensor")
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a 2-D row-major view")
    return t.data_ptr()


__all__ = ["AttunerError", "Context", "ModelCfg", "bf16_to_device", "bf16_to_host", "MAX_REQUESTS", "MAX_RANK"]
