"""Reference definitions of the suffix-prefill path, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).  Each function names the
passage of the paper it follows.

Notation: Hq query heads, Hkv key/value heads (G = Hq / Hkv query heads share a
KV head), head dimension d, L_art cached artifact tokens, S suffix tokens.

Parity status: every function here is pinned by the CPU test suite against a
closed form, an invariant, a brute-force loop or a library routine (the
oracle-pin tests).  The paper prints no kernel-level worked example; the small
worked examples under ``tests/golden`` are derived by hand from the definitions.
The decoder layer and stack (``decoder_layer``, ``first_token``), whose
structure the paper does not give, are pinned against the transformers
library's Qwen3 implementation run in float64 (the paper's base models) and
against a brute-force loop in plain Python sums.
"""

from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


# ----------------------------------------------------------------------------
# storage
# ----------------------------------------------------------------------------

def decode_bf16(bits) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exact float64 values.

    A bfloat16 value is the upper 16 bits of an IEEE binary32 word, so shifting
    the pattern left by 16 gives the binary32 word of the same value.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# O1/O2  cache construction and assembly (integer / copy work)
# ----------------------------------------------------------------------------

def page_valid_counts(n_tokens: int, page_tokens: int) -> List[int]:
    """Tokens held by each page of an artifact of n_tokens (section 2, the PIC box:
    each artifact's KV is stored once, independently).  Page p holds tokens
    [p*T, min((p+1)*T, n)); every page but the last is full."""
    if n_tokens <= 0:
        raise ValueError("an artifact holds at least one token")
    full, rem = divmod(n_tokens, page_tokens)
    return [page_tokens] * full + ([rem] if rem else [])


def block_table(artifact_lengths: Sequence[int],
                requests: Sequence[Tuple[Sequence[int], int]],
                page_tokens: int):
    """Logical block table of a batch of requests (section 2, the PIC box:
    cached blocks are put together in prompt order; appendix A.3, "Cache
    construction and reuse").

    ``requests`` is a list of (ordered artifact ids, suffix capacity).  Request r
    owns rows [cu_ctx[r], cu_ctx[r+1]) of the assembled cache: first its
    artifacts back to back in the given order (no holes), then ``suffix
    capacity`` rows for the online tokens.

    Returns (entries, cu_ctx) where entries is an int64 array of rows
    (artifact_id, page_index_in_artifact, n_valid, request, dst_row), in request
    order, then artifact order, then page order; dst_row is the global row of
    the page's first token.
    """
    entries = []
    cu_ctx = [0]
    for r, (ids, cap) in enumerate(requests):
        row = cu_ctx[-1]
        for a in ids:
            for p, nv in enumerate(page_valid_counts(int(artifact_lengths[a]), page_tokens)):
                entries.append((int(a), p, nv, r, row))
                row += nv
        cu_ctx.append(row + int(cap))
    return np.asarray(entries, dtype=np.int64).reshape(-1, 5), np.asarray(cu_ctx, dtype=np.int64)


def assemble(artifact_k: Dict[int, np.ndarray], artifact_v: Dict[int, np.ndarray],
             requests: Sequence[Tuple[Sequence[int], int]], n_kv: int, head_dim: int,
             fill=0) -> Tuple[np.ndarray, np.ndarray]:
    """Assembled request cache (section 2, the PIC box: stored blocks are
    reused in prompt order without re-encoding; appendix C.1, PIC: artifact
    tokens are not recomputed and keep their local-position rotation).

    artifact_k[a] / artifact_v[a]: [n_layers][L_a][Hkv][d] (any dtype; copied
    exactly).  Returns (cache, cu_ctx) with cache laid out as
    [n_layers][2 (K, V)][Hkv][T_total][d]:  row cu_ctx[r] + off_j + t holds token t
    of the request's j-th artifact, off_j being the summed length of the
    artifacts before it.  Suffix rows hold ``fill``.
    """
    any_a = next(iter(artifact_k.values()))
    n_layers, dt = any_a.shape[0], any_a.dtype
    cu = [0]
    for ids, cap in requests:
        cu.append(cu[-1] + sum(artifact_k[a].shape[1] for a in ids) + int(cap))
    cache = np.full((n_layers, 2, n_kv, cu[-1], head_dim), fill, dtype=dt)
    for r, (ids, cap) in enumerate(requests):
        parts_k = [artifact_k[a] for a in ids]
        parts_v = [artifact_v[a] for a in ids]
        if not parts_k:
            continue
        kk = np.concatenate(parts_k, axis=1)  # [layers][L_art][Hkv][d]
        vv = np.concatenate(parts_v, axis=1)
        L = kk.shape[1]
        cache[:, 0, :, cu[r]:cu[r] + L, :] = kk.transpose(0, 2, 1, 3)
        cache[:, 1, :, cu[r]:cu[r] + L, :] = vv.transpose(0, 2, 1, 3)
    return cache, np.asarray(cu, dtype=np.int64)


# ----------------------------------------------------------------------------
# O3  query-side LoRA projection (section 4, eq. 4)
# ----------------------------------------------------------------------------

def qproj_lora(x: np.ndarray, w: np.ndarray, a: Optional[np.ndarray] = None,
               b: Optional[np.ndarray] = None, scale: float = 1.0,
               lora_cols: Optional[int] = None) -> np.ndarray:
    """out = x W^T + scale * (x A^T) B^T   (section 4, eq. 4, with scale = alpha / r).

    x [T][H], W [N][H], A [r][H], B [lora_cols][r].  The low-rank term is added to
    the first ``lora_cols`` output columns only (the query block of a fused
    q/k/v weight: keys and values are never adapted, section 4, "Query
    Adaptation with Fixed Artifact KV").  rank 0 (A or B empty/None) gives the
    plain projection.
    """
    x = np.asarray(x, np.float64)
    out = x @ np.asarray(w, np.float64).T
    if a is not None and b is not None and np.asarray(a).size and np.asarray(b).size:
        a = np.asarray(a, np.float64)
        b = np.asarray(b, np.float64)
        nl = b.shape[0] if lora_cols is None else int(lora_cols)
        down = x @ a.T                   # A h   [T][r]
        out[:, :nl] += scale * (down @ b[:nl].T)   # (alpha/r) B (A h)
    return out


# ----------------------------------------------------------------------------
# O4/O5  per-head QK-RMSNorm and rotary embedding (section 4: after the
#        adapted projection, the query goes through the base model's own
#        per-head q-norm and rotary embedding, unchanged)
# ----------------------------------------------------------------------------

def rms_norm_heads(u: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis (one head):  gamma * u / sqrt(mean(u^2) + eps)."""
    u = np.asarray(u, np.float64)
    ms = np.mean(u * u, axis=-1, keepdims=True)
    return np.asarray(gamma, np.float64) * u / np.sqrt(ms + eps)


def rope(u: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotary position embedding in the half-split pairing used by Qwen3:
    dimension j is paired with j + d/2 and rotated by angle p * theta^(-2j/d).

    u [T][heads][d], positions [T] (integers).
    """
    u = np.asarray(u, np.float64)
    d = u.shape[-1]
    half = d // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * j / d)                              # [d/2]
    ang = np.asarray(positions, np.float64)[:, None] * inv_freq[None, :]   # [T][d/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    lo, hi = u[..., :half], u[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


# ----------------------------------------------------------------------------
# O6  attention over the assembled context (section 3.2, eq. 3 gives the form:
#     softmax(q K^T / sqrt(d_k) + M_t) V with the causal mask M_t; appendix A.5,
#     Deployment: scaled dot-product attention with causal masks and position
#     ids of the assembled context)
# ----------------------------------------------------------------------------

def _scores(q: np.ndarray, k: np.ndarray, art_len: int, rows: np.ndarray) -> List[np.ndarray]:
    """Masked scaled scores per query head: list over h of [len(rows)][n_keys]."""
    S, Hq, d = q.shape
    n_keys, Hkv, _ = k.shape
    G = Hq // Hkv
    visible = (np.arange(n_keys)[None, :] <= (art_len + rows)[:, None])    # row i sees j <= L_art + i
    out = []
    for h in range(Hq):
        g = h // G                                                    # query head h reads KV head h // G
        z = (q[rows, h, :] @ k[:, g, :].T) / math.sqrt(d)
        out.append(np.where(visible, z, -np.inf))
    return out


def attention_probs(q, k, art_len: int, rows=None) -> np.ndarray:
    """Attention weights P [len(rows)][Hq][n_keys] (rows sum to one)."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    rows = np.arange(q.shape[0]) if rows is None else np.asarray(rows)
    ps = []
    for z in _scores(q, k, art_len, rows):
        m = z.max(axis=1, keepdims=True)
        e = np.exp(z - m)
        ps.append(e / e.sum(axis=1, keepdims=True))
    return np.stack(ps, axis=1)


def attention(q, k, v, art_len: int, rows=None, return_lse: bool = False):
    """Multi-segment GQA attention of the suffix queries over the assembled keys.

    q [S][Hq][d] (normalised, rotated suffix queries), k/v [n_keys][Hkv][d] with
    n_keys >= art_len + S: rows [0, art_len) are the cached artifact keys, row
    art_len + i is suffix token i.  Suffix row i attends to keys 0 .. art_len + i:
    every artifact key, and the suffix causally.  Returns O [len(rows)][Hq][d]
    and, if asked, the natural-log sum of exponentials of the scaled scores,
    lse [len(rows)][Hq].
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    rows = np.arange(q.shape[0]) if rows is None else np.asarray(rows)
    Hq, Hkv = q.shape[1], k.shape[1]
    G = Hq // Hkv
    o = np.empty((len(rows), Hq, q.shape[2]))
    lse = np.empty((len(rows), Hq))
    for h, z in enumerate(_scores(q, k, art_len, rows)):
        m = z.max(axis=1, keepdims=True)
        e = np.exp(z - m)
        den = e.sum(axis=1, keepdims=True)
        o[:, h, :] = (e / den) @ v[:, h // G, :]
        lse[:, h] = (m + np.log(den))[:, 0]
    return (o, lse) if return_lse else o


# ----------------------------------------------------------------------------
# one layer of suffix prefill, and full prefill
# ----------------------------------------------------------------------------

def suffix_layer(x, wq, wk, wv, a, b, scale, gamma_q, gamma_k, k_art, v_art,
                 pos0: int, n_q_heads: int, n_kv_heads: int, theta: float, eps: float,
                 rows=None) -> Dict[str, np.ndarray]:
    """One layer of Attuner online prefill over a frozen artifact cache.

    Section 4, eq. 4: adapted queries q = W_q h + scale * B A h; keys and values of
    the online tokens use the unadapted projections.  Section 4: q and k pass
    through the per-head RMSNorm and RoPE; suffix token i sits at position
    pos0 + i.  Appendix A.3 and C.1: the artifact keys/values (k_art, v_art
    [L_art][Hkv][d], already normalised and rotated at their local positions)
    are used unchanged.  Attention as in :func:`attention`.

    Returns q_hat [S][Hq][d], k_hat and v [S][Hkv][d] (the suffix rows written to
    the cache) and O, lse for ``rows`` (default all suffix rows).
    """
    x = np.asarray(x, np.float64)
    S = x.shape[0]
    d = np.asarray(gamma_q).shape[0]
    q = qproj_lora(x, wq, a, b, scale).reshape(S, n_q_heads, d)
    k = qproj_lora(x, wk).reshape(S, n_kv_heads, d)
    v = qproj_lora(x, wv).reshape(S, n_kv_heads, d)
    pos = pos0 + np.arange(S)
    q_hat = rope(rms_norm_heads(q, gamma_q, eps), pos, theta)
    k_hat = rope(rms_norm_heads(k, gamma_k, eps), pos, theta)
    k_art = np.asarray(k_art, np.float64).reshape(-1, n_kv_heads, d)
    v_art = np.asarray(v_art, np.float64).reshape(-1, n_kv_heads, d)
    L = k_art.shape[0]
    keys = np.concatenate([k_art, k_hat], axis=0)
    vals = np.concatenate([v_art, v], axis=0)
    o, lse = attention(q_hat, keys, vals, L, rows=rows, return_lse=True)
    return {"q": q, "k": k, "q_hat": q_hat, "k_hat": k_hat, "v": v, "o": o, "lse": lse}


def full_prefill(x, wq, wk, wv, gamma_q, gamma_k, pos0: int, n_q_heads: int,
                 n_kv_heads: int, theta: float, eps: float, a=None, b=None,
                 scale: float = 0.0, rows=None) -> Dict[str, np.ndarray]:
    """Full-context prefill of one layer (section 2, eq. 2, Full; appendix C.1,
    Full): every token is computed, causally, at positions pos0 .. pos0 + N - 1.
    With pos0 = 0 on an artifact alone this is also the artifact encoder of the
    PIC construction (eq. 2, PIC: local positions from zero, adapters off).
    Returns O, lse and the normalised/rotated keys and raw values of all N rows.
    """
    d = np.asarray(gamma_q).shape[0]
    empty = np.zeros((0, n_kv_heads, d))
    return suffix_layer(x, wq, wk, wv, a, b, scale, gamma_q, gamma_k, empty, empty,
                        pos0, n_q_heads, n_kv_heads, theta, eps, rows=rows)


# ----------------------------------------------------------------------------
# the decoder layer around the path (the base models of section 5.1 are
# Qwen3 decoder stacks; the paper times prefill up to the greedy first token,
# appendix A.2).  The layer structure is Qwen3's: pre-norm RMSNorm, attention,
# residual, RMSNorm, SwiGLU MLP, residual; a final RMSNorm and the LM head.
# ----------------------------------------------------------------------------

def silu(z: np.ndarray) -> np.ndarray:
    """silu(z) = z / (1 + e^-z) (the gate activation of the SwiGLU MLP)."""
    z = np.asarray(z, np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def linear(x: np.ndarray, w: np.ndarray, residual: Optional[np.ndarray] = None) -> np.ndarray:
    """x W^T (+ residual): o_proj and down_proj, with the residual connection."""
    out = np.asarray(x, np.float64) @ np.asarray(w, np.float64).T
    return out if residual is None else out + np.asarray(residual, np.float64)


def swiglu(x: np.ndarray, w_gate: np.ndarray, w_up: np.ndarray) -> np.ndarray:
    """silu(x W_gate^T) * (x W_up^T): the MLP's gated hidden activation."""
    return silu(linear(x, w_gate)) * linear(x, w_up)


def decoder_layer(h, w: Dict[str, np.ndarray], k_art, v_art, pos0: int, n_q_heads: int,
                  n_kv_heads: int, theta: float, eps: float, scale: float = 0.0) -> Dict[str, np.ndarray]:
    """One decoder layer around the adapted attention of :func:`suffix_layer`.

    h [S][H] is the residual stream of the suffix tokens; w holds wq, wk, wv,
    a, b (or None), gamma_q, gamma_k (the path), gamma_in, wo, gamma_post,
    w_gate, w_up, w_down:
        x  = RMSNorm(h) * gamma_in
        o  = attention of the suffix over the artifacts (suffix_layer on x)
        h1 = h + o W_o^T
        h2 = h1 + down(silu(x2 W_gate^T) * (x2 W_up^T)),  x2 = RMSNorm(h1) * gamma_post
    Returns h2 and the pieces (x, o, h1, x2, mlp hidden, and the suffix K/V).
    """
    h = np.asarray(h, np.float64)
    S = h.shape[0]
    x = rms_norm_heads(h, w["gamma_in"], eps)
    att = suffix_layer(x, w["wq"], w["wk"], w["wv"], w.get("a"), w.get("b"), scale, w["gamma_q"],
                       w["gamma_k"], k_art, v_art, pos0, n_q_heads, n_kv_heads, theta, eps)
    o = att["o"].reshape(S, -1)
    h1 = linear(o, w["wo"], h)
    x2 = rms_norm_heads(h1, w["gamma_post"], eps)
    g = swiglu(x2, w["w_gate"], w["w_up"])
    h2 = linear(g, w["w_down"], h1)
    return {"x": x, "o": o, "h1": h1, "x2": x2, "mlp": g, "h": h2, "k_hat": att["k_hat"], "v": att["v"]}


def first_token(h_last: np.ndarray, gamma_final: np.ndarray, w_lm: np.ndarray, eps: float):
    """Greedy first token of each request: argmax over the vocabulary of
    RMSNorm(h_last) * gamma_final W_lm^T (smallest index on ties).  h_last
    [n][H] holds the last suffix token of each request.  Returns (ids, logits)."""
    logits = linear(rms_norm_heads(h_last, gamma_final, eps), w_lm)
    return np.argmax(logits, axis=-1), logits


# ----------------------------------------------------------------------------
# interleaved online spans (appendix A.3, the request layouts: system text,
# headers, separators and the question sit between and around the cached
# artifacts and are computed online; appendix A.5: attention with the causal
# mask over the assembled context and its position ids)
# ----------------------------------------------------------------------------

def interleaved_layer(segments, x, wq, wk, wv, a, b, scale, gamma_q, gamma_k, art_k, art_v,
                      n_q_heads: int, n_kv_heads: int, theta: float, eps: float) -> Dict[str, np.ndarray]:
    """One layer of online prefill for a prompt that interleaves cached
    artifacts with online spans.

    segments: the prompt in order; an entry >= 0 is a cached artifact id
    (art_k[id], art_v[id]: [L][Hkv][d], frozen, normalised and rotated at
    their own local positions), an entry -n < 0 is an online span of n tokens.
    x [n_online][H]: the hidden states of all online tokens, spans in order.
    An online token at assembled position p (its offset in the whole prompt)
    gets the adapted query and unadapted key/value projections, the per-head
    norms and RoPE at position p, and attends to every assembled key at a
    position <= p (cached keys as stored, online keys as just computed).
    Returns o [n_online][Hq][d], q_hat, k_hat, v, the position of every online
    token and the assembled keys/values [n_pos][Hkv][d].
    """
    x = np.asarray(x, np.float64)
    d = np.asarray(gamma_q).shape[0]
    pos = []
    p = 0
    for s in segments:
        if s >= 0:
            p += np.asarray(art_k[s]).shape[0]
        else:
            pos.extend(range(p, p - s))
            p -= s
    pos = np.asarray(pos, dtype=np.int64)
    n = x.shape[0]
    assert n == len(pos), "x must hold one row per online token"
    q = qproj_lora(x, wq, a, b, scale).reshape(n, n_q_heads, d)
    k = qproj_lora(x, wk).reshape(n, n_kv_heads, d)
    v = qproj_lora(x, wv).reshape(n, n_kv_heads, d)
    q_hat = rope(rms_norm_heads(q, gamma_q, eps), pos, theta)
    k_hat = rope(rms_norm_heads(k, gamma_k, eps), pos, theta)
    keys, vals = [], []
    t = 0
    for s in segments:
        if s >= 0:
            keys.append(np.asarray(art_k[s], np.float64))
            vals.append(np.asarray(art_v[s], np.float64))
        else:
            keys.append(k_hat[t:t - s])
            vals.append(v[t:t - s])
            t -= s
    keys = np.concatenate(keys) if keys else np.zeros((0, n_kv_heads, d))
    vals = np.concatenate(vals) if vals else np.zeros((0, n_kv_heads, d))
    G = n_q_heads // n_kv_heads
    visible = np.arange(keys.shape[0])[None, :] <= pos[:, None]
    o = np.empty((n, n_q_heads, d))
    for h in range(n_q_heads):
        z = (q_hat[:, h, :] @ keys[:, h // G, :].T) / math.sqrt(d)
        z = np.where(visible, z, -np.inf)
        e = np.exp(z - z.max(axis=1, keepdims=True))
        o[:, h, :] = (e / e.sum(axis=1, keepdims=True)) @ vals[:, h // G, :]
    return {"o": o, "q_hat": q_hat, "k_hat": k_hat, "v": v, "pos": pos, "keys": keys, "vals": vals}


def block_table_segments(artifact_lengths: Sequence[int], requests: Sequence[Sequence[int]], page_tokens: int):
    """Logical block table of a batch whose prompts interleave cached
    artifacts with online spans (appendix A.3: cached KV is put together in
    the original prompt order; the text between and around the artifacts is
    computed online).

    Each request is a list of segments: an entry >= 0 is an artifact id, an
    entry -n < 0 an online span of n tokens.  Request r owns rows [cu_ctx[r],
    cu_ctx[r+1]) holding its whole prompt in order: artifact pages where the
    artifacts sit, and rows left for the online spans where they sit.

    Returns (entries, cu_ctx, spans): entries as in :func:`block_table`
    (artifact_id, page_index, n_valid, request, dst_row); spans an int64 array
    of rows (request, offset of the span in its request, length), in request
    and prompt order.
    """
    entries, spans = [], []
    cu_ctx = [0]
    for r, segs in enumerate(requests):
        base = cu_ctx[-1]
        off = 0
        for s in segs:
            if s >= 0:
                for p, nv in enumerate(page_valid_counts(int(artifact_lengths[s]), page_tokens)):
                    entries.append((int(s), p, nv, r, base + off))
                    off += nv
            else:
                spans.append((r, off, -int(s)))
                off += -int(s)
        cu_ctx.append(base + off)
    return (np.asarray(entries, dtype=np.int64).reshape(-1, 5), np.asarray(cu_ctx, dtype=np.int64),
            np.asarray(spans, dtype=np.int64).reshape(-1, 3))


def merge_lora(w: np.ndarray, a: np.ndarray, b: np.ndarray, scale: float, lora_cols: int) -> np.ndarray:
    """Deployment form of the adapter (appendix A.5: the update is merged into
    the query projection, W_Q <- W_Q + (alpha / r) B A): rows below lora_cols
    get scale * B A added, the other rows (keys, values) are unchanged."""
    w = np.array(w, np.float64)
    w[:lora_cols] += scale * (np.asarray(b, np.float64) @ np.asarray(a, np.float64))
    return w
