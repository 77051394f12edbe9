"""Synthetic workloads shaped like the paper's Qwen3-4B / Qwen3-8B settings.

The paper evaluates on seven public benchmarks that are not available here; the
workloads below stand in for them with the shapes the method sees: a handful of
cached artifacts per request (the paper's requests hold one to eight), a suffix
of online tokens, and Qwen3 attention geometry (32 query heads, 8 KV heads,
head dimension 128, rotary base 1e6).

Every tensor is drawn from its own PCG64 stream keyed by
``(workload index, purpose, ids...)``, so any single layer, artifact or request
can be regenerated alone.  Values are drawn in float32, scaled by the stated
standard deviation and stored as bfloat16 bits.

Artifact keys: the cache holds keys that were rotated at their local positions
when the artifact was encoded.  Each rotation acts on (j, j+64) pairs as an
orthogonal 2x2 matrix, and a pair of independent standard normals has a
rotation-invariant law, so i.i.d. N(0, 1) draws already follow the law of
"N(0, 1) keys rotated at local positions".  The keys are therefore drawn
directly; no rotation happens here.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

from .bf16 import f32_to_bf16_bits

# purposes (second seed word)
_STRUCT, _WEIGHTS, _ARTIFACT, _SUFFIX, _PREFILL, _GAMMA, _DECODER, _LMHEAD, _TOKENS = 0, 1, 2, 3, 4, 5, 6, 7, 8


@dataclass(frozen=True)
class ModelShape:
    hidden: int
    n_q_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6
    page_tokens: int = 16

    @property
    def q_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def kv_dim(self) -> int:
        return self.n_kv_heads * self.head_dim


@dataclass(frozen=True)
class Request:
    artifact_ids: Tuple[int, ...]
    suffix_len: int
    pos0: Optional[int] = None  # None: first suffix position = total artifact length


@dataclass(frozen=True)
class Workload:
    name: str
    index: int  # seed root
    shape: ModelShape
    n_layers: int
    rank: int
    scale: float
    artifact_lengths: Tuple[int, ...]
    requests: Tuple[Request, ...]
    w_std: float = 0.02
    b_std: float = 0.01
    gamma: str = "ones"  # "ones" | "uniform" (U(0.5, 1.5)) | "sharp" (gamma_q = 8)

    def art_len(self, req: Request) -> int:
        return int(sum(self.artifact_lengths[a] for a in req.artifact_ids))

    def pos0(self, req: Request) -> int:
        return self.art_len(req) if req.pos0 is None else int(req.pos0)

    @property
    def a_std(self) -> float:
        return 1.0 / float(np.sqrt(self.shape.hidden))

    @property
    def total_suffix(self) -> int:
        return int(sum(r.suffix_len for r in self.requests))


def _rng(*words: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(w) for w in words])))


def _normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x)


# ----------------------------------------------------------------------------
# the five configurations
# ----------------------------------------------------------------------------

QWEN3_4B = ModelShape(hidden=2560)
QWEN3_8B = ModelShape(hidden=4096)


def _c1() -> Workload:
    # 1 layer, 4B shapes, two 256-token artifacts, 64-token suffix at 512..575, rank 8.
    return Workload("c1_qwen3_4b_1layer_2x256_s64_r8", 1, QWEN3_4B, 1, 8, 2.0,
                    (256, 256), (Request((0, 1), 64),))


def _c2() -> Workload:
    # 36 layers, 4B shapes, eight 1024-token artifacts, 256-token suffix, rank 16.
    return Workload("c2_qwen3_4b_36layer_8x1024_s256_r16", 2, QWEN3_4B, 36, 16, 1.0,
                    (1024,) * 8, (Request(tuple(range(8)), 256),))


def _c3() -> Workload:
    # 36 layers, 8B shapes, sixteen artifacts of U{512..2048} tokens in seeded random
    # order, 512-token suffix, rank 16.
    rng = _rng(3, _STRUCT)
    lengths = tuple(int(v) for v in rng.integers(512, 2049, size=16))
    order = tuple(int(v) for v in rng.permutation(16))
    return Workload("c3_qwen3_8b_36layer_16xU512_2048_s512_r16", 3, QWEN3_8B, 36, 16, 1.0,
                    lengths, (Request(order, 512),))


def _zipf_draw(rng: np.random.Generator, weights: np.ndarray, n: int) -> List[int]:
    """n distinct indices by sequential weighted sampling without replacement."""
    w = weights.astype(np.float64).copy()
    out = []
    for _ in range(n):
        p = w / w.sum()
        k = int(rng.choice(len(w), p=p))
        out.append(k)
        w[k] = 0.0
    return out


def _c4() -> Workload:
    # 1 layer, 8B shapes; a pool of 64 artifacts of U{256..1536} tokens in 16-token pages;
    # 16 requests, each drawing 4..12 distinct artifacts with Zipf(1.1) popularity in
    # random order, suffix U{64..512}.  The LoRA rank is not given for this batch; 16 is
    # used, as in the other 8B configurations.
    rng = _rng(4, _STRUCT)
    lengths = tuple(int(v) for v in rng.integers(256, 1537, size=64))
    rank_to_artifact = rng.permutation(64)
    zipf = 1.0 / np.arange(1, 65, dtype=np.float64) ** 1.1
    reqs = []
    for _ in range(16):
        n = int(rng.integers(4, 13))
        ranks = _zipf_draw(rng, zipf, n)
        ids = [int(rank_to_artifact[k]) for k in ranks]
        ids = [ids[i] for i in rng.permutation(n)]
        s = int(rng.integers(64, 513))
        reqs.append(Request(tuple(ids), s))
    return Workload("c4_qwen3_8b_1layer_batch16_pool64_zipf", 4, QWEN3_8B, 1, 16, 1.0,
                    lengths, tuple(reqs))


def _c5() -> Workload:
    # 36 layers, 8B shapes, thirty-two 1024-token artifacts, 1024-token suffix, rank 32.
    return Workload("c5_qwen3_8b_36layer_32x1024_s1024_r32", 5, QWEN3_8B, 36, 32, 0.5,
                    (1024,) * 32, (Request(tuple(range(32)), 1024),))


WORKLOADS = {"c1": _c1, "c2": _c2, "c3": _c3, "c4": _c4, "c5": _c5}


def make_workload(name: str, **overrides) -> Workload:
    """Build one of c1..c5, optionally overriding fields (e.g. n_layers, gamma, scale)."""
    wl = WORKLOADS[name]()
    if overrides:
        d = {f: getattr(wl, f) for f in wl.__dataclass_fields__}
        d.update(overrides)
        wl = Workload(**d)
    return wl


def custom_workload(name: str, index: int, shape: ModelShape, artifact_lengths, requests,
                    n_layers: int = 1, rank: int = 8, scale: float = 1.0, **kw) -> Workload:
    """A workload of arbitrary (e.g. tiny) shape, for tests."""
    return Workload(name, index, shape, n_layers, rank, scale, tuple(int(v) for v in artifact_lengths),
                    tuple(requests), **kw)


# ----------------------------------------------------------------------------
# draws
# ----------------------------------------------------------------------------

def layer_weights(wl: Workload, layer: int) -> Dict[str, np.ndarray]:
    """bf16 bits of one layer's weights.

    wq [q_dim][hidden], wk/wv [kv_dim][hidden] ~ N(0, w_std);  A [rank][hidden] ~
    N(0, 1/sqrt(hidden));  B [q_dim][rank] ~ N(0, b_std);  gamma_q, gamma_k [head_dim].
    """
    s, H = wl.shape, wl.shape.hidden
    out = {
        "wq": _normal_bf16(_rng(wl.index, _WEIGHTS, layer, 0), (s.q_dim, H), wl.w_std),
        "wk": _normal_bf16(_rng(wl.index, _WEIGHTS, layer, 1), (s.kv_dim, H), wl.w_std),
        "wv": _normal_bf16(_rng(wl.index, _WEIGHTS, layer, 2), (s.kv_dim, H), wl.w_std),
        "a": _normal_bf16(_rng(wl.index, _WEIGHTS, layer, 3), (wl.rank, H), wl.a_std),
        "b": _normal_bf16(_rng(wl.index, _WEIGHTS, layer, 4), (s.q_dim, wl.rank), wl.b_std),
    }
    d = s.head_dim
    if wl.gamma == "ones":
        gq = np.ones(d, np.float32)
        gk = np.ones(d, np.float32)
    elif wl.gamma == "uniform":
        r = _rng(wl.index, _GAMMA, layer)
        gq = r.uniform(0.5, 1.5, size=d).astype(np.float32)
        gk = r.uniform(0.5, 1.5, size=d).astype(np.float32)
    elif wl.gamma == "sharp":
        r = _rng(wl.index, _GAMMA, layer)
        gq = np.full(d, 8.0, np.float32)
        gk = r.uniform(0.5, 1.5, size=d).astype(np.float32)
    else:
        raise ValueError(wl.gamma)
    out["gamma_q"] = f32_to_bf16_bits(gq)
    out["gamma_k"] = f32_to_bf16_bits(gk)
    return out


def artifact_kv(wl: Workload, artifact_id: int, layer: int) -> Tuple[np.ndarray, np.ndarray]:
    """bf16 bits of one artifact's cached K and V for one layer: [L_a][n_kv][head_dim] each."""
    s = wl.shape
    L = wl.artifact_lengths[artifact_id]
    shp = (L, s.n_kv_heads, s.head_dim)
    k = _normal_bf16(_rng(wl.index, _ARTIFACT, artifact_id, layer, 0), shp, 1.0)
    v = _normal_bf16(_rng(wl.index, _ARTIFACT, artifact_id, layer, 1), shp, 1.0)
    return k, v


def suffix_hidden(wl: Workload, request_index: int, layer: int) -> np.ndarray:
    """bf16 bits of one request's suffix hidden states for one layer: [S][hidden] ~ N(0, 1)."""
    S = wl.requests[request_index].suffix_len
    return _normal_bf16(_rng(wl.index, _SUFFIX, request_index, layer), (S, wl.shape.hidden), 1.0)


def prefill_hidden(wl: Workload, request_index: int, layer: int) -> np.ndarray:
    """bf16 bits of the hidden states a full-context prefill of the whole request
    (artifacts and suffix, L_art + S tokens) would see at one layer, ~ N(0, 1)."""
    req = wl.requests[request_index]
    n = wl.art_len(req) + req.suffix_len
    return _normal_bf16(_rng(wl.index, _PREFILL, request_index, layer), (n, wl.shape.hidden), 1.0)


# ----------------------------------------------------------------------------
# the decoder layer around the path (o_proj, MLP, norms, embedding, LM head)
# ----------------------------------------------------------------------------

def _gamma(wl: Workload, n: int, *words: int) -> np.ndarray:
    if wl.gamma == "ones":
        return f32_to_bf16_bits(np.ones(n, np.float32))
    return f32_to_bf16_bits(_rng(wl.index, _GAMMA, *words).uniform(0.5, 1.5, size=n).astype(np.float32))


def decoder_weights(wl: Workload, layer: int, intermediate: int) -> Dict[str, np.ndarray]:
    """bf16 bits of one layer's weights outside the attention path.

    wo [hidden][q_dim], w_gate / w_up [intermediate][hidden], w_down
    [hidden][intermediate], each ~ N(0, 1/sqrt(fan_in)) (N(0, 0.02) at the 4B
    hidden size, and unit-scale activations at any test size); gamma_in,
    gamma_post [hidden] as the workload's gamma setting.
    """
    s, H, I = wl.shape, wl.shape.hidden, int(intermediate)
    d = lambda k, shape, fan: _normal_bf16(_rng(wl.index, _DECODER, layer, k), shape, 1.0 / float(np.sqrt(fan)))
    return {"wo": d(0, (H, s.q_dim), s.q_dim), "w_gate": d(1, (I, H), H), "w_up": d(2, (I, H), H),
            "w_down": d(3, (H, I), I), "gamma_in": _gamma(wl, H, 1000 + layer, 0),
            "gamma_post": _gamma(wl, H, 1000 + layer, 1)}


def lm_weights(wl: Workload, vocab: int) -> Dict[str, np.ndarray]:
    """bf16 bits of the embedding table [vocab][hidden] ~ N(0, 0.25), the LM
    head [vocab][hidden] ~ N(0, 1/sqrt(hidden)) and the final norm's gamma
    [hidden].  The embedding rows are deliberately not of unit RMS: a decoder
    layer's input RMSNorm then rescales them by about 4, so a stack that
    skipped that norm would be visibly wrong (with unit-RMS rows the norm is
    nearly the identity)."""
    H = wl.shape.hidden
    return {"embed": _normal_bf16(_rng(wl.index, _LMHEAD, 0), (vocab, H), 0.25),
            "w_lm": _normal_bf16(_rng(wl.index, _LMHEAD, 1), (vocab, H), 1.0 / float(np.sqrt(H))),
            "gamma_final": _gamma(wl, H, 2000)}


def suffix_tokens(wl: Workload, request_index: int, vocab: int) -> np.ndarray:
    """Token ids of one request's suffix, uniform over the vocabulary (int32)."""
    S = wl.requests[request_index].suffix_len
    return _rng(wl.index, _TOKENS, request_index).integers(0, vocab, size=S).astype(np.int32)
