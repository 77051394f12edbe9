"""Pins of the oracle's decoder layer and stack (the layer around the
suffix path) against things other than the oracle itself.

The paper names its base models (Qwen3-4B / Qwen3-8B, section 5.1) but says
nothing of their layer structure; the oracle's composition (pre-norm
RMSNorm, attention with per-head q/k RMSNorm and RoPE, o_proj + residual,
RMSNorm, SwiGLU MLP + residual, final RMSNorm, LM head) is Qwen3's.  Three
pins fix it:

* the published Qwen3 implementation of the transformers library, run in
  float64 on the CPU with random weights, a pre-filled cache that plays the
  artifact keys/values and the suffix at its assembled positions: it fixes
  norm placement, the roles of gamma_in / gamma_post / gamma_q / gamma_k,
  the residual connections, the gate/up order and the merged adapter
  (appendix A.5 serves with W_q + (alpha/r) B A);
* a brute-force per-token loop in plain Python sums on tiny shapes (<= 1e-12);
* planted mistakes (no input norm, post-attention norm taken from h instead
  of h1, gamma_in and gamma_post swapped, a dropped residual) that the stack
  bar used by the GPU stack test must reject, while it accepts the bf16
  storage the GPU path does at every stored intermediate.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from synthdata.workloads import ModelShape, Request, custom_workload
from tests._tol import assert_stack_close


# ----------------------------------------------------------------------------
# the transformers Qwen3 implementation in float64
# ----------------------------------------------------------------------------

def _qwen3_case(seed=41, H=64, I=96, Hq=8, Hkv=2, d=16, V=50, NL=2, S=6, L=9, rank=4, scale=2.0):
    rng = np.random.default_rng(seed)
    f = lambda *shape, std=1.0: rng.standard_normal(shape) * std
    u = lambda *shape: rng.uniform(0.5, 1.5, shape)
    layers = []
    for _ in range(NL):
        layers.append({"wq": f(Hq * d, H, std=H ** -0.5), "wk": f(Hkv * d, H, std=H ** -0.5),
                       "wv": f(Hkv * d, H, std=H ** -0.5), "a": f(rank, H, std=H ** -0.5),
                       "b": f(Hq * d, rank, std=0.3), "gamma_q": u(d), "gamma_k": u(d), "gamma_in": u(H),
                       "wo": f(H, Hq * d, std=(Hq * d) ** -0.5), "gamma_post": u(H),
                       "w_gate": f(I, H, std=H ** -0.5), "w_up": f(I, H, std=H ** -0.5),
                       "w_down": f(H, I, std=I ** -0.5)})
    art = [(f(L, Hkv, d), f(L, Hkv, d)) for _ in range(NL)]
    top = {"embed": f(V, H), "gamma_final": u(H), "w_lm": f(V, H, std=H ** -0.5)}
    dims = dict(H=H, I=I, Hq=Hq, Hkv=Hkv, d=d, V=V, NL=NL, S=S, L=L, scale=scale)
    return layers, art, top, dims, rng


def _hf_forward(layers, art, top, dims, tokens, pos0):
    transformers = pytest.importorskip("transformers")
    from transformers import Qwen3Config, Qwen3ForCausalLM
    from transformers.cache_utils import DynamicCache

    D = dims
    cfg = Qwen3Config(vocab_size=D["V"], hidden_size=D["H"], intermediate_size=D["I"],
                      num_hidden_layers=D["NL"], num_attention_heads=D["Hq"], num_key_value_heads=D["Hkv"],
                      head_dim=D["d"], rope_theta=1e6, rms_norm_eps=1e-6, max_position_embeddings=4096,
                      tie_word_embeddings=False, attn_implementation="eager")
    model = Qwen3ForCausalLM(cfg).to(torch.float64).eval()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))
    with torch.no_grad():
        model.model.embed_tokens.weight.copy_(t(top["embed"]))
        model.model.norm.weight.copy_(t(top["gamma_final"]))
        model.lm_head.weight.copy_(t(top["w_lm"]))
        for l, w in enumerate(layers):
            m = model.model.layers[l]
            # the deployment form of the adapter: merged into the query projection
            m.self_attn.q_proj.weight.copy_(t(w["wq"] + D["scale"] * (w["b"] @ w["a"])))
            m.self_attn.k_proj.weight.copy_(t(w["wk"]))
            m.self_attn.v_proj.weight.copy_(t(w["wv"]))
            m.self_attn.o_proj.weight.copy_(t(w["wo"]))
            m.self_attn.q_norm.weight.copy_(t(w["gamma_q"]))
            m.self_attn.k_norm.weight.copy_(t(w["gamma_k"]))
            m.input_layernorm.weight.copy_(t(w["gamma_in"]))
            m.post_attention_layernorm.weight.copy_(t(w["gamma_post"]))
            m.mlp.gate_proj.weight.copy_(t(w["w_gate"]))
            m.mlp.up_proj.weight.copy_(t(w["w_up"]))
            m.mlp.down_proj.weight.copy_(t(w["w_down"]))
        cache = DynamicCache(config=cfg)
        for l, (ka, va) in enumerate(art):
            # the cache holds keys after k-norm and RoPE, as the stored artifacts do
            cache.update(t(ka).permute(1, 0, 2)[None], t(va).permute(1, 0, 2)[None], l)
        S = len(tokens)
        pos = torch.arange(pos0, pos0 + S)[None]
        out = model(input_ids=torch.as_tensor(np.asarray(tokens))[None], past_key_values=cache, position_ids=pos,
                    use_cache=True, output_hidden_states=True)
    hs = [h[0].numpy() for h in out.hidden_states]
    # the suffix keys/values the model appended to each layer's cache
    new_kv = []
    for l in range(D["NL"]):
        k_all, v_all = cache.layers[l].keys, cache.layers[l].values
        new_kv.append((k_all[0, :, D["L"]:].permute(1, 0, 2).numpy(), v_all[0, :, D["L"]:].permute(1, 0, 2).numpy()))
    return hs, out.logits[0].numpy(), new_kv


def _oracle_stack(layers, art, top, dims, tokens, pos0):
    D = dims
    h = top["embed"][np.asarray(tokens)]
    outs = []
    for l, w in enumerate(layers):
        r = oracle.decoder_layer(h, w, art[l][0], art[l][1], pos0, D["Hq"], D["Hkv"], 1e6, 1e-6, D["scale"])
        outs.append(r)
        h = r["h"]
    logits = oracle.linear(oracle.rms_norm_heads(h, top["gamma_final"], 1e-6), top["w_lm"])
    return outs, logits


# transformers evaluates RMSNorm and the rotary angles in float32 even in a
# float64 model; 1e-5 of the largest magnitude covers that, while every
# composition mistake tried below moves the output by far more.
HF_REL = 1e-5


def _rel(a, b):
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b))) / np.max(np.abs(np.asarray(b))))


@pytest.mark.parametrize("pos_shift", [0, 13])
def test_decoder_stack_matches_transformers_qwen3(pos_shift):
    layers, art, top, D, rng = _qwen3_case()
    tokens = rng.integers(0, D["V"], D["S"])
    pos0 = D["L"] + pos_shift
    hs, logits_hf, new_kv = _hf_forward(layers, art, top, D, tokens, pos0)
    outs, logits = _oracle_stack(layers, art, top, D, tokens, pos0)
    # hidden_states: the embeddings, the output of every layer but the last,
    # then the last layer's output after the final norm
    assert _rel(outs[0]["h"], hs[1]) <= HF_REL
    assert _rel(oracle.rms_norm_heads(outs[-1]["h"], top["gamma_final"], 1e-6), hs[-1]) <= HF_REL
    assert _rel(logits, logits_hf) <= HF_REL
    # the suffix keys (normed + rotated at the assembled positions) and values
    for l in range(D["NL"]):
        assert _rel(outs[l]["k_hat"], new_kv[l][0]) <= HF_REL
        assert _rel(outs[l]["v"], new_kv[l][1]) <= HF_REL
    # the greedy first token of the last suffix row
    ids, _ = oracle.first_token(outs[-1]["h"][-1:], top["gamma_final"], top["w_lm"], 1e-6)
    assert int(ids[0]) == int(np.argmax(logits_hf[-1]))


def _variant_layer(h, w, k_art, v_art, pos0, D, mistake=None, rnd=None):
    """A decoder layer recomposed from the oracle's primitives, with one
    planted mistake and optional storage rounding (rnd) of every intermediate
    the GPU path stores in bf16."""
    r = rnd or (lambda t: t)
    Hq, Hkv, eps, th = D["Hq"], D["Hkv"], 1e-6, 1e6
    g_in, g_post = (w["gamma_post"], w["gamma_in"]) if mistake == "swap_gammas" else (w["gamma_in"], w["gamma_post"])
    x = r(h * g_in if mistake == "no_input_norm" else oracle.rms_norm_heads(h, g_in, eps))
    S, d = h.shape[0], w["gamma_q"].shape[0]
    q = r(oracle.qproj_lora(x, w["wq"], w.get("a"), w.get("b"), D["scale"])).reshape(S, Hq, d)
    k = r(oracle.qproj_lora(x, w["wk"])).reshape(S, Hkv, d)
    v = r(oracle.qproj_lora(x, w["wv"])).reshape(S, Hkv, d)
    pos = pos0 + np.arange(S)
    q_hat = r(oracle.rope(oracle.rms_norm_heads(q, w["gamma_q"], eps), pos, th))
    k_hat = r(oracle.rope(oracle.rms_norm_heads(k, w["gamma_k"], eps), pos, th))
    o = r(oracle.attention(q_hat, np.concatenate([k_art, k_hat]), np.concatenate([v_art, v]), k_art.shape[0]))
    o = o.reshape(S, -1)
    h1 = r(oracle.linear(o, w["wo"], None if mistake == "drop_attn_residual" else h))
    x2 = r(oracle.rms_norm_heads(h if mistake == "post_norm_from_h" else h1, g_post, eps))
    g = r(oracle.swiglu(x2, w["w_gate"], w["w_up"]))
    h2 = r(oracle.linear(g, w["w_down"], None if mistake == "drop_mlp_residual" else h1))
    return {"h": h2, "k_hat": k_hat, "v": v}


def test_variant_layer_without_mistake_is_the_oracle_layer():
    layers, art, top, D, rng = _qwen3_case()
    h = top["embed"][rng.integers(0, D["V"], D["S"])]
    w = layers[0]
    ref = oracle.decoder_layer(h, w, art[0][0], art[0][1], 11, D["Hq"], D["Hkv"], 1e6, 1e-6, D["scale"])
    got = _variant_layer(h, w, art[0][0], art[0][1], 11, D)
    assert np.max(np.abs(got["h"] - ref["h"])) <= 1e-12 * np.max(np.abs(ref["h"]))


@pytest.mark.parametrize("mistake", ["no_input_norm", "post_norm_from_h", "swap_gammas", "drop_attn_residual",
                                     "drop_mlp_residual"])
def test_transformers_pin_rejects_composition_mistakes(mistake):
    # the library pin is tight enough to see every plausible composition mistake
    layers, art, top, D, rng = _qwen3_case()
    tokens = rng.integers(0, D["V"], D["S"])
    hs, _, _ = _hf_forward(layers, art, top, D, tokens, D["L"])
    h = top["embed"][np.asarray(tokens)]
    bad = _variant_layer(h, layers[0], art[0][0], art[0][1], D["L"], D, mistake)
    assert _rel(bad["h"], hs[1]) > 100 * HF_REL


# ----------------------------------------------------------------------------
# brute force: one decoder layer in plain Python sums
# ----------------------------------------------------------------------------

def _brute_layer(h, w, k_art, v_art, pos0, Hq, Hkv, theta, eps, scale):
    S, H = len(h), len(h[0])
    d = len(w["gamma_q"])
    G = Hq // Hkv
    rank = len(w["a"])

    def norm(row, gamma):
        ms = sum(t * t for t in row) / len(row)
        return [gamma[i] * row[i] / math.sqrt(ms + eps) for i in range(len(row))]

    def matvec(W, row):
        return [sum(W[o][i] * row[i] for i in range(len(row))) for o in range(len(W))]

    def rot(vec, p):
        half = d // 2
        out = [0.0] * d
        for j in range(half):
            ang = p * theta ** (-2.0 * j / d)
            c, s_ = math.cos(ang), math.sin(ang)
            out[j] = vec[j] * c - vec[j + half] * s_
            out[j + half] = vec[j + half] * c + vec[j] * s_
        return out

    keys = [[list(k_art[t][g]) for g in range(Hkv)] for t in range(len(k_art))]
    vals = [[list(v_art[t][g]) for g in range(Hkv)] for t in range(len(v_art))]
    L = len(keys)
    xs, qs = [], []
    for i in range(S):
        x = norm(h[i], w["gamma_in"])
        xs.append(x)
        q = matvec(w["wq"], x)
        down = matvec(w["a"], x)
        for o in range(len(q)):
            q[o] += scale * sum(w["b"][o][j] * down[j] for j in range(rank))
        k = matvec(w["wk"], x)
        v = matvec(w["wv"], x)
        p = pos0 + i
        qs.append([rot(norm(q[hh * d:(hh + 1) * d], w["gamma_q"]), p) for hh in range(Hq)])
        keys.append([rot(norm(k[g * d:(g + 1) * d], w["gamma_k"]), p) for g in range(Hkv)])
        vals.append([v[g * d:(g + 1) * d] for g in range(Hkv)])
    out = []
    for i in range(S):
        o = []
        for hh in range(Hq):
            g = hh // G
            z = [sum(qs[i][hh][e] * keys[j][g][e] for e in range(d)) / math.sqrt(d) for j in range(L + i + 1)]
            m = max(z)
            ex = [math.exp(t - m) for t in z]
            den = sum(ex)
            o += [sum(ex[j] * vals[j][g][e] for j in range(len(z))) / den for e in range(d)]
        h1 = [h[i][c] + sum(w["wo"][c][e] * o[e] for e in range(len(o))) for c in range(H)]
        x2 = norm(h1, w["gamma_post"])
        gate = matvec(w["w_gate"], x2)
        up = matvec(w["w_up"], x2)
        act = [gate[j] / (1.0 + math.exp(-gate[j])) * up[j] for j in range(len(gate))]
        out.append([h1[c] + sum(w["w_down"][c][j] * act[j] for j in range(len(act))) for c in range(H)])
    return out


def test_decoder_layer_brute_force():
    layers, art, top, D, rng = _qwen3_case(seed=43, H=12, I=10, Hq=4, Hkv=2, d=8, S=4, L=3, rank=2)
    w = layers[0]
    h = rng.standard_normal((D["S"], D["H"])) * 1.7
    pos0 = 5
    ref = oracle.decoder_layer(h, w, art[0][0], art[0][1], pos0, D["Hq"], D["Hkv"], 1e6, 1e-6, D["scale"])
    wl = {k: v.tolist() for k, v in w.items()}
    got = np.array(_brute_layer(h.tolist(), wl, art[0][0].tolist(), art[0][1].tolist(), pos0, D["Hq"], D["Hkv"],
                                1e6, 1e-6, D["scale"]))
    assert np.max(np.abs(got - ref["h"])) <= 1e-12 * max(1.0, np.max(np.abs(ref["h"])))


# ----------------------------------------------------------------------------
# the stack bar against planted mistakes (the GPU stack test's shapes)
# ----------------------------------------------------------------------------

def _stack_bar_case():
    # the shapes and seeds of the GPU two-layer stack test
    shape = ModelShape(hidden=256)
    wl = custom_workload("stack", 92, shape, [40, 17, 64], [Request((0, 1), 20), Request((2, 0), 33)],
                         n_layers=2, rank=16, scale=1.0, gamma="uniform")
    return wl, 512, 1024


def _stack_run(wl, I, V, mistake=None, bf16=False):
    s = wl.shape
    rnd = (lambda t: oracle.decode_bf16(sd.f32_to_bf16_bits(np.asarray(t, np.float32)))) if bf16 else None
    D = {"Hq": s.n_q_heads, "Hkv": s.n_kv_heads, "scale": wl.scale}
    ws = []
    for l in range(2):
        w = {k: oracle.decode_bf16(v) for k, v in sd.layer_weights(wl, l).items()}
        w.update({k: oracle.decode_bf16(v) for k, v in sd.decoder_weights(wl, l, I).items()})
        ws.append(w)
    emb = oracle.decode_bf16(sd.lm_weights(wl, V)["embed"])
    hs = []
    for r, req in enumerate(wl.requests):
        h = emb[sd.suffix_tokens(wl, r, V)]
        for l in range(2):
            kv = [sd.artifact_kv(wl, a, l) for a in req.artifact_ids]
            ka = np.concatenate([oracle.decode_bf16(k) for k, _ in kv])
            va = np.concatenate([oracle.decode_bf16(v) for _, v in kv])
            h = _variant_layer(h, ws[l], ka, va, wl.pos0(req), D, mistake, rnd)["h"]
        hs.append(h)
    return np.concatenate(hs)


def test_stack_bar_accepts_bf16_storage_and_rejects_composition_mistakes():
    wl, I, V = _stack_bar_case()
    ref = _stack_run(wl, I, V)
    # what the GPU path does: every stored intermediate rounded to bf16
    assert_stack_close(_stack_run(wl, I, V, bf16=True), ref, 2)
    for mistake in ["no_input_norm", "post_norm_from_h", "swap_gammas", "drop_attn_residual", "drop_mlp_residual"]:
        bad = _stack_run(wl, I, V, mistake=mistake, bf16=True)
        with pytest.raises(AssertionError):
            assert_stack_close(bad, ref, 2, mistake)
