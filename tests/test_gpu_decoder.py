"""GPU parity of the decoder layer around the suffix path (embedding rows,
RMSNorm, o_proj / down_proj with the residual, the SwiGLU gate/up GEMM, the
LM head with the greedy pick, and a two-layer stack chained through them,
prefill and decode) against the fp64 oracle, through the C ABI.  The oracle
only ever takes the seeded inputs.

Bars: the embedding lookup bit-exact; bf16-stored outputs of one step within
the intermediate bar (max|err| <= 1e-2 max|ref|, mean|err| <= 2^-8
mean|ref|); the stack run end to end from the embedding within the stack
bar of tests/_tol.py (L * 2^-7 of mean|ref| and of max|ref| after L layers:
twice the oracle's model of the eight bf16 stores of each layer; the
decoder-pin tests show it rejects every composition mistake tried).  The
greedy token, an argmax decided in floating
point: for the same bf16 input, the chosen id's exact logit is within the
fp32 accumulation bound of the exact maximum, and equals the exact argmax
wherever the exact top-two gap exceeds twice that bound; after the stack,
the same with the bound widened by what the stack bar lets the input move.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from synthdata.workloads import ModelShape, Request, custom_workload
from tests._tol import assert_intermediate_close, assert_stack_close, stack_bar

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload, dev_bf16, host_f64
    from paper_2609_36722_amd.api import AttunerError, Context, ModelCfg, bf16_to_host
    from paper_2609_36722_amd.decoder import DecoderStack, LayerWeights, StackWeights


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _bits(rng, shape, std=1.0):
    return sd.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * np.float32(std))


def _fp32_bound(x, w):
    """Bound on |fp32 dot - exact dot| for each output of x w^T with K terms:
    K * 2^-24 * sum_k |x_k w_k| (one rounding per product-add, and a margin)."""
    K = x.shape[-1]
    return 2.0 * K * 2.0 ** -24 * (np.abs(x) @ np.abs(w).T)


# ----------------------------------------------------------------------------
# embedding rows (bit-exact) and RMSNorm rows
# ----------------------------------------------------------------------------

def test_embed_bit_exact():
    _say("embed")
    rng = np.random.default_rng(31)
    V, H = 1000, 256
    table = rng.integers(0, 2 ** 16, size=(V, H), dtype=np.uint16)
    ids = np.concatenate([[0, V - 1, 5, 5], rng.integers(0, V, size=77)]).astype(np.int32)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        out = torch.empty(len(ids), H, dtype=torch.bfloat16, device="cuda")
        ctx.embed(ids.tolist(), dev_bf16(table), out)
        torch.cuda.synchronize()
        assert np.array_equal(bf16_to_host(out), table[ids])
        with pytest.raises(AttunerError) as e:
            ctx.embed([3, V], dev_bf16(table), out)
        assert e.value.status == -5


@pytest.mark.parametrize("H,n,rows", [(2560, 37, None), (4096, 300, None), (2560, 9, [8, 0, 5, 5, 1]),
                                      (8192, 3, [2])])
def test_rms_norm_rows(H, n, rows):
    _say(f"rms_norm H={H} n={n} rows={rows}")
    rng = np.random.default_rng(H + n)
    x = _bits(rng, (n, H), 3.0)
    g = sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, H).astype(np.float32))
    m = n if rows is None else len(rows)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        out = torch.empty(m, H, dtype=torch.bfloat16, device="cuda")
        ctx.rms_norm(dev_bf16(x), dev_bf16(g), out, rows=rows)
        torch.cuda.synchronize()
        got = host_f64(out)
    sel = np.arange(n) if rows is None else np.array(rows)
    ref = oracle.rms_norm_heads(oracle.decode_bf16(x)[sel], oracle.decode_bf16(g), 1e-6)
    assert_intermediate_close(got, ref, "rms_norm")


# ----------------------------------------------------------------------------
# plain GEMM epilogues: bf16, + residual (in place), SwiGLU, fp32 logits
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("T,K,N,res", [
    (1, 256, 64, "none"),
    (37, 2560, 4096, "none"),
    (300, 4096, 2560, "separate"),   # o_proj of the 4B stack (K = Hq d), ragged tokens
    (256, 9728, 2560, "inplace"),    # down_proj of the 4B stack, residual read and written in place
    (513, 12288, 4096, "inplace"),   # down_proj of the 8B stack
    # products the tile plan gives to the two-k-group kernel (6144 outputs):
    (450, 4096, 6144, "none"),       # 128 x 96 tile, ragged last token tile
    (256, 4096, 6144, "separate"),   # 128 x 96 tile in 2 key splits (fp32 partials + reduce)
    (96, 4096, 6144, "inplace"),     # 128 x 96 tile in 4 key splits, fewer tokens than a tile
])
def test_linear_parity(T, K, N, res):
    _say(f"linear T={T} K={K} N={N} residual={res}")
    rng = np.random.default_rng(T + K + N)
    x, w = _bits(rng, (T, K)), _bits(rng, (N, K), 1 / math.sqrt(K))
    r = _bits(rng, (T, N)) if res != "none" else None
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        if res == "inplace":
            out = dev_bf16(r)
            ctx.linear(dev_bf16(x), dev_bf16(w), out, residual=out)
        else:
            out = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
            ctx.linear(dev_bf16(x), dev_bf16(w), out, residual=dev_bf16(r) if r is not None else None)
        torch.cuda.synchronize()
        got = host_f64(out)
    ref = oracle.linear(oracle.decode_bf16(x), oracle.decode_bf16(w),
                        oracle.decode_bf16(r) if r is not None else None)
    assert_intermediate_close(got, ref, "linear")


@pytest.mark.parametrize("seed", [501, 502, 503, 504, 505, 506])
def test_linear_random_shapes(seed):
    # Seeded random shapes (tokens 1-16 or 17-1200, k and outputs multiples
    # of 64) and residual forms: the plan's tile, its key split (a plain
    # product may split the k range when its tiles leave CUs idle) and the
    # few-token paths vary with the shape.
    rng = np.random.default_rng(seed)
    T = int(rng.integers(1, 17)) if seed % 3 == 0 else int(rng.integers(17, 1201))
    K, N = 64 * int(rng.integers(1, 81)), 64 * int(rng.integers(1, 81))
    res = ["none", "separate", "inplace"][int(rng.integers(0, 3))]
    _say(f"linear random shape seed {seed}: T={T} K={K} N={N} residual={res}")
    x, w = _bits(rng, (T, K)), _bits(rng, (N, K), 1 / math.sqrt(K))
    r = _bits(rng, (T, N)) if res != "none" else None
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        if res == "inplace":
            out = dev_bf16(r)
            ctx.linear(dev_bf16(x), dev_bf16(w), out, residual=out)
        else:
            out = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
            ctx.linear(dev_bf16(x), dev_bf16(w), out, residual=dev_bf16(r) if r is not None else None)
        torch.cuda.synchronize()
        got = host_f64(out)
    ref = oracle.linear(oracle.decode_bf16(x), oracle.decode_bf16(w),
                        oracle.decode_bf16(r) if r is not None else None)
    assert_intermediate_close(got, ref, "linear")


@pytest.mark.parametrize("T,K,I", [(1, 2560, 9728), (100, 2560, 9728), (513, 4096, 12288), (64, 256, 32),
                                   (1000, 4096, 12288)])   # the last: two-k-group 128 x 192 tile, ragged
def test_gate_up_swiglu_parity(T, K, I):
    _say(f"gate_up_swiglu T={T} K={K} I={I}")
    rng = np.random.default_rng(T + K + I)
    x = _bits(rng, (T, K))
    wg, wu = _bits(rng, (I, K), 1 / math.sqrt(K)), _bits(rng, (I, K), 1 / math.sqrt(K))
    w_gu = np.stack([wg, wu], axis=1).reshape(2 * I, K)
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        out = torch.empty(T, I, dtype=torch.bfloat16, device="cuda")
        ctx.gate_up_swiglu(dev_bf16(x), dev_bf16(np.ascontiguousarray(w_gu)), out)
        torch.cuda.synchronize()
        got = host_f64(out)
    d = oracle.decode_bf16
    assert_intermediate_close(got, oracle.swiglu(d(x), d(wg), d(wu)), "swiglu")


def _check_pick(ids, max_logit, x, w):
    """The greedy pick against the exact logits of the same bf16 x and w."""
    exact = oracle.linear(x, w)
    bound = _fp32_bound(x, w)
    for r in range(exact.shape[0]):
        top = int(np.argmax(exact[r]))
        i = int(ids[r])
        assert 0 <= i < w.shape[0]
        assert exact[r, i] >= exact[r, top] - 2 * bound[r].max(), f"row {r}: id {i} is not a maximum"
        assert abs(max_logit[r] - exact[r, i]) <= bound[r, i] + 1e-30
        second = np.partition(exact[r], -2)[-2]
        if exact[r, top] - second > 2 * bound[r].max():
            assert i == top, f"row {r}: id {i}, exact argmax {top} with a clear gap"


@pytest.mark.parametrize("n,H,V", [(1, 256, 1024), (5, 2560, 151936), (16, 512, 4096)])
def test_lm_head_argmax(n, H, V):
    _say(f"lm_head_argmax n={n} H={H} V={V}")
    rng = np.random.default_rng(n + H + V)
    x, w = _bits(rng, (n, H)), _bits(rng, (V, H), 1 / math.sqrt(H))
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        ids = torch.empty(n, dtype=torch.int32, device="cuda")
        mx = torch.empty(n, dtype=torch.float32, device="cuda")
        ctx.lm_head_argmax(dev_bf16(x), dev_bf16(w), ids, mx)
        torch.cuda.synchronize()
        _check_pick(ids.cpu().numpy(), mx.cpu().numpy().astype(np.float64), oracle.decode_bf16(x),
                    oracle.decode_bf16(w))


def test_lm_head_argmax_tie_takes_smallest_index():
    # a copy of the winning vocabulary row at a smaller index gives the same
    # fp32 logit (same products, same order): the smaller index must win
    _say("lm_head_argmax tie")
    rng = np.random.default_rng(33)
    n, H, V = 3, 256, 2048
    x, w = _bits(rng, (n, H)), _bits(rng, (V, H), 1 / math.sqrt(H))
    exact = oracle.linear(oracle.decode_bf16(x), oracle.decode_bf16(w))
    top = int(np.argmax(exact[0]))
    dup = 7 if top > 7 else V - 1
    w[dup] = w[top]
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        ids = torch.empty(n, dtype=torch.int32, device="cuda")
        ctx.lm_head_argmax(dev_bf16(x), dev_bf16(w), ids)
        torch.cuda.synchronize()
        got = ids.cpu().numpy()
    exact2 = oracle.linear(oracle.decode_bf16(x), oracle.decode_bf16(w))
    gap = np.sort(exact2[0])[-1] - np.sort(exact2[0])[-3]   # the top two are the tie
    assert gap > 2 * _fp32_bound(oracle.decode_bf16(x), oracle.decode_bf16(w))[0].max(), "seed gives no clear tie"
    assert got[0] == min(top, dup)


# ----------------------------------------------------------------------------
# a two-layer stack chained through the calls
# ----------------------------------------------------------------------------

def _stack_case():
    shape = ModelShape(hidden=256)
    wl = custom_workload("stack", 92, shape, [40, 17, 64], [Request((0, 1), 20), Request((2, 0), 33)],
                         n_layers=2, rank=16, scale=1.0, gamma="uniform")
    return wl, 512, 1024     # intermediate, vocab


def _oracle_weights(wl, l, I):
    w = {k: oracle.decode_bf16(v) for k, v in sd.layer_weights(wl, l).items()}
    w.update({k: oracle.decode_bf16(v) for k, v in sd.decoder_weights(wl, l, I).items()})
    return w


def _pick_bound(x_ref, w):
    """Bound on |logit_v(x) - logit_v(x_ref)| for an x within the two-layer
    stack bar of x_ref (max|x - x_ref| <= b max|x_ref| per element, b =
    max(1e-2, stack_bar(2))): sum_k |dx_k| |w_vk| <= b max|x_ref| * max_v
    sum_k |w_vk|, plus the fp32 accumulation bound."""
    b = max(1e-2, stack_bar(2))
    return b * np.abs(x_ref).max() * np.abs(w).sum(axis=1).max() + _fp32_bound(x_ref, w).max()


def _check_pick_near(ids, x_ref, w):
    """ids from a GPU x close to x_ref: each id's exact logit at x_ref is within
    twice the bound of the exact maximum (the two logits each move by at most
    the bound), and equals the exact argmax where the top-two gap exceeds it."""
    logits = oracle.linear(x_ref, w)
    for r in range(logits.shape[0]):
        b = _pick_bound(x_ref[r:r + 1], w)
        top = int(np.argmax(logits[r]))
        assert logits[r, int(ids[r])] >= logits[r, top] - 2 * b, f"row {r}: id {ids[r]} far from the maximum"
        second = np.partition(logits[r], -2)[-2]
        if logits[r, top] - second > 2 * b:
            assert int(ids[r]) == top, f"row {r}: id {ids[r]}, exact argmax {top} with a clear gap"


def test_decoder_stack_two_layers_then_decode():
    # the whole stack on the GPU against the whole stack in the oracle, both
    # from the same seeded token ids: prefill of the suffix to the first
    # token, then two decode steps with seeded next tokens (the oracle takes
    # no GPU value as input)
    _say("decoder stack 2 layers + 2 decode steps")
    wl, I, V = _stack_case()
    s = wl.shape
    n_dec = 2
    g = GpuWorkload(wl, layers=[0, 1], suffix_extra=n_dec)
    n_req = len(wl.requests)
    tokens = [sd.suffix_tokens(wl, r, V) for r in range(n_req)]
    dec_tokens = np.random.default_rng(96).integers(0, V, size=(n_dec, n_req))
    try:
        layers = []
        for l in range(2):
            w, dw = sd.layer_weights(wl, l), sd.decoder_weights(wl, l, I)
            layers.append(LayerWeights(
                wqkv=dev_bf16(np.concatenate([w["wq"], w["wk"], w["wv"]])), gamma_q=dev_bf16(w["gamma_q"]),
                gamma_k=dev_bf16(w["gamma_k"]), gamma_in=dev_bf16(dw["gamma_in"]), wo=dev_bf16(dw["wo"]),
                gamma_post=dev_bf16(dw["gamma_post"]),
                w_gu=dev_bf16(np.ascontiguousarray(np.stack([dw["w_gate"], dw["w_up"]], 1).reshape(2 * I, -1))),
                w_down=dev_bf16(dw["w_down"]), a=dev_bf16(w["a"]), b=dev_bf16(w["b"])))
        lm = sd.lm_weights(wl, V)
        sw = StackWeights(embed=dev_bf16(lm["embed"]), gamma_final=dev_bf16(lm["gamma_final"]),
                          w_lm=dev_bf16(lm["w_lm"]), layers=layers, rank=wl.rank, scale=wl.scale)
        stack = DecoderStack(g.ctx, sw, [r.suffix_len for r in wl.requests])
        stack.embed(np.concatenate(tokens).tolist())
        h_emb = host_f64(stack.h)
        stack.layers(g.cu_ctx, g.art_len, g.pos0, g.req_kv, g.rows)
        ids = stack.first_token().cpu().numpy()
        h_pre, x_last = host_f64(stack.h), host_f64(stack.x_last)
        # the same prefill with layer 0's pages gathered first and layer 1's
        # copied inside layer 0's attention launch: h, the first tokens and
        # the cache bit for bit as above
        _say("decoder stack: pages copied inside the attention launches")
        kv2, bt2 = torch.zeros_like(g.req_kv), torch.zeros_like(g.block_table)
        g.ctx.assemble_table(g.requests, g.suffix_cap, bt2, g.rows)
        g.ctx.gather_layers(bt2, g.n_entries, 0, 1, kv2, g.rows)
        stack.embed(np.concatenate(tokens).tolist())
        stack.layers(g.cu_ctx, g.art_len, g.pos0, kv2, g.rows, gather=(bt2, g.n_entries))
        assert np.array_equal(stack.first_token().cpu().numpy(), ids)
        assert np.array_equal(host_f64(stack.h), h_pre)
        assert torch.equal(kv2.view(torch.int16), g.req_kv.view(torch.int16))
        del kv2, bt2
        dec = []
        for j in range(n_dec):
            ctx_len = [g.art_len[r] + wl.requests[r].suffix_len + j for r in range(n_req)]
            ids_j = stack.decode(dec_tokens[j].tolist(), g.cu_ctx, ctx_len, g.req_kv, g.rows).cpu().numpy()
            dec.append((host_f64(stack.hd), host_f64(stack.x_last), ids_j))
        torch.cuda.synchronize()
    finally:
        g.close()

    emb = oracle.decode_bf16(lm["embed"])
    h0 = np.concatenate([emb[t] for t in tokens])
    assert np.array_equal(h_emb, h0), "embedding rows"
    ws = [_oracle_weights(wl, l, I) for l in range(2)]
    gf, w_lm = oracle.decode_bf16(lm["gamma_final"]), oracle.decode_bf16(lm["w_lm"])
    args = lambda r, l, keys, vals, p0: (keys, vals, p0, s.n_q_heads, s.n_kv_heads, s.rope_theta, s.rms_eps, wl.scale)
    # prefill in the oracle: every layer's keys/values of the context kept per request
    ctx_k, ctx_v, h_ref, x_ref = [], [], [], []
    for r, req in enumerate(wl.requests):
        lo, hi = g.cu_q[r], g.cu_q[r + 1]
        h = h0[lo:hi]
        ks, vs = [], []
        for l in range(2):
            ka = np.concatenate([oracle.decode_bf16(g.art_k[a][l]) for a in req.artifact_ids])
            va = np.concatenate([oracle.decode_bf16(g.art_v[a][l]) for a in req.artifact_ids])
            out = oracle.decoder_layer(h, ws[l], *args(r, l, ka, va, wl.pos0(req)))
            ks.append(np.concatenate([ka, out["k_hat"]]))
            vs.append(np.concatenate([va, out["v"]]))
            h = out["h"]
        ctx_k.append(ks)
        ctx_v.append(vs)
        h_ref.append(h)
        x_ref.append(oracle.rms_norm_heads(h[-1:], gf, s.rms_eps))
    assert_stack_close(h_pre, np.concatenate(h_ref), 2, "two-layer stack h")
    x_ref = np.concatenate(x_ref)
    assert_stack_close(x_last, x_ref, 2, "final norm of the last rows")
    _check_pick_near(ids, x_ref, w_lm)
    # two decode steps in the oracle over its own growing context
    for j in range(n_dec):
        hd_ref, xd_ref = [], []
        for r, req in enumerate(wl.requests):
            h = emb[dec_tokens[j, r]][None, :]
            p0 = g.art_len[r] + req.suffix_len + j
            for l in range(2):
                out = oracle.decoder_layer(h, ws[l], *args(r, l, ctx_k[r][l], ctx_v[r][l], p0))
                ctx_k[r][l] = np.concatenate([ctx_k[r][l], out["k_hat"]])
                ctx_v[r][l] = np.concatenate([ctx_v[r][l], out["v"]])
                h = out["h"]
            hd_ref.append(h)
            xd_ref.append(oracle.rms_norm_heads(h, gf, s.rms_eps))
        hd, xd, ids_j = dec[j]
        assert_stack_close(hd, np.concatenate(hd_ref), 2, f"decode step {j} h")
        _check_pick_near(ids_j, np.concatenate(xd_ref), w_lm)


# ----------------------------------------------------------------------------
# the few-token path (at most 16 tokens: the weight-streaming GEMV) in every mode
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("T,rank", [(1, 16), (2, 8), (3, 48), (5, 0), (8, 32), (7, 5), (12, 16), (16, 0), (9, 64)])
def test_few_token_qproj_lora(T, rank):
    _say(f"few-token qproj T={T} r={rank}")
    rng = np.random.default_rng(100 + T + rank)
    H, N, lora_cols = 2560, 6144, 4096
    x, w = _bits(rng, (T, H)), _bits(rng, (N, H), 0.02)
    a = _bits(rng, (max(rank, 1), H), 1 / math.sqrt(H))[:rank]
    b = _bits(rng, (lora_cols, max(rank, 1)), 1.0)[:, :rank]     # B ~ N(0, 1): the update is visible
    scale = 16.0 / max(rank, 1)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        out = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), dev_bf16(w), dev_bf16(np.ascontiguousarray(a)) if rank else None,
                       dev_bf16(np.ascontiguousarray(b)) if rank else None, rank, scale, lora_cols, out)
        torch.cuda.synchronize()
        got = host_f64(out)
    d = oracle.decode_bf16
    ref = oracle.qproj_lora(d(x), d(w), d(a) if rank else None, d(b) if rank else None, scale, lora_cols)
    assert_intermediate_close(got[:, :lora_cols], ref[:, :lora_cols], "q columns")
    assert_intermediate_close(got[:, lora_cols:], ref[:, lora_cols:], "k/v columns")


@pytest.mark.parametrize("T", [2, 4, 6, 8, 10, 16])
def test_few_token_modes(T):
    _say(f"few-token modes T={T}")
    rng = np.random.default_rng(200 + T)
    d = oracle.decode_bf16
    with Context(ModelCfg(n_layers=1, hidden=512), pool_pages=0) as ctx:
        # down projection with the residual in place (K = 9728)
        g, wd, h = _bits(rng, (T, 9728)), _bits(rng, (512, 9728), 1 / math.sqrt(9728)), _bits(rng, (T, 512))
        hd = dev_bf16(h)
        ctx.linear(dev_bf16(g), dev_bf16(wd), hd, residual=hd)
        # gate/up SwiGLU
        x, wg, wu = _bits(rng, (T, 512)), _bits(rng, (1024, 512), 1 / math.sqrt(512)), _bits(rng, (1024, 512), 1 / math.sqrt(512))
        sw = torch.empty(T, 1024, dtype=torch.bfloat16, device="cuda")
        ctx.gate_up_swiglu(dev_bf16(x), dev_bf16(np.ascontiguousarray(np.stack([wg, wu], 1).reshape(2048, 512))), sw)
        # greedy pick over fp32 logits
        wl = _bits(rng, (4096, 512), 1 / math.sqrt(512))
        ids = torch.empty(T, dtype=torch.int32, device="cuda")
        mx = torch.empty(T, dtype=torch.float32, device="cuda")
        ctx.lm_head_argmax(dev_bf16(x), dev_bf16(wl), ids, mx)
        torch.cuda.synchronize()
        assert_intermediate_close(host_f64(hd), oracle.linear(d(g), d(wd), d(h)), "down + residual")
        assert_intermediate_close(host_f64(sw), oracle.swiglu(d(x), d(wg), d(wu)), "swiglu")
        _check_pick(ids.cpu().numpy(), mx.cpu().numpy().astype(np.float64), d(x), d(wl))


@pytest.mark.parametrize("T", [3, 12])
def test_few_token_k_not_a_multiple_of_128(T):
    # k = 320 (a multiple of 64, not of 128): 12 tokens stay on the dot-product
    # GEMV instead of the matrix-core one; the residual added in place
    _say(f"few-token K=320 T={T}")
    rng = np.random.default_rng(400 + T)
    d = oracle.decode_bf16
    with Context(ModelCfg(n_layers=1, hidden=320), pool_pages=0) as ctx:
        x, w, h = _bits(rng, (T, 320)), _bits(rng, (512, 320), 1 / math.sqrt(320)), _bits(rng, (T, 512))
        hd = dev_bf16(h)
        ctx.linear(dev_bf16(x), dev_bf16(w), hd, residual=hd)
        torch.cuda.synchronize()
        assert_intermediate_close(host_f64(hd), oracle.linear(d(x), d(w), d(h)), "linear + residual")
