"""Graph capture of whole-stack decode steps across a RoPE-table boundary.

A context builds its RoPE table for 4096 positions; later calls extend it
and grow their workspaces without waiting for the device, and attuner_reserve
sizes everything up front.  Here a two-layer stack decodes eight tokens at
positions 4092..4099 (the cached artifacts fill 4088 rows, the suffix 4):
- the eager steps match the fp64 oracle's stack (the stack bar);
- with the context reserved first, one HIP graph per step captures the
  layers, the final norm and the greedy pick, and every replay reproduces
  the eager step bit for bit;
- without a reservation, capturing a step past the table fails with ERANGE
  (nothing is enqueued), and the same step run eagerly extends the table and
  gives the reserved context's result bit for bit.
"""

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from synthdata.workloads import ModelShape, Request, custom_workload
from tests._tol import assert_stack_close

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload, dev_bf16, host_f64
    from paper_2609_36722_amd.api import AttunerError
    from paper_2609_36722_amd.decoder import DecoderStack, LayerWeights, StackWeights

I, V, N_DEC = 512, 1024, 8


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _case():
    shape = ModelShape(hidden=256)
    return custom_workload("graph", 94, shape, [1022, 1022, 1022, 1022], [Request((0, 1, 2, 3), 4)],
                           n_layers=2, rank=16, scale=1.0, gamma="uniform")


def _stack(wl, g):
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
    return DecoderStack(g.ctx, sw, [r.suffix_len for r in wl.requests]), lm


def _prefill(wl, g, stack):
    stack.embed(sd.suffix_tokens(wl, 0, V).tolist())
    stack.layers(g.cu_ctx, g.art_len, g.pos0, g.req_kv, g.rows)
    stack.first_token()


def _ctx_len(wl, g, j):
    return [g.art_len[0] + wl.requests[0].suffix_len + j]


def _dec_tokens():
    return np.random.default_rng(97).integers(0, V, size=N_DEC)


def test_decode_graph_capture_across_rope_boundary():
    wl = _case()
    toks = _dec_tokens()
    g = GpuWorkload(wl, layers=[0, 1], suffix_extra=N_DEC)
    try:
        assert g.art_len[0] + wl.requests[0].suffix_len == 4092
        stack, lm = _stack(wl, g)
        g.ctx.reserve(max_tokens=16, max_position=8192, max_rank=wl.rank, max_out=2 * I, max_lm_rows=1,
                      max_vocab=V)
        _prefill(wl, g, stack)
        _say("eager decode of 8 steps at positions 4092..4099")
        eager = []
        for j in range(N_DEC):
            ids = stack.decode([int(toks[j])], g.cu_ctx, _ctx_len(wl, g, j), g.req_kv, g.rows)
            torch.cuda.synchronize()
            eager.append((host_f64(stack.hd), int(ids.cpu()[0])))
        _say("capture one graph per step")
        graphs = []
        for j in range(N_DEC):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                stack.decode_layers(g.cu_ctx, _ctx_len(wl, g, j), g.req_kv, g.rows)
                stack.decode_token()
            graphs.append(gr)
        torch.cuda.synchronize()
        _say("replay each step twice, eager work and syncs in between")
        for rep in range(2):
            for j in range(N_DEC):
                stack.decode_embed([int(toks[j])])
                graphs[j].replay()
                torch.cuda.synchronize()
                hd = host_f64(stack.hd)
                assert np.array_equal(hd, eager[j][0]), f"replay {rep} step {j}: h differs from the eager step"
                assert int(stack.ids.cpu()[0]) == eager[j][1], f"replay {rep} step {j}: token"
    finally:
        g.close()

    _say("oracle stack: prefill + 8 decode steps")
    s = wl.shape
    ws = []
    for l in range(2):
        w = {k: oracle.decode_bf16(v) for k, v in sd.layer_weights(wl, l).items()}
        w.update({k: oracle.decode_bf16(v) for k, v in sd.decoder_weights(wl, l, I).items()})
        ws.append(w)
    emb = oracle.decode_bf16(lm["embed"])
    req = wl.requests[0]
    h = emb[sd.suffix_tokens(wl, 0, V)]
    ks, vs = [], []
    for l in range(2):
        ka = np.concatenate([oracle.decode_bf16(sd.artifact_kv(wl, a, l)[0]) for a in req.artifact_ids])
        va = np.concatenate([oracle.decode_bf16(sd.artifact_kv(wl, a, l)[1]) for a in req.artifact_ids])
        out = oracle.decoder_layer(h, ws[l], ka, va, wl.pos0(req), s.n_q_heads, s.n_kv_heads, s.rope_theta,
                                   s.rms_eps, wl.scale)
        ks.append(np.concatenate([ka, out["k_hat"]]))
        vs.append(np.concatenate([va, out["v"]]))
        h = out["h"]
    for j in range(N_DEC):
        h = emb[toks[j]][None, :]
        p = 4092 + j
        for l in range(2):
            out = oracle.decoder_layer(h, ws[l], ks[l], vs[l], p, s.n_q_heads, s.n_kv_heads, s.rope_theta,
                                       s.rms_eps, wl.scale)
            ks[l] = np.concatenate([ks[l], out["k_hat"]])
            vs[l] = np.concatenate([vs[l], out["v"]])
            h = out["h"]
        assert_stack_close(eager[j][0], h, 2, f"decode step {j} (position {p}) h")


def test_capture_past_the_rope_table_fails_and_eager_growth_matches():
    wl = _case()
    toks = _dec_tokens()
    results = {}
    for reserved in (True, False):
        g = GpuWorkload(wl, layers=[0, 1], suffix_extra=N_DEC)
        try:
            stack, _ = _stack(wl, g)
            if reserved:
                g.ctx.reserve(max_tokens=16, max_position=8192, max_rank=wl.rank, max_out=2 * I, max_lm_rows=1,
                              max_vocab=V)
            _prefill(wl, g, stack)
            # steps 0..3 (positions 4092..4095) fit the initial table; they also size the workspaces
            for j in range(4):
                stack.decode([int(toks[j])], g.cu_ctx, _ctx_len(wl, g, j), g.req_kv, g.rows)
            torch.cuda.synchronize()
            if not reserved:
                _say("capture of a step at position 4096 without a reservation")
                stack.decode_embed([int(toks[4])])
                gr = torch.cuda.CUDAGraph()
                with pytest.raises(AttunerError) as e:
                    with torch.cuda.graph(gr):
                        stack.decode_layers(g.cu_ctx, _ctx_len(wl, g, 4), g.req_kv, g.rows)
                assert e.value.status == -5 and "RoPE" in str(e.value)
                torch.cuda.synchronize()
            _say(f"eager steps 4..7 ({'reserved' if reserved else 'growing the table'})")
            for j in range(4, N_DEC):
                ids = stack.decode([int(toks[j])], g.cu_ctx, _ctx_len(wl, g, j), g.req_kv, g.rows)
            torch.cuda.synchronize()
            results[reserved] = (host_f64(stack.hd), int(ids.cpu()[0]))
        finally:
            g.close()
    assert np.array_equal(results[True][0], results[False][0])
    assert results[True][1] == results[False][1]


def test_reserve_then_capture_prefill_without_warmup():
    # a reservation alone (no eager call first) must size every workspace the
    # suffix path needs: capture three layers of the Qwen3-4B-shaped step and
    # a full prefill of 600 tokens with a rank-48 adapter (the separate
    # down-projection), replay twice, compare with the eager calls bit for bit
    import synthdata as sd
    wl = sd.make_workload("c2", gamma="uniform")
    s = wl.shape
    g = GpuWorkload(wl, layers=[0, 17, 35])
    try:
        T = wl.requests[0].suffix_len
        nq, nkv = s.q_dim, s.kv_dim
        n_out = nq + 2 * nkv
        ins = []
        for li in range(3):
            w, x = g.layer_inputs(li)
            ins.append((dev_bf16(x), dev_bf16(np.concatenate([w["wq"], w["wk"], w["wv"]])), dev_bf16(w["a"]),
                        dev_bf16(w["b"]), dev_bf16(w["gamma_q"]), dev_bf16(w["gamma_k"])))
        rng = np.random.default_rng(5)
        N, r = 600, 48
        xf = dev_bf16(sd.f32_to_bf16_bits(rng.standard_normal((N, s.hidden)).astype(np.float32)))
        af = dev_bf16(sd.f32_to_bf16_bits((rng.standard_normal((r, s.hidden)) / np.sqrt(s.hidden)).astype(np.float32)))
        bfm = dev_bf16(sd.f32_to_bf16_bits((rng.standard_normal((nq, r)) * 0.01).astype(np.float32)))
        g.ctx.reserve(max_tokens=N, max_position=max(g.rows, N), max_rank=r)

        def run(outs):
            for li, (x, w, a, b, gq, gk) in enumerate(ins):
                qkv, o, lse = outs[li]
                g.ctx.qproj_lora(x, w, a, b, wl.rank, wl.scale, nq, qkv)
                g.ctx.suffix_attn(li, g.cu_q, g.cu_ctx, g.art_len, g.pos0, qkv[:, :nq], n_out, qkv[:, nq:nq + nkv],
                                  qkv[:, nq + nkv:], n_out, gq, gk, g.req_kv, g.rows, o, lse)
            of, kf, vf = outs[3]
            g.ctx.full_prefill(0, xf, ins[0][1], af, bfm, r, 0.5, ins[0][4], ins[0][5], of, kf, vf)

        def buffers():
            bufs = [(torch.empty(T, n_out, dtype=torch.bfloat16, device="cuda"),
                     torch.empty(T, s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda"),
                     torch.empty(T, s.n_q_heads, dtype=torch.float32, device="cuda")) for _ in range(3)]
            bufs.append((torch.empty(N, s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda"),
                         torch.empty(s.n_kv_heads, N, s.head_dim, dtype=torch.bfloat16, device="cuda"),
                         torch.empty(s.n_kv_heads, N, s.head_dim, dtype=torch.bfloat16, device="cuda")))
            return bufs

        _say("capture after a reservation, no eager call first")
        cap = buffers()
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            run(cap)
        torch.cuda.synchronize()
        _say("eager reference")
        ref = buffers()
        run(ref)
        torch.cuda.synchronize()
        for rep in range(2):
            for t in cap:
                for u in t:
                    u.zero_()
            torch.cuda.synchronize()
            gr.replay()
            torch.cuda.synchronize()
            for i, (a_, b_) in enumerate(zip(cap, ref)):
                for u, v in zip(a_, b_):
                    assert torch.equal(u, v), f"replay {rep}: buffer set {i} differs from the eager calls"
    finally:
        g.close()
