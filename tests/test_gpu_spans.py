"""GPU parity of prompts that interleave cached artifacts with online spans
(system text, separators, questions between and around the artifacts),
through the C ABI: the segment block table and gathered artifact rows
bit-exact against the oracle; the online spans' normalised keys and values
within the intermediate bar; O within the O bar over the
batch (each request within it or the relative bar of a bf16-stored value).
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from tests._tol import assert_intermediate_close, assert_o_close, assert_o_close_per_request

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import dev_bf16, host_f64
    from paper_2609_36722_amd.api import AttunerError, Context, ModelCfg, bf16_to_host

HQ, HKV, D = 32, 8, 128


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _bits(rng, shape, std=1.0):
    return sd.f32_to_bf16_bits(rng.standard_normal(shape).astype(np.float32) * np.float32(std))


@pytest.mark.parametrize("H,rank,layer", [(512, 16, 1), (2560, 8, 0)])
def test_interleaved_spans(H, rank, layer):
    _say(f"interleaved spans H={H} r={rank} layer={layer}")
    # prompts in order: artifacts by index, online spans as -n
    _run_interleaved(H, rank, layer, [40, 17, 64, 1, 300],
                     [[-7, 0, -3, 1, -20], [2, -5], [-9], [3, 3, -1, 0], [4, -64, 2, -70]], 70 + H + rank)


@pytest.mark.parametrize("seed", [301, 302, 303])
def test_interleaved_random_prompts(seed):
    # Seeded random prompts: 1-6 prompts of 1-7 segments each, artifacts of
    # 1-400 tokens (repeats allowed) between online spans of 1-80 tokens,
    # every prompt with at least one online span.
    rng = np.random.default_rng(seed)
    lengths = [int(rng.integers(1, 401)) for _ in range(int(rng.integers(1, 7)))]
    prompts = []
    for _ in range(int(rng.integers(1, 7))):
        segs = [int(rng.integers(0, len(lengths))) if rng.random() < 0.5 else -int(rng.integers(1, 81))
                for _ in range(int(rng.integers(1, 8)))]
        if all(x >= 0 for x in segs):
            segs.insert(int(rng.integers(0, len(segs) + 1)), -int(rng.integers(1, 81)))
        prompts.append(segs)
    _say(f"interleaved random prompts seed {seed}: lengths {lengths}, prompts {prompts}")
    _run_interleaved(512, 16, int(rng.integers(0, 2)), lengths, prompts, seed)


def _run_interleaved(H, rank, layer, lengths, prompts, seed):
    rng = np.random.default_rng(seed)
    n_layers = 2
    scale = 16.0 / rank
    with Context(ModelCfg(n_layers=n_layers, hidden=H), pool_pages=sum(math.ceil(L / 16) for L in lengths)) as ctx:
        art_k, art_v, ids = {}, {}, {}
        for a, L in enumerate(lengths):
            k, v = _bits(rng, (n_layers, HKV, L, D)), _bits(rng, (n_layers, HKV, L, D))
            ids[a] = ctx.store_artifact(dev_bf16(k), dev_bf16(v))
            art_k[a], art_v[a] = k, v
        segs = [[ids[s] if s >= 0 else s for s in p] for p in prompts]
        ne, rows, ns = ctx.assemble_segments_plan(segs)
        bt = torch.zeros(max(1, ne) * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(n_layers * 2 * HKV * rows * D, dtype=torch.bfloat16, device="cuda")
        cu, spans = ctx.assemble_segments(segs, bt, kv, rows)
        assert len(spans) == ns

        # the plan against the oracle's segment table (physical pages mapped in)
        e, cu_ref, sp_ref = oracle.block_table_segments(lengths, prompts, 16)
        phys = {a: ctx.artifact_pages(ids[a])[0] for a in ids}
        want = np.array([[phys[a][p], nv, dst, r] for a, p, nv, r, dst in e.tolist()], np.int32).reshape(-1, 4)
        assert np.array_equal(bt.cpu().numpy().reshape(-1, 4)[:len(want)], want)
        assert cu == cu_ref.tolist() and [list(s) for s in spans] == sp_ref.tolist()

        n_on = sum(l for _, _, l in spans)
        x = _bits(rng, (n_on, H))
        wq, wk, wv = _bits(rng, (HQ * D, H), 0.02), _bits(rng, (HKV * D, H), 0.02), _bits(rng, (HKV * D, H), 0.02)
        a, b = _bits(rng, (rank, H), 1 / math.sqrt(H)), _bits(rng, (HQ * D, rank), 0.01)
        gq = sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, D).astype(np.float32))
        gk = sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, D).astype(np.float32))
        n_out = (HQ + 2 * HKV) * D
        qkv = torch.empty(n_on, n_out, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), dev_bf16(np.concatenate([wq, wk, wv])), dev_bf16(a), dev_bf16(b), rank, scale,
                       HQ * D, qkv)
        cu_q = [0]
        for _, _, l in spans:
            cu_q.append(cu_q[-1] + l)
        o = torch.empty(n_on, HQ, D, dtype=torch.bfloat16, device="cuda")
        ctx.span_attn(layer, cu_q, [cu[r] for r, _, _ in spans], [off for _, off, _ in spans], None,
                      qkv[:, :HQ * D], n_out, qkv[:, HQ * D:(HQ + HKV) * D], qkv[:, (HQ + HKV) * D:], n_out,
                      dev_bf16(gq), dev_bf16(gk), kv, rows, o)
        torch.cuda.synchronize()
        got_o = host_f64(o)
        cache = bf16_to_host(kv).reshape(n_layers, 2, HKV, rows, D)

    # artifact rows bit-exact at their offsets, on every layer
    for a_idx, p, nv, r, dst in e.tolist():
        src = slice(16 * p, 16 * p + nv)
        assert np.array_equal(cache[:, 0, :, dst:dst + nv], art_k[a_idx][:, :, src]), f"K rows of artifact {a_idx}"
        assert np.array_equal(cache[:, 1, :, dst:dst + nv], art_v[a_idx][:, :, src]), f"V rows of artifact {a_idx}"

    d = oracle.decode_bf16
    refs, t0 = [], 0
    for r, p in enumerate(prompts):
        n_r = sum(-s for s in p if s < 0)
        ak = {i: d(art_k[i][layer]).transpose(1, 0, 2) for i in range(len(lengths))}
        av = {i: d(art_v[i][layer]).transpose(1, 0, 2) for i in range(len(lengths))}
        ref = oracle.interleaved_layer(p, d(x[t0:t0 + n_r]), d(wq), d(wk), d(wv), d(a), d(b), scale, d(gq), d(gk),
                                       ak, av, HQ, HKV, 1e6, 1e-6)
        # the online rows of the cache: normalised keys and values
        rows_r = cu[r] + ref["pos"]
        assert_intermediate_close(d(cache[layer, 0][:, rows_r]).transpose(1, 0, 2), ref["k_hat"], f"request {r} k_hat")
        assert_intermediate_close(d(cache[layer, 1][:, rows_r]).transpose(1, 0, 2), ref["v"], f"request {r} v")
        assert_o_close_per_request(got_o[t0:t0 + n_r], ref["o"], f"request {r} O")
        refs.append(ref["o"])
        t0 += n_r
    assert_o_close(got_o, np.concatenate(refs), "batch O")


def test_span_errors():
    _say("span errors")
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=1) as ctx:
        with pytest.raises(AttunerError) as e:
            ctx.assemble_segments_plan([[5]])          # unknown artifact id
        assert e.value.status == -3
        kv = torch.zeros(2 * HKV * 10 * D, dtype=torch.bfloat16, device="cuda")
        q = torch.zeros(4, (HQ + 2 * HKV) * D, dtype=torch.bfloat16, device="cuda")
        g = torch.ones(D, dtype=torch.bfloat16, device="cuda")
        ld = q.shape[1]
        with pytest.raises(AttunerError) as e:
            # 10 cache rows; a span of 4 at offset 7 would end at row 11
            ctx.span_attn(0, [0, 4], [0], [7], None, q[:, :HQ * D], ld, q[:, HQ * D:(HQ + HKV) * D],
                          q[:, (HQ + HKV) * D:], ld, g, g, kv, 10, torch.empty(4, HQ, D, dtype=torch.bfloat16,
                                                                                 device="cuda"))
        assert e.value.status == -1


def test_interleaved_c2_prompt():
    # the c2 request with online text around its artifacts (a 32-token system
    # span, 8 tokens between consecutive artifacts, the 256-token suffix), as
    # bench.py --spans 8 times it, in its launch plan; every online row's O
    # against the oracle (a few seconds of fp64)
    _say("interleaved c2 prompt")
    rng = np.random.default_rng(77)
    H, rank, scale, layer = 2560, 16, 1.0, 0
    lengths = [1024] * 8
    prompt = [-32]
    for j in range(8):
        if j:
            prompt.append(-8)
        prompt.append(j)
    prompt.append(-256)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=8 * 64) as ctx:
        art_k, art_v, ids = {}, {}, {}
        for a, L in enumerate(lengths):
            k, v = _bits(rng, (1, HKV, L, D)), _bits(rng, (1, HKV, L, D))
            ids[a] = ctx.store_artifact(dev_bf16(k), dev_bf16(v))
            art_k[a], art_v[a] = k, v
        segs = [[ids[s] if s >= 0 else s for s in prompt]]
        ne, rows, ns = ctx.assemble_segments_plan(segs)
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * HKV * rows * D, dtype=torch.bfloat16, device="cuda")
        cu, spans = ctx.assemble_segments(segs, bt, kv, rows)
        n_on = sum(l for _, _, l in spans)
        x = _bits(rng, (n_on, H))
        wq, wk, wv = _bits(rng, (HQ * D, H), 0.02), _bits(rng, (HKV * D, H), 0.02), _bits(rng, (HKV * D, H), 0.02)
        a, b = _bits(rng, (rank, H), 1 / math.sqrt(H)), _bits(rng, (HQ * D, rank), 0.01)
        g1 = sd.f32_to_bf16_bits(np.ones(D, np.float32))
        n_out = (HQ + 2 * HKV) * D
        qkv = torch.empty(n_on, n_out, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), dev_bf16(np.concatenate([wq, wk, wv])), dev_bf16(a), dev_bf16(b), rank, scale,
                       HQ * D, qkv)
        cu_q = [0]
        for _, _, l in spans:
            cu_q.append(cu_q[-1] + l)
        o = torch.empty(n_on, HQ, D, dtype=torch.bfloat16, device="cuda")
        ctx.span_attn(layer, cu_q, [cu[r] for r, _, _ in spans], [off for _, off, _ in spans], None,
                      qkv[:, :HQ * D], n_out, qkv[:, HQ * D:(HQ + HKV) * D], qkv[:, (HQ + HKV) * D:], n_out,
                      dev_bf16(g1), dev_bf16(g1), kv, rows, o)
        torch.cuda.synchronize()
        got_o = host_f64(o)
        cache = bf16_to_host(kv).reshape(1, 2, HKV, rows, D)
    d = oracle.decode_bf16
    ak = {i: d(art_k[i][0]).transpose(1, 0, 2) for i in range(8)}
    av = {i: d(art_v[i][0]).transpose(1, 0, 2) for i in range(8)}
    ref = oracle.interleaved_layer(prompt, d(x), d(wq), d(wk), d(wv), d(a), d(b), scale, d(g1), d(g1), ak, av,
                                   HQ, HKV, 1e6, 1e-6)
    assert_o_close(got_o, ref["o"], "O")
    t0 = 0
    for _, _, l in spans:
        assert_o_close_per_request(got_o[t0:t0 + l], ref["o"][t0:t0 + l], f"span at row {t0}")
        t0 += l
    # cached rows of the first and last artifact stayed put
    for j, off in ((0, 32), (7, 32 + 7 * (1024 + 8))):
        assert np.array_equal(cache[0, 0, :, off:off + 1024], art_k[j][0]), f"artifact {j} keys"


def test_spans_given_out_of_prompt_order():
    # the same prompt's spans listed last-first (rows of the question before
    # the header's): positions no longer grow along the rows, so the spans
    # must not share query blocks.  Both orders against the oracle; the raw
    # q/k/v rows are the seeded inputs, passed to the oracle through identity
    # projections (W_q = [I 0 0] etc. over the 6144 q|k|v columns)
    _say("spans out of prompt order")
    rng = np.random.default_rng(78)
    H, L = 512, 100
    n_out = (HQ + 2 * HKV) * D
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=8) as ctx:
        k, v = _bits(rng, (1, HKV, L, D)), _bits(rng, (1, HKV, L, D))
        aid = ctx.store_artifact(dev_bf16(k), dev_bf16(v))
        ne, rows, ns = ctx.assemble_segments_plan([[-5, aid, -7]])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * HKV * rows * D, dtype=torch.bfloat16, device="cuda")
        cu, spans = ctx.assemble_segments([[-5, aid, -7]], bt, kv, rows)
        raw = _bits(rng, (12, n_out))
        g = torch.ones(D, dtype=torch.bfloat16, device="cuda")

        def run(order):
            rows_in = np.concatenate([raw[0:5], raw[5:12]] if order == "in" else [raw[5:12], raw[0:5]])
            q = dev_bf16(rows_in)
            o = torch.empty(12, HQ, D, dtype=torch.bfloat16, device="cuda")
            cq, offs = ([0, 5, 12], [0, 5 + L]) if order == "in" else ([0, 7, 12], [5 + L, 0])
            ctx.span_attn(0, cq, [0, 0], offs, None, q[:, :HQ * D], n_out, q[:, HQ * D:(HQ + HKV) * D],
                          q[:, (HQ + HKV) * D:], n_out, g, g, kv, rows, o)
            torch.cuda.synchronize()
            return host_f64(o)
        a = run("in")
        b = run("out")
    eye = np.eye(n_out)
    d = oracle.decode_bf16
    ref = oracle.interleaved_layer([-5, 0, -7], d(raw), eye[:HQ * D], eye[HQ * D:(HQ + HKV) * D],
                                   eye[(HQ + HKV) * D:], None, None, 0.0, np.ones(D), np.ones(D),
                                   {0: d(k[0]).transpose(1, 0, 2)}, {0: d(v[0]).transpose(1, 0, 2)}, HQ, HKV,
                                   1e6, 1e-6)["o"]
    assert_o_close(a, ref, "in order")
    assert_o_close(np.concatenate([b[7:12], b[0:7]]), ref, "out of order")
