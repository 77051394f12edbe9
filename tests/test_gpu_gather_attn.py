"""attuner_suffix_attn_gather (one layer's suffix attention with another
layer's artifact-page copy riding in the attention launch) against the same
work as separate calls: attuner_assemble_kv for every layer, then
attuner_suffix_attn layer by layer.  Every layer's O and LSE and the whole
request cache must agree bit for bit, and each request's cached rows must
hold its artifacts in order (the oracle's assembly: rows cu_ctx[r] ..
cu_ctx[r] + art_len[r] - 1).

Cases (the library's launch tracer tells which path ran): a three-layer
batch of four requests (ragged last pages, an artifact twice in one
request; the copy rides, partly after the tile loop where a request's key
range is short); the Qwen3-4B and the long-context Qwen3-8B shapes over two
layers (the launches the step times, with key splits); the three-layer
batch with short suffixes and suffixes of one to three tokens over long
artifacts (too few key tiles to carry the copy: a gather launch of its own);
an artifact in the host pool (likewise); a batch with no suffix tokens; the
argument errors; and the chained layer loop captured in a HIP graph and
replayed."""

import numpy as np
import pytest
import torch

import synthdata as sd
from synthdata.workloads import ModelShape, Request, custom_workload

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload, dev_bf16
    from paper_2609_36722_amd.api import AttunerError, bf16_to_host


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _three_layer(index=96, suffixes=(400, 300, 257, 129)):
    return custom_workload("gather-3l", index, ModelShape(hidden=2560), [700, 1500, 333, 64, 16],
                           [Request((0, 1), suffixes[0]), Request((2,), suffixes[1]), Request((3, 1, 0), suffixes[2]),
                            Request((4, 4), suffixes[3])],
                           n_layers=3, rank=8, scale=2.0, gamma="uniform")


def _short_suffix():
    return custom_workload("gather-short", 97, ModelShape(hidden=2560), [2000, 3100, 517],
                           [Request((0, 1), 1), Request((2, 0), 3), Request((1,), 2)],
                           n_layers=2, rank=8, scale=1.0, gamma="uniform")


def _qkv(g, li):
    s = g.wl.shape
    w, x = g.layer_inputs(li)
    T = x.shape[0]
    nq, nkv = s.q_dim, s.kv_dim
    qkv = torch.empty(T, nq + 2 * nkv, dtype=torch.bfloat16, device="cuda")
    g.ctx.qproj_lora(dev_bf16(x), dev_bf16(np.concatenate([w["wq"], w["wk"], w["wv"]])),
                     dev_bf16(w["a"]) if g.wl.rank else None, dev_bf16(w["b"]) if g.wl.rank else None, g.wl.rank,
                     g.wl.scale, nq, qkv)
    return qkv, dev_bf16(w["gamma_q"]), dev_bf16(w["gamma_k"]), T


def _call(g, li, ins, kv, gather_layer=None, bt=None, cu_q=None):
    s = g.wl.shape
    qkv, gq, gk, T = ins
    nq, nkv = s.q_dim, s.kv_dim
    ld = nq + 2 * nkv
    o = torch.empty(T, s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(T, s.n_q_heads, dtype=torch.float32, device="cuda")
    args = (li, g.cu_q if cu_q is None else cu_q, g.cu_ctx, g.art_len, g.pos0, qkv[:, :nq], ld,
            qkv[:, nq:nq + nkv], qkv[:, nq + nkv:], ld, gq, gk, kv, g.rows, o)
    if gather_layer is None:
        g.ctx.suffix_attn(*args, lse)
    else:
        g.ctx.suffix_attn_gather(*args, bt, g.n_entries, gather_layer, lse)
    return o, lse


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _check_artifact_rows(g, kv_host):
    """Each request's cached rows hold its artifacts' K and V, in order, in every layer."""
    s = g.wl.shape
    cache = kv_host.reshape(len(g.layers), 2, s.n_kv_heads, g.rows, s.head_dim)
    for r, req in enumerate(g.wl.requests):
        if not req.artifact_ids:
            continue
        for plane, arts in ((0, g.art_k), (1, g.art_v)):
            want = np.concatenate([arts[a] for a in req.artifact_ids], axis=1)  # [layers][L][n_kv][d]
            lo, n = g.cu_ctx[r], g.art_len[r]
            assert np.array_equal(cache[:, plane, :, lo:lo + n], want.transpose(0, 2, 1, 3)), \
                f"request {r} plane {plane}"


def _chain(g, name, fused):
    """Reference: cache assembled for every layer, then suffix_attn per layer.
    Chained: layer 0's pages, then layer l's attention copies layer l + 1's
    (the last layer's copies layer 0 again, which leaves it unchanged)."""
    L = len(g.layers)
    ins = [_qkv(g, li) for li in range(L)]
    _say(f"{name}: reference (assemble_kv, suffix_attn per layer)")
    ref = [_call(g, li, ins[li], g.req_kv) for li in range(L)]
    torch.cuda.synchronize()
    kv_ref = bf16_to_host(g.req_kv)
    _check_artifact_rows(g, kv_ref)

    kv = torch.zeros_like(g.req_kv)
    bt = torch.zeros_like(g.block_table)
    cu, al = g.ctx.assemble_table(g.requests, g.suffix_cap, bt, g.rows)
    assert list(cu) == list(g.cu_ctx) and list(al) == list(g.art_len)
    g.ctx.gather_layers(bt, g.n_entries, 0, 1, kv, g.rows)
    got = []
    g.ctx.trace_begin()
    for li in range(L):
        nxt = li + 1 if li + 1 < L else 0
        _say(f"{name}: suffix_attn_gather layer {li}, copy layer {nxt}")
        got.append(_call(g, li, ins[li], kv, nxt, bt))
    torch.cuda.synchronize()
    launches = {k: v[0] for k, v in g.ctx.trace_end().items()}
    _say(f"{name}: launches {launches}")
    # which path ran: the copy inside every attention launch, or (short key
    # ranges, host pages) a gather launch of its own before each attention
    if fused is True:
        assert launches.get("attention_gather_kernel") == L and "gather_kernel" not in launches, launches
    elif fused is False:
        assert launches.get("gather_kernel") == L and "attention_gather_kernel" not in launches, launches
    for li in range(L):
        assert torch.equal(_bits(got[li][0]), _bits(ref[li][0])), f"{name}: O of layer {li}"
        assert torch.equal(_bits(got[li][1]), _bits(ref[li][1])), f"{name}: LSE of layer {li}"
    kv_got = bf16_to_host(kv)
    assert np.array_equal(kv_got, kv_ref), f"{name}: request cache"
    return launches


def test_gather_attn_three_layers_bit_exact():
    g = GpuWorkload(_three_layer(), layers=(0, 1, 2))
    try:
        _chain(g, "3-layer batch", fused=True)
    finally:
        g.close()


def test_gather_attn_short_batch_three_layers():
    g = GpuWorkload(_three_layer(101, (40, 100, 7, 129)), layers=(0, 1, 2))
    try:
        _chain(g, "3-layer batch, short suffixes", fused=False)
    finally:
        g.close()


def test_gather_attn_c2_two_layers():
    g = GpuWorkload(sd.make_workload("c2", gamma="uniform"), layers=(0, 1))
    try:
        _chain(g, "c2 layers 0-1", fused=True)
    finally:
        g.close()


def test_gather_attn_long_context_two_layers():
    g = GpuWorkload(sd.make_workload("c5", gamma="uniform"), layers=(0, 1))
    try:
        _chain(g, "c5 layers 0-1", fused=True)
    finally:
        g.close()


def test_gather_attn_short_suffixes():
    g = GpuWorkload(_short_suffix(), layers=(0, 1))
    try:
        _chain(g, "1-3 token suffixes", fused=False)
    finally:
        g.close()


def test_gather_attn_host_pages_fall_back():
    g = GpuWorkload(_three_layer(98), layers=(0, 1, 2), host_artifacts=(1,))
    try:
        _chain(g, "host-pool artifact", fused=False)
        # a call rejected after the copy was set apart enqueues nothing
        _say("host-pool artifact: rejected call")
        kv = torch.zeros_like(g.req_kv)
        bt = torch.zeros_like(g.block_table)
        g.ctx.assemble_table(g.requests, g.suffix_cap, bt, g.rows)
        ins = _qkv(g, 0)
        with pytest.raises(AttunerError) as e:
            _call(g, 3, ins, kv, 1, bt)                     # no layer 3 to attend over
        assert e.value.status == -1
        torch.cuda.synchronize()
        assert not bf16_to_host(kv).any()
    finally:
        g.close()


def test_gather_attn_no_suffix_and_errors():
    g = GpuWorkload(_three_layer(99), layers=(0, 1, 2))
    try:
        ins = _qkv(g, 0)
        kv = torch.zeros_like(g.req_kv)
        bt = torch.zeros_like(g.block_table)
        g.ctx.assemble_table(g.requests, g.suffix_cap, bt, g.rows)
        _say("no suffix tokens: the copy alone")
        zero_q = [0] * len(g.cu_q)
        empty = (ins[0][:0], ins[1], ins[2], 0)
        _call(g, 0, empty, kv, 2, bt, cu_q=zero_q)
        torch.cuda.synchronize()
        s = g.wl.shape
        got = bf16_to_host(kv).reshape(3, 2, s.n_kv_heads, g.rows, s.head_dim)
        want = bf16_to_host(g.req_kv).reshape(got.shape)
        assert np.array_equal(got[2], want[2]) and not got[:2].any()
        _say("argument errors")
        with pytest.raises(AttunerError) as e:
            _call(g, 1, ins, kv, 1, bt)                     # copies the layer it attends over
        assert e.value.status == -1
        with pytest.raises(AttunerError) as e:
            _call(g, 0, ins, kv, 3, bt)                     # no layer 3
        assert e.value.status == -5
        with pytest.raises(AttunerError) as e:
            _call(g, 0, ins, kv, 1, bt.clone())             # not the last assembled table
        assert e.value.status == -1
        torch.cuda.synchronize()
        assert not bf16_to_host(kv).reshape(got.shape)[:2].any()   # the rejected calls wrote nothing
    finally:
        g.close()


def test_gather_attn_graph_replays():
    """The chained layer loop captured in one HIP graph (layer 0's gather,
    then each layer's attention copying the next layer's pages), replayed
    three times into a cleared cache with eager work between the replays:
    every replay gives the eager chain's O, LSE and cache bit for bit."""
    g = GpuWorkload(_three_layer(100), layers=(0, 1, 2))
    try:
        L = len(g.layers)
        ins = [_qkv(g, li) for li in range(L)]
        kv = torch.zeros_like(g.req_kv)
        bt = torch.zeros_like(g.block_table)
        g.ctx.assemble_table(g.requests, g.suffix_cap, bt, g.rows)
        s = g.wl.shape
        outs = [(torch.empty(ins[li][3], s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda"),
                 torch.empty(ins[li][3], s.n_q_heads, dtype=torch.float32, device="cuda")) for li in range(L)]

        def chain(stream=None):
            g.ctx.gather_layers(bt, g.n_entries, 0, 1, kv, g.rows, stream=stream)
            nq, nkv = s.q_dim, s.kv_dim
            ld = nq + 2 * nkv
            for li in range(L):
                qkv, gq, gk, _ = ins[li]
                args = (li, g.cu_q, g.cu_ctx, g.art_len, g.pos0, qkv[:, :nq], ld, qkv[:, nq:nq + nkv],
                        qkv[:, nq + nkv:], ld, gq, gk, kv, g.rows, outs[li][0])
                if li + 1 < L:
                    g.ctx.suffix_attn_gather(*args, bt, g.n_entries, li + 1, outs[li][1], stream=stream)
                else:
                    g.ctx.suffix_attn(*args, outs[li][1], stream=stream)

        _say("graph of the chained layer loop: eager reference")
        chain()
        torch.cuda.synchronize()
        want = [(o.clone(), l.clone()) for o, l in outs]
        kv_want = kv.clone()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=cap):
            chain(stream=cap)
        torch.cuda.synchronize()
        for rep in range(3):
            _say(f"graph replay {rep}")
            kv.zero_()
            for o, l in outs:
                o.zero_()
                l.zero_()
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            for li in range(L):
                assert torch.equal(_bits(outs[li][0]), _bits(want[li][0])), f"replay {rep}: O of layer {li}"
                assert torch.equal(_bits(outs[li][1]), _bits(want[li][1])), f"replay {rep}: LSE of layer {li}"
            assert torch.equal(kv.view(torch.int16), kv_want.view(torch.int16)), f"replay {rep}: cache"
            _ = (torch.ones(1 << 20, device="cuda") * 2).sum().item()   # eager work between replays
        del graph
    finally:
        g.close()


@pytest.mark.parametrize("seed", [601, 602, 603, 604])
def test_gather_attn_random_batches(seed):
    """Random batches (1-5 requests, 1-4 artifacts each of 1-2500 tokens,
    suffixes of 1-700 tokens, 2-3 layers, the 4B or 8B head layout): the
    chained calls give O, LSE and cache bit for bit as the separate ones,
    whichever path the library takes."""
    rng = np.random.default_rng(seed)
    n_art = int(rng.integers(2, 7))
    lengths = [int(v) for v in rng.integers(1, 2500, size=n_art)]
    reqs = []
    for _ in range(int(rng.integers(1, 6))):
        arts = tuple(int(a) for a in rng.integers(0, n_art, size=int(rng.integers(1, 5))))
        reqs.append(Request(arts, int(rng.integers(1, 700))))
    hidden = 2560 if seed % 2 else 4096
    wl = custom_workload(f"gather-rand-{seed}", seed, ModelShape(hidden=hidden), lengths, reqs,
                         n_layers=3, rank=8, scale=1.0, gamma="uniform")
    layers = (0, 1, 2) if seed % 3 else (0, 1)
    _say(f"seed {seed}: artifacts {lengths}, requests {[(r.artifact_ids, r.suffix_len) for r in reqs]}")
    g = GpuWorkload(wl, layers=layers)
    try:
        launches = _chain(g, f"random batch {seed}", fused=None)
        assert launches.get("attention_gather_kernel", 0) + launches.get("gather_kernel", 0) == len(layers)
    finally:
        g.close()
