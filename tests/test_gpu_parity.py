"""GPU parity of every step of the suffix-prefill path against the fp64 oracle,
through the C ABI of libattuner (HIP kernels on gfx950).

Bars: the KV gather and block tables bit-exact; attention output O within
max|err| <= 1e-2 max|ref| and mean|err| <= 1e-3; bf16-stored intermediates
within max|err| <= 1e-2 max|ref| and mean|err| <= 2^-8 mean|ref| (see _tol).
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from synthdata.workloads import ModelShape, Request, custom_workload
from tests._tol import assert_intermediate_close, assert_o_close, assert_o_close_per_request, lse_bar

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload, dev_bf16, host_f64
    from paper_2609_36722_amd.api import AttunerError, Context, ModelCfg, bf16_to_host


def _say(msg):
    print(f"[case] {msg}", flush=True)


# ----------------------------------------------------------------------------
# K1: block table and gather (bit-exact)
# ----------------------------------------------------------------------------

def _check_assembly(g: "GpuWorkload"):
    wl = g.wl
    # block table: oracle's logical table mapped through the pool's physical pages
    lengths = list(wl.artifact_lengths)
    reqs = [(list(r.artifact_ids), r.suffix_len) for r in wl.requests]
    entries, cu = oracle.block_table(lengths, reqs, 16)
    phys = {a: g.ctx.artifact_pages(g.ids[a])[0] for a in g.ids}
    want = np.array([[phys[a][p], nv, dst, r] for a, p, nv, r, dst in entries.tolist()], np.int32).reshape(-1, 4)
    got = g.block_table.cpu().numpy().reshape(-1, 4)[: len(want)]
    assert np.array_equal(got, want), "block table differs"
    assert g.cu_ctx == cu.tolist()
    # gathered cache: every artifact row bit-exact; compare in the oracle's layout
    cache, cu2 = oracle.assemble(g.art_k, g.art_v, reqs, wl.shape.n_kv_heads, wl.shape.head_dim)
    assert cu2.tolist() == g.cu_ctx
    got_c = g.cache_view()
    for r, req in enumerate(wl.requests):
        lo, n = g.cu_ctx[r], g.art_len[r]
        assert np.array_equal(got_c[:, :, :, lo:lo + n], cache[:, :, :, lo:lo + n]), f"request {r} rows differ"


def test_gather_c1_bit_exact():
    _say("gather c1")
    g = GpuWorkload(sd.make_workload("c1"))
    try:
        _check_assembly(g)
    finally:
        g.close()


def test_gather_ragged_multilayer_multirequest_bit_exact():
    # partial last pages, single-token artifact, duplicates, an empty request,
    # several layers and requests
    _say("gather ragged 3 layers")
    shape = ModelShape(hidden=256)
    wl = custom_workload("ragged", 90, shape, [1, 15, 17, 33, 16, 200],
                         [Request((2, 0, 5), 7), Request((), 5), Request((3, 3, 1), 0), Request((4,), 32)],
                         n_layers=3)
    g = GpuWorkload(wl, layers=[0, 1, 2])
    try:
        _check_assembly(g)
    finally:
        g.close()


def test_gather_layers_split_from_table_bit_exact():
    # a1 and a2 as separate calls: the table once, then layers gathered out of
    # order on two streams; every artifact row bit-exact against the oracle's
    # assembly, a one-layer gather touches no other layer, and a table other
    # than the last one written is refused
    _say("assemble_table + gather_layers")
    cfg = ModelCfg(n_layers=3, hidden=256)
    rng = np.random.default_rng(11)
    lengths = {0: 17, 1: 40, 2: 1, 3: 16}
    with Context(cfg, pool_pages=16) as ctx:
        art_k, art_v, ids = {}, {}, {}
        for a, L in lengths.items():
            k = rng.integers(0, 2 ** 16, size=(3, 8, L, 128), dtype=np.uint16)
            v = rng.integers(0, 2 ** 16, size=(3, 8, L, 128), dtype=np.uint16)
            ids[a] = ctx.store_artifact(dev_bf16(k), dev_bf16(v))
            art_k[a], art_v[a] = k.transpose(0, 2, 1, 3), v.transpose(0, 2, 1, 3)   # [layers][L][Hkv][d]
        reqs = [([1, 0, 3], 5), ([], 3), ([2, 2, 1], 0)]
        requests, caps = [[ids[a] for a in r] for r, _ in reqs], [c for _, c in reqs]
        ne, rows = ctx.assemble_plan(requests, caps)
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(3 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        cu, al = ctx.assemble_table(requests, caps, bt, rows)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        ctx.gather_layers(bt, ne, 2, 1, kv, rows, stream=side)
        ctx.gather_layers(bt, ne, 0, 2, kv, rows)
        torch.cuda.synchronize()
        want, cu2 = oracle.assemble(art_k, art_v, reqs, 8, 128)
        assert cu == cu2.tolist()
        got = bf16_to_host(kv).reshape(3, 2, 8, rows, 128)
        for r in range(len(reqs)):
            lo, n = cu[r], al[r]
            assert np.array_equal(got[:, :, :, lo:lo + n], want[:, :, :, lo:lo + n]), f"request {r} rows differ"
        one = torch.zeros_like(kv)
        ctx.gather_layers(bt, ne, 1, 1, one, rows)
        torch.cuda.synchronize()
        got1 = bf16_to_host(one).reshape(3, 2, 8, rows, 128)
        assert not got1[0].any() and not got1[2].any()
        for r in range(len(reqs)):
            lo, n = cu[r], al[r]
            assert np.array_equal(got1[1, :, :, lo:lo + n], want[1, :, :, lo:lo + n]), f'layer 1, request {r}'
        with pytest.raises(AttunerError) as e:
            ctx.gather_layers(bt, ne, 2, 2, kv, rows)      # past the last layer
        assert e.value.status == -5
        other = torch.zeros_like(bt)
        with pytest.raises(AttunerError) as e:
            ctx.gather_layers(other, ne, 0, 1, kv, rows)   # not the table assemble_table wrote
        assert e.value.status == -1
        big = torch.zeros(3 * 2 * 8 * (rows + 1) * 128, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(AttunerError) as e:
            ctx.gather_layers(bt, ne, 0, 1, big, rows + 1)  # other cache geometry
        assert e.value.status == -1


def test_pool_reuse_after_release_bit_exact():
    _say("pool release and reuse")
    shape = ModelShape(hidden=256)
    cfg = ModelCfg(n_layers=2, hidden=256)
    rng = np.random.default_rng(3)
    with Context(cfg, pool_pages=6) as ctx:
        def art(L):
            k = rng.integers(0, 2 ** 16, size=(2, 8, L, 128), dtype=np.uint16)
            v = rng.integers(0, 2 ** 16, size=(2, 8, L, 128), dtype=np.uint16)
            return k, v, ctx.store_artifact(dev_bf16(k), dev_bf16(v))
        k0, v0, a0 = art(40)   # 3 pages
        k1, v1, a1 = art(20)   # 2 pages
        with pytest.raises(AttunerError) as e:
            art(20)             # needs 2 pages, 1 free
        assert e.value.status == -2
        ctx.release_artifact(a0)
        k2, v2, a2 = art(33)   # reuses freed pages
        ne, rows = ctx.assemble_plan([[a2, a1]], [4])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        cu, al = ctx.assemble_kv([[a2, a1]], [4], bt, kv, rows)
        torch.cuda.synchronize()
        got = bf16_to_host(kv).reshape(2, 2, 8, rows, 128)
        assert np.array_equal(got[:, 0, :, :33], k2) and np.array_equal(got[:, 1, :, :33], v2)
        assert np.array_equal(got[:, 0, :, 33:53], k1) and np.array_equal(got[:, 1, :, 33:53], v1)
        assert al == [53] and cu == [0, 57]


# ----------------------------------------------------------------------------
# K2: projection GEMM with fused LoRA epilogue
# ----------------------------------------------------------------------------

def _gemm_case(M, H, N, rank, lora_cols, seed, b_std=0.01):
    rng = np.random.default_rng(seed)
    f = lambda *s, std=1.0: sd.f32_to_bf16_bits(rng.standard_normal(s).astype(np.float32) * std)
    x, w = f(M, H), f(N, H, std=0.02)
    a, b = f(max(rank, 1), H, std=1 / math.sqrt(H))[:rank], f(max(lora_cols, 1), max(rank, 1), std=b_std)[:lora_cols, :rank]
    return x, w, np.ascontiguousarray(a), np.ascontiguousarray(b)


@pytest.mark.parametrize("M,H,N,rank,lora_cols", [
    (64, 2560, 6144, 8, 4096),     # c1 shapes
    (1, 512, 256, 16, 128),        # single token
    (37, 256, 384, 5, 256),        # ragged tokens, rank not a multiple of 8
    (300, 1024, 1280, 32, 1024),   # several token tiles with a ragged tail
    (1024, 512, 512, 64, 512),     # 128-token tiles, maximum rank
    (130, 256, 256, 0, 0),         # no adapter (merged deployment form)
    # token counts at which the launcher picks each larger tile (tokens x features)
    (1000, 512, 6144, 32, 4096),   # two-k-group 128 x 192, ragged last token tile, LoRA-down fused
    (500, 512, 6144, 16, 4096),    # two-k-group 128 x 96 (four waves)
    (1024, 2560, 6144, 48, 4096),  # two-k-group 128 x 192 reading t (rank > 32: 3 hidden slices, the last partial)
    (2048, 256, 2560, 8, 2048),    # 128 x 256
    (2100, 256, 6144, 16, 4096),   # 256 x 256, ragged; t from the separate down-projection
    (1024, 256, 1280, 12, 1024),   # 128 x 128; rank 12 reads B element by element
])
def test_qproj_lora_parity(M, H, N, rank, lora_cols):
    _say(f"qproj M={M} H={H} N={N} r={rank}")
    scale = 16.0 / max(rank, 1)
    x, w, a, b = _gemm_case(M, H, N, rank, lora_cols, seed=M + N)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), dev_bf16(w), dev_bf16(a) if rank else None, dev_bf16(b) if rank else None,
                       rank, scale, lora_cols, out)
        torch.cuda.synchronize()
        got = host_f64(out)
    ref = oracle.qproj_lora(oracle.decode_bf16(x), oracle.decode_bf16(w), oracle.decode_bf16(a) if rank else None,
                            oracle.decode_bf16(b) if rank else None, scale, lora_cols)
    assert_intermediate_close(got, ref, "q/k/v projection")


@pytest.mark.parametrize("seed", [401, 402, 403, 404, 405, 406])
def test_qproj_lora_random_shapes(seed):
    # Seeded random shapes (tokens 1-16 or 17-1600, hidden a multiple of 64,
    # outputs a multiple of 128, rank 0-64, adapted columns a multiple of
    # 32): the launcher's tile, the fused or separate down-projection and the
    # few-token GEMV paths vary with the shape.  B ~ N(0, 1) so that the
    # low-rank term is not lost in the base term's rounding.
    rng = np.random.default_rng(seed)
    M = int(rng.integers(1, 17)) if seed % 3 == 0 else int(rng.integers(17, 1601))   # every third: the GEMV
    H = 64 * int(rng.integers(2, 33))
    N = 128 * int(rng.integers(1, 33))
    rank = int(rng.integers(0, 65))
    lora_cols = 32 * int(rng.integers(1, N // 32 + 1)) if rank else 0
    _say(f"qproj random shape seed {seed}: M={M} H={H} N={N} r={rank} lora_cols={lora_cols}")
    scale = 16.0 / max(rank, 1)
    x, w, a, b = _gemm_case(M, H, N, rank, lora_cols, seed=seed, b_std=1.0)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), dev_bf16(w), dev_bf16(a) if rank else None, dev_bf16(b) if rank else None,
                       rank, scale, lora_cols, out)
        torch.cuda.synchronize()
        got = host_f64(out)
    ref = oracle.qproj_lora(oracle.decode_bf16(x), oracle.decode_bf16(w), oracle.decode_bf16(a) if rank else None,
                            oracle.decode_bf16(b) if rank else None, scale, lora_cols)
    assert_intermediate_close(got, ref, "q/k/v projection")


@pytest.mark.parametrize("rank", [8, 16, 32])
def test_lora_delta(rank):
    # B ~ N(0, 1) makes the low-rank term dominate, so a dropped, mis-scaled or
    # mis-indexed update cannot hide inside the bf16 rounding of the base term
    _say(f"lora delta r={rank}")
    M, H, N = 96, 2560, 6144
    scale = 16.0 / rank
    x, w, a, b = _gemm_case(M, H, N, rank, 4096, seed=rank, b_std=1.0)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        base = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), dev_bf16(w), dev_bf16(a), dev_bf16(b), rank, scale, 4096, out)
        ctx.qproj_lora(dev_bf16(x), dev_bf16(w), None, None, 0, 0.0, 0, base)
        torch.cuda.synchronize()
        delta = host_f64(out) - host_f64(base)
    xf, af, bf = oracle.decode_bf16(x), oracle.decode_bf16(a), oracle.decode_bf16(b)
    want = scale * (xf @ af.T) @ bf.T
    assert np.abs(delta[:, 4096:]).max() == 0.0, "keys/values must stay unadapted"
    err = np.abs(delta[:, :4096] - want)
    assert err.max() <= 1e-2 * np.abs(want).max()
    assert err.mean() <= 2.0 ** -7 * np.abs(want).mean()


# ----------------------------------------------------------------------------
# K3: QK-RMSNorm + RoPE
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("pos0,gamma", [(512, "uniform"), (0, "ones"), (40000, "uniform")])
def test_qk_norm_rope_parity(pos0, gamma):
    _say(f"qk_norm_rope pos0={pos0}")
    rng = np.random.default_rng(pos0 + 1)
    T, n_q, n_kv, d = 70, 32, 8, 128
    f = lambda *s: sd.f32_to_bf16_bits(rng.standard_normal(s).astype(np.float32))
    qkv = f(T, (n_q + 2 * n_kv) * d)
    gq = sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, d).astype(np.float32) if gamma == "uniform" else np.ones(d, np.float32))
    gk = sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, d).astype(np.float32) if gamma == "uniform" else np.ones(d, np.float32))
    art_len, cap = 33, 80
    rows = art_len + cap
    with Context(ModelCfg(n_layers=2, hidden=256), pool_pages=0) as ctx:
        qkv_d = dev_bf16(qkv)
        q_hat = torch.empty(T, n_q, d, dtype=torch.bfloat16, device="cuda")
        kv = torch.zeros(2 * 2 * n_kv * rows * d, dtype=torch.bfloat16, device="cuda")
        ld = (n_q + 2 * n_kv) * d
        ctx.qk_norm_rope(1, [0, T], [0, rows], [art_len], [pos0], qkv_d[:, :n_q * d], ld,
                         qkv_d[:, n_q * d:(n_q + n_kv) * d], qkv_d[:, (n_q + n_kv) * d:], ld, dev_bf16(gq),
                         dev_bf16(gk), q_hat, kv, rows)
        torch.cuda.synchronize()
        got_q = host_f64(q_hat)
        cache = bf16_to_host(kv).reshape(2, 2, n_kv, rows, d)
    x = oracle.decode_bf16(qkv)
    pos = pos0 + np.arange(T)
    want_q = oracle.rope(oracle.rms_norm_heads(x[:, :n_q * d].reshape(T, n_q, d), oracle.decode_bf16(gq), 1e-6), pos, 1e6)
    want_k = oracle.rope(oracle.rms_norm_heads(x[:, n_q * d:(n_q + n_kv) * d].reshape(T, n_kv, d),
                                               oracle.decode_bf16(gk), 1e-6), pos, 1e6)
    assert_intermediate_close(got_q, want_q, "q_hat")
    got_k = oracle.decode_bf16(cache[1, 0, :, art_len:art_len + T]).transpose(1, 0, 2)
    assert_intermediate_close(got_k, want_k, "k_hat")
    # values are copied bit for bit; other rows and layer 0 untouched
    want_v = qkv[:, (n_q + n_kv) * d:].reshape(T, n_kv, d).transpose(1, 0, 2)
    assert np.array_equal(cache[1, 1, :, art_len:art_len + T], want_v)
    assert not cache[0].any() and not cache[1, :, :, :art_len].any() and not cache[1, :, :, art_len + T:].any()


# ----------------------------------------------------------------------------
# K4 alone: attention on identical bf16 inputs
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("reqs", [
    [(512, 64)],                       # c1-like: 2 splits
    [(8192, 256)],                     # c2 layer: split-KV
    [(0, 300)],                        # plain causal, ragged block
    [(37, 1), (1000, 45), (0, 5), (2047, 64), (3, 130)],   # varlen batch, S = 1, tiny art
    [(8192, 64)],                      # 8 blocks: 16 key splits, the most the merge takes
    [(100, 7), (50, 0), (0, 0), (700, 33)],                # zero-length suffixes inside a batch
    [(16 * (i % 5), 1 + (i % 3)) for i in range(64)],      # the maximum of 64 requests
])
def test_attention_parity(reqs):
    _say(f"attention {reqs}")
    rng = np.random.default_rng(len(reqs) * 7 + reqs[0][0])
    n_q, n_kv, d = 32, 8, 128
    cu_q, cu_ctx, art_len = [0], [0], []
    for L, S in reqs:
        cu_q.append(cu_q[-1] + S)
        cu_ctx.append(cu_ctx[-1] + L + S + 3)   # 3 spare rows after each request
        art_len.append(L)
    T, rows = cu_q[-1], cu_ctx[-1]
    f = lambda *s: sd.f32_to_bf16_bits(rng.standard_normal(s).astype(np.float32))
    q = f(T, n_q, d)
    cache = f(1, 2, n_kv, rows, d)
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        o = torch.empty(T, n_q, d, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(T, n_q, dtype=torch.float32, device="cuda")
        ctx.attention(0, cu_q, cu_ctx, art_len, dev_bf16(q), dev_bf16(cache), rows, o, lse)
        torch.cuda.synchronize()
        got, got_lse = host_f64(o), lse.cpu().numpy()
    qf, cf = oracle.decode_bf16(q), oracle.decode_bf16(cache)
    for r, (L, S) in enumerate(reqs):
        if S == 0:
            continue
        kk = cf[0, 0, :, cu_ctx[r]:cu_ctx[r] + L + S].transpose(1, 0, 2)
        vv = cf[0, 1, :, cu_ctx[r]:cu_ctx[r] + L + S].transpose(1, 0, 2)
        ref, ref_lse = oracle.attention(qf[cu_q[r]:cu_q[r + 1]], kk, vv, L, return_lse=True)
        assert_o_close(got[cu_q[r]:cu_q[r + 1]], ref, f"O request {r}")
        assert np.abs(got_lse[cu_q[r]:cu_q[r + 1]] - ref_lse).max() <= 1e-3 * max(1.0, np.abs(ref_lse).max())


@pytest.mark.parametrize("seed", [101, 102, 103, 104])
def test_attention_random_batches(seed):
    # Seeded random batches (1-24 requests, 0-3000 cached keys, 0-300 suffix
    # rows): the key-split plan and the launch order (request order or
    # longest first, whichever the host's model prefers) vary from batch to
    # batch; every request's rows against the oracle.
    rng = np.random.default_rng(seed)
    n_req = int(rng.integers(1, 25))
    reqs = [(int(rng.integers(0, 3001)), int(rng.integers(0, 301))) for _ in range(n_req)]
    if all(S == 0 for _, S in reqs):
        reqs[0] = (reqs[0][0], 17)
    _say(f"attention random batch seed {seed}: {reqs}")
    n_q, n_kv, d = 32, 8, 128
    cu_q, cu_ctx, art_len = [0], [0], []
    for L, S in reqs:
        cu_q.append(cu_q[-1] + S)
        cu_ctx.append(cu_ctx[-1] + L + S + int(rng.integers(0, 5)))   # a few spare rows, varying
        art_len.append(L)
    T, rows = cu_q[-1], cu_ctx[-1]
    f = lambda *s: sd.f32_to_bf16_bits(rng.standard_normal(s).astype(np.float32))
    q = f(T, n_q, d)
    cache = f(1, 2, n_kv, rows, d)
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        o = torch.empty(T, n_q, d, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(T, n_q, dtype=torch.float32, device="cuda")
        ctx.attention(0, cu_q, cu_ctx, art_len, dev_bf16(q), dev_bf16(cache), rows, o, lse)
        torch.cuda.synchronize()
        got, got_lse = host_f64(o), lse.cpu().numpy()
    qf, cf = oracle.decode_bf16(q), oracle.decode_bf16(cache)
    for r, (L, S) in enumerate(reqs):
        if S == 0:
            continue
        kk = cf[0, 0, :, cu_ctx[r]:cu_ctx[r] + L + S].transpose(1, 0, 2)
        vv = cf[0, 1, :, cu_ctx[r]:cu_ctx[r] + L + S].transpose(1, 0, 2)
        ref, ref_lse = oracle.attention(qf[cu_q[r]:cu_q[r + 1]], kk, vv, L, return_lse=True)
        assert_o_close(got[cu_q[r]:cu_q[r + 1]], ref, f"O request {r}")
        assert np.abs(got_lse[cu_q[r]:cu_q[r + 1]] - ref_lse).max() <= 1e-3 * max(1.0, np.abs(ref_lse).max())


@pytest.mark.parametrize("kind", ["rising", "spike"])
def test_attention_scores_outrun_first_tile(kind):
    # Scores that grow along the keys ("rising": by about 40 log2 units over
    # the artifact) or one key far above the rest ("spike": about 260 log2
    # units, past the fp32 range of 2^(s - m) for the first tile's m): the
    # exponentials of later tiles against the first tile's reference would
    # exceed any fixed bound, so the result rests on the kernel's redo with a
    # row max per tile.
    _say(f"attention scores outrunning the first tile: {kind}")
    rng = np.random.default_rng(23 if kind == "rising" else 29)
    n_q, n_kv, d = 32, 8, 128
    reqs = [(2048, 64), (4096, 100), (300, 20)]
    cu_q, cu_ctx, art_len = [0], [0], []
    for L, S in reqs:
        cu_q.append(cu_q[-1] + S)
        cu_ctx.append(cu_ctx[-1] + L + S)
        art_len.append(L)
    T, rows = cu_q[-1], cu_ctx[-1]
    q = rng.standard_normal((T, n_q, d)).astype(np.float32) * 0.5 + 1.0
    kc = rng.standard_normal((n_kv, rows, d)).astype(np.float32)
    for r, (L, S) in enumerate(reqs):
        pos = np.arange(L + S)
        if kind == "rising":   # mean score grows by ~ 40 log2 units over the artifact
            kc[:, cu_ctx[r]:cu_ctx[r] + L + S, :] += (3.0 * pos / max(L, 1))[None, :, None]
        else:                  # one artifact key far above all others
            kc[:, cu_ctx[r] + (2 * L) // 3, :] = 16.0
    vc = rng.standard_normal((n_kv, rows, d)).astype(np.float32)
    q = sd.f32_to_bf16_bits(q)
    cache = sd.f32_to_bf16_bits(np.stack([kc, vc])[None])
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        o = torch.empty(T, n_q, d, dtype=torch.bfloat16, device="cuda")
        lse = torch.empty(T, n_q, dtype=torch.float32, device="cuda")
        ctx.attention(0, cu_q, cu_ctx, art_len, dev_bf16(q), dev_bf16(cache), rows, o, lse)
        torch.cuda.synchronize()
        got, got_lse = host_f64(o), lse.cpu().numpy()
    assert np.isfinite(got).all() and np.isfinite(got_lse).all()
    qf, cf = oracle.decode_bf16(q), oracle.decode_bf16(cache)
    for r, (L, S) in enumerate(reqs):
        kk = cf[0, 0, :, cu_ctx[r]:cu_ctx[r] + L + S].transpose(1, 0, 2)
        vv = cf[0, 1, :, cu_ctx[r]:cu_ctx[r] + L + S].transpose(1, 0, 2)
        ref, ref_lse = oracle.attention(qf[cu_q[r]:cu_q[r + 1]], kk, vv, L, return_lse=True)
        assert_o_close(got[cu_q[r]:cu_q[r + 1]], ref, f"O request {r}")
        assert np.abs(got_lse[cu_q[r]:cu_q[r + 1]] - ref_lse).max() <= 1e-3 * max(1.0, np.abs(ref_lse).max())


def test_attention_never_reads_future_suffix_rows():
    # a huge value planted at suffix row j must not move any row i < j
    _say("attention future-row probe")
    rng = np.random.default_rng(11)
    n_q, n_kv, d, L, S = 32, 8, 128, 200, 64
    rows = L + S
    f = lambda *s: sd.f32_to_bf16_bits(rng.standard_normal(s).astype(np.float32))
    q, cache = f(S, n_q, d), f(1, 2, n_kv, rows, d)
    j = 40
    planted = cache.copy()
    planted[0, 1, :, L + j, :] = sd.f32_to_bf16_bits(np.full(d, 3.0e4, np.float32))
    planted[0, 0, :, L + j, :] = sd.f32_to_bf16_bits(np.full(d, 30.0, np.float32))
    outs = []
    with Context(ModelCfg(n_layers=1, hidden=256), pool_pages=0) as ctx:
        for c in (cache, planted):
            o = torch.empty(S, n_q, d, dtype=torch.bfloat16, device="cuda")
            ctx.attention(0, [0, S], [0, rows], [L], dev_bf16(q), dev_bf16(c), rows, o)
            torch.cuda.synchronize()
            outs.append(bf16_to_host(o))
    assert np.array_equal(outs[0][:j], outs[1][:j])
    assert not np.array_equal(outs[0][j:], outs[1][j:])


# ----------------------------------------------------------------------------
# the whole suffix layer (a2..a5) against the oracle
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("gamma,scale", [("uniform", None), ("ones", 0.0), ("uniform", 1.0)])
def test_suffix_layer_c1(gamma, scale):
    _say(f"suffix layer c1 gamma={gamma} scale={scale}")
    kw = {"gamma": gamma}
    if scale is not None:
        kw["scale"] = scale
    g = GpuWorkload(sd.make_workload("c1", **kw))
    try:
        out = g.run_layer(0)
        ref = g.oracle_layer(0, 0)
        assert_intermediate_close(host_f64(out["qkv"][:, :4096]), ref["q"].reshape(64, -1), "q")
        assert_o_close(host_f64(out["o"]), ref["o"])
        # the suffix keys and values now sit after the artifacts in the cache
        c = g.cache_view()
        L = g.art_len[0]
        keys = np.concatenate([oracle.decode_bf16(g.art_k[a][0]) for a in g.wl.requests[0].artifact_ids])
        bar = lse_bar(ref["q_hat"], np.concatenate([keys, ref["k_hat"]]), 32, 8)
        assert np.abs(out["lse"].cpu().numpy() - ref["lse"]).max() <= bar
        assert_intermediate_close(oracle.decode_bf16(c[0, 0, :, L:L + 64]).transpose(1, 0, 2), ref["k_hat"], "k_hat")
    finally:
        g.close()


def test_suffix_layer_lora_delta_c1():
    # paper-scale B is small; B ~ N(0, 1) makes the adapter visible in O
    _say("suffix layer c1 big B")
    g = GpuWorkload(sd.make_workload("c1", gamma="uniform", b_std=1.0))
    try:
        out = g.run_layer(0)
        assert_o_close(host_f64(out["o"]), g.oracle_layer(0, 0)["o"])
    finally:
        g.close()


def test_suffix_layer_varlen_batch():
    _say("suffix layer varlen batch")
    shape = ModelShape(hidden=512)
    wl = custom_workload("varlen", 91, shape, [256, 700, 33, 1024, 16, 513],
                         [Request((1, 0), 64), Request((), 17), Request((3, 5, 2, 4), 200), Request((2,), 1),
                          Request((5, 5), 96, pos0=5000)], rank=16, scale=1.0, gamma="uniform")
    g = GpuWorkload(wl)
    try:
        out = g.run_layer(0)
        got = host_f64(out["o"])
        for r in range(len(wl.requests)):
            ref = g.oracle_layer(0, r)
            assert_o_close(got[g.cu_q[r]:g.cu_q[r + 1]], ref["o"], f"O request {r}")
    finally:
        g.close()


# ----------------------------------------------------------------------------
# full prefill (a6), and PIC at offset zero == Full (single artifact)
# ----------------------------------------------------------------------------

def _full_inputs(H, N, rank, seed):
    rng = np.random.default_rng(seed)
    f = lambda *s, std=1.0: sd.f32_to_bf16_bits(rng.standard_normal(s).astype(np.float32) * std)
    return dict(x=f(N, H), wq=f(4096, H, std=0.02), wk=f(1024, H, std=0.02), wv=f(1024, H, std=0.02),
                a=f(max(rank, 1), H, std=1 / math.sqrt(H))[:rank], b=f(4096, max(rank, 1), std=0.01)[:, :rank],
                gq=sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, 128).astype(np.float32)),
                gk=sd.f32_to_bf16_bits(rng.uniform(0.5, 1.5, 128).astype(np.float32)))


def _gpu_full(ctx, inp, pos0, rank, scale, rows=None):
    x = inp["x"] if rows is None else inp["x"][rows]
    N = x.shape[0]
    wqkv = dev_bf16(np.concatenate([inp["wq"], inp["wk"], inp["wv"]]))
    o = torch.empty(N, 32, 128, dtype=torch.bfloat16, device="cuda")
    k = torch.empty(8, N, 128, dtype=torch.bfloat16, device="cuda")
    v = torch.empty(8, N, 128, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(N, 32, dtype=torch.float32, device="cuda")
    ctx.full_prefill(pos0, dev_bf16(x), wqkv, dev_bf16(np.ascontiguousarray(inp["a"])) if rank else None,
                     dev_bf16(np.ascontiguousarray(inp["b"])) if rank else None, rank, scale, dev_bf16(inp["gq"]),
                     dev_bf16(inp["gk"]), o, k, v, lse)
    torch.cuda.synchronize()
    return o, k, v, lse


@pytest.mark.parametrize("N,pos0,rank", [(300, 0, 0), (129, 1000, 8)])
def test_full_prefill_parity(N, pos0, rank):
    _say(f"full prefill N={N} pos0={pos0} r={rank}")
    H = 512
    inp = _full_inputs(H, N, rank, seed=N)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        o, k, v, lse = _gpu_full(ctx, inp, pos0, rank, 2.0)
    d = {n: oracle.decode_bf16(inp[n]) for n in inp}
    ref = oracle.full_prefill(d["x"], d["wq"], d["wk"], d["wv"], d["gq"], d["gk"], pos0, 32, 8, 1e6, 1e-6,
                              a=d["a"] if rank else None, b=d["b"] if rank else None, scale=2.0)
    assert_o_close(host_f64(o), ref["o"])
    assert_intermediate_close(host_f64(k).transpose(1, 0, 2), ref["k_hat"], "k_hat")
    assert_intermediate_close(host_f64(v).transpose(1, 0, 2), ref["v"], "v")
    assert np.abs(lse.cpu().numpy() - ref["lse"]).max() <= lse_bar(ref["q_hat"], ref["k_hat"], 32, 8)


def test_encode_store_assemble_equals_full_prefill():
    # one artifact at offset 0: encode it alone with full_prefill, store it, and
    # run the suffix over it; the suffix rows must match a full prefill of
    # artifact + suffix (the single-layer PIC == Full identity), on the GPU
    _say("encode -> store -> suffix == full")
    H, La, S = 512, 200, 50
    inp = _full_inputs(H, La + S, 0, seed=5)
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=32) as ctx:
        _, ka, va, _ = _gpu_full(ctx, inp, 0, 0, 0.0, rows=slice(0, La))
        aid = ctx.store_artifact(ka.unsqueeze(0).contiguous(), va.unsqueeze(0).contiguous())
        ne, rows = ctx.assemble_plan([[aid]], [S])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        cu, al = ctx.assemble_kv([[aid]], [S], bt, kv, rows)
        wqkv = dev_bf16(np.concatenate([inp["wq"], inp["wk"], inp["wv"]]))
        qkv = torch.empty(S, 6144, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(inp["x"][La:]), wqkv, None, None, 0, 0.0, 0, qkv)
        o = torch.empty(S, 32, 128, dtype=torch.bfloat16, device="cuda")
        ctx.suffix_attn(0, [0, S], cu, al, [La], qkv[:, :4096], 6144, qkv[:, 4096:5120], qkv[:, 5120:], 6144,
                        dev_bf16(inp["gq"]), dev_bf16(inp["gk"]), kv, rows, o)
        o_full, _, _, _ = _gpu_full(ctx, inp, 0, 0, 0.0)
        torch.cuda.synchronize()
        got_sfx, got_full = host_f64(o), host_f64(o_full)[La:]
    d = {n: oracle.decode_bf16(inp[n]) for n in inp}
    ref = oracle.full_prefill(d["x"], d["wq"], d["wk"], d["wv"], d["gq"], d["gk"], 0, 32, 8, 1e6, 1e-6)["o"][La:]
    assert_o_close(got_sfx, ref, "suffix over stored artifact")
    assert_o_close(got_full, ref, "full prefill suffix rows")


# ----------------------------------------------------------------------------
# errors forced from the host
# ----------------------------------------------------------------------------

def test_error_codes():
    _say("error codes")
    cfg = ModelCfg(n_layers=1, hidden=256)
    with Context(cfg, pool_pages=2) as ctx:
        k = torch.zeros(1, 8, 20, 128, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(AttunerError) as e:
            ctx.store_artifact(k, k, n_tokens=0)
        assert e.value.status == -1
        with pytest.raises(AttunerError) as e:
            ctx.store_artifact(torch.zeros(1, 8, 40, 128, dtype=torch.bfloat16, device="cuda"),
                               torch.zeros(1, 8, 40, 128, dtype=torch.bfloat16, device="cuda"))
        assert e.value.status == -2  # 3 pages > 2
        aid = ctx.store_artifact(k, k)
        with pytest.raises(AttunerError) as e:
            ctx.assemble_plan([[aid, 12345]], [0])
        assert e.value.status == -3
        with pytest.raises(AttunerError) as e:
            ctx.release_artifact(777)
        assert e.value.status == -3
        with pytest.raises(AttunerError) as e:
            ctx.assemble_plan([[aid]] * 65, [0] * 65)
        assert e.value.status == -5
        ne, rows = ctx.assemble_plan([[aid]], [4])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * 8 * (rows + 1) * 128, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(AttunerError) as e:   # cache_rows that disagrees with the plan
            ctx.assemble_kv([[aid]], [4], bt, kv, rows + 1)
        assert e.value.status == -5
        x = torch.zeros(4, 256, dtype=torch.bfloat16, device="cuda")
        w = torch.zeros(256, 256, dtype=torch.bfloat16, device="cuda")
        out = torch.zeros(4, 256, dtype=torch.bfloat16, device="cuda")
        a = torch.zeros(65, 256, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(AttunerError) as e:
            ctx.qproj_lora(x, w, a, a, 65, 1.0, 128, out)
        assert e.value.status == -5
        with pytest.raises(AttunerError) as e:
            ctx.qproj_lora(x, torch.zeros(100, 256, dtype=torch.bfloat16, device="cuda"), None, None, 0, 0.0, 0, out)
        assert e.value.status == -1
        q = torch.zeros(4, 32, 128, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(AttunerError) as e:   # suffix longer than its reserved rows
            ctx.attention(0, [0, 4], [0, rows], [rows - 2], q, kv, rows, q)
        assert e.value.status == -1
        with pytest.raises(AttunerError) as e:
            ctx.attention(1, [0, 4], [0, rows], [1], q, kv, rows, q)
        assert e.value.status == -1
        # q/k/v rows must be 16-byte aligned with row strides a multiple of 8
        g = torch.ones(128, dtype=torch.bfloat16, device="cuda")
        for ld, off in ((48 * 128 + 8, 1), (48 * 128 + 4, 0)):   # shifted start; row stride not a multiple of 8
            qkv = torch.zeros(4, ld, dtype=torch.bfloat16, device="cuda")
            q_raw, k_raw, v_raw = qkv[:, off:], qkv[:, 32 * 128:], qkv[:, 40 * 128:]
            with pytest.raises(AttunerError) as e:
                ctx.qk_norm_rope(0, [0, 4], [0, rows], [1], [1], q_raw, ld, k_raw, v_raw, ld, g, g, q, kv, rows)
            assert e.value.status == -1
            with pytest.raises(AttunerError) as e:
                ctx.suffix_attn(0, [0, 4], [0, rows], [1], [1], q_raw, ld, k_raw, v_raw, ld, g, g, kv, rows, q)
            assert e.value.status == -1


def test_suffix_attn_64_requests():
    # 64 requests in one call (the work list's capacity): empty, one-token and
    # multi-block suffixes over shared and private artifacts
    _say("suffix attention 64 requests")
    shape = ModelShape(hidden=256)
    rng = np.random.default_rng(93)
    lengths = [int(v) for v in rng.integers(1, 300, size=12)]
    reqs = []
    for i in range(64):
        k = int(rng.integers(0, 3))
        reqs.append(Request(tuple(int(a) for a in rng.choice(12, size=k, replace=False)),
                            int(rng.choice([0, 1, 5, 64, 70]))))
    wl = custom_workload("batch64", 94, shape, lengths, reqs, rank=8, scale=2.0, gamma="uniform")
    g = GpuWorkload(wl)
    try:
        out = g.run_layer(0, with_lse=False)
        got = host_f64(out["o"])
        refs = []
        for r in range(64):
            if wl.requests[r].suffix_len == 0:
                continue
            ref = g.oracle_layer(0, r)["o"]
            assert_o_close_per_request(got[g.cu_q[r]:g.cu_q[r + 1]], ref, f"O request {r}")
            refs.append(ref)
        assert_o_close(got, np.concatenate(refs), "batch O")
    finally:
        g.close()
