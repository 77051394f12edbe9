"""Artifact caches kept in CPU RAM (the pinned host pool): assembly gathers
host pages over the host link into the request cache, bit-exact against the
oracle's assembly, mixed with HBM-pool artifacts, all layers at once and
layer by layer, and in an interleaved prompt; pages are reused after a
release.  The copy-engine route (host pages copied into an HBM staging pool,
then gathered) gives the same cache, eagerly and from a replayed graph."""

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import dev_bf16
    from paper_2609_36722_amd.api import AttunerError, Context, ModelCfg, bf16_to_host
    from paper_2609_36722_amd._lib import HOST_PAGE_FLAG, STAGE_PAGE_FLAG


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _store_mixed(ctx, rng, lengths, host_set, n_layers):
    art_k, art_v, ids = {}, {}, {}
    for a, L in enumerate(lengths):
        k = rng.integers(0, 2 ** 16, size=(n_layers, 8, L, 128), dtype=np.uint16)
        v = rng.integers(0, 2 ** 16, size=(n_layers, 8, L, 128), dtype=np.uint16)
        store = ctx.store_artifact_host if a in host_set else ctx.store_artifact
        ids[a] = store(dev_bf16(k), dev_bf16(v))
        art_k[a], art_v[a] = k.transpose(0, 2, 1, 3), v.transpose(0, 2, 1, 3)   # [layers][L][Hkv][d]
    return art_k, art_v, ids


def test_host_pool_assembly_bit_exact():
    _say("host pool assembly")
    rng = np.random.default_rng(81)
    lengths = [17, 40, 1, 33, 300]
    host = {1, 2, 4}
    with Context(ModelCfg(n_layers=3, hidden=256), pool_pages=8) as ctx:
        ctx.host_pool_create(40)
        art_k, art_v, ids = _store_mixed(ctx, rng, lengths, host, 3)
        assert ctx.host_pool_info() == (40, 40 - 3 - 1 - 19)
        for a in host:
            pages, _ = ctx.artifact_pages(ids[a])
            assert all(p & HOST_PAGE_FLAG for p in pages)
        reqs = [([1, 0, 4], 5), ([], 3), ([2, 2, 3, 1], 0)]
        requests, caps = [[ids[a] for a in r] for r, _ in reqs], [c for _, c in reqs]
        ne, rows = ctx.assemble_plan(requests, caps)
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(3 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        cu, al = ctx.assemble_kv(requests, caps, bt, kv, rows)
        torch.cuda.synchronize()
        entries, cu2 = oracle.block_table(lengths, reqs, 16)
        phys = {a: ctx.artifact_pages(ids[a])[0] for a in ids}
        want = np.array([[phys[a][p], nv, dst, r] for a, p, nv, r, dst in entries.tolist()], np.int32).reshape(-1, 4)
        assert np.array_equal(bt.cpu().numpy().reshape(-1, 4), want)
        cache, _ = oracle.assemble(art_k, art_v, reqs, 8, 128)
        got = bf16_to_host(kv).reshape(3, 2, 8, rows, 128)
        for r in range(len(reqs)):
            lo, n = cu[r], al[r]
            assert np.array_equal(got[:, :, :, lo:lo + n], cache[:, :, :, lo:lo + n]), f"request {r}"
        # layer by layer on a second stream, from the same table
        kv2 = torch.zeros_like(kv)
        cu3, al3 = ctx.assemble_table(requests, caps, bt, rows)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        for l in (2, 0, 1):
            ctx.gather_layers(bt, ne, l, 1, kv2, rows, stream=side)
        torch.cuda.synchronize()
        got2 = bf16_to_host(kv2).reshape(3, 2, 8, rows, 128)
        for r in range(len(reqs)):
            lo, n = cu[r], al[r]
            assert np.array_equal(got2[:, :, :, lo:lo + n], cache[:, :, :, lo:lo + n]), f"request {r} per layer"
        # release a host artifact and reuse its pages for a new one
        ctx.release_artifact(ids[4])
        assert ctx.host_pool_info()[1] == 40 - 3 - 1
        k = rng.integers(0, 2 ** 16, size=(3, 8, 200, 128), dtype=np.uint16)
        nid = ctx.store_artifact_host(dev_bf16(k), dev_bf16(k))
        ne, rows = ctx.assemble_plan([[nid]], [0])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(3 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        ctx.assemble_kv([[nid]], [0], bt, kv, rows)
        torch.cuda.synchronize()
        got = bf16_to_host(kv).reshape(3, 2, 8, rows, 128)
        assert np.array_equal(got[:, 0], k) and np.array_equal(got[:, 1], k)


def test_host_pool_segments_and_errors():
    _say("host pool segments + errors")
    rng = np.random.default_rng(82)
    lengths = [50, 20]
    with Context(ModelCfg(n_layers=2, hidden=256), pool_pages=4) as ctx:
        with pytest.raises(AttunerError) as e:
            ctx.store_artifact_host(torch.zeros(2, 8, 4, 128, dtype=torch.bfloat16, device="cuda"),
                                    torch.zeros(2, 8, 4, 128, dtype=torch.bfloat16, device="cuda"))
        assert e.value.status == -1                 # no host pool yet
        ctx.host_pool_create(8)
        with pytest.raises(AttunerError) as e:
            ctx.host_pool_create(8)                 # a second one
        assert e.value.status == -1
        art_k, art_v, ids = _store_mixed(ctx, rng, lengths, {0}, 2)
        with pytest.raises(AttunerError) as e:
            ctx.store_artifact_host(torch.zeros(2, 8, 100, 128, dtype=torch.bfloat16, device="cuda"),
                                    torch.zeros(2, 8, 100, 128, dtype=torch.bfloat16, device="cuda"))
        assert e.value.status == -2                 # host pool full (7 pages needed, 4 free)
        prompts = [[-3, 0, -2, 1, -4]]
        segs = [[ids[s] if s >= 0 else s for s in p] for p in prompts]
        ne, rows, ns = ctx.assemble_segments_plan(segs)
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        cu, spans = ctx.assemble_segments(segs, bt, kv, rows)
        torch.cuda.synchronize()
        e2, _, _ = oracle.block_table_segments(lengths, prompts, 16)
        got = bf16_to_host(kv).reshape(2, 2, 8, rows, 128)
        for a_idx, p, nv, r, dst in e2.tolist():
            src = slice(16 * p, 16 * p + nv)
            assert np.array_equal(got[:, 0, :, dst:dst + nv], art_k[a_idx][:, src].transpose(0, 2, 1, 3))
            assert np.array_equal(got[:, 1, :, dst:dst + nv], art_v[a_idx][:, src].transpose(0, 2, 1, 3))


# ----------------------------------------------------------------------------
# copy-engine route: host pages -> HBM staging pool -> request cache
# ----------------------------------------------------------------------------

def _staged_table_want(ctx, ids, lengths, reqs):
    """The block table the staged assembly must write: the oracle's entries
    through the physical pages, the i-th smallest distinct host page renamed
    to staging page i; and the distinct count."""
    entries, _ = oracle.block_table(lengths, reqs, 16)
    phys = {a: ctx.artifact_pages(ids[a])[0] for a in ids}
    host = sorted({phys[a][p] for a, p, _, _, _ in entries.tolist() if phys[a][p] & HOST_PAGE_FLAG})
    slot = {pg: i for i, pg in enumerate(host)}
    rows = []
    for a, p, nv, r, dst in entries.tolist():
        pg = phys[a][p]
        if pg & HOST_PAGE_FLAG:
            pg = slot[pg] | STAGE_PAGE_FLAG
        rows.append([pg, nv, dst, r])
    return np.array(rows, np.int32).reshape(-1, 4), len(slot)


def _check_cache(kv, cache, cu, al, n_layers, rows, what):
    got = bf16_to_host(kv).reshape(n_layers, 2, 8, rows, 128)
    for r in range(len(cu) - 1):
        lo, n = cu[r], al[r]
        assert np.array_equal(got[:, :, :, lo:lo + n], cache[:, :, :, lo:lo + n]), f"{what}: request {r}"


def test_staged_assembly_bit_exact():
    _say("staged host pool assembly")
    rng = np.random.default_rng(83)
    lengths = [17, 40, 1, 33, 300]
    host = {1, 2, 4}
    with Context(ModelCfg(n_layers=3, hidden=256), pool_pages=8) as ctx:
        ctx.host_pool_create(40)
        art_k, art_v, ids = _store_mixed(ctx, rng, lengths, host, 3)
        reqs = [([1, 0, 4], 5), ([], 3), ([2, 2, 3, 1], 0)]
        requests, caps = [[ids[a] for a in r] for r, _ in reqs], [c for _, c in reqs]
        ne, rows = ctx.assemble_plan(requests, caps)
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        with pytest.raises(AttunerError) as e:
            ctx.assemble_table_staged(requests, caps, bt, rows)
        assert e.value.status == -1                 # no staging pool yet
        ctx.stage_pool_create(23)                   # the batch's distinct host pages: 3 + 1 + 19
        with pytest.raises(AttunerError) as e:
            ctx.stage_pool_create(23)
        assert e.value.status == -1
        cu, al, staged = ctx.assemble_table_staged(requests, caps, bt, rows)
        torch.cuda.synchronize()
        want, n_distinct = _staged_table_want(ctx, ids, lengths, reqs)
        assert staged == n_distinct == 23
        assert np.array_equal(bt.cpu().numpy().reshape(-1, 4), want)
        pages, runs = ctx.stage_pool_info()
        assert pages == 23 and runs == 1             # host pages 0..22: one copy per layer
        cache, cu_o = oracle.assemble(art_k, art_v, reqs, 8, 128)
        assert list(cu) == list(cu_o)
        # layer by layer: copies on one stream, each layer's gather on a
        # second one after that layer's copies (event)
        kv = torch.zeros(3 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        copy, side = torch.cuda.Stream(), torch.cuda.Stream()
        copy.wait_stream(torch.cuda.current_stream())
        side.wait_stream(torch.cuda.current_stream())
        for l in (2, 0, 1):
            ctx.stage_layers(l, 1, stream=copy)
            ev = torch.cuda.Event()
            ev.record(copy)
            side.wait_event(ev)
            ctx.gather_layers(bt, ne, l, 1, kv, rows, stream=side)
        torch.cuda.synchronize()
        _check_cache(kv, cache, cu, al, 3, rows, "per layer")
        # all layers at once, one stream
        kv.zero_()
        ctx.stage_layers(0, 3)
        ctx.gather_layers(bt, ne, 0, 3, kv, rows)
        torch.cuda.synchronize()
        _check_cache(kv, cache, cu, al, 3, rows, "all layers")
        # host pages with a gap (artifact 2's page left out): two copy runs
        reqs3 = [([4, 0, 1], 2)]
        req3 = [[ids[a] for a in r] for r, _ in reqs3]
        ne3, rows3 = ctx.assemble_plan(req3, [2])
        bt3 = torch.zeros(ne3 * 4, dtype=torch.int32, device="cuda")
        cu3, al3, n3 = ctx.assemble_table_staged(req3, [2], bt3, rows3)
        want3, _ = _staged_table_want(ctx, ids, lengths, reqs3)
        assert n3 == 22 and ctx.stage_pool_info()[1] == 2
        kv3 = torch.zeros(3 * 2 * 8 * rows3 * 128, dtype=torch.bfloat16, device="cuda")
        ctx.stage_layers(0, 3)
        ctx.gather_layers(bt3, ne3, 0, 3, kv3, rows3)
        torch.cuda.synchronize()
        assert np.array_equal(bt3.cpu().numpy().reshape(-1, 4), want3)
        _check_cache(kv3, oracle.assemble(art_k, art_v, reqs3, 8, 128)[0], cu3, al3, 3, rows3, "two runs")
        # a repeated host artifact is staged once
        req2 = requests + [[ids[4], ids[1]]]
        ne2, rows2 = ctx.assemble_plan(req2, caps + [0])
        bt2 = torch.zeros(ne2 * 4, dtype=torch.int32, device="cuda")
        assert ctx.assemble_table_staged(req2, caps + [0], bt2, rows2)[2] == 23
        # errors: layers out of range, staging after a plain assembly
        cu, al, _ = ctx.assemble_table_staged(requests, caps, bt, rows)
        with pytest.raises(AttunerError) as e:
            ctx.stage_layers(2, 2)
        assert e.value.status == -5
        ctx.assemble_table(requests, caps, bt, rows)
        with pytest.raises(AttunerError) as e:
            ctx.stage_layers(0, 1)
        assert e.value.status == -1
        assert ctx.stage_pool_info()[1] == 0


@pytest.mark.parametrize("seed", [91, 92])
def test_random_store_release_assemble_bit_exact(seed):
    # A seeded sequence of stores (1-200 tokens, into HBM or pinned host
    # pages) and releases fragments both pools; every few operations a random
    # batch (repeats allowed) is assembled three ways: all layers at once
    # (host pages read over the link), layer by layer from the same table,
    # and staged through HBM by bulk copies.  Block tables and caches must
    # equal the oracle's, bit for bit.
    rng = np.random.default_rng(seed)
    n_layers = 2
    _say(f"random store/release/assemble, seed {seed}")
    with Context(ModelCfg(n_layers=n_layers, hidden=256), pool_pages=48) as ctx:
        ctx.host_pool_create(48)
        ctx.stage_pool_create(48)
        live = {}   # artifact id -> (length, k, v) in the oracle's [layers][L][Hkv][d] layout
        checks = 0
        for op in range(40):
            if live and (rng.random() < 0.3 or op % 9 == 8):
                victim = int(rng.choice(sorted(live)))
                ctx.release_artifact(victim)
                del live[victim]
            else:
                L = int(rng.integers(1, 201))
                k = rng.integers(0, 2 ** 16, size=(n_layers, 8, L, 128), dtype=np.uint16)
                v = rng.integers(0, 2 ** 16, size=(n_layers, 8, L, 128), dtype=np.uint16)
                store = ctx.store_artifact_host if rng.random() < 0.5 else ctx.store_artifact
                try:
                    aid = store(dev_bf16(k), dev_bf16(v))
                except AttunerError as e:
                    assert e.status == -2   # that pool is full: ENOMEM, nothing stored
                    continue
                live[aid] = (L, k.transpose(0, 2, 1, 3), v.transpose(0, 2, 1, 3))
            if op % 5 != 4 or not live:
                continue
            order = sorted(live)
            reqs = [([int(a) for a in rng.choice(order, int(rng.integers(0, 5)))], int(rng.integers(0, 21)))
                    for _ in range(int(rng.integers(1, 6)))]
            requests, caps = [r for r, _ in reqs], [c for _, c in reqs]
            lengths = {a: live[a][0] for a in order}
            # the oracle indexes artifacts 0..n-1: map ids to positions
            pos = {a: i for i, a in enumerate(order)}
            oreqs = [([pos[a] for a in r], c) for r, c in reqs]
            olen = [lengths[a] for a in order]
            art_k = {pos[a]: live[a][1] for a in order}
            art_v = {pos[a]: live[a][2] for a in order}
            entries, cu_o = oracle.block_table(olen, oreqs, 16)
            cache, _ = oracle.assemble(art_k, art_v, oreqs, 8, 128)
            phys = {pos[a]: ctx.artifact_pages(a)[0] for a in order}
            want = np.array([[phys[a][p], nv, dst, r] for a, p, nv, r, dst in entries.tolist()],
                            np.int32).reshape(-1, 4)
            ne, rows = ctx.assemble_plan(requests, caps)
            bt = torch.zeros(max(1, ne) * 4, dtype=torch.int32, device="cuda")
            kv = torch.zeros(n_layers * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
            cu, al = ctx.assemble_kv(requests, caps, bt, kv, rows)
            torch.cuda.synchronize()
            assert list(cu) == list(cu_o)
            assert np.array_equal(bt.cpu().numpy().reshape(-1, 4)[:ne], want), f"op {op}: block table"
            _check_cache(kv, cache, cu, al, n_layers, rows, f"op {op}, all layers")
            kv.zero_()
            ctx.assemble_table(requests, caps, bt, rows)
            for l in rng.permutation(n_layers):
                ctx.gather_layers(bt, ne, int(l), 1, kv, rows)
            torch.cuda.synchronize()
            _check_cache(kv, cache, cu, al, n_layers, rows, f"op {op}, per layer")
            kv.zero_()
            ctx.assemble_table_staged(requests, caps, bt, rows)
            ctx.stage_layers(0, n_layers)
            ctx.gather_layers(bt, ne, 0, n_layers, kv, rows)
            torch.cuda.synchronize()
            _check_cache(kv, cache, cu, al, n_layers, rows, f"op {op}, staged")
            checks += 1
        assert checks >= 5


def test_staged_assembly_capacity():
    _say("staged assembly: staging pool too small")
    rng = np.random.default_rng(84)
    with Context(ModelCfg(n_layers=2, hidden=256), pool_pages=0) as ctx:
        ctx.host_pool_create(8)
        ctx.stage_pool_create(3)
        _, _, ids = _store_mixed(ctx, rng, [40, 20], {0, 1}, 2)   # 3 + 2 host pages
        ne, rows = ctx.assemble_plan([[ids[0]]], [0])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        assert ctx.assemble_table_staged([[ids[0]]], [0], bt, rows)[2] == 3
        ne, rows = ctx.assemble_plan([[ids[0], ids[1]]], [0])
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        with pytest.raises(AttunerError) as e:
            ctx.assemble_table_staged([[ids[0], ids[1]]], [0], bt, rows)
        assert e.value.status == -5
        with pytest.raises(AttunerError) as e:      # the failed plan left nothing to stage
            ctx.stage_layers(0, 1)
        assert e.value.status == -1


def test_staged_assembly_graph_replays():
    """Copies and gathers captured in one HIP graph, replayed three times with
    eager work and synchronisations between replays: every replay rebuilds
    the cache the oracle assembles."""
    _say("staged assembly in a captured graph")
    rng = np.random.default_rng(85)
    lengths = [64, 48, 100, 16]
    with Context(ModelCfg(n_layers=2, hidden=256), pool_pages=8) as ctx:
        ctx.host_pool_create(16)
        ctx.stage_pool_create(16)
        art_k, art_v, ids = _store_mixed(ctx, rng, lengths, {0, 2, 3}, 2)
        reqs = [([0, 1, 2], 7), ([3, 0], 4)]
        requests, caps = [[ids[a] for a in r] for r, _ in reqs], [c for _, c in reqs]
        ne, rows = ctx.assemble_plan(requests, caps)
        bt = torch.zeros(ne * 4, dtype=torch.int32, device="cuda")
        kv = torch.zeros(2 * 2 * 8 * rows * 128, dtype=torch.bfloat16, device="cuda")
        cu, al, _ = ctx.assemble_table_staged(requests, caps, bt, rows)
        cache, _ = oracle.assemble(art_k, art_v, reqs, 8, 128)
        torch.cuda.synchronize()
        cap, copy = torch.cuda.Stream(), torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(graph, stream=cap):
            copy.wait_stream(cap)
            for l in range(2):
                ctx.stage_layers(l, 1, stream=copy)
                ev = torch.cuda.Event()
                ev.record(copy)
                cap.wait_event(ev)
                ctx.gather_layers(bt, ne, l, 1, kv, rows, stream=cap)
        torch.cuda.synchronize()
        for rep in range(3):
            kv.zero_()
            ctx.assemble_table_staged(requests, caps, bt, rows)   # same plan each time
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            _check_cache(kv, cache, cu, al, 2, rows, f"replay {rep}")


# ----------------------------------------------------------------------------
# merged deployment: W_Q + s B A, then the rank-0 projection
# ----------------------------------------------------------------------------

@pytest.mark.parametrize("rank,H", [(16, 2560), (5, 512), (64, 256)])
def test_merge_lora_then_rank0_projection(rank, H):
    _say(f"merge lora r={rank} H={H}")
    import math
    import synthdata as sd
    from tests._gpu import host_f64
    from tests._tol import assert_intermediate_close
    rng = np.random.default_rng(90 + rank)
    N, lora_cols, T = 6144, 4096, 37
    f = lambda *s_, std=1.0: sd.f32_to_bf16_bits(rng.standard_normal(s_).astype(np.float32) * np.float32(std))
    w, a, b, x = f(N, H, std=0.02), f(rank, H, std=1 / math.sqrt(H)), f(lora_cols, rank, std=0.3), f(T, H)
    scale = 16.0 / rank
    d = oracle.decode_bf16
    with Context(ModelCfg(n_layers=1, hidden=H), pool_pages=0) as ctx:
        wm = torch.empty(N, H, dtype=torch.bfloat16, device="cuda")
        ctx.merge_lora(dev_bf16(w), dev_bf16(a), dev_bf16(b), rank, scale, lora_cols, wm)
        out = torch.empty(T, N, dtype=torch.bfloat16, device="cuda")
        ctx.qproj_lora(dev_bf16(x), wm, None, None, 0, 0.0, 0, out)
        torch.cuda.synchronize()
        got_w = host_f64(wm)
        got = host_f64(out)
    ref_w = oracle.merge_lora(d(w), d(a), d(b), scale, lora_cols)
    # one bf16 rounding of a value summed in fp32: one unit in the last place
    # of the exact value, plus the fp32 sum's own error ((rank + 2) roundings
    # of at most 2^-24 of the magnitudes involved), which a cancellation
    # (w + update ~ 0) can make the larger of the two
    ulp = np.exp2(np.floor(np.log2(np.maximum(np.abs(ref_w), 1e-30))) - 7)
    mag = np.abs(d(w))
    mag[:lora_cols] += abs(scale) * (np.abs(d(b)) @ np.abs(d(a)))
    bound = ulp + (rank + 2) * 2.0 ** -24 * mag
    assert np.all(np.abs(got_w - ref_w) <= bound), "merged weights beyond one bf16 rounding of the fp32 sum"
    assert np.array_equal(bf16_to_host(wm)[lora_cols:], w[lora_cols:]), "k/v rows must be copied unchanged"
    ref = oracle.qproj_lora(d(x), d(w), d(a), d(b), scale, lora_cols)
    assert_intermediate_close(got, ref, "merged projection")
