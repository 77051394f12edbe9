"""Parity at the full workload sizes, in the launch configurations bench.py
times (same shapes, so the same tile/split choices), against the fp64 oracle.

Attention is checked on sampled suffix rows the oracle computes one by one
(every head, every dimension of each sampled row), the gather bit-exact on
every row of three layers, and the 16-request varlen batch on all rows.
"""

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from tests._tol import assert_intermediate_close, assert_o_close

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload, host_f64
    from paper_2609_36722_amd.api import bf16_to_device


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _sample_rows(S, n=12, seed=0):
    rng = np.random.default_rng(seed)
    rows = {0, 1, S // 2, S - 2, S - 1} | set(int(v) for v in rng.integers(0, S, size=n))
    return np.array(sorted(r for r in rows if 0 <= r < S))


def _check_gather(g):
    wl = g.wl
    reqs = [(list(r.artifact_ids), r.suffix_len) for r in wl.requests]
    cache, cu = oracle.assemble(g.art_k, g.art_v, reqs, wl.shape.n_kv_heads, wl.shape.head_dim)
    got = g.cache_view()
    for r in range(len(wl.requests)):
        lo, n = g.cu_ctx[r], g.art_len[r]
        assert np.array_equal(got[:, :, :, lo:lo + n], cache[:, :, :, lo:lo + n]), f"gather request {r}"


@pytest.mark.parametrize("name,layers", [("c2", [0, 17, 35]), ("c5", [0]), ("c3", [35])])
def test_stack_layers_sampled_rows(name, layers):
    wl = sd.make_workload(name, gamma="uniform")
    _say(f"{name} layers {layers}: gather bit-exact, O on sampled rows")
    g = GpuWorkload(wl, layers=layers)
    try:
        _check_gather(g)
        S = wl.requests[0].suffix_len
        rows = _sample_rows(S, seed=len(layers))
        for li, l in enumerate(layers):
            out = g.run_layer(li)
            ref = g.oracle_layer(li, 0, rows=rows)
            assert_intermediate_close(host_f64(out["qkv"][:, :wl.shape.q_dim]), ref["q"].reshape(S, -1),
                                      f"{name} layer {l} q")
            assert_o_close(host_f64(out["o"])[rows], ref["o"], f"{name} layer {l} O")
    finally:
        g.close()


def test_varlen_batch_all_rows():
    wl = sd.make_workload("c4", gamma="uniform")
    _say("c4: 16 requests, every row")
    g = GpuWorkload(wl)
    try:
        _check_gather(g)
        out = g.run_layer(0)
        got = host_f64(out["o"])
        for r in range(len(wl.requests)):
            ref = g.oracle_layer(0, r)
            assert_o_close(got[g.cu_q[r]:g.cu_q[r + 1]], ref["o"], f"c4 request {r}")
    finally:
        g.close()


def test_full_prefill_c2_size_sampled_rows():
    # the speed baseline: 8448 tokens, rank 0, same kernels as the bench
    wl = sd.make_workload("c2", gamma="uniform")
    _say("full prefill 8448 tokens, sampled rows")
    s = wl.shape
    w = sd.layer_weights(wl, 0)
    x = sd.prefill_hidden(wl, 0, 0)
    N = x.shape[0]
    g = GpuWorkload(sd.make_workload("c1"))  # any context with the same geometry
    try:
        from paper_2609_36722_amd.api import Context, ModelCfg
        with Context(ModelCfg(n_layers=1, hidden=s.hidden), pool_pages=0) as ctx:
            wqkv = bf16_to_device(np.concatenate([w["wq"], w["wk"], w["wv"]]))
            o = torch.empty(N, s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda")
            k = torch.empty(s.n_kv_heads, N, s.head_dim, dtype=torch.bfloat16, device="cuda")
            v = torch.empty_like(k)
            ctx.full_prefill(0, bf16_to_device(x), wqkv, None, None, 0, 0.0, bf16_to_device(w["gamma_q"]),
                             bf16_to_device(w["gamma_k"]), o, k, v)
            torch.cuda.synchronize()
            got = host_f64(o)
        rows = _sample_rows(N, n=10, seed=3)
        d = {n: oracle.decode_bf16(t) for n, t in w.items()}
        ref = oracle.full_prefill(oracle.decode_bf16(x), d["wq"], d["wk"], d["wv"], d["gamma_q"], d["gamma_k"], 0,
                                  s.n_q_heads, s.n_kv_heads, s.rope_theta, s.rms_eps, rows=rows)
        assert_o_close(got[rows], ref["o"], "full prefill O")
    finally:
        g.close()
