"""Parity at the full workload sizes, in the launch configurations bench.py
times (same shapes, so the same tile/split choices), against the fp64 oracle.

The 36-layer stacks are checked at layers 0, 17 and 35 on every suffix row
(the q projection, O and the LSE; the oracle runs its attention over blocks
of rows), the gather bit-exact on every row of those layers, the
16-request varlen batch on all rows, and the full prefill of the Qwen3-4B
and long-context sizes on sampled rows the oracle computes one by one.
"""

import numpy as np
import pytest
import torch

import oracle
import synthdata as sd
from tests._tol import assert_intermediate_close, assert_o_close, lse_bar

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


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name", ["c2", "c3", "c5"])
def test_stack_layers_all_rows(name):
    layers = [0, 17, 35]
    wl = sd.make_workload(name, gamma="uniform")
    s = wl.shape
    _say(f"{name} layers {layers}: gather bit-exact; q, O and LSE on every row")
    g = GpuWorkload(wl, layers=layers)
    try:
        _check_gather(g)
        S = wl.requests[0].suffix_len
        for li, l in enumerate(layers):
            out = g.run_layer(li)
            got_q = host_f64(out["qkv"][:, :s.q_dim])
            got_o = host_f64(out["o"])
            got_lse = out["lse"].cpu().numpy().astype(np.float64)
            _say(f"{name} layer {l}: GPU done, oracle running")
            ref = g.oracle_layer_blocks(li, 0, say=_say)
            assert_intermediate_close(got_q, ref["q"].reshape(S, -1), f"{name} layer {l} q")
            assert_o_close(got_o, ref["o"], f"{name} layer {l} O")
            bar = lse_bar(ref["q_hat"], ref["keys"], s.n_q_heads, s.n_kv_heads)
            lse_err = float(np.abs(got_lse - ref["lse"]).max())
            assert lse_err <= bar, f"{name} layer {l} LSE max|err| {lse_err:.3e} > {bar:.3e}"
            _say(f"{name} layer {l}: q, O and LSE within bars")
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


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["c2", "c5"])
def test_full_prefill_sampled_rows(name):
    # the speed baseline at the bench's sizes (8448 and 33792 tokens), rank 0,
    # the same kernels and launch plan as the bench
    wl = sd.make_workload(name, gamma="uniform")
    s = wl.shape
    w = sd.layer_weights(wl, 0)
    x = sd.prefill_hidden(wl, 0, 0)
    N = x.shape[0]
    _say(f"full prefill of {N} tokens ({name} size), sampled rows")
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
        got_k = host_f64(k)
    rows = _sample_rows(N, n=10, seed=3)
    _say(f"full prefill of {N} tokens: GPU done, oracle running")
    d = {n: oracle.decode_bf16(t) for n, t in w.items()}
    ref = oracle.full_prefill(oracle.decode_bf16(x), d["wq"], d["wk"], d["wv"], d["gamma_q"], d["gamma_k"], 0,
                              s.n_q_heads, s.n_kv_heads, s.rope_theta, s.rms_eps, rows=rows)
    assert_o_close(got[rows], ref["o"], f"full prefill O ({N} tokens)")
    assert_intermediate_close(got_k.transpose(1, 0, 2)[rows], ref["k_hat"][rows], f"full prefill k_hat ({N} tokens)")
