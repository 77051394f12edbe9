"""attuner_suffix_attn_noalloc (key-split partials in the library's fixed
device buffer, no allocation) against attuner_suffix_attn on the same
inputs, through the C ABI.

Two noalloc calls run back to back after the reference calls: first the
long-context Qwen3-8B layer (1024 suffix rows over 33,792 keys, two key
splits: 16.5 MiB of partials), then a smaller three-request batch whose
requests have different split counts, so the second call runs over the
first one's leftovers in the buffer.  O is held to the parity bar against
the other entry point's output (and, as both take the same split plan
here, equals it bit for bit), the LSE likewise.  A position past the RoPE
table is rejected with ERANGE.
"""

import numpy as np
import pytest
import torch

import synthdata as sd
from synthdata.workloads import ModelShape, Request, custom_workload
from tests._tol import assert_o_close

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload, dev_bf16, host_f64
    from paper_2609_36722_amd.api import AttunerError


def _say(msg):
    print(f"[case] {msg}", flush=True)


def _inputs(g):
    s = g.wl.shape
    w, x = g.layer_inputs(0)
    T = x.shape[0]
    nq, nkv = s.q_dim, s.kv_dim
    qkv = torch.empty(T, nq + 2 * nkv, dtype=torch.bfloat16, device="cuda")
    g.ctx.qproj_lora(dev_bf16(x), dev_bf16(np.concatenate([w["wq"], w["wk"], w["wv"]])),
                     dev_bf16(w["a"]) if g.wl.rank else None, dev_bf16(w["b"]) if g.wl.rank else None, g.wl.rank,
                     g.wl.scale, nq, qkv)
    return qkv, dev_bf16(w["gamma_q"]), dev_bf16(w["gamma_k"]), T


def _attn(g, qkv, gq, gk, T, noalloc):
    s = g.wl.shape
    nq, nkv = s.q_dim, s.kv_dim
    o = torch.empty(T, s.n_q_heads, s.head_dim, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(T, s.n_q_heads, dtype=torch.float32, device="cuda")
    g.ctx.suffix_attn(0, g.cu_q, g.cu_ctx, g.art_len, g.pos0, qkv[:, :nq], nq + 2 * nkv, qkv[:, nq:nq + nkv],
                      qkv[:, nq + nkv:], nq + 2 * nkv, gq, gk, g.req_kv, g.rows, o, lse, noalloc=noalloc)
    return o, lse


def _small_batch():
    shape = ModelShape(hidden=2560)
    return custom_workload("noalloc-small", 95, shape, [700, 1500, 333, 64],
                           [Request((0, 1), 40), Request((2,), 100), Request((3, 1, 0), 7)],
                           n_layers=1, rank=8, scale=2.0, gamma="uniform")


def test_noalloc_matches_suffix_attn_two_calls_second_smaller():
    cases = [("c5 layer 0", sd.make_workload("c5", gamma="uniform")), ("3-request batch", _small_batch())]
    gs, ins, ref = [], [], []
    try:
        for name, wl in cases:
            g = GpuWorkload(wl)
            g.ctx.reserve(max_position=max(g.pos0[r] + wl.requests[r].suffix_len for r in range(len(wl.requests))))
            gs.append(g)
            ins.append(_inputs(g))
            _say(f"{name}: attuner_suffix_attn")
            ref.append(_attn(g, *ins[-1], noalloc=False))
        torch.cuda.synchronize()
        got = []
        for (name, _), g, x in zip(cases, gs, ins):
            _say(f"{name}: attuner_suffix_attn_noalloc")
            got.append(_attn(g, *x, noalloc=True))
        torch.cuda.synchronize()
        for (name, _), (o, lse), (o_ref, lse_ref) in zip(cases, got, ref):
            a, b = host_f64(o), host_f64(o_ref)
            assert_o_close(a, b, f"{name}: O of the allocation-free call")
            la, lb = lse.cpu().numpy(), lse_ref.cpu().numpy()
            assert np.all(np.abs(la - lb) <= 1e-3 * np.maximum(1.0, np.abs(lb))), f"{name}: LSE"
            # the same split plan on both sides here: identical arithmetic
            assert np.array_equal(a, b) and np.array_equal(la, lb), f"{name}: not bit-identical"
    finally:
        for g in gs:
            g.close()


def test_noalloc_rejects_a_position_past_the_rope_table():
    wl = sd.make_workload("c1", gamma="uniform")
    g = GpuWorkload(wl)
    try:
        qkv, gq, gk, T = _inputs(g)
        g.pos0 = [4096 - 10]   # rows 4086 .. 4149: past the 4096-position table
        with pytest.raises(AttunerError) as e:
            _attn(g, qkv, gq, gk, T, noalloc=True)
        assert e.value.status == -5 and "RoPE" in str(e.value)
    finally:
        g.close()
