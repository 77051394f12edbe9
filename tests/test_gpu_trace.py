"""The library's launch tracer (attuner_trace_begin/end) through the C ABI."""

import pytest
import torch

import synthdata as sd

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests._gpu import GpuWorkload
    from paper_2609_36722_amd.api import AttunerError


def test_trace_counts_every_kernel_of_a_layer():
    print("[case] trace c1 layer", flush=True)
    g = GpuWorkload(sd.make_workload("c1"))
    try:
        g.ctx.trace_begin()
        g.run_layer(0)
        g.run_layer(0)
        times = g.ctx.trace_end()
        # two layers: GEMM (LoRA down-projection fused at rank 8), norm+rope,
        # attention (+ split merge) each
        for k in ("gemm_lora_kernel", "qk_norm_rope_kernel", "attention_kernel"):
            assert times[k][0] == 2, (k, times)
            assert 0.0 < times[k][1] < 1000.0 and times[k][2] <= times[k][1]
        assert "lora_down_kernel" not in times, times
        with pytest.raises(AttunerError):
            g.ctx.trace_end()   # no trace open any more
        g.run_layer(0)          # untraced launches still work
    finally:
        g.close()
