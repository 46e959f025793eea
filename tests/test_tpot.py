"""The multi-layer decode-step harness (paper_2606_00024_amd.tpot)."""
from __future__ import annotations

import pytest
import torch

from paper_2606_00024_amd import tpot


def test_llama3_8b_parameter_count():
    """Llama-3-8B's published size is 8.03e9 parameters: the weights one step
    reads plus the input embedding table (the same size as the LM head)."""
    m = tpot.MODELS["llama3_8b"]
    params = m.weight_bytes() // 2 + m.vocab * m.hidden
    assert abs(params - 8.03e9) / 8.03e9 < 2e-3


def test_kv_bytes():
    m = tpot.MODELS["llama3_8b"]
    # 32 layers x 8 sequences x 32K tokens x 8 KV heads x (K + V) x 128 x bf16
    assert m.kv_bytes(8, 32768) == 32 * 8 * 32768 * 8 * 2 * 128 * 2


def test_tp4_share_is_a_quarter_of_the_heads():
    m = tpot.MODELS["llama3_70b_tp4"]
    assert (m.q_heads * 4, m.kv_heads * 4, m.ffn * 4) == (64, 8, 28672)


@pytest.mark.gpu
def test_step_runs_and_attention_matches_a_direct_call():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_00024_amd import api
    m = tpot.ModelShape("tiny", layers=2, hidden=512, q_heads=8, kv_heads=2, ffn=1024, vocab=1000)
    step = tpot.Step(m, batch=2, seq_len=4096)
    for mode in ("nodet", "off", "on"):
        x = step.run(mode)
        torch.cuda.synchronize()
        assert torch.isfinite(x.float()).all()
    # the step's attention call of layer 1 gives what a direct call gives
    step.attention("on", 1)
    torch.cuda.synchronize()
    got = step.out.clone()
    wl = step.layers[1]["wl"]
    ref, _, stop = api.decode_workload(wl, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(got, ref)
    assert torch.equal(step.stop[1], stop)
    ms = step.time_ms("on", steps=2, warmup=1)
    assert (ms > 0).all()
