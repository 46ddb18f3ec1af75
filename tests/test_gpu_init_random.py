"""cllm_model_init_random draws the seeded synthetic weights on the GPU from the published
counter-based generator (SplitMix64 keys, Box-Muller in double, fp32 then bf16 rounding). The
host generator (workload.make_weights) implements the same definition, so a context created from
a seed computes exactly what a context loaded with the host-drawn weights of that seed computes:
prefill logits and Jacobi-step logits are compared bit for bit, and the decoded tokens are equal.
A different seed gives different logits."""
import numpy as np
import pytest

from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import LLAMA7B, SMALL, TINY
from tests.parity import log

pytestmark = pytest.mark.gpu


def _logits_after(m, prompt, block):
    m.debug_logits(True)
    y0 = m.prefill(prompt)
    pre = m.last_logits(len(prompt))[-1].copy()
    b = np.array([y0] + list(block), dtype=np.int32)
    out, a = m.jacobi_step(b)
    step = m.last_logits(len(b)).copy()
    m.debug_logits(False)
    return y0, pre, out, step


@pytest.mark.parametrize("cfg", [TINY, SMALL, LLAMA7B], ids=["tiny-f32", "small-bf16", "llama7b-bf16"])
def test_init_random_equals_host_weights(cfg):
    from paper_2403_00835_amd import binding
    prompt = workload.make_prompt(cfg, 24, seed=4)
    block = workload.make_prompt(cfg, 7, seed=8)
    log(f"[init-random] {cfg.n_layers} layers, d {cfg.d_model}: device-drawn context")
    a = binding.Model(cfg, max_ctx=128, max_block=16, max_new=64, random_seed=0)
    ra = _logits_after(a, prompt, block)
    dec_a, _ = a.jacobi_decode(prompt, 8, 32)
    bytes_a = a.streamed_weight_bytes()
    a.close()
    log("  host-drawn weights")
    ws = workload.make_weights(cfg, seed=0)
    b = binding.Model(cfg, max_ctx=128, max_block=16, max_new=64, weights=ws)
    del ws
    rb = _logits_after(b, prompt, block)
    dec_b, _ = b.jacobi_decode(prompt, 8, 32)
    assert b.streamed_weight_bytes() == bytes_a
    b.close()
    assert ra[0] == rb[0]
    assert np.array_equal(ra[1], rb[1]), np.abs(ra[1] - rb[1]).max()
    assert np.array_equal(ra[2], rb[2])
    assert np.array_equal(ra[3], rb[3]), np.abs(ra[3] - rb[3]).max()
    assert np.array_equal(dec_a, dec_b)
    if cfg is not LLAMA7B:
        c = binding.Model(cfg, max_ctx=128, max_block=16, max_new=64, random_seed=1)
        rc = _logits_after(c, prompt, block)
        c.close()
        assert not np.array_equal(ra[1], rc[1])
