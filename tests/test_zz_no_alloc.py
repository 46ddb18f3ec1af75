"""GPU check of cllm_hidden_rows_noalloc, the entry point that allocates nothing (its staging rows
live in the library's fixed per-GPU scratch array): through the C ABI, two calls in a row, the
second with a smaller block, each against cllm_hidden_rows on the same state, bit for bit; also
on a second context of the same GPU (the array is shared by every context of a device)."""
import numpy as np
import pytest

from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import SMALL, TINY
from tests.parity import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [TINY, SMALL], ids=["tiny-f32", "small-bf16"])
def test_hidden_rows_noalloc_equals_allocating_entry_point(cfg):
    from paper_2403_00835_amd import binding
    ws = workload.make_weights(cfg)
    m1 = binding.Model(cfg, max_ctx=256, max_block=16, max_new=32, weights=ws)
    m2 = binding.Model(cfg, max_ctx=256, max_block=16, max_new=32, max_batch=2, weights=ws)
    try:
        prompt = workload.make_prompt(cfg, 37, seed=41)
        for model, seq in ((m1, 0), (m2, 1)):
            model.prefill(prompt, seq=seq)
            for m in (16, 5):  # the second call smaller than the first
                blk = workload.make_prompt(cfg, m, seed=42 + m)
                ref = model.hidden_rows(blk, seq=seq)
                got = model.hidden_rows_noalloc(blk, seq=seq)
                log(f"[no-alloc] {cfg.dtype} slot {seq} m={m}: max|d| {np.abs(ref - got).max():.3g}")
                assert got.shape == (m, cfg.d_model)
                np.testing.assert_array_equal(got, ref)
                assert np.isfinite(got).all()
            L, _ = model.seq_state(seq=seq)
            assert L == 37  # nothing committed
    finally:
        m2.close()
        m1.close()


def test_hidden_rows_noalloc_argument_errors():
    from paper_2403_00835_amd import binding
    cfg = TINY
    m = binding.Model(cfg, max_ctx=64, max_block=8, max_new=8, weights=workload.make_weights(cfg))
    try:
        blk = np.arange(4, dtype=np.int32)
        with pytest.raises(binding.CllmError, match="ERR_STATE"):
            m.hidden_rows_noalloc(blk)  # before prefill
        m.prefill(np.arange(10, dtype=np.int32))
        with pytest.raises(binding.CllmError, match="ERR_ARG"):
            m.hidden_rows_noalloc(np.arange(9, dtype=np.int32))  # m above max_block
        with pytest.raises(binding.CllmError, match="ERR_ARG"):
            m.hidden_rows_noalloc(np.array([0, cfg.vocab], dtype=np.int32))  # id out of range
    finally:
        m.close()
