"""GPU checks of the caller-owned iteration workspace (cllm_runtime_opts.workspace): a context
whose workspace is a PyTorch tensor on the GPU decodes exactly as one whose workspace the library
allocates (bit-identical tokens and iteration counts, logits of a step), through the C ABI; and
the creation checks reject a workspace that is too small, misaligned or not device memory."""
import ctypes

import numpy as np
import pytest

from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import GUESS_STREAM_REINJECT, GUESS_UNIFORM, SMALL, TINY
from tests.parity import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [TINY, SMALL], ids=["tiny-f32", "small-bf16"])
def test_torch_workspace_decodes_identically(cfg):
    import torch
    from paper_2403_00835_amd import binding
    kw = dict(max_ctx=512, max_block=16, max_new=64, max_batch=2)
    nbytes = binding.workspace_bytes(cfg, **kw)
    log(f"[workspace] {cfg.dtype}: {nbytes} bytes of caller workspace")
    buf = torch.full((nbytes,), 0x7f, dtype=torch.uint8, device="cuda:0")  # not zero: the library zeroes it
    torch.cuda.synchronize()
    ws = workload.make_weights(cfg)
    own = binding.Model(cfg, weights=ws, **kw)
    ext = binding.Model(cfg, weights=ws, workspace=(buf.data_ptr(), nbytes), **kw)
    try:
        prompt = workload.make_prompt(cfg, 40, seed=31)
        ar_own, _ = own.ar_decode(prompt, 64)
        ar_ext, _ = ext.ar_decode(prompt, 64)
        np.testing.assert_array_equal(ar_own, ar_ext)
        for pol in (GUESS_UNIFORM, GUESS_STREAM_REINJECT):
            a, sa = own.jacobi_decode(prompt, 16, 64, policy=pol, stream=ar_own, p=0.3, seed=4, seq=1)
            b, sb = ext.jacobi_decode(prompt, 16, 64, policy=pol, stream=ar_own, p=0.3, seed=4, seq=1)
            np.testing.assert_array_equal(a, b)
            np.testing.assert_array_equal(a, ar_own)
            assert sa["steps"] == sb["steps"]
        # a host-driven step: logits bit for bit
        outs = []
        for m in (own, ext):
            m.debug_logits(True)
            y0 = m.prefill(prompt)
            blk = np.concatenate([[y0], ar_own[1:12]]).astype(np.int32)
            out, acc = m.jacobi_step(blk)
            outs.append((out, acc, m.last_logits(blk.size)))
            m.debug_logits(False)
        np.testing.assert_array_equal(outs[0][0], outs[1][0])
        assert outs[0][1] == outs[1][1]
        np.testing.assert_array_equal(outs[0][2], outs[1][2])
    finally:
        ext.close()
        own.close()
    torch.cuda.synchronize()
    del buf


def test_workspace_creation_errors():
    import torch
    from paper_2403_00835_amd import binding
    cfg = TINY
    kw = dict(max_ctx=256, max_block=8, max_new=32)
    nbytes = binding.workspace_bytes(cfg, **kw)
    buf = torch.empty(nbytes + 4096, dtype=torch.uint8, device="cuda:0")
    host = np.zeros(nbytes, dtype=np.uint8)
    cases = [((buf.data_ptr(), nbytes - 256), "ERR_CAPACITY"),  # too small
             ((buf.data_ptr() + 16, nbytes), "ERR_ARG"),        # not 256-byte aligned
             ((host.ctypes.data, nbytes), "ERR_ARG")]           # host memory
    for ws, err in cases:
        with pytest.raises(binding.CllmError) as ei:
            binding.Model(cfg, workspace=ws, **kw)
        assert err in str(ei.value), str(ei.value)
    m = binding.Model(cfg, workspace=(buf.data_ptr(), nbytes), **kw)  # exactly enough
    m.close()
    torch.cuda.synchronize()
    del buf
