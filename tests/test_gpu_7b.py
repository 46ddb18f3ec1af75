"""GPU checks at the LLaMA-2-7B shape (32 layers, d 4096, 32 x 128 heads, FFN 11008, vocab
32000, bf16), the shape the benchmark times.

- Oracle parity, teacher-forced: a 40-token prompt (the oracle's fp64 forward at this shape
  costs ~13 GFLOP per row, so a 512-token prefill is out of a test's reach), then Jacobi
  iterations of 16 rows: logits within 2e-2 of the oracle, tokens bit-exact outside the tie
  margin.
- Properties at full size, in the benchmark's launch configuration (prompt 512, n = 16, 256 new
  tokens, guesses re-drawn at p = 0.3, shrink): GPU Jacobi equals GPU AR bit-exactly under every
  guess and block policy, iterations accept >= 1 token and at most the block, the run is
  deterministic, the 512-row prompt pass gives the same values as 64-row passes; and the long
  workload (prompt 2048, n = 64, 512 new).
"""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import (BLOCK_SHRINK, BLOCK_SLIDE, GUESS_STREAM, GUESS_STREAM_REINJECT,
                                          GUESS_UNIFORM, LLAMA7B)
from tests.parity import TOL, check_rows, log

pytestmark = pytest.mark.gpu

CFG = LLAMA7B


@pytest.fixture(scope="module")
def weights():
    log("[gpu7b] drawing 7B weights")
    return workload.make_weights(CFG)


@pytest.fixture(scope="module")
def gpu(weights):
    from paper_2403_00835_amd import binding
    log("[gpu7b] creating the 7B context (max_ctx 2752, max_block 64, max_new 512)")
    return binding.Model(CFG, max_ctx=2048 + 512 + 64 + 128, max_block=64, max_new=512, weights=weights)


def test_7b_teacher_forced_iterations_vs_oracle(gpu, weights):
    tol = TOL["bf16"]
    log("[gpu7b] oracle model (fp32 copies of the bf16 weights)")
    orc = oracle.Model(CFG, [workload.as_f32(CFG, t) for t in weights])
    prompt = workload.make_prompt(CFG, 40, seed=21)
    st = oracle.State(orc, 128)
    gpu.debug_logits(True)
    try:
        log("[gpu7b] prefill 40 tokens on both sides")
        y0 = gpu.prefill(prompt)
        g0 = gpu.last_logits(40)[39]
        _, lg0 = st.prefill(prompt, want_logits=True)
        err = np.abs(g0 - lg0).max()
        log(f"  prefill max|dlogit| = {err:.3g}")
        assert err <= tol
        check_rows([y0], lg0[None], tol, "prefill")
        spec = oracle.GuessSpec(GUESS_UNIFORM, 0, None, seed=5)
        z = np.array([y0] + [oracle.guess(spec, 0, j, 0, CFG.vocab) for j in range(1, 16)], dtype=np.int32)
        worst = err
        for it in range(2):
            log(f"[gpu7b] iteration {it}: 16 rows on both sides")
            out, a = gpu.jacobi_step(z)
            lg_g = gpu.last_logits(z.size)
            lg_o = st.eval_block(z)
            e = np.abs(lg_g - lg_o).max()
            worst = max(worst, e)
            log(f"  max|dlogit| = {e:.3g}, a = {a}")
            assert e <= tol
            check_rows(out, lg_o, tol, f"iteration {it}")
            assert a == oracle.accept_len(z, out)
            st.commit(a, int(out[a - 1]))
            z = np.concatenate([[out[a - 1]], out[a:a + 15]]).astype(np.int32)
            if z.size < 16:
                z = np.concatenate([z, np.arange(16 - z.size, dtype=np.int32) + 7])
        log(f"  worst max|dlogit| = {worst:.3g} (tolerance {tol})")
    finally:
        gpu.debug_logits(False)
        del orc


def test_7b_full_size_jacobi_equals_ar(gpu):
    prompt = workload.make_prompt(CFG, 512)
    log("[gpu7b] AR decode, prompt 512, 256 tokens")
    ar, st_ar = gpu.ar_decode(prompt, 256)
    assert st_ar["steps"] == 256
    for pol, bp in [(GUESS_STREAM_REINJECT, BLOCK_SHRINK), (GUESS_STREAM, BLOCK_SHRINK),
                    (GUESS_STREAM_REINJECT, BLOCK_SLIDE), (GUESS_UNIFORM, BLOCK_SHRINK)]:
        log(f"[gpu7b] Jacobi decode n=16 policy={pol} block={bp}")
        out, st = gpu.jacobi_decode(prompt, 16, 256, policy=pol, block_policy=bp, stream=ar, p=0.3, seed=3)
        np.testing.assert_array_equal(out, ar)
        hist = np.array(st["accept_hist"])
        assert hist[0] == 0 and hist[17:].sum() == 0
        assert (np.arange(hist.size) * hist).sum() == 256 and st["steps"] == hist.sum() <= 256
        log(f"  iterations {st['steps']}, mean accepted {256 / st['steps']:.2f}")
    out2, st2 = gpu.jacobi_decode(prompt, 16, 256, policy=GUESS_STREAM_REINJECT, stream=ar, p=0.3, seed=3)
    out3, st3 = gpu.jacobi_decode(prompt, 16, 256, policy=GUESS_STREAM_REINJECT, stream=ar, p=0.3, seed=3)
    np.testing.assert_array_equal(out2, out3)
    assert st2["steps"] == st3["steps"]


def test_7b_prompt_chunking_leaves_values_unchanged(gpu):
    # The benchmark's prefill (one 512-row pass of the prompt GEMM and the chunk-parallel
    # attention) against eight 64-row passes of a second context with bit-identical weights
    # (drawn on the device): the prompt's last logits, a 16-row iteration's logits over the
    # cache it left and a 64-token decode are bit-identical.
    from paper_2403_00835_amd import binding
    prompt = workload.make_prompt(CFG, 512, seed=4)
    blk = workload.make_prompt(CFG, 15, seed=5)
    res = []
    for chunk, ctx in [(0, gpu), (64, None)]:
        if ctx is None:
            log("[gpu7b] second context: weights drawn on the device, 64-row prefill passes")
            ctx = binding.Model(CFG, max_ctx=704, max_block=16, max_new=64, random_seed=workload.SEED_WEIGHTS,
                                prefill_chunk=chunk)
        try:
            ctx.debug_logits(True)
            y0 = ctx.prefill(prompt)
            pre = ctx.last_logits(64)[(512 - 1) % 64].copy()
            out, a = ctx.jacobi_step(np.concatenate([[y0], blk]).astype(np.int32))
            step = ctx.last_logits(16).copy()
            ctx.debug_logits(False)
            dec, _ = ctx.jacobi_decode(prompt, 16, 64, policy=GUESS_UNIFORM, seed=6)
            res.append((y0, pre, out.copy(), a, step, dec.copy()))
        finally:
            if ctx is not gpu:
                ctx.close()
    log(f"  y0 {res[0][0]} / {res[1][0]}, accepted {res[0][3]} / {res[1][3]}")
    assert res[0][0] == res[1][0] and res[0][3] == res[1][3]
    for i in (1, 2, 4, 5):
        np.testing.assert_array_equal(res[0][i], res[1][i])


def test_7b_exact_guesses_and_step_api(gpu):
    prompt = workload.make_prompt(CFG, 512, seed=2)
    log("[gpu7b] AR 64 tokens, then exact guesses converge in one iteration per block")
    ar, _ = gpu.ar_decode(prompt, 64)
    out, st = gpu.jacobi_decode(prompt, 16, 64, policy=GUESS_STREAM, stream=ar, p=0.0)
    np.testing.assert_array_equal(out, ar)
    assert st["steps"] == 4 and st["accept_hist"][16] == 4
    # the host-driven step API on the same cache: a block of the true continuation is accepted whole
    y0 = gpu.prefill(prompt)
    assert y0 == ar[0]
    blk, a = gpu.jacobi_step(ar[:16])
    assert a == 16
    np.testing.assert_array_equal(blk[:15], ar[1:16])
    L, pend = gpu.seq_state()
    assert L == 512 + 16 and pend == blk[15] == ar[16]


def test_7b_long_context_block_64(gpu):
    prompt = workload.make_prompt(CFG, 2048, seed=3)
    log("[gpu7b] long: prompt 2048, AR 512 tokens")
    ar, _ = gpu.ar_decode(prompt, 512)
    log("[gpu7b] long: Jacobi n=64, re-drawn guesses p=0.3")
    out, st = gpu.jacobi_decode(prompt, 64, 512, policy=GUESS_STREAM_REINJECT, stream=ar, p=0.3, seed=7)
    np.testing.assert_array_equal(out, ar)
    log(f"  iterations {st['steps']}, mean accepted {512 / st['steps']:.2f}")
    assert st["steps"] <= 512
