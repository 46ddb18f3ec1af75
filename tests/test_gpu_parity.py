"""GPU parity of the HIP path (through the C ABI) against the oracle, on the tiny fp32 and the
small bf16 configurations: prefill logits, teacher-forced Jacobi iterations (logits within the
tolerance, tokens bit-exact outside the tie margin, accepted length by the acceptance rule),
whole decodes checked as valid greedy continuations, and bit-exact equality of GPU AR and GPU
Jacobi decoding."""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import (BLOCK_SHRINK, BLOCK_SLIDE, GUESS_STREAM, GUESS_STREAM_REINJECT,
                                          GUESS_UNIFORM, SMALL, TINY)
from tests.parity import TOL, check_rows, log, verify_greedy_sequence

pytestmark = pytest.mark.gpu


class Pair:
    def __init__(self, cfg, max_ctx, max_block, max_new, prefill_chunk=0):
        from paper_2403_00835_amd import binding
        self.cfg = cfg
        ws = workload.make_weights(cfg)
        self.gpu = binding.Model(cfg, max_ctx=max_ctx, max_block=max_block, max_new=max_new, weights=ws,
                                 prefill_chunk=prefill_chunk)
        self.orc = oracle.Model(cfg, [workload.as_f32(cfg, t) for t in ws])
        self.tol = TOL[cfg.dtype]
        self.max_ctx = max_ctx


@pytest.fixture(scope="module")
def tiny():
    log("[gpu] building tiny fp32 pair")
    return Pair(TINY, max_ctx=256, max_block=64, max_new=128)


@pytest.fixture(scope="module")
def tiny_chunked():
    log("[gpu] building tiny fp32 pair with 64-row prefill chunks")
    return Pair(TINY, max_ctx=256, max_block=64, max_new=128, prefill_chunk=64)


@pytest.fixture(scope="module")
def small():
    log("[gpu] building small bf16 pair")
    return Pair(SMALL, max_ctx=512, max_block=64, max_new=256)


def _teacher_forced(pair, prompt, n, steps, stream=None, p=0.3, seed=5, policy=GUESS_STREAM_REINJECT):
    gpu, orc, tol, V = pair.gpu, pair.orc, pair.tol, pair.cfg.vocab
    spec = oracle.GuessSpec(GUESS_UNIFORM if stream is None else policy, 0, stream, p=p, seed=seed)
    gpu.debug_logits(True)
    try:
        y0 = gpu.prefill(prompt)
        st = oracle.State(orc, pair.max_ctx)
        _, lg0 = st.prefill(prompt, want_logits=True)
        P = len(prompt)
        last = (P - 1) % 64
        g0 = gpu.last_logits(last + 1)[last]
        err0 = np.abs(g0 - lg0).max()
        log(f"  prefill: y0={y0} max|dlogit|={err0:.3g}")
        assert err0 <= tol
        check_rows([y0], lg0[None], tol, "prefill")
        e, pending, worst, inside = 0, y0, err0, 0
        z = np.array([pending] + [oracle.guess(spec, 0, j, 0, V) for j in range(1, n)], dtype=np.int32)
        for it in range(steps):
            m = z.size
            out, a = gpu.jacobi_step(z)
            lg_g = gpu.last_logits(m)
            lg_o = st.eval_block(z)
            err = np.abs(lg_g - lg_o).max()
            worst = max(worst, err)
            assert err <= tol, f"iteration {it}: max|dlogit| {err} > {tol}"
            inside += check_rows(out, lg_o, tol, f"iteration {it}")
            assert a == oracle.accept_len(z, out)
            assert 1 <= a <= m
            st.commit(a, int(out[a - 1]))
            L, pend = gpu.seq_state()
            assert L == st.L and pend == int(out[a - 1])
            e += a
            pending = int(out[a - 1])
            # next state: shrink within a block of n; re-drawn guesses when a stream is given
            left = m - a
            if left == 0:
                left = n
            nz = [pending]
            for j in range(1, left):
                if stream is not None:
                    nz.append(oracle.guess(spec, 0, e + j, it + 1, V))
                else:
                    nz.append(int(out[a - 1 + j]) if a - 1 + j < m else oracle.guess(spec, 0, e + j, 0, V))
            z = np.array(nz, dtype=np.int32)
        log(f"  {steps} iterations, {e} tokens, worst max|dlogit|={worst:.3g}, rows inside margin={inside}")
    finally:
        gpu.debug_logits(False)


def test_tiny_teacher_forced_iterations(tiny):
    log("[gpu] tiny teacher-forced iterations n=8")
    prompt = workload.make_prompt(TINY, 16)
    _teacher_forced(tiny, prompt, n=8, steps=20)


def test_tiny_long_prompt_spans_chunks(tiny_chunked):
    # 150-token prompt in 64-row prefill chunks: three chunks, several attention chunks, ragged tails.
    log("[gpu] tiny teacher-forced, prompt 150 in 64-row prefill chunks, n=13")
    prompt = workload.make_prompt(TINY, 150, seed=7)
    _teacher_forced(tiny_chunked, prompt, n=13, steps=8)


@pytest.mark.parametrize("cfg", [TINY, SMALL], ids=["tiny", "small"])
def test_prefill_chunk_size_leaves_values_unchanged(cfg):
    # The prefill's rows are computed with reduction orders fixed by the model shape, so the
    # chunk size (64-row passes, 128-row passes, one pass of the whole prompt) changes no value:
    # the prompt's last logits, the KV cache (seen through the next iteration's logits) and a
    # whole decode are bit-identical.
    from paper_2403_00835_amd import binding
    log(f"[gpu] {cfg.dtype} d={cfg.d_model}: prefill chunk sizes 64 / 128 / default give identical values")
    ws = workload.make_weights(cfg)
    prompt = workload.make_prompt(cfg, 300, seed=17)
    res = []
    for chunk in (64, 128, 0):
        m = binding.Model(cfg, max_ctx=512, max_block=16, max_new=64, weights=ws, prefill_chunk=chunk)
        try:
            m.debug_logits(True)
            y0 = m.prefill(prompt)
            pre = m.last_logits(64)[(len(prompt) - 1) % 64].copy()
            blk = np.array([y0] + list(workload.make_prompt(cfg, 15, seed=18)), dtype=np.int32)
            out, a = m.jacobi_step(blk)
            step = m.last_logits(blk.size).copy()
            m.debug_logits(False)
            m.reset()
            dec, _ = m.jacobi_decode(prompt, 16, 64, policy=GUESS_UNIFORM, seed=6)
            res.append((y0, pre, out.copy(), a, step, dec.copy()))
        finally:
            m.close()
    for r in res[1:]:
        assert r[0] == res[0][0] and r[3] == res[0][3]
        np.testing.assert_array_equal(r[1], res[0][1])
        np.testing.assert_array_equal(r[2], res[0][2])
        np.testing.assert_array_equal(r[4], res[0][4])
        np.testing.assert_array_equal(r[5], res[0][5])


def test_tiny_full_block_of_64(tiny):
    log("[gpu] tiny teacher-forced, n=64 (four row groups)")
    prompt = workload.make_prompt(TINY, 40, seed=8)
    _teacher_forced(tiny, prompt, n=64, steps=3)


def test_tiny_decode_equals_oracle(tiny):
    log("[gpu] tiny decode vs oracle AR")
    prompt = workload.make_prompt(TINY, 16)
    ar_o = tiny.orc.ar_decode(prompt, 32)
    out, st = tiny.gpu.jacobi_decode(prompt, 8, 32, policy=GUESS_UNIFORM, seed=2)
    log(f"  steps={st['steps']} blocks={st['blocks']}")
    inside = verify_greedy_sequence(tiny.orc, prompt, out, tiny.tol)
    if inside == 0:
        np.testing.assert_array_equal(out, ar_o)
    assert st["tokens"] == 32 and st["steps"] <= 32
    assert sum(a * c for a, c in enumerate(st["accept_hist"])) == 32
    # per-iteration device times: ordered percentiles, full blocks (m = n) among them
    assert 0 < st["iter_ms_p10"] <= st["iter_ms_p50"] <= st["iter_ms_p90"]
    assert 0 < st["iter_ms_full_p10"] <= st["iter_ms_full_p50"] <= st["iter_ms_full_p90"]
    assert st["decode_ms"] > 0 and st["prefill_ms"] > 0


def test_tiny_short_decodes_equal_ar(tiny):
    # The decode loop queues rounds of iterations it knows are needed and reads the sequence
    # state while a round's last iteration runs: decodes of 1-3 tokens, a block longer than the
    # output and an output one longer than a block end with exactly max_new tokens, the greedy ones.
    log("[gpu] tiny short decodes (max_new 1-3, n up to 64) vs GPU AR")
    prompt = workload.make_prompt(TINY, 9, seed=12)
    ar, _ = tiny.gpu.ar_decode(prompt, 17)
    for n, max_new in [(1, 1), (8, 1), (8, 2), (64, 3), (16, 17), (2, 17)]:
        out, st = tiny.gpu.jacobi_decode(prompt, n, max_new, policy=GUESS_UNIFORM, seed=n)
        np.testing.assert_array_equal(out, ar[:max_new])
        assert st["tokens"] == max_new and 1 <= st["steps"] <= max_new


@pytest.mark.parametrize("policy,block_policy", [(GUESS_UNIFORM, BLOCK_SHRINK), (GUESS_STREAM, BLOCK_SHRINK),
                                                 (GUESS_STREAM_REINJECT, BLOCK_SHRINK),
                                                 (GUESS_STREAM_REINJECT, BLOCK_SLIDE), (GUESS_STREAM, BLOCK_SLIDE)])
def test_tiny_gpu_ar_equals_gpu_jacobi(tiny, policy, block_policy):
    log(f"[gpu] tiny AR == Jacobi policy={policy} block={block_policy}")
    prompt = workload.make_prompt(TINY, 16, seed=3)
    ar, _ = tiny.gpu.ar_decode(prompt, 100)
    for n in (1, 5, 8, 16, 64):
        out, st = tiny.gpu.jacobi_decode(prompt, n, 100, policy=policy, block_policy=block_policy, stream=ar, p=0.3,
                                         seed=4)
        np.testing.assert_array_equal(out, ar)
        # the oracle's Jacobi loop under the same guess policy takes the same iterations
        spec = oracle.GuessSpec(policy, block_policy, ar, p=0.3, seed=4)
        _, so = tiny.orc.jacobi_decode(prompt, n, 100, spec)
        assert so["steps"] == st["steps"] and so["blocks"] == st["blocks"], (n, so["steps"], st["steps"])


def test_tiny_exact_and_fully_corrupted_guesses(tiny):
    log("[gpu] tiny special cases of the guess stream")
    prompt = workload.make_prompt(TINY, 16, seed=5)
    ar, _ = tiny.gpu.ar_decode(prompt, 40)
    out, st = tiny.gpu.jacobi_decode(prompt, 8, 40, policy=GUESS_STREAM, stream=ar, p=0.0)
    np.testing.assert_array_equal(out, ar)
    assert st["steps"] == 5 and st["accept_hist"][8] == 5
    out, st = tiny.gpu.jacobi_decode(prompt, 8, 40, policy=GUESS_STREAM_REINJECT, block_policy=BLOCK_SLIDE,
                                     stream=ar, p=1.0)
    np.testing.assert_array_equal(out, ar)
    assert st["steps"] == 40 and st["accept_hist"][1] == 40


def test_small_teacher_forced_iterations(small):
    log("[gpu] small bf16 teacher-forced iterations n=16")
    prompt = workload.make_prompt(SMALL, 128)
    ar = small.orc.ar_decode(prompt, 96)
    _teacher_forced(small, prompt, n=16, steps=10, stream=ar, p=0.3)


def test_small_ragged_prompt_vs_oracle(small):
    # 300 prompt rows in one pass of the prompt GEMM: five 64-row tiles, the last one ragged
    # (44 live rows), and the chunk-parallel attention; then teacher-forced iterations.
    log("[gpu] small bf16 teacher-forced, prompt 300 (ragged prompt tiles), n=16")
    prompt = workload.make_prompt(SMALL, 300, seed=23)
    _teacher_forced(small, prompt, n=16, steps=4)


def test_bf16_ragged_widths_vs_oracle():
    # Output widths that are not multiples of the GEMM column groups: QKV 960 and gate/up 1728
    # columns (the prompt GEMM's 256-column groups and the decode GEMM's tile groups end ragged),
    # O and down 320 columns (2.5 prompt groups), a 1000-token LM head; a 150-token prompt in one
    # prompt pass of three 64-row tiles, the last ragged; then teacher-forced iterations.
    from paper_2403_00835_amd.configs import ModelConfig
    cfg = ModelConfig(n_layers=2, d_model=320, n_heads=5, head_dim=64, ffn_dim=864, vocab=1000)
    log("[gpu] bf16 ragged widths (d 320, FFN 864, vocab 1000), prompt 150, n=12")
    pair = Pair(cfg, max_ctx=256, max_block=16, max_new=64)
    try:
        prompt = workload.make_prompt(cfg, 150, seed=29)
        _teacher_forced(pair, prompt, n=12, steps=5)
    finally:
        pair.gpu.close()


@pytest.mark.parametrize("dtype,hd", [("bf16", 32), ("bf16", 256), ("f32", 32), ("f32", 64), ("f32", 128)])
def test_head_widths_vs_oracle(dtype, hd):
    # The head widths the library accepts beside those of the tiny, small and 7B configurations
    # (bf16 32 and 256, fp32 32, 64 and 128: other attention and RoPE instances; 256 takes the
    # chunk-parallel attention in every iteration). Prompt 150 (three 64-key chunks, a ragged
    # prompt tile), then blocks of 40 rows whose guesses come from the greedy continuation
    # corrupted at p = 0.1, so they shrink by several tokens per iteration: one-tile GEMM
    # launches sized for 64 rows that run 3, 2 or 1 live 16-row groups.
    from paper_2403_00835_amd.configs import ModelConfig
    H = 4 if hd <= 64 else 2
    cfg = ModelConfig(n_layers=2, d_model=H * hd, n_heads=H, head_dim=hd, ffn_dim=344, vocab=1000, dtype=dtype)
    log(f"[gpu] {dtype} head_dim {hd} ({H} heads), prompt 150, n=40")
    pair = Pair(cfg, max_ctx=512, max_block=40, max_new=256)
    try:
        prompt = workload.make_prompt(cfg, 150, seed=31)
        stream, _ = pair.gpu.ar_decode(prompt, 256)
        _teacher_forced(pair, prompt, n=40, steps=8, stream=stream, p=0.1)
    finally:
        pair.gpu.close()


def test_tiny_largest_context_ar_equals_jacobi():
    # The longest context the library accepts (65,408 positions: 1,022 64-key chunks): a 65,200-
    # token prompt in 512-row prefill passes, then GPU AR and GPU Jacobi decoding (n = 64, guesses
    # from the AR continuation corrupted at p = 0.3) give the same 128 tokens; every iteration
    # combines over 1,019 or more chunks (the chunk-parallel attention).
    from paper_2403_00835_amd import binding
    max_ctx = 65408
    ws = workload.make_weights(TINY)
    gpu = binding.Model(TINY, max_ctx=max_ctx, max_block=64, max_new=128, weights=ws, prefill_chunk=512)
    try:
        prompt = workload.make_prompt(TINY, 65200, seed=41)
        log("[gpu] tiny, prompt 65200 (largest context), AR vs Jacobi n=64, 128 new")
        ar, _ = gpu.ar_decode(prompt, 128)
        out, st = gpu.jacobi_decode(prompt, 64, 128, policy=GUESS_STREAM_REINJECT, stream=ar, p=0.3, seed=6)
        np.testing.assert_array_equal(out, ar)
        log(f"  {st['steps']} Jacobi iterations")
        assert st["steps"] < 128
        with pytest.raises(binding.CllmError):  # one position past the capacity
            gpu.ar_decode(workload.make_prompt(TINY, max_ctx - 127, seed=41), 128)
    finally:
        gpu.close()


def test_small_decode_is_valid_greedy(small):
    log("[gpu] small bf16 decode, stream re-drawn p=0.3, n=16, 96 new")
    prompt = workload.make_prompt(SMALL, 128)
    ar_o = small.orc.ar_decode(prompt, 96)
    out, st = small.gpu.jacobi_decode(prompt, 16, 96, policy=GUESS_STREAM_REINJECT, stream=ar_o, p=0.3, seed=3)
    log(f"  steps={st['steps']} mean a={96 / st['steps']:.2f}")
    inside = verify_greedy_sequence(small.orc, prompt, out, small.tol)
    log(f"  positions inside the tie margin: {inside}")
    ar_g, _ = small.gpu.ar_decode(prompt, 96)
    np.testing.assert_array_equal(out, ar_g)


def test_small_gpu_ar_equals_gpu_jacobi(small):
    log("[gpu] small bf16 AR == Jacobi over n")
    prompt = workload.make_prompt(SMALL, 128, seed=2)
    ar, _ = small.gpu.ar_decode(prompt, 128)
    for n, pol, bp in [(16, GUESS_STREAM_REINJECT, BLOCK_SHRINK), (16, GUESS_STREAM, BLOCK_SHRINK),
                       (32, GUESS_STREAM_REINJECT, BLOCK_SLIDE), (64, GUESS_UNIFORM, BLOCK_SHRINK),
                       (7, GUESS_STREAM_REINJECT, BLOCK_SLIDE)]:
        out, st = small.gpu.jacobi_decode(prompt, n, 128, policy=pol, block_policy=bp, stream=ar, p=0.3, seed=9)
        np.testing.assert_array_equal(out, ar)


def test_small_acceptance_closed_form(small):
    # Re-drawn guesses are right independently with probability 1-p, so a full window accepts
    # E[a] = 1 + (1-p)(1-(1-p)^(n-1))/p tokens per iteration.
    log("[gpu] small acceptance under re-drawn guesses vs closed form")
    prompt = workload.make_prompt(SMALL, 128, seed=4)
    ar, _ = small.gpu.ar_decode(prompt, 256)
    n, p = 16, 0.3
    out, st = small.gpu.jacobi_decode(prompt, n, 256, policy=GUESS_STREAM_REINJECT, block_policy=BLOCK_SLIDE,
                                      stream=ar, p=p, seed=12)
    np.testing.assert_array_equal(out, ar)
    hist = np.array(st["accept_hist"], dtype=np.float64)
    a = np.arange(hist.size)
    steps = hist.sum()
    mean_a = (a * hist).sum() / steps
    sd = np.sqrt(((a - mean_a) ** 2 * hist).sum() / (steps - 1))
    expect = 1 + (1 - p) * (1 - (1 - p) ** (n - 1)) / p
    log(f"  steps={int(steps)} mean a={mean_a:.3f} closed form={expect:.3f} se={sd / np.sqrt(steps):.3f}")
    # the last few windows are shorter than n, which only lowers the mean slightly
    assert expect - 4 * sd / np.sqrt(steps) - 0.3 < mean_a < expect + 4 * sd / np.sqrt(steps)


def test_determinism_run_twice(small):
    log("[gpu] small decode twice, identical")
    prompt = workload.make_prompt(SMALL, 100, seed=6)
    a1, s1 = small.gpu.jacobi_decode(prompt, 16, 64, policy=GUESS_UNIFORM, seed=1)
    a2, s2 = small.gpu.jacobi_decode(prompt, 16, 64, policy=GUESS_UNIFORM, seed=1)
    np.testing.assert_array_equal(a1, a2)
    assert s1["steps"] == s2["steps"]


def test_abi_errors_on_device(tiny):
    from paper_2403_00835_amd import binding
    log("[gpu] ABI error paths")
    g = binding.Model(TINY, max_ctx=64, max_block=8, max_new=16, weights=workload.make_weights(TINY))
    with pytest.raises(binding.CllmError) as e:
        g.jacobi_step(np.array([1, 2], dtype=np.int32))
    assert e.value.status == 2  # before prefill
    prompt = workload.make_prompt(TINY, 10)
    y0 = g.prefill(prompt)
    with pytest.raises(binding.CllmError) as e:
        g.jacobi_step(np.array([(y0 + 1) % 256, 2], dtype=np.int32))
    assert e.value.status == 2  # block_in[0] is not the pending token
    empty = np.zeros(0, dtype=np.int32)
    for call in (lambda: g.jacobi_step(empty), lambda: g.prefill(empty), lambda: g.jacobi_decode(empty, 8, 16),
                 lambda: g.jacobi_decode(prompt, 0, 16), lambda: g.jacobi_decode(prompt, 8, 0),
                 lambda: g.ar_decode(prompt, 0)):
        with pytest.raises(binding.CllmError) as e:
            call()
        assert e.value.status == 1  # empty block or prompt, n = 0, max_new = 0
    assert g.prefill(prompt) == y0  # (the empty prefill changed nothing)
    with pytest.raises(binding.CllmError) as e:
        g.jacobi_step(np.array([y0] + [0] * 8, dtype=np.int32))
    assert e.value.status == 1  # m > max_block
    with pytest.raises(binding.CllmError) as e:
        g.jacobi_step(np.array([y0, 999], dtype=np.int32))
    assert e.value.status == 1  # id out of range
    with pytest.raises(binding.CllmError) as e:
        g.prefill(np.zeros(70, dtype=np.int32))
    assert e.value.status == 3  # prompt beyond max_ctx
    with pytest.raises(binding.CllmError) as e:
        g.jacobi_decode(prompt, 8, 17)
    assert e.value.status == 3  # max_new beyond the context's max_new
    with pytest.raises(binding.CllmError) as e:
        g.jacobi_decode(prompt, 8, 16, policy=GUESS_STREAM, stream=np.zeros(4, dtype=np.int32))
    assert e.value.status == 1  # stream too short
    # state unchanged by the failures: a valid iteration still works
    out, a = g.jacobi_step(np.array([y0, 3, 4], dtype=np.int32))
    assert 1 <= a <= 3


def test_nan_logits_are_reported():
    # A NaN logit is an error, not a token: the embeddings of ids 128..255 are NaN, so a prompt
    # holding one fails in the prefill, and a clean prompt whose uniform-random guesses (or the
    # model's own predictions) bring one into a block fails in the decode, alone or batched; the
    # status is ERR_NUMERIC and a clean prefill works afterwards.
    from paper_2403_00835_amd import binding
    log("[gpu] NaN logits: prefill, decode and batched decode report ERR_NUMERIC")
    ws = workload.make_weights(TINY)
    ws[0] = ws[0].copy()
    ws[0][128:] = np.nan
    g = binding.Model(TINY, max_ctx=128, max_block=8, max_new=32, max_batch=2, weights=ws)
    try:
        clean = workload.make_prompt(TINY, 12) % 128
        bad = clean.copy()
        bad[5] = 200
        with pytest.raises(binding.CllmError) as e:
            g.prefill(bad)
        assert e.value.status == 8
        with pytest.raises(binding.CllmError) as e:
            g.jacobi_decode(clean, 8, 32, policy=GUESS_UNIFORM, seed=5)
        assert e.value.status == 8
        with pytest.raises(binding.CllmError) as e:
            g.jacobi_decode_batch([0, 1], [clean, clean[:7]], 8, 32)
        assert e.value.status == 8
        y0 = g.prefill(clean)
        assert 0 <= y0 < 256
    finally:
        g.close()


def test_weight_file_roundtrip(tiny, tmp_path):
    from paper_2403_00835_amd import binding
    log("[gpu] weight file load")
    ws = workload.make_weights(TINY)
    path = tmp_path / "tiny.bin"
    binding.write_weight_file(str(path), TINY, ws)
    g = binding.Model(TINY, max_ctx=256, max_block=64, max_new=128, path=str(path))
    prompt = workload.make_prompt(TINY, 16)
    a, _ = g.ar_decode(prompt, 24)
    b, _ = tiny.gpu.ar_decode(prompt, 24)
    np.testing.assert_array_equal(a, b)


def test_kernel_timing_sampling(tiny):
    """The measurement hook: with a sampling stride, one eligible launch in `every` is timed;
    every timed launch has a positive duration; a bad stride is rejected."""
    from paper_2403_00835_amd import binding
    log("[gpu] kernel timing sampling stride")
    g = tiny.gpu
    prompt = workload.make_prompt(TINY, 16, seed=9)
    ar, _ = g.ar_decode(prompt, 40)
    out = {}
    for every in (1, 3):
        g.timing_enable("gate_up", max_rows=8, every=every)
        res, st = g.jacobi_decode(prompt, 8, 40)
        launches, ms = g.timing_read()
        g.timing_enable(-1)
        np.testing.assert_array_equal(res, ar)
        out[every] = (launches, ms, st["steps"])
    # one gate/up launch per layer and queued iteration (iterations queued past the end launch too)
    assert out[1][0] >= out[1][2] * TINY.n_layers
    assert out[3][0] == (out[1][0] + 2) // 3  # the same decode: launches 0, 3, 6, ... are timed
    assert out[1][1] > 0 and out[3][1] > 0
    with pytest.raises(binding.CllmError) as e:
        g.timing_enable("gate_up", max_rows=8, every=0)
    assert e.value.status == 1


@pytest.mark.parametrize("policy,block_policy", [(GUESS_STREAM, 0), (GUESS_STREAM_REINJECT, 0), (GUESS_STREAM, 1)])
def test_tiny_trajectory_equals_oracle(tiny, policy, block_policy):
    """The GPU's recorded trajectory (every iteration's L, e, block start, m, a, z and
    predictions) equals the oracle's, and so do the fast-forward and stationary counts."""
    from paper_2403_00835_amd import binding
    log(f"[gpu] tiny trajectory vs oracle policy={policy} block={block_policy}")
    prompt = workload.make_prompt(TINY, 16, seed=12)
    ar, _ = tiny.gpu.ar_decode(prompt, 64)
    g = tiny.gpu
    g.trace_enable(True)
    try:
        out, st = g.jacobi_decode(prompt, 8, 64, policy=policy, block_policy=block_policy, stream=ar, p=0.3, seed=4)
        traj = g.trace_read()
    finally:
        g.trace_enable(False)
    spec = oracle.GuessSpec(policy, block_policy, ar, p=0.3, seed=4)
    out_o, st_o = tiny.orc.jacobi_decode(prompt, 8, 64, spec, trace=True)
    np.testing.assert_array_equal(out, out_o)
    assert len(traj) == st["steps"] == st_o["steps"]
    for t, (r, ro) in enumerate(zip(traj, st_o["trajectory"])):
        assert {k: r[k] for k in ("L", "e", "b0", "m", "a")} == {k: ro[k] for k in ("L", "e", "b0", "m", "a")}, t
        np.testing.assert_array_equal(r["z"], ro["z"])
        np.testing.assert_array_equal(r["pred"], ro["pred"])
    c = binding.trace_count(traj, out, 8, block_policy)
    co = oracle.trajectory_counts(st_o["trajectory"], out_o, 8, block_policy)
    assert (c["iterations"], c["stationary"], c["windows"]) == (co["iterations"], co["stationary"], co["windows"])
    # a decode without recording leaves no records
    g.jacobi_decode(prompt, 8, 64, policy=policy, block_policy=block_policy, stream=ar, p=0.3, seed=4)
    assert g.trace_read() == []
