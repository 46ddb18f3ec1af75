"""GPU checks of the batched ragged iteration (the blocks of several sequences in one forward
pass, each against its own cache, with its own committed length and block size), through the
C ABI.

Every row of a batched iteration is computed exactly as a single-sequence iteration computes
it (fixed reduction orders that do not depend on the rows sharing the pass), so:
- tiny fp32 and small bf16: batched steps give bit-identical tokens, accepted lengths and logits
  to single-sequence steps on a context with one slot (the single-sequence launches take the
  one-kernel attention, the batched ones the chunk-parallel pair, so this also pins the two
  attention paths to each other bit for bit); a batched decode of sequences with
  different prompt lengths and guess policies equals, per sequence, the single-sequence GPU AR
  decode; prompts longer than 64 rows run as one row-tiled prefill chunk, and a batched decode
  packs its prompts into shared prefill passes (a prompt may span passes); on tiny the result is
  also the oracle's greedy AR continuation.
- LLaMA-2-7B shape at the batched workload's full size (16 sequences, prompts uniform in
  [256, 1024], n = 32, 256 new tokens, corruption rates uniform in [0.1, 0.6]): batched Jacobi
  equals batched AR bit-exactly, and slot 0 equals the single-sequence AR of the same context.
"""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import (ModelConfig, BLOCK_SHRINK, BLOCK_SLIDE, GUESS_STREAM, GUESS_STREAM_REINJECT,
                                          GUESS_UNIFORM, LLAMA7B, SMALL, TINY, WORKLOADS)
from tests.parity import log

pytestmark = pytest.mark.gpu


def _models(cfg, max_ctx, max_block, max_new, max_batch):
    from paper_2403_00835_amd import binding
    ws = workload.make_weights(cfg)
    batched = binding.Model(cfg, max_ctx=max_ctx, max_block=max_block, max_new=max_new, max_batch=max_batch,
                            weights=ws)
    single = binding.Model(cfg, max_ctx=max_ctx, max_block=max_block, max_new=max_new, weights=ws)
    return ws, batched, single


@pytest.fixture(scope="module")
def tiny():
    log("[gpu-batch] tiny fp32: batched context (8 slots, row capacity 128) and a one-slot context")
    return _models(TINY, max_ctx=256, max_block=16, max_new=64, max_batch=8)


@pytest.fixture(scope="module")
def small():
    log("[gpu-batch] small bf16: batched context (4 slots x 32 rows) and a one-slot context")
    return _models(SMALL, max_ctx=512, max_block=32, max_new=64, max_batch=4)


def _specs(prompts, ars, pol):
    out = []
    for b, (pr, ar) in enumerate(zip(prompts, ars)):
        policy, block, p = pol[b % len(pol)]
        out.append(dict(policy=policy, block_policy=block, stream=None if policy == GUESS_UNIFORM else ar, p=p,
                        seed=11 + b))
    return out


POLICIES = [(GUESS_UNIFORM, BLOCK_SHRINK, 0.0), (GUESS_STREAM, BLOCK_SHRINK, 0.3),
            (GUESS_STREAM_REINJECT, BLOCK_SHRINK, 0.5), (GUESS_STREAM_REINJECT, BLOCK_SLIDE, 0.2)]


def _batched_steps_equal_single(cfg, batched, single, prompts, n, iters, seed):
    V = cfg.vocab
    B = len(prompts)
    rng = np.random.default_rng(seed)
    y0s = [batched.prefill(p, seq=b) for b, p in enumerate(prompts)]
    # the blocks of every iteration: pending token + random guesses, of varying size
    batched.debug_logits(True)
    rec = []
    pend = list(y0s)
    try:
        for it in range(iters):
            ms = [int(rng.integers(1, n + 1)) for _ in range(B)]
            blocks = [np.concatenate([[pend[b]], rng.integers(0, V, ms[b] - 1)]).astype(np.int32) for b in range(B)]
            res = batched.jacobi_step_batch(list(range(B)), blocks)
            lg = batched.last_logits(sum(ms))
            r0 = np.concatenate([[0], np.cumsum(ms)])
            rec.append([(blocks[b], res[b][0], res[b][1], lg[r0[b]:r0[b + 1]]) for b in range(B)])
            for b in range(B):
                out, a = res[b]
                pend[b] = int(out[a - 1])
    finally:
        batched.debug_logits(False)
    single.debug_logits(True)
    try:
        for b in range(B):
            assert single.prefill(prompts[b]) == y0s[b]
            for it in range(iters):
                blk, out_b, a_b, lg_b = rec[it][b]
                out, a = single.jacobi_step(blk)
                np.testing.assert_array_equal(out, out_b)
                assert a == a_b
                np.testing.assert_array_equal(single.last_logits(blk.size), lg_b)
    finally:
        single.debug_logits(False)


def _batched_decode_equals_ar(cfg, batched, single, prompts, n, max_new, check_oracle=None):
    ars = []
    for p in prompts:
        ar, _ = single.ar_decode(p, max_new)
        ars.append(ar)
    if check_oracle is not None:
        for p, ar in zip(prompts, ars):
            np.testing.assert_array_equal(check_oracle.ar_decode(p, max_new), ar)
    B = len(prompts)
    out, stats = batched.jacobi_decode_batch(list(range(B)), prompts, n, max_new,
                                             specs=_specs(prompts, ars, POLICIES))
    for b in range(B):
        np.testing.assert_array_equal(out[b], ars[b])
        hist = np.array(stats[b]["accept_hist"])
        assert hist[0] == 0 and (np.arange(hist.size) * hist).sum() == max_new
        assert stats[b]["steps"] == hist.sum() <= max_new
    log("  iterations per sequence: " + ", ".join(str(s["steps"]) for s in stats))
    # batched AR (blocks of one token for every sequence)
    out1, _ = batched.jacobi_decode_batch(list(range(B)), prompts, 1, max_new)
    for b in range(B):
        np.testing.assert_array_equal(out1[b], ars[b])


def test_tiny_batched_steps_equal_single(tiny):
    ws, batched, single = tiny
    prompts = [workload.make_prompt(TINY, L, seed=31, seq=b) for b, L in enumerate([5, 37, 16, 100, 64, 1])]
    log("[gpu-batch] tiny: 6 sequences, 5 batched steps vs single steps")
    _batched_steps_equal_single(TINY, batched, single, prompts, 16, 5, seed=1)


def test_tiny_batched_decode(tiny):
    ws, batched, single = tiny
    orc = oracle.Model(TINY, [workload.as_f32(TINY, t) for t in ws])
    prompts = [workload.make_prompt(TINY, L, seed=32, seq=b) for b, L in enumerate([9, 120, 33, 70, 16, 2, 50, 81])]
    log("[gpu-batch] tiny: batched decode of 8 sequences (n=8, 48 new) vs single AR and oracle AR")
    _batched_decode_equals_ar(TINY, batched, single, prompts, 8, 48, check_oracle=orc)


def test_tiny_batch_subsets_and_errors(tiny):
    from paper_2403_00835_amd import binding
    ws, batched, single = tiny
    p = workload.make_prompt(TINY, 20, seed=33)
    ar, _ = single.ar_decode(p, 32)
    # a slot decoded alone, through the single-sequence call, in a batched context
    out, _ = batched.jacobi_decode(p, 8, 32, seq=5, policy=GUESS_STREAM_REINJECT, stream=ar, p=0.4, seed=2)
    np.testing.assert_array_equal(out, ar)
    # a batch of slots in arbitrary order
    out, _ = batched.jacobi_decode_batch([6, 2], [p, p], 8, 32)
    np.testing.assert_array_equal(out[0], ar)
    np.testing.assert_array_equal(out[1], ar)
    with pytest.raises(binding.CllmError) as e:
        batched.jacobi_decode_batch([1, 1], [p, p], 8, 32)
    assert e.value.status == 1
    with pytest.raises(binding.CllmError) as e:
        batched.jacobi_decode_batch([8], [p], 8, 32)
    assert e.value.status == 1
    batched.reset(3)
    with pytest.raises(binding.CllmError) as e:
        batched.jacobi_step(np.array([1], dtype=np.int32), seq=3)
    assert e.value.status == 2


def test_small_batched_steps_equal_single(small):
    ws, batched, single = small
    prompts = [workload.make_prompt(SMALL, L, seed=34, seq=b) for b, L in enumerate([50, 130, 200, 77])]
    log("[gpu-batch] small: 4 sequences, 4 batched steps vs single steps")
    _batched_steps_equal_single(SMALL, batched, single, prompts, 32, 4, seed=2)


def test_narrow_bf16_batched_steps_equal_single():
    # d_model 64 in bf16: two k-steps per product, fewer than the class-pair split's four, so
    # iterations of more than 64 rows take gemm_kernel over the row tiles for QKV, O, gate/up and
    # the LM head (and the row-tiled kernel for the down ranges); rows keep the single-step bits
    cfg = ModelConfig(n_layers=2, d_model=64, n_heads=2, head_dim=32, ffn_dim=172, vocab=256, dtype="bf16")
    ws, batched, single = _models(cfg, max_ctx=256, max_block=32, max_new=64, max_batch=4)
    try:
        prompts = [workload.make_prompt(cfg, L, seed=38, seq=b) for b, L in enumerate([20, 45, 90, 7])]
        log("[gpu-batch] narrow bf16 (d 64): 4 sequences of 32-row blocks, 6 batched steps vs single steps")
        _batched_steps_equal_single(cfg, batched, single, prompts, 32, 6, seed=3)
    finally:
        batched.close()
        single.close()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_max_batch_and_block(dtype):
    # The largest batched iteration the library takes: 64 sequences with blocks of up to 64 rows
    # (4096 rows, 64 row tiles; bf16 products through the class-pair split, fp32 through
    # gemm_kernel over the row tiles). Batched steps equal single steps bit for bit (logits
    # included), and a batched decode of the 64 sequences equals their single-sequence AR decodes.
    if dtype == "f32":
        cfg = TINY
    else:
        cfg = ModelConfig(n_layers=2, d_model=256, n_heads=4, head_dim=64, ffn_dim=688, vocab=1000, dtype="bf16")
    ws, batched, single = _models(cfg, max_ctx=320, max_block=64, max_new=64, max_batch=64)
    try:
        lens = np.random.default_rng(40).integers(1, 130, 64)
        prompts = [workload.make_prompt(cfg, int(L), seed=40, seq=b) for b, L in enumerate(lens)]
        log(f"[gpu-batch] {dtype}: 64 sequences x blocks of up to 64 rows, 3 batched steps vs single steps")
        _batched_steps_equal_single(cfg, batched, single, prompts, 64, 3, seed=4)
        log(f"[gpu-batch] {dtype}: batched decode of 64 sequences (n=64, 48 new) vs single AR")
        _batched_decode_equals_ar(cfg, batched, single, prompts, 64, 48)
    finally:
        batched.close()
        single.close()


def test_small_batched_decode(small):
    ws, batched, single = small
    prompts = [workload.make_prompt(SMALL, L, seed=35, seq=b) for b, L in enumerate([60, 140, 200, 90])]
    log("[gpu-batch] small: batched decode of 4 sequences (n=16, 64 new) vs single AR")
    _batched_decode_equals_ar(SMALL, batched, single, prompts, 16, 64)


def test_small_packed_prefill_passes():
    # A batched decode prefills its prompts packed into passes of the prefill chunk: with a chunk
    # of 128 rows, prompts of 60..260 tokens share passes, span passes, and several end in one
    # pass (the LM head then runs on each 64-row tile that holds a prompt's last row). Every
    # sequence equals its single-sequence AR decode, whose prefill runs one prompt at a time in
    # passes of 512 rows.
    from paper_2403_00835_amd import binding
    ws = workload.make_weights(SMALL)
    packed = binding.Model(SMALL, max_ctx=512, max_block=16, max_new=48, max_batch=6, weights=ws, prefill_chunk=128)
    single = binding.Model(SMALL, max_ctx=512, max_block=16, max_new=48, weights=ws)
    try:
        lens = [60, 140, 30, 260, 20, 90]
        prompts = [workload.make_prompt(SMALL, L, seed=36, seq=b) for b, L in enumerate(lens)]
        log("[gpu-batch] small: 6 prompts packed into 128-row prefill passes, batched decode (n=16, 48 new) vs single AR")
        _batched_decode_equals_ar(SMALL, packed, single, prompts, 16, 48)
    finally:
        packed.close()
        single.close()


def test_7b_batched_ragged_full_size():
    from paper_2403_00835_amd import binding
    wl = WORKLOADS["7b_batched"]
    cfg = wl.model
    prompts, ps = workload.make_batch(cfg, wl.batch, wl.prompt_len_range, wl.p_range)
    B = len(prompts)
    log(f"[gpu-batch] 7B: {B} sequences, prompt lengths {min(map(len, prompts))}..{max(map(len, prompts))}")
    ws = workload.make_weights(cfg)
    m = binding.Model(cfg, max_ctx=wl.prompt_len_range[1] + wl.max_new + wl.n + 64, max_block=wl.n,
                      max_new=wl.max_new, max_batch=B, weights=ws)
    del ws
    log("[gpu-batch] 7B: batched AR (blocks of one token)")
    ar, _ = m.jacobi_decode_batch(list(range(B)), prompts, 1, wl.max_new)
    log("[gpu-batch] 7B: batched Jacobi, n=32, re-drawn guesses at per-sequence p")
    specs = [dict(policy=GUESS_STREAM_REINJECT, block_policy=BLOCK_SHRINK, stream=ar[b], p=float(ps[b]), seed=3)
             for b in range(B)]
    out, stats = m.jacobi_decode_batch(list(range(B)), prompts, wl.n, wl.max_new, specs=specs)
    np.testing.assert_array_equal(out, ar)
    log("  iterations per sequence: " + ", ".join(str(s["steps"]) for s in stats))
    log("[gpu-batch] 7B: slot 0 by the single-sequence AR call")
    single, _ = m.ar_decode(prompts[0], wl.max_new, seq=0)
    np.testing.assert_array_equal(single, ar[0])
    m.close()


def test_tiny_batched_trajectories_equal_single(tiny):
    """Trajectory records of a batched decode, per sequence slot, equal the records of the same
    sequence decoded alone in the same slot (the guess draws depend on the slot id; every row
    is computed as in a single-sequence iteration)."""
    ws, batched, single = tiny
    slots = (4, 1, 6)
    prompts = [workload.make_prompt(TINY, L, seed=36, seq=b) for b, L in enumerate([12, 70, 33])]
    ars = [single.ar_decode(p, 40)[0] for p in prompts]
    specs = _specs(prompts, ars, POLICIES)
    log("[gpu-batch] tiny: trajectories of a batched decode vs single decodes")
    batched.trace_enable(True)
    try:
        out, stats = batched.jacobi_decode_batch(list(slots), prompts, 8, 40, specs=specs)
        trajs = [batched.trace_read(q) for q in slots]
        for b, p in enumerate(prompts):
            sp = specs[b]
            o1, _ = batched.jacobi_decode(p, 8, 40, seq=slots[b], policy=sp["policy"], block_policy=sp["block_policy"],
                                          stream=sp["stream"], p=sp["p"], seed=sp["seed"])
            np.testing.assert_array_equal(out[b], o1)
            t1 = batched.trace_read(slots[b])
            assert len(t1) == len(trajs[b]) == stats[b]["steps"]
            for r, r1 in zip(trajs[b], t1):
                assert {k: r[k] for k in ("L", "e", "b0", "m", "a")} == {k: r1[k] for k in ("L", "e", "b0", "m", "a")}
                np.testing.assert_array_equal(r["z"], r1["z"])
                np.testing.assert_array_equal(r["pred"], r1["pred"])
    finally:
        batched.trace_enable(False)


def test_tiny_trajectory_collection_equals_oracle(tiny):
    """Algorithm 1 over 10 prompts (two batches of the 8 slots): every block's states, fixed
    point and augmented copy equal the oracle's collection from its own decode of the prompt in
    the same slot."""
    from paper_2403_00835_amd import collect
    ws, batched, single = tiny
    orc = oracle.Model(TINY, [workload.as_f32(TINY, t) for t in ws])
    prompts = [workload.make_prompt(TINY, L, seed=37, seq=i) for i, L in enumerate([9, 20, 31, 5, 64, 12, 40, 17, 3, 50])]
    ars = [single.ar_decode(p, 32)[0] for p in prompts]
    specs = [dict(policy=GUESS_STREAM_REINJECT if i % 2 else GUESS_UNIFORM, block_policy=BLOCK_SHRINK,
                  stream=ars[i] if i % 2 else None, p=0.4, seed=50 + i) for i in range(len(prompts))]
    log("[gpu-batch] tiny: trajectory collection of 10 prompts vs oracle")
    entries = collect.collect(batched, prompts, 8, 32, specs=specs, rate=0.5, seed=77)
    k = 0
    for i, p in enumerate(prompts):
        sp = specs[i]
        spec = oracle.GuessSpec(sp["policy"], BLOCK_SHRINK, sp["stream"], p=sp["p"], seed=sp["seed"])
        out_o, st_o = orc.jacobi_decode(p, 8, 32, spec, seq=i % batched.max_batch, trace=True)
        np.testing.assert_array_equal(out_o, ars[i])
        for blk in oracle.collect_trajectories(st_o["trajectory"], out_o, 8, 0.5, 77 + i):
            e = entries[k]
            k += 1
            assert e["prompt"] == i
            np.testing.assert_array_equal(e["prefix"], np.concatenate([p, out_o[:blk["b0"]]]))
            np.testing.assert_array_equal(e["fixed"], blk["fixed"])
            np.testing.assert_array_equal(e["states"], np.stack(blk["states"]))
            np.testing.assert_array_equal(e["augmented"], np.stack(blk["augmented"]))
    assert k == len(entries)
