"""GPU against the oracle at the sizes and in the kernel paths the benchmark runs (teacher-forced
protocol: the oracle is fed the GPU's blocks and commits, and every iteration's logits, tokens
and accepted length are compared).

- LLaMA-2-7B shape, prompt 512, iterations of 16 rows: the headline's own prefill (one 512-row
  pass of the prompt GEMMs and the chunk-parallel attention) and decode iterations at contexts
  of 513..593 keys, where the one-kernel attention gives its waves a second 64-key chunk and
  the rows of one iteration straddle a chunk boundary.
- A two-layer model of the 7B width (d 4096, 32 x 128 heads, FFN 11008, vocab 32000), prompt
  2048, blocks of 64 rows: four prompt passes of 512 rows, then iterations whose contexts span
  more than 32 chunks (the two-kernel attention) through the 64-row GEMM tiles and the 64-row
  K-split down product.
- The same two-layer model, batched ragged iterations of five sequences (prompts 90..1100 tokens,
  blocks of 7..64 rows, 160 and 111 rows in all): row-tiled GEMMs over several 64-row tiles, the
  batched attention grid, compared per sequence with one oracle state per sequence.

Each test logs its worst max|dlogit|; the tolerance is the bf16 one (2e-2), tokens must agree
wherever the oracle's top-1 margin exceeds it.
"""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import LLAMA7B, ModelConfig
from tests.parity import TOL, check_rows, log

pytestmark = pytest.mark.gpu

WIDE2 = ModelConfig(n_layers=2, d_model=4096, n_heads=32, head_dim=128, ffn_dim=11008, vocab=32000)


def _oracle_model(cfg, ws):
    return oracle.Model(cfg, [workload.as_f32(cfg, t) for t in ws])


def _next_block(out, a, stream, e, m, vocab, corrupt_every=0):
    """The next block after an iteration that emitted up to output position e: the pending token
    out[a - 1], then the reference continuation stream[e + 1 ..] (every corrupt_every-th guess
    replaced by a different id)."""
    z = [int(out[a - 1])] + [int(t) for t in stream[e + 1:e + m]]
    if corrupt_every:
        for j in range(corrupt_every, len(z), corrupt_every):
            z[j] = (z[j] + 1 + j) % vocab
    return np.array(z, dtype=np.int32)


def _oracle_prefill(st, prompt, chunk, what):
    """The oracle's prefill in chunks of `chunk` prompt rows (each chunk a cached block forward
    over the rows before it, which equals one forward over the whole prompt), logging each
    chunk. Returns y0 and the logits of the last prompt row."""
    P = len(prompt)
    if P <= chunk:
        return st.prefill(prompt, want_logits=True)
    st.prefill(prompt[:chunk])
    for c0 in range(chunk, P, chunk):
        blk = prompt[c0:c0 + chunk]
        lg = st.eval_block(blk)
        y = oracle.argmax(lg[-1])
        st.commit(blk.size, int(prompt[c0 + blk.size]) if c0 + blk.size < P else y)
        log(f"  {what}: oracle prompt rows {c0 + blk.size} / {P}")
    return y, lg[-1]


def _compare(lg_g, lg_o, out, a, z, tol, what):
    e = float(np.abs(lg_g - lg_o).max())
    inside = check_rows(out, lg_o, tol, what)
    if inside == 0:
        assert a == oracle.accept_len(z, out), what
    log(f"  {what}: rows {z.size}, max|dlogit| {e:.4g}, accepted {a}, rows inside the margin {inside}")
    assert e <= tol, f"{what}: max|dlogit| {e:.4g} > {tol}"
    return e


@pytest.mark.timeout(1200)
def test_7b_prompt512_iterations_vs_oracle():
    from paper_2403_00835_amd import binding
    cfg, tol = LLAMA7B, TOL["bf16"]
    log("[oracle-full] 7B: drawing weights, creating the GPU context")
    ws = workload.make_weights(cfg)
    gpu = binding.Model(cfg, max_ctx=704, max_block=16, max_new=128, weights=ws)
    prompt = workload.make_prompt(cfg, 512)  # the benchmark's prompt
    ar, _ = gpu.ar_decode(prompt, 128)
    gpu.debug_logits(True)
    log("[oracle-full] 7B: GPU prefill (512 rows) and 6 iterations of 16 rows")
    y0 = gpu.prefill(prompt)
    assert y0 == ar[0]
    g_pre = gpu.last_logits(64)[511 % 64].copy()
    spec = oracle.GuessSpec(0, 0, None, seed=5)
    z = np.array([y0] + [oracle.guess(spec, 0, j, 0, cfg.vocab) for j in range(1, 16)], dtype=np.int32)
    its, e = [], 0
    for it in range(6):
        out, a = gpu.jacobi_step(z)
        its.append((z.copy(), out.copy(), a, gpu.last_logits(z.size).copy()))
        e += a
        # exact guesses advance the context 16 keys per iteration; the last two are corrupted
        z = _next_block(out, a, ar, e, 16, cfg.vocab, corrupt_every=0 if it < 3 else 5)
    L, _ = gpu.seq_state()
    gpu.debug_logits(False)
    gpu.close()
    log(f"[oracle-full] 7B: committed length after the iterations {L}")

    log("[oracle-full] 7B: oracle prefill of 512 rows (fp64, host threads)")
    orc = _oracle_model(cfg, ws)
    st = oracle.State(orc, 704)
    y0_o, lg0 = _oracle_prefill(st, prompt, 128, "7B")
    worst = _compare(g_pre[None], lg0[None], np.array([y0]), 1, np.array([y0]), tol, "prefill row 511")
    for it, (z, out, a, lg_g) in enumerate(its):
        lg_o = st.eval_block(z)
        worst = max(worst, _compare(lg_g, lg_o, out, a, z, tol, f"iteration {it} at L={st.L}"))
        st.commit(a, int(out[a - 1]))
    assert st.L == L
    log(f"[oracle-full] 7B: worst max|dlogit| {worst:.4g} (tolerance {tol})")


@pytest.fixture(scope="module")
def wide2():
    log("[oracle-full] 7B-width two-layer model: weights and oracle copy")
    ws = workload.make_weights(WIDE2, seed=7)
    return ws, _oracle_model(WIDE2, ws)


@pytest.mark.timeout(900)
def test_7b_width_prompt2048_blocks_of_64_vs_oracle(wide2):
    from paper_2403_00835_amd import binding
    ws, orc = wide2
    tol = TOL["bf16"]
    gpu = binding.Model(WIDE2, max_ctx=2048 + 320, max_block=64, max_new=256, weights=ws)
    prompt = workload.make_prompt(WIDE2, 2048, seed=8)
    ar, _ = gpu.ar_decode(prompt, 256)
    gpu.debug_logits(True)
    log("[oracle-full] width-2: GPU prefill (2048 rows in four passes) and 3 iterations of 64 rows")
    y0 = gpu.prefill(prompt)
    g_pre = gpu.last_logits(64)[2047 % 64].copy()
    spec = oracle.GuessSpec(0, 0, None, seed=6)
    z = np.array([y0] + [oracle.guess(spec, 0, j, 0, WIDE2.vocab) for j in range(1, 64)], dtype=np.int32)
    its, e = [], 0
    for it in range(3):
        out, a = gpu.jacobi_step(z)
        its.append((z.copy(), out.copy(), a, gpu.last_logits(z.size).copy()))
        e += a
        z = _next_block(out, a, ar, e, 64, WIDE2.vocab, corrupt_every=0 if it == 0 else 9)
    gpu.debug_logits(False)
    gpu.close()

    log("[oracle-full] width-2: oracle prefill of 2048 rows")
    st = oracle.State(orc, 2048 + 320)
    y0_o, lg0 = _oracle_prefill(st, prompt, 512, "width-2")
    worst = _compare(g_pre[None], lg0[None], np.array([y0]), 1, np.array([y0]), tol, "prefill row 2047")
    for it, (z, out, a, lg_g) in enumerate(its):
        nch = (st.L + z.size - 1) // 64 + 1
        lg_o = st.eval_block(z)
        worst = max(worst, _compare(lg_g, lg_o, out, a, z, tol, f"iteration {it} at L={st.L} ({nch} chunks)"))
        st.commit(a, int(out[a - 1]))
    log(f"[oracle-full] width-2: worst max|dlogit| {worst:.4g} (tolerance {tol})")


@pytest.mark.timeout(900)
def test_7b_width_batched_ragged_vs_oracle(wide2):
    from paper_2403_00835_amd import binding
    ws, orc = wide2
    tol = TOL["bf16"]
    lens = [300, 1100, 90, 700, 513]
    sizes = [[16, 64, 7, 40, 33], [32, 5, 50, 1, 23]]  # 160 and 111 rows: three and two 64-row tiles
    B = len(lens)
    gpu = binding.Model(WIDE2, max_ctx=1100 + 192 + 64, max_block=64, max_new=192, max_batch=B, weights=ws)
    prompts = [workload.make_prompt(WIDE2, n, seed=20 + b) for b, n in enumerate(lens)]
    ars = [gpu.ar_decode(p, 192, seq=b)[0] for b, p in enumerate(prompts)]
    gpu.debug_logits(True)
    log("[oracle-full] batched: GPU prefills of five sequences, two batched iterations")
    pre = []
    for b, p in enumerate(prompts):
        y0 = gpu.prefill(p, seq=b)
        pre.append((y0, gpu.last_logits(64)[(len(p) - 1) % 64].copy()))
    spec = oracle.GuessSpec(0, 0, None, seed=9)
    blocks = [np.array([pre[b][0]] + [oracle.guess(spec, b, j, 0, WIDE2.vocab) for j in range(1, sizes[0][b])],
                       dtype=np.int32) for b in range(B)]
    steps, e = [], [0] * B
    for s, sz in enumerate(sizes):
        res = gpu.jacobi_step_batch(list(range(B)), blocks)
        lg = gpu.last_logits(sum(sz)).copy()
        r0 = np.concatenate([[0], np.cumsum(sz)[:-1]])
        steps.append([(blocks[b].copy(), res[b][0].copy(), res[b][1], lg[r0[b]:r0[b] + sz[b]]) for b in range(B)])
        if s + 1 < len(sizes):
            nxt = []
            for b in range(B):
                out, a = res[b]
                e[b] += a
                nxt.append(_next_block(out, a, ars[b], e[b], sizes[s + 1][b], WIDE2.vocab, corrupt_every=4))
            blocks = nxt
    gpu.debug_logits(False)
    gpu.close()

    worst = 0.0
    for b in range(B):
        log(f"[oracle-full] batched: oracle sequence {b} (prompt {lens[b]})")
        st = oracle.State(orc, 1100 + 192 + 64)
        y0_o, lg0 = _oracle_prefill(st, prompts[b], 512, f"seq {b}")
        worst = max(worst, _compare(pre[b][1][None], lg0[None], np.array([pre[b][0]]), 1, np.array([pre[b][0]]), tol,
                                    f"seq {b} prefill"))
        for s in range(len(sizes)):
            z, out, a, lg_g = steps[s][b]
            lg_o = st.eval_block(z)
            worst = max(worst, _compare(lg_g, lg_o, out, a, z, tol, f"seq {b} batched iteration {s}"))
            st.commit(a, int(out[a - 1]))
    log(f"[oracle-full] batched: worst max|dlogit| {worst:.4g} (tolerance {tol})")
