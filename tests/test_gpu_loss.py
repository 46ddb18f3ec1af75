"""GPU checks of the CLLM training loss at the LM head (Section 3.2.2: the global consistency
loss, a forward KL between the fixed point's and the trajectory state's token distributions, plus
omega times the AR loss) against the oracle's fp64 loss_head, through cllm_loss_head.

Inputs: the model's own LM-head weights (N(0, 0.02), bf16 or fp32) and seeded rows scaled so the
logits have standard deviation ~3 (workload.make_head_rows; every fourth student row equals its
teacher row, so its KL and gradient vanish).

Tolerances. The fp32 path (rows and weights fp32, fp32 MFMA accumulation) gets the fp32 bar,
1e-4. In bf16 the rows enter the GEMM as hi + lo bf16 planes (16 significant bits, relative error
<= 2^-16) against exact bf16 weights with fp32 accumulation, so each logit is within ~2^-16 of
its scale (~3 here) of the fp64 value, i.e. ~5e-5; the log-softmax moves by at most twice that,
a KL or NLL by at most ~4x (times 1 + its value), and the gradients (softmax differences times
W or H, fp32 MFMA) by the same relative amount of their scale. 1e-3 covers this with a margin of
~5, and stays two orders of magnitude below what a dropped term, a wrong sign or a swapped
operand would change (those are pinned in the oracle's own tests).

Every value is checked per row as |gpu - oracle| <= tol * (1 + |oracle|). A gradient element,
a sum of products of softmax terms and rows or weights, is checked against the same sum over
absolute values (the usual forward-error form: a converged pair has an exact gradient of zero,
which the GPU reaches only up to rounding): for dH[i, k] = sum_v D[i, v] W[v, k] the scale is
sum_v |dD|[i, v] |W[v, k]| with |dD| = p + q for a pair and omega (c + onehot) for an AR row, and
for dW[v, k] the scale is sum_i |dD|[i, v] |H[i, k]|.
"""
import numpy as np
import pytest

import oracle
from paper_2403_00835_amd import workload
from paper_2403_00835_amd.configs import SMALL, ModelConfig
from tests.parity import log

pytestmark = pytest.mark.gpu

# fp32 head with a vocabulary that is not a multiple of the 64-column LM-head tile (1000 -> 1024)
HEAD_F32 = ModelConfig(n_layers=1, d_model=64, n_heads=4, head_dim=16, ffn_dim=172, vocab=1000, dtype="f32")
# bf16 head whose width is not a multiple of the dW kernel's 128-column block (192), ragged vocabulary
HEAD_BF16 = ModelConfig(n_layers=1, d_model=192, n_heads=3, head_dim=64, ffn_dim=512, vocab=1000, dtype="bf16")
TOLS = {"f32": 1e-4, "bf16": 1e-3}

CASES = [  # (teacher/student pairs, AR rows, omega)
    (5, 3, 1.0),
    (0, 7, 2.0),      # AR rows only
    (9, 0, 1.0),      # consistency pairs only
    (1, 0, 1.0),
    (0, 1, 0.5),
    (40, 24, 1.0),    # 64 loss rows, 104 GEMM rows: two 64-row tiles
    (16, 16, 0.0),    # omega 0: the AR rows are reported but carry no gradient
    (64, 0, 1.0),     # the most pairs: 128 GEMM rows, two full row tiles
    (0, 64, 1.0),     # the most AR rows
]


@pytest.fixture(scope="module", params=[HEAD_F32, HEAD_BF16, SMALL], ids=["f32-v1000", "bf16-d192-v1000", "small-bf16"])
def head(request):
    from paper_2403_00835_amd import binding
    cfg = request.param
    log(f"[loss] context {cfg.dtype} d={cfg.d_model} V={cfg.vocab}")
    ws = workload.make_weights(cfg)
    m = binding.Model(cfg, max_ctx=64, max_block=8, max_new=8, weights=ws)
    W = workload.as_f32(cfg, ws[-1]).astype(np.float64)
    yield cfg, m, W
    m.close()


def _close_rows(g, o, tol, what):
    err = np.abs(np.asarray(g, np.float64) - o)
    bound = tol * (1.0 + np.abs(o))
    assert np.all(err <= bound), f"{what}: worst {err.max():.3g} (bound {bound[err.argmax()]:.3g})"
    return float(err.max()) if err.size else 0.0


def _softmax(z):
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def _grad_scales(W, t, s, ar, tg, omega):
    """Absolute-value sums bounding the gradients' rounding (see the module docstring)."""
    aW = np.abs(W)
    dp = _softmax(t.astype(np.float64) @ W.T) + _softmax(s.astype(np.float64) @ W.T)
    da = _softmax(ar.astype(np.float64) @ W.T)
    da[np.arange(tg.size), tg] += 1.0
    da *= abs(omega)
    return dp @ aW, da @ aW, dp.T @ np.abs(s) + da.T @ np.abs(ar)


def _close_array(g, o, scale, tol, what):
    if o.size == 0:
        return 0.0
    err = np.abs(np.asarray(g, np.float64) - o)
    ratio = err / np.maximum(scale, 1e-300)
    assert np.all(err <= tol * scale), f"{what}: worst err/scale {ratio.max():.3g} (err {err.max():.3g})"
    return float(ratio.max())


@pytest.mark.parametrize("P,A,omega", CASES)
def test_loss_head_vs_oracle(head, P, A, omega):
    cfg, m, W = head
    tol = TOLS[cfg.dtype]
    t, s, ar, tg = workload.make_head_rows(cfg, P, A, seed=100 + 7 * P + A)
    log(f"[loss] {cfg.dtype} P={P} A={A} omega={omega}")
    g = m.loss_head(t, s, ar, tg, omega, want_dw=True)
    o = oracle.loss_head(W, t, s, ar, tg, omega)
    e_kl = _close_rows(g["kl"], o["kl"], tol, "kl")
    e_nll = _close_rows(g["nll"], o["nll"], tol, "nll")
    terms = np.abs(o["kl"]).sum() + abs(omega) * np.abs(o["nll"]).sum()
    assert abs(g["loss"] - o["loss"]) <= tol * (1.0 + terms), (g["loss"], o["loss"])
    sc_s, sc_a, sc_w = _grad_scales(W, t, s, ar, tg, omega)
    r_s = _close_array(g["d_student"], o["d_student"], sc_s, tol, "d_student")
    r_a = _close_array(g["d_ar"], o["d_ar"], sc_a, tol, "d_ar")
    r_w = _close_array(g["d_W"], o["d_W"], sc_w, tol, "d_W")
    log(f"  max err kl {e_kl:.2g} nll {e_nll:.2g}; rel grad err student {r_s:.2g} ar {r_a:.2g} W {r_w:.2g}")
    if P:
        conv = np.arange(0, P, 4)  # student rows equal to their teacher rows
        assert np.all(np.abs(g["kl"][conv]) <= tol), g["kl"][conv]
    if omega == 0.0 and A:
        assert np.all(g["d_ar"] == 0.0)
    assert np.all(g["kl"] >= -tol)  # a KL divergence is non-negative
    assert np.all(g["nll"] >= 0.0)


def test_loss_head_repeat_is_deterministic(head):
    """Every sum runs in a fixed order: two calls return identical bits, and a call with a
    smaller batch in between does not disturb the next one."""
    cfg, m, W = head
    t, s, ar, tg = workload.make_head_rows(cfg, 12, 6, seed=5)
    a = m.loss_head(t, s, ar, tg, 1.0, want_dw=True)
    m.loss_head(t[:2], s[:2], ar[:1], tg[:1], 3.0, want_dw=True)
    b = m.loss_head(t, s, ar, tg, 1.0, want_dw=True)
    for k in ("kl", "nll", "d_student", "d_ar", "d_W"):
        assert np.array_equal(a[k], b[k]), k
    assert a["loss"] == b["loss"]


def test_loss_head_without_dw_matches(head):
    cfg, m, W = head
    t, s, ar, tg = workload.make_head_rows(cfg, 6, 4, seed=9)
    a = m.loss_head(t, s, ar, tg, 1.0, want_dw=True)
    b = m.loss_head(t, s, ar, tg, 1.0, want_dw=False)
    assert "d_W" not in b
    for k in ("kl", "nll", "d_student", "d_ar"):
        assert np.array_equal(a[k], b[k]), k


def test_loss_head_argument_errors(head):
    from paper_2403_00835_amd import binding
    cfg, m, W = head
    t, s, ar, tg = workload.make_head_rows(cfg, 40, 25, seed=11)
    with pytest.raises(binding.CllmError):
        m.loss_head(t[:0], s[:0], ar[:0], tg[:0], 1.0)       # no rows
    with pytest.raises(binding.CllmError):
        m.loss_head(t, s, ar, tg, 1.0)                       # 65 loss rows
    bad = tg[:3].copy()
    bad[1] = cfg.vocab
    with pytest.raises(binding.CllmError):
        m.loss_head(t[:2], s[:2], ar[:3], bad, 1.0)          # target out of range
    with pytest.raises(binding.CllmError):
        m.loss_head(t[:2], s[:2], ar[:3], tg[:3], float("nan"))
    # the context still works after rejected calls
    g = m.loss_head(t[:2], s[:2], ar[:3], tg[:3], 1.0)
    o = oracle.loss_head(W, t[:2], s[:2], ar[:3], tg[:3], 1.0)
    _close_rows(g["kl"], o["kl"], TOLS[cfg.dtype], "kl after errors")


def _dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def test_loss_head_device_equals_host(head):
    """cllm_loss_head_device on device arrays returns the host entry point's results bit for bit,
    on two calls in a row, the second smaller (the workspace keeps the first call's contents)."""
    import torch
    cfg, m, W = head
    d, V = cfg.d_model, cfg.vocab
    for P, A in ((12, 20), (3, 2)):
        t, s, ar, tg = workload.make_head_rows(cfg, P, A, seed=31 + P)
        h = m.loss_head(t, s, ar, tg, 1.5, want_dw=True)
        T, S, Ar, TG = _dev(t), _dev(s), _dev(ar), _dev(tg)
        nan = float("nan")
        kl, nll = torch.full((P,), nan, device="cuda"), torch.full((A,), nan, device="cuda")
        ds, da = torch.full((P, d), nan, device="cuda"), torch.full((A, d), nan, device="cuda")
        dw = torch.full((V, d), nan, device="cuda")
        loss = torch.full((1,), nan, dtype=torch.float64, device="cuda")
        torch.cuda.synchronize()
        m.loss_head_device(P, A, 1.5, T, S, Ar, TG, kl, nll, ds, da, dw, loss)
        torch.cuda.synchronize()
        assert np.array_equal(kl.cpu().numpy(), h["kl"]) and np.array_equal(nll.cpu().numpy(), h["nll"])
        assert np.array_equal(ds.cpu().numpy(), h["d_student"]) and np.array_equal(da.cpu().numpy(), h["d_ar"])
        assert np.array_equal(dw.cpu().numpy(), h["d_W"])
        assert loss.item() == h["loss"]


def test_loss_head_device_bad_target_and_host_memory(head):
    """On device arrays a target outside the vocabulary gives a NaN loss and gradient for that AR
    row only; pageable host memory is rejected before anything runs."""
    import torch
    from paper_2403_00835_amd import binding
    cfg, m, W = head
    d = cfg.d_model
    t, s, ar, tg = workload.make_head_rows(cfg, 2, 3, seed=41)
    h = m.loss_head(t, s, ar, tg, 1.0)
    bad = tg.copy()
    bad[1] = cfg.vocab + 5
    T, S, Ar, TG = _dev(t), _dev(s), _dev(ar), _dev(bad)
    kl, nll = torch.zeros(2, device="cuda"), torch.zeros(3, device="cuda")
    ds, da = torch.zeros(2, d, device="cuda"), torch.zeros(3, d, device="cuda")
    torch.cuda.synchronize()
    m.loss_head_device(2, 3, 1.0, T, S, Ar, TG, kl, nll, ds, da)
    torch.cuda.synchronize()
    nll_h, da_h = nll.cpu().numpy(), da.cpu().numpy()
    assert np.isnan(nll_h[1]) and np.all(np.isnan(da_h[1]))
    assert np.array_equal(nll_h[[0, 2]], h["nll"][[0, 2]]) and np.array_equal(da_h[[0, 2]], h["d_ar"][[0, 2]])
    assert np.array_equal(kl.cpu().numpy(), h["kl"]) and np.array_equal(ds.cpu().numpy(), h["d_student"])
    host_rows = np.ascontiguousarray(t)
    with pytest.raises(binding.CllmError):
        m.loss_head_device(2, 3, 1.0, host_rows.ctypes.data, S, Ar, TG, kl, nll, ds, da)
    with pytest.raises(ValueError):
        m.loss_head_device(2, 3, 1.0, T, S, Ar, TG, kl, nll[:2], ds, da)  # too few rows


def test_loss_head_7b_bench_configuration():
    """The benchmark's configuration at full size: the LLaMA-2-7B LM head (32000 x 4096 bf16, a
    one-layer context drawn on the device), 16 pairs + 48 AR rows through the device entry point
    with the weight gradient; every output (per-row KL and NLL, the total, dH and all of dW)
    against the oracle, to the bf16 bar of this file."""
    import dataclasses

    import torch
    from paper_2403_00835_amd import binding
    from paper_2403_00835_amd.configs import LLAMA7B
    cfg = dataclasses.replace(LLAMA7B, n_layers=1)
    d, V = cfg.d_model, cfg.vocab
    P, A, omega = 16, 48, 1.0
    log("[loss] 7B head: device-drawn context, host-drawn head for the oracle")
    m = binding.Model(cfg, max_ctx=64, max_block=16, max_new=16, random_seed=0)
    W = workload.as_f32(cfg, workload.make_tensor(cfg, workload.tensor_specs(cfg)[-1])).astype(np.float64)
    t, s, ar, tg = workload.make_head_rows(cfg, P, A, seed=1)
    T, S, Ar, TG = _dev(t), _dev(s), _dev(ar), _dev(tg)
    kl, nll = torch.empty(P, device="cuda"), torch.empty(A, device="cuda")
    ds, da = torch.empty(P, d, device="cuda"), torch.empty(A, d, device="cuda")
    dw = torch.empty(V, d, device="cuda")
    loss = torch.empty(1, dtype=torch.float64, device="cuda")
    torch.cuda.synchronize()
    m.loss_head_device(P, A, omega, T, S, Ar, TG, kl, nll, ds, da, dw, loss)
    torch.cuda.synchronize()
    m.close()
    log("  oracle")
    o = oracle.loss_head(W, t, s, ar, tg, omega)
    tol = TOLS["bf16"]
    e_kl = _close_rows(kl.cpu().numpy(), o["kl"], tol, "kl")
    e_nll = _close_rows(nll.cpu().numpy(), o["nll"], tol, "nll")
    terms = np.abs(o["kl"]).sum() + omega * np.abs(o["nll"]).sum()
    assert abs(loss.item() - o["loss"]) <= tol * (1.0 + terms)
    sc_s, sc_a, sc_w = _grad_scales(W, t, s, ar, tg, omega)
    r_s = _close_array(ds.cpu().numpy(), o["d_student"], sc_s, tol, "d_student")
    r_a = _close_array(da.cpu().numpy(), o["d_ar"], sc_a, tol, "d_ar")
    r_w = _close_array(dw.cpu().numpy(), o["d_W"], sc_w, tol, "d_W")
    log(f"  max err kl {e_kl:.2g} nll {e_nll:.2g}; rel grad err student {r_s:.2g} ar {r_a:.2g} W {r_w:.2g}")
