"""Seeded synthetic inputs shared by the GPU path and the CPU oracle.

Only random numbers are drawn here (weights, prompts, batch lengths); none of the decoding
method's arithmetic lives in this module. The C generator in gen.c is built into
libcllm_workload.so next to this file.
"""
import ctypes
import os
import subprocess

import numpy as np

from ..configs import SEED_BATCH, ModelConfig, SEED_PROMPT, SEED_WEIGHTS

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gen.c")
# CLLM_HOST_SANITIZE=1: the build with address and undefined-behaviour checks (build_host_sanitized)
_SANITIZE = os.environ.get("CLLM_HOST_SANITIZE") == "1"
_LIB = os.path.join(_HERE, "libcllm_workload.hostsan.so" if _SANITIZE else "libcllm_workload.so")
_lib = None

WEIGHT_STD = 0.02


def build(verbose=False):
    """Compile gen.c into libcllm_workload.so (always recompiles)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", _LIB + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    global _lib
    _lib = None


def build_host_sanitized(clang, verbose=False):
    """Compile gen.c with address and undefined-behaviour checks into libcllm_workload.hostsan.so."""
    out = os.path.join(_HERE, "libcllm_workload.hostsan.so")
    cmd = [clang, "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-shared-libasan",
           "-fopenmp", "-fPIC", "-shared", "-o", out + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            if _SANITIZE:
                raise RuntimeError(f"{_LIB} is not built (build.py --host-sanitize)")
            build()
        L = ctypes.CDLL(_LIB)
        u64, i64, i32, dbl = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
        vp = ctypes.c_void_p
        L.wl_bits.restype = u64
        L.wl_bits.argtypes = [u64, u64, u64]
        L.wl_fill_normal_f32.argtypes = [u64, u64, dbl, vp, i64]
        L.wl_fill_normal_bf16.argtypes = [u64, u64, dbl, vp, i64]
        L.wl_fill_uniform_ids.argtypes = [u64, u64, i32, vp, i64]
        L.wl_fill_uniform_range.argtypes = [u64, u64, i32, i32, vp, i64]
        L.wl_fill_uniform_f64.argtypes = [u64, u64, vp, i64]
        L.wl_fill_const_f32.argtypes = [ctypes.c_float, vp, i64]
        L.wl_fill_const_bf16.argtypes = [ctypes.c_float, vp, i64]
        _lib = L
    return _lib


def bits(seed, stream, index):
    return int(lib().wl_bits(seed, stream, index))


def tensor_specs(cfg: ModelConfig):
    """Fixed tensor order of the weight set: (name, shape, stream id, kind).

    Order: embedding [V, d]; per layer: attn_norm [d], wq, wk, wv, wo [d, d], ffn_norm [d],
    w_gate [F, d], w_up [F, d], w_down [d, F]; final_norm [d]; lm_head [V, d].
    Matrices are row-major [out, in]; kind "normal" is N(0, 0.02), "ones" is the norm gain 1.0.
    """
    d, f, v = cfg.d_model, cfg.ffn_dim, cfg.vocab
    specs = [("embed", (v, d), 1, "normal")]
    for l in range(cfg.n_layers):
        b = 1000 * (l + 1)
        specs += [
            (f"l{l}.attn_norm", (d,), b + 0, "ones"),
            (f"l{l}.wq", (d, d), b + 1, "normal"),
            (f"l{l}.wk", (d, d), b + 2, "normal"),
            (f"l{l}.wv", (d, d), b + 3, "normal"),
            (f"l{l}.wo", (d, d), b + 4, "normal"),
            (f"l{l}.ffn_norm", (d,), b + 5, "ones"),
            (f"l{l}.w_gate", (f, d), b + 6, "normal"),
            (f"l{l}.w_up", (f, d), b + 7, "normal"),
            (f"l{l}.w_down", (d, f), b + 8, "normal"),
        ]
    specs += [("final_norm", (d,), 2, "ones"), ("lm_head", (v, d), 3, "normal")]
    return specs


def make_tensor(cfg: ModelConfig, spec, seed=SEED_WEIGHTS):
    """One weight tensor: matrices are uint16 bf16 bit patterns for bf16 models and float32 for
    f32 models; norm gains are always float32."""
    name, shape, stream, kind = spec
    n = int(np.prod(shape))
    L = lib()
    if kind == "ones":
        out = np.empty(shape, dtype=np.float32)
        L.wl_fill_const_f32(1.0, out.ctypes.data, n)
    elif cfg.dtype == "bf16":
        out = np.empty(shape, dtype=np.uint16)
        L.wl_fill_normal_bf16(seed, stream, WEIGHT_STD, out.ctypes.data, n)
    else:
        out = np.empty(shape, dtype=np.float32)
        L.wl_fill_normal_f32(seed, stream, WEIGHT_STD, out.ctypes.data, n)
    return out


def make_weights(cfg: ModelConfig, seed=SEED_WEIGHTS):
    """All weight tensors in the fixed order of tensor_specs."""
    return [make_tensor(cfg, s, seed) for s in tensor_specs(cfg)]


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (a.astype(np.uint32) << 16).view(np.float32)


def as_f32(cfg: ModelConfig, t: np.ndarray) -> np.ndarray:
    """float32 view of a weight tensor (bf16 bit patterns are widened exactly)."""
    return bf16_bits_to_f32(t) if t.dtype == np.uint16 else t


def make_prompt(cfg: ModelConfig, length, seed=SEED_PROMPT, seq=0):
    """Uniform-random prompt ids in [0, vocab); sequence `seq` uses its own stream."""
    out = np.empty(length, dtype=np.int32)
    lib().wl_fill_uniform_ids(seed, 100 + seq, cfg.vocab, out.ctypes.data, length)
    return out


def make_uniform_range(lo, hi, n, seed, stream):
    out = np.empty(n, dtype=np.int32)
    lib().wl_fill_uniform_range(seed, stream, lo, hi, out.ctypes.data, n)
    return out


def make_uniform_f64(n, seed, stream):
    out = np.empty(n, dtype=np.float64)
    lib().wl_fill_uniform_f64(seed, stream, out.ctypes.data, n)
    return out


def make_normal_f32(shape, std, seed, stream):
    """float32 array of the given shape with N(0, std^2) entries from stream `stream`."""
    out = np.empty(shape, dtype=np.float32)
    lib().wl_fill_normal_f32(seed, stream, float(std), out.ctypes.data, out.size)
    return out


def make_head_rows(cfg: ModelConfig, n_pairs, n_ar, seed, logit_std=3.0, student_mix=0.5):
    """Synthetic LM-head input rows for the training loss: teacher [P, d], student [P, d], AR
    rows [A, d] and AR targets [A]. Entries are normal, scaled so that with the N(0, 0.02) head
    weights the logits have standard deviation about `logit_std`; a student row is its teacher row
    plus `student_mix` times an independent row (the state's hidden rows lie near the fixed
    point's), and every fourth student row equals its teacher row (a converged position)."""
    d = cfg.d_model
    s = logit_std / (WEIGHT_STD * np.sqrt(d))
    t = make_normal_f32((n_pairs, d), s, seed, 201)
    st = t + np.float32(student_mix) * make_normal_f32((n_pairs, d), s, seed, 202)
    st[::4] = t[::4]
    ar = make_normal_f32((n_ar, d), s, seed, 203)
    tg = np.empty(n_ar, dtype=np.int32)
    lib().wl_fill_uniform_ids(seed, 204, cfg.vocab, tg.ctypes.data, n_ar)
    return t, st.astype(np.float32), ar, tg


def make_batch(cfg: ModelConfig, batch, len_range, p_range, seed=SEED_BATCH):
    """Ragged batch: `batch` prompt lengths uniform in [len_range[0], len_range[1]] (inclusive) and
    corruption rates uniform in [p_range[0], p_range[1]); prompt b is make_prompt(..., seq=b)."""
    lens = make_uniform_range(len_range[0], len_range[1], batch, seed, 1)
    u = make_uniform_f64(batch, seed, 2)
    ps = p_range[0] + (p_range[1] - p_range[0]) * u
    prompts = [make_prompt(cfg, int(n), seq=b) for b, n in enumerate(lens)]
    return prompts, ps
