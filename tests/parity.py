"""Parity helpers shared by the GPU tests: compare the HIP path with the oracle under the
teacher-forced protocol. Where floating point decides a token (the argmax), positions whose
oracle top-1 margin is within the tolerance may legitimately differ; everywhere else the
tokens must be identical."""
import sys

import numpy as np

import oracle

TOL = {"f32": 1e-4, "bf16": 2e-2}


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def margins(lg):
    """top-1 minus top-2 of each row, on the fp32-rounded oracle logits."""
    x = np.asarray(lg, dtype=np.float32)
    part = np.partition(x, -2, axis=-1)
    return part[..., -1].astype(np.float64) - part[..., -2].astype(np.float64)


def oracle_argmax_rows(lg):
    return np.array([oracle.argmax(r) for r in lg], dtype=np.int64)


def check_rows(gpu_tokens, orc_logits, tol, what=""):
    """Each GPU token is the oracle's argmax where the oracle's margin exceeds tol, and otherwise
    within tol of the oracle's maximum logit. Returns the number of rows inside the margin."""
    orc_logits = np.atleast_2d(orc_logits)
    mg = margins(orc_logits)
    am = oracle_argmax_rows(orc_logits)
    inside = 0
    for i, tok in enumerate(np.atleast_1d(gpu_tokens)):
        if mg[i] > tol:
            assert tok == am[i], f"{what} row {i}: gpu {tok} != oracle {am[i]} (margin {mg[i]:.3g})"
        else:
            inside += 1
            gap = orc_logits[i, am[i]] - orc_logits[i, tok]
            assert gap <= tol, f"{what} row {i}: gpu token {tok} is {gap:.3g} below the max (tol {tol})"
    return inside


def verify_greedy_sequence(orc_model, prompt, tokens, tol, what="decode"):
    """tokens (y0 first) is a valid greedy continuation of prompt under the oracle: one
    uncached forward over prompt + tokens[:-1] scores every position at once."""
    seq = np.concatenate([np.asarray(prompt), np.asarray(tokens[:-1])]).astype(np.int32)
    lg = orc_model.forward_full(seq)
    P = len(prompt)
    return check_rows(tokens, lg[P - 1:P - 1 + len(tokens)], tol, what)
