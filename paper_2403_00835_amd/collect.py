"""Jacobi trajectory collection over a prompt set (the paper's Algorithm 1, Section 3.2.1): the
prompts are decoded in batches of the context's sequence slots with trajectory recording on
(one device-resident batched loop per batch, every row computed in the library's kernels); each
sequence's records become, per n-token block, the trajectory of block states from the first
guess to the fixed point, plus a copy with false tokens corrected at random (cllm_collect_states).
This module only orders the calls; it adds no arithmetic of its own.
"""
import numpy as np

from . import binding
from .configs import BLOCK_SHRINK


def collect(model, prompts, n, max_new, specs=None, rate=0.0, seed=0):
    """Returns one entry per prompt and block: dict(prompt index, prefix = the prompt followed by
    the earlier blocks' fixed points (the x of the next Jacobi decoding), fixed point, states
    [J, nb], augmented [J, nb]). specs: per prompt dict(policy, block_policy, stream, p, seed) as
    for Model.jacobi_decode_batch (the shrink block policy is required); the augmentation seed of
    prompt i is seed + i."""
    if specs is not None and any(sp.get("block_policy", BLOCK_SHRINK) != BLOCK_SHRINK for sp in specs):
        raise ValueError("trajectory collection takes the shrink block policy")
    entries = []
    B = model.max_batch
    model.trace_enable(True)
    try:
        for i0 in range(0, len(prompts), B):
            chunk = prompts[i0:i0 + B]
            slots = list(range(len(chunk)))
            out, _ = model.jacobi_decode_batch(slots, chunk, n, max_new,
                                               specs=None if specs is None else specs[i0:i0 + B])
            for b, q in enumerate(slots):
                traj = model.trace_read(q)
                st, au, bs = binding.collect_states(traj, out[b], n, rate, seed + i0 + b)
                j = 0
                while j < len(bs):
                    b0 = int(bs[j])
                    k = j
                    while k < len(bs) and bs[k] == b0:
                        k += 1
                    nb = int((st[k - 1] >= 0).sum())
                    entries.append({"prompt": i0 + b,
                                    "prefix": np.concatenate([np.asarray(chunk[b], dtype=np.int32), out[b][:b0]]),
                                    "fixed": st[k - 1, :nb].copy(), "states": st[j:k, :nb].copy(),
                                    "augmented": au[j:k, :nb].copy()})
                    j = k
    finally:
        model.trace_enable(False)
    return entries
