"""Bit-exactness of the multi-row decode GEMMs against gemm_kernel, through the standalone kernel
driver's check mode: seeded random weights, operands and RMSNorm inputs at the LLaMA-2-7B shape,
each product (QKV, O, gate/up, down, LM head) launched as iterations launch it (with several row
tiles: the class-pair K split for QKV, gate/up and the LM head, the row-tiled kernel for the down
product's K ranges, each taking gemm_kernel's body when the live rows fit one tile) and through
gemm_kernel over the same row tiles. Every output (Q operand, cached keys and values, residual
rows, next RMSNorm operand and its sums of squares, SwiGLU rows, argmax partials) must be
bit-identical, from one 16-row group to eight 64-row tiles, ragged tails included (a one-tile
launch and the last tile of a split launch run only their live 16-row groups, 1 to 4 of them): the
split and the row-tiled kernels keep gemm_kernel's reduction order, which is what makes batched,
Jacobi and AR decoding give the same bits for a row."""
import os
import subprocess

import pytest

from paper_2403_00835_amd import build
from tests.parity import log

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rows", [16, 17, 33, 48, 64, 65, 96, 120, 160, 200, 289, 512])
def test_multi_row_gemms_bit_identical(rows):
    exe = build.KERNEL_BENCH
    if not os.path.exists(exe):
        pytest.fail("the kernel driver is not built (python -c 'import __graft_entry__; __graft_entry__.build()')")
    log(f"[kernel-check] {rows} rows")
    r = subprocess.run([exe, "check", str(rows)], capture_output=True, text=True, timeout=120)
    for line in r.stdout.splitlines():
        log("  " + line)
    assert r.returncode == 0 and "check ok" in r.stdout, r.stdout + r.stderr
