"""MI355X (gfx950) Jacobi-decoding hot path of CLLMs (arXiv 2403.00835).

The product is the HIP library libcllm.so behind the C ABI in include/cllm.h; binding.py is
its thin ctypes binding. Import `paper_2403_00835_amd.binding` for the GPU path.
"""
from .configs import ModelConfig, Workload, WORKLOADS, TINY, SMALL, LLAMA7B  # noqa: F401
