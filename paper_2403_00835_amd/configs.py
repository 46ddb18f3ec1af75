"""Model shapes and decode workloads.

The paper runs LLaMA-2-7B and Deepseek-coder-7B (Section 4, experimental setup) but prints no
architecture; these shapes follow the LLaMA-style decoder the experiments name: pre-norm
RMSNorm, rotate-half RoPE, multi-head attention without GQA, SwiGLU FFN, untied LM head,
no biases. Weights are seeded N(0, 0.02), norm gains 1.0.
"""
from dataclasses import dataclass, field, asdict


@dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    rms_eps: float = 1e-6
    rope_base: float = 10000.0
    dtype: str = "bf16"  # "bf16" or "f32"

    def __post_init__(self):
        if self.n_heads * self.head_dim != self.d_model:
            raise ValueError("n_heads * head_dim must equal d_model")
        if self.head_dim % 2:
            raise ValueError("head_dim must be even for rotate-half RoPE")
        if self.dtype not in ("bf16", "f32"):
            raise ValueError("dtype must be 'bf16' or 'f32'")

    @property
    def dtype_code(self) -> int:
        return 1 if self.dtype == "bf16" else 0

    @property
    def n_tensors(self) -> int:
        return 3 + 9 * self.n_layers

    def streamed_params(self) -> int:
        """Parameters read by one forward pass (the embedding is only gathered)."""
        d, f = self.d_model, self.ffn_dim
        per_layer = 4 * d * d + 3 * d * f + 2 * d
        return self.n_layers * per_layer + d + self.vocab * d

    def kv_bytes_per_token(self) -> int:
        elem = 2 if self.dtype == "bf16" else 4
        return 2 * self.n_layers * self.d_model * elem

    def as_dict(self):
        return asdict(self)


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelConfig
    prompt_len: int
    n: int
    max_new: int
    p: tuple = ()  # corruption rates of the guess stream
    batch: int = 1
    prompt_len_range: tuple = ()  # (lo, hi) for ragged batches
    p_range: tuple = ()


TINY = ModelConfig(n_layers=2, d_model=64, n_heads=4, head_dim=16, ffn_dim=172, vocab=256, dtype="f32")
SMALL = ModelConfig(n_layers=12, d_model=768, n_heads=12, head_dim=64, ffn_dim=2048, vocab=32000)
LLAMA7B = ModelConfig(n_layers=32, d_model=4096, n_heads=32, head_dim=128, ffn_dim=11008, vocab=32000)

WORKLOADS = {
    "tiny": Workload("tiny-f32", TINY, prompt_len=16, n=8, max_new=32),
    "small": Workload("small-bf16", SMALL, prompt_len=128, n=16, max_new=256, p=(0.3,)),
    "7b": Workload("llama7b-bf16", LLAMA7B, prompt_len=512, n=16, max_new=256, p=(0.1, 0.3, 0.6)),
    "7b_long": Workload("llama7b-bf16-long", LLAMA7B, prompt_len=2048, n=64, max_new=512, p=(0.3,)),
    "7b_batched": Workload("llama7b-bf16-batched", LLAMA7B, prompt_len=1024, n=32, max_new=256,
                           batch=16, prompt_len_range=(256, 1024), p_range=(0.1, 0.6)),
}

# Seeds of the synthetic inputs (one per purpose).
SEED_WEIGHTS = 0
SEED_PROMPT = 1
SEED_GUESS = 2      # uniform-random initial guesses
SEED_CORRUPT = 3    # corruption of the guess stream
SEED_BATCH = 4      # ragged batch lengths and per-sequence p

# Guess and block policies (mirrored in the C ABI).
GUESS_UNIFORM = 0
GUESS_STREAM = 1
GUESS_STREAM_REINJECT = 2
BLOCK_SHRINK = 0
BLOCK_SLIDE = 1
