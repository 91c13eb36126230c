"""Model shapes and workloads used as synthetic stand-ins for the paper's setting.

The paper (Sec. 4, experimental setup) measures trained Qwen2.5/Qwen3 targets on
MATH-500, GSM8K, HumanEval and MT-Bench on A100.  None of those weights or
datasets is used here: the workloads below are random-init decoders of the named
shapes with seeded synthetic prompts, drafts and drafter confidences.
"""
from dataclasses import dataclass, field


@dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    dtype: str  # "f32" | "bf16" (storage and operand type)
    rms_eps: float = 1e-5
    rope_base: float = 10000.0
    init_std: float = 0.02

    @property
    def n_qkv(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def matmul_params(self) -> int:
        """Parameters of every matmul on the verify path, LM head included."""
        d, hd = self.d_model, self.head_dim
        per_layer = d * self.n_qkv + self.n_q_heads * hd * d + 3 * d * self.d_ff
        return self.n_layers * per_layer + d * self.vocab

    def with_layers(self, n_layers: int, name: str | None = None) -> "ModelShape":
        from dataclasses import replace
        return replace(self, n_layers=n_layers, name=name or f"{self.name}-{n_layers}L")


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    batch: int
    context: tuple  # ("fixed", C) or ("uniform", lo, hi)
    G: int  # drafted tokens available per sequence
    conf: tuple  # ("uniform", decay) or ("beta", a, b, decay); position index i starts at 1
    accept: str  # "greedy" | "sample" | "greedy+sample"
    temperature: float = 0.0
    cost: tuple = ("measured",)  # ("affine", a, c) -> cost[d] = a + c*d ; or measured
    seed: int = 0
    extra: dict = field(default_factory=dict)


TINY_F32 = ModelShape("tiny-f32", 2, 256, 4, 4, 64, 688, 1024, "f32")
LLAMA3_8B = ModelShape("llama3-8b", 32, 4096, 32, 8, 128, 14336, 128256, "bf16")
QWEN25_32B = ModelShape("qwen2.5-32b", 64, 5120, 40, 8, 128, 27648, 152064, "bf16")
LLAMA3_70B = ModelShape("llama3-70b", 80, 8192, 64, 8, 128, 28672, 128256, "bf16")
# Test-only shapes: small enough for the oracle, but exercising the bf16 kernels
# (grouped-query attention, head_dim 64 and 128, ragged tails).
TINY_BF16 = ModelShape("tiny-bf16-gqa", 2, 256, 4, 2, 64, 688, 1024, "bf16")
SMALL_BF16 = ModelShape("small-bf16-hd128", 2, 1024, 8, 2, 128, 2816, 4096, "bf16")

MODELS = {m.name: m for m in (TINY_F32, LLAMA3_8B, QWEN25_32B, LLAMA3_70B, TINY_BF16, SMALL_BF16)}

WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny-f32-b1-c128", TINY_F32, 1, ("fixed", 128), 16, ("uniform", 0.9), "greedy",
                 cost=("affine", 1.0, 0.05), seed=1),
        Workload("llama3-8b-b1-c2048", LLAMA3_8B, 1, ("fixed", 2048), 16, ("beta", 8.0, 2.0, 0.92), "greedy",
                 seed=2),
        Workload("llama3-8b-b8-ragged", LLAMA3_8B, 8, ("uniform", 1024, 8192), 32, ("beta", 6.0, 3.0, 0.9),
                 "greedy", seed=3),
        Workload("qwen2.5-32b-b4-sample", QWEN25_32B, 4, ("fixed", 4096), 16, ("beta", 8.0, 2.0, 0.92),
                 "sample", temperature=1.0, seed=4),
        Workload("llama3-70b-b4", LLAMA3_70B, 4, ("fixed", 8192), 32, ("beta", 5.0, 3.0, 0.9),
                 "greedy+sample", temperature=0.7, seed=5),
    )
}
