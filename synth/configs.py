"""The five synthetic workloads: layer shapes, rank count, chunk, steps,
hyperparameters and gradient distributions.

Shapes are those of the models' decoder layers (one flat state segment per
layer, tensors concatenated in the order listed).  Values are synthetic: the
FP32 master is N(0, 0.02), moments start at zero, gradients are fresh
N(0, sigma) draws per step and rank, rounded to BF16.  The paper's workloads
train real Qwen3 / Qwen2.5 checkpoints on C4 (Evaluation, setup); those are
stood in for by these layer-shaped states.
"""
from dataclasses import dataclass, field
from typing import List, Tuple

NORM_TILE = 65536  # elements per norm partial


@dataclass(frozen=True)
class Segment:
    name: str
    tensors: Tuple[Tuple[str, Tuple[int, ...]], ...]

    @property
    def numel(self) -> int:
        n = 0
        for _, shape in self.tensors:
            k = 1
            for d in shape:
                k *= d
            n += k
        return n


@dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    mode: str                      # "device" or "streamed"
    segments: Tuple[Segment, ...]
    ranks: int
    chunk: int                     # elements per chunk
    steps: int
    sigma: float                   # gradient standard deviation
    outlier_p: float = 0.0         # probability that a gradient is scaled
    outlier_scale: float = 1.0
    master_sigma: float = 0.02
    lr: float = 1e-5
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.01
    max_grad_norm: float = 1.0

    @property
    def numel(self) -> int:
        return sum(s.numel for s in self.segments)

    def hparams(self, step: int) -> dict:
        return dict(lr=self.lr, beta1=self.beta1, beta2=self.beta2,
                    eps=self.eps, weight_decay=self.weight_decay,
                    max_grad_norm=self.max_grad_norm, step=step)


def decoder_layer(name: str, hidden: int, kv: int, ffn: int) -> Segment:
    """Attention q/k/v/o, MLP gate/up/down and two RMSNorm weight vectors."""
    return Segment(name, (
        ("q_proj", (hidden, hidden)),
        ("k_proj", (kv, hidden)),
        ("v_proj", (kv, hidden)),
        ("o_proj", (hidden, hidden)),
        ("gate_proj", (ffn, hidden)),
        ("up_proj", (ffn, hidden)),
        ("down_proj", (hidden, ffn)),
        ("input_layernorm", (hidden,)),
        ("post_attention_layernorm", (hidden,)),
    ))


QWEN3_8B_LAYER = decoder_layer("qwen3_8b_layer", 4096, 1024, 12288)
QWEN3_14B_LAYER = decoder_layer("qwen3_14b_layer", 5120, 1024, 17408)
QWEN25_72B_LAYER = decoder_layer("qwen2.5_72b_layer", 8192, 1024, 29568)
VOCAB_QWEN3 = 151936


def _qwen3_14b_full() -> Tuple[Segment, ...]:
    segs: List[Segment] = [Segment("embed_tokens", (("embed_tokens", (VOCAB_QWEN3, 5120)),))]
    for i in range(40):
        segs.append(Segment(f"layer{i}", QWEN3_14B_LAYER.tensors))
    segs.append(Segment("lm_head", (("lm_head", (VOCAB_QWEN3, 5120)),)))
    return tuple(segs)


WORKLOADS: Tuple[Workload, ...] = (
    Workload(0, "tiny_1024x1024_r2", "device",
             (Segment("W", (("W", (1024, 1024)),)),),
             ranks=2, chunk=1048576, steps=3, sigma=1e-3),
    Workload(1, "qwen3_8b_layer_r4_device", "device", (QWEN3_8B_LAYER,),
             ranks=4, chunk=16 * 1048576, steps=10, sigma=1e-3,
             outlier_p=0.01, outlier_scale=100.0),
    Workload(2, "qwen3_14b_layer_r4_streamed", "streamed", (QWEN3_14B_LAYER,),
             ranks=4, chunk=32 * 1048576, steps=5, sigma=1e-3),
    Workload(3, "qwen3_14b_full_r2_streamed", "streamed", _qwen3_14b_full(),
             ranks=2, chunk=32 * 1048576, steps=2, sigma=1e-3),
    Workload(4, "qwen2.5_72b_layer_r8_device", "device", (QWEN25_72B_LAYER,),
             ranks=8, chunk=64 * 1048576, steps=3, sigma=5e-4,
             weight_decay=0.1),
)


def workload(cid: int) -> Workload:
    return WORKLOADS[cid]
