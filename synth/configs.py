"""Model shapes and the synthetic workloads the tests and the benchmark run.

Shapes follow Llama-3 (GQA with contiguous query-head groups, SwiGLU FFN, RMSNorm, rotary
embeddings with base 500000). Weights are seeded N(0, 0.02) draws, not trained checkpoints.
"""
from dataclasses import dataclass, replace

__all__ = ["Shape", "Workload", "TINY", "LLAMA3_8B", "LLAMA3_70B", "WORKLOADS", "tiny_shape"]


@dataclass(frozen=True)
class Shape:
    n_layers: int
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    d_ffn: int
    vocab: int = 0          # 0: no LM head (a bare layer stack)
    rope_theta: float = 500000.0
    rms_eps: float = 1e-5

    @property
    def group_size(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def with_layers(self, n: int, vocab: int | None = None) -> "Shape":
        return replace(self, n_layers=n, vocab=self.vocab if vocab is None else vocab)


# Tiny single layer: hidden 512, 8 query / 2 KV heads, head_dim 64, SwiGLU 1536.
TINY = Shape(n_layers=1, d_model=512, n_q_heads=8, n_kv_heads=2, head_dim=64, d_ffn=1536)
# Llama-3-8B geometry: hidden 4096, 32/8 heads, head_dim 128, SwiGLU 14336, vocab 128256.
LLAMA3_8B = Shape(n_layers=32, d_model=4096, n_q_heads=32, n_kv_heads=8, head_dim=128,
                  d_ffn=14336, vocab=128256)
# Llama-3-70B geometry: hidden 8192, 64/8 heads, head_dim 128, SwiGLU 28672, vocab 128256.
LLAMA3_70B = Shape(n_layers=80, d_model=8192, n_q_heads=64, n_kv_heads=8, head_dim=128,
                   d_ffn=28672, vocab=128256)


def tiny_shape(d=16, hq=4, hkv=2, dh=4, f=8, layers=1, vocab=0, theta=500000.0):
    """Very small shapes for brute-force and exhaustive checks."""
    return Shape(n_layers=layers, d_model=d, n_q_heads=hq, n_kv_heads=hkv, head_dim=dh,
                 d_ffn=f, vocab=vocab, rope_theta=theta)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: Shape
    batch: int
    pos: int            # prior positions in the cache (decode writes at index pos)
    prefill_tokens: int = 0
    mask_seeds: tuple = (1,)
    include_dense: bool = True
    kind: str = "decode"    # "decode" (decode / prefill steps), "mask" (mask construction),
                            # "request" (prefill of prefill_tokens, then n_new greedy decode steps),
                            # "router" (routing of user turns; the stack gives the path latencies),
                            # "shared" (batch-1 decode from the shared groupwise store)
    n_new: int = 0
    granule: int = 1024     # SwiGLU channels per candidate group (mask construction)


WORKLOADS = {
    # one tiny layer, batch 1, 128 prior positions; 6/8 heads and 1024/1536 channels kept
    "tiny_layer": Workload("tiny_layer", TINY, batch=1, pos=128, mask_seeds=(1,)),
    # one Llama-3-8B-shaped layer, batch 1, 2048 prior positions, 43%-reduction masks
    "llama3_8b_layer": Workload("llama3_8b_layer", LLAMA3_8B.with_layers(1, vocab=0), batch=1,
                                pos=2048, mask_seeds=(1, 2, 3, 4, 5)),
    # 32-layer Llama-3-8B-shaped stack with BF16 LM head, 4096 prior positions
    "llama3_8b_stack": Workload("llama3_8b_stack", LLAMA3_8B, batch=1, pos=4096,
                                mask_seeds=(1, 2, 3, 4, 5)),
    # 80-layer Llama-3-70B-shaped stack with BF16 LM head, 4096 prior positions
    "llama3_70b_stack": Workload("llama3_70b_stack", LLAMA3_70B, batch=1, pos=4096,
                                 mask_seeds=(1,)),
    # one 8B-shaped layer: 512-token prefill from an empty cache
    "llama3_8b_prefill512": Workload("llama3_8b_prefill512", LLAMA3_8B.with_layers(1, vocab=0),
                                     batch=1, pos=0, prefill_tokens=512, mask_seeds=(1,)),
    # one 8B-shaped layer: the request's 2048-token prefill from an empty cache
    "llama3_8b_prefill2048": Workload("llama3_8b_prefill2048", LLAMA3_8B.with_layers(1, vocab=0),
                                      batch=1, pos=0, prefill_tokens=2048, mask_seeds=(1,)),
    # one 70B-shaped layer: the request's 2048-token prefill from an empty cache
    "llama3_70b_prefill2048": Workload("llama3_70b_prefill2048", LLAMA3_70B.with_layers(1, vocab=0),
                                       batch=1, pos=0, prefill_tokens=2048, mask_seeds=(1,)),
    # the paper's timed request: 2048-token prompt, then 256 greedy decode steps, one plan
    "llama3_8b_request": Workload("llama3_8b_request", LLAMA3_8B, batch=1, pos=0,
                                  prefill_tokens=2048, kind="request", n_new=256),
    "llama3_70b_request": Workload("llama3_70b_request", LLAMA3_70B, batch=1, pos=0,
                                   prefill_tokens=2048, kind="request", n_new=256),
    # greedy mask construction over the 80-layer 70B candidate set (64 heads + 28 groups of
    # 1024 channels per layer, 7360 candidates) at the 0.57 active-FLOP target
    "llama3_70b_mask": Workload("llama3_70b_mask", LLAMA3_70B, batch=0, pos=0, kind="mask",
                                granule=1024),
    # the router (2048 hashed bins -> 256, MLP 512 / 256, 5 tasks) on 2048-token-sized prompts
    # and a mix of the five task families; the mixture latency uses the sparse and dense decode
    # of the 32-layer 8B stack at 4096 prior positions
    "router_llama3_8b": Workload("router_llama3_8b", LLAMA3_8B, batch=1, pos=4096,
                                 mask_seeds=(1,), kind="router"),
    # one 8B-shaped layer from the shared groupwise store (BF16 scales per 128 inputs), batch 1,
    # 2048 prior positions, seed-1 mask
    "llama3_8b_layer_shared": Workload("llama3_8b_layer_shared", LLAMA3_8B.with_layers(1, vocab=0),
                                       batch=1, pos=2048, mask_seeds=(1,), kind="shared"),
    # the 80-layer 70B-shaped stack from one shared groupwise store (plans own no weight bytes),
    # batch 1, 4096 prior positions: seed-1 mask and the dense plan
    "llama3_70b_stack_shared": Workload("llama3_70b_stack_shared", LLAMA3_70B, batch=1, pos=4096,
                                        mask_seeds=(1,), kind="shared"),
    # one 8B-shaped layer: batch-8 decode, every sequence at 8192 prior positions
    "llama3_8b_batch8": Workload("llama3_8b_batch8", LLAMA3_8B.with_layers(1, vocab=0),
                                 batch=8, pos=8192, mask_seeds=(1,)),
}
