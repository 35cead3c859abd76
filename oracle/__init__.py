"""CPU oracle for the decode-step Attention/FFN operators.

TEST INFRASTRUCTURE ONLY. Nothing on the product path imports this package:
only the tests, the smoke check and the benchmark's CPU-baseline leg may call
it. It shares no code with the HIP library; both sides receive the same inputs
from the seeded generator and nothing else.

Every function is the plain mathematical definition written out in float64
with PyTorch CPU ops (a matmul, an exp, a sort are the only library steps).
There is no splitting, fusion or reordering beyond the definition. bf16 inputs
are widened exactly; nothing is rounded on the way; results are float64.

The paper (AFlex, "Energy-Efficient LLM Serving via Disaggregated
Attention-FFN and Flexible Frequency Scaling") names the operators it
disaggregates -- decode Attention over the growing KV cache and the FFN of a
dense model (Qwen3-32B) and of an MoE model (Mixtral-8x7B) (section 1,
section 2, section 6.1) -- but prints no formula for them. The definitions
below are the standard ones of those architectures; every reading taken where
the paper is silent is listed in the module that takes it.

Pinned by the ``-m "not gpu"`` tests in ``tests/test_oracle_*.py`` (closed
forms, invariants, brute force, independent library routines). No function
here is "parity unpinned".
"""
from .attention import attention_decode, attention_weights, gather_sequence  # noqa: F401
from .ffn import silu, swiglu_ffn  # noqa: F401
from .moe import route_topk, routing_tables, moe_ffn  # noqa: F401
from .pipeline import af_decode_layer_steps, af_layer_steps  # noqa: F401
from .block import kv_append, kv_write, linear, moe_block, rmsnorm  # noqa: F401
from .prefill import attention_prefill  # noqa: F401
