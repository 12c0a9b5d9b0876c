"""CPU oracle for the target model's tree-verification step (Dovetail,
arXiv 2412.18934, Section 3.1 "CPU/GPU Heterogeneous Architecture").

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library: it takes plain numpy arrays (weights, cached keys/values, token ids,
tree parents) and evaluates the definition directly, in float64 unless asked
for another dtype.

Pinned (see ``tests/test_oracle_*.py``): every function here is checked against
something other than itself: an independent Llama implementation from the
``transformers`` library, ``torch.nn.functional.scaled_dot_product_attention``,
sequential decoding, per-path decoding, brute-force acceptance, greedy-decoding
losslessness, hand-derived closed forms and, for sampled acceptance, the
distribution it must reproduce (Monte Carlo) and its greedy limit.
"""
from .verify import (  # noqa: F401
    OracleModel, TreeInfo, tree_info, round_cache, bf16_to_f64, rmsnorm, rope,
    attention_node, forward_tree, argmax_lowest, greedy_accept, verify_step, commit,
    prefill, greedy_decode, softmax_t, sample_inverse_cdf, accept_sampled, dequantize_rows,
)
