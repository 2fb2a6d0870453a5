"""fp64 CPU oracle for one MoE layer's forward and backward (FlowMoE, Sec. 2.1).

TEST INFRASTRUCTURE ONLY. Only the test-suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path never
does. It shares no code with the HIP implementation: it is plain numpy in
float64, written from the paper's statement of the MoE layer, one function per
step, with no blocking, fusion or reordering beyond the definitions.

Pins (what each function is checked against, in tests/test_oracle_pins.py):
  capacity        exact rational arithmetic; hand-worked integer cases
  gate_logits     library matmul; all-zero token gives all-equal logits
  topk_select     brute-force over all k-subsets (tiny E); closed form
                  sum_j w = 1 and w == 1 for k = 1; renormalised full softmax
  route           brute-force O((T*k)^2) position count; invariants
                  (counts <= C, bijection, C = 0 / C >= T*k special cases)
  dispatch        exact copy (bitwise)
  expert_ffn(+bwd) dense torch-fp64 autograd formulation; central finite
                  differences; closed-form derivatives of GELU and SiLU
  expert_bias_grads  the same autograd formulation and finite differences
                  with biased experts; zero weights give y = b2 per kept
                  assignment (closed form)
  combine(+bwd)   identity experts give (sum of kept w) * x; k = E with no
                  drops equals the dense softmax mixture of experts
  gate_bwd        torch autograd of the masked dense formulation; finite
                  differences at locally constant routing
  layer (chunked) concatenation of per-chunk calls; with no drops the weight
                  gradients equal the unchunked ones (microbatch equivalence,
                  App. H, Eqs. 19-23)
  attention(+bwd), mha_fwd(+bwd)
                  (attention of AT_r) torch's fp64 scaled_dot_product_attention
                  and its autograd gradients; central finite differences;
                  closed forms: W^Q = 0 gives uniform weights (the mean, or
                  for causal attention the prefix mean, of V) and
                  lse = log(number of visible tokens); one-token sequences
                  give I W^V W^O; non-causal attention is equivariant under
                  a permutation of a sequence's tokens
No function here is pinned to values printed in the paper: the paper prints
no numeric output of an MoE layer.
"""
from .moe_ref import (  # noqa: F401
    capacity, rows_capacity, gate_logits, topk_select, route, dispatch,
    expert_ffn, combine, combine_bwd, expert_ffn_bwd, expert_bias_grads, dispatch_bwd, gate_bwd,
    gelu, gelu_grad, silu, silu_grad, layer_chunk, layer_fwd_bwd,
)
from .mha_ref import attention, attention_bwd, mha_fwd, mha_bwd  # noqa: F401
