"""CPU oracle for one Blockwise Parallel Transformer (BPT) layer — TEST INFRASTRUCTURE.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package. The HIP library never calls it, shares no code with it
and has no fallback to it.

Contents
--------
``layer``      The plain, unblocked definition in float64: pre-LayerNorm GPT
               block with exact softmax attention (paper, Section 2, eq. 1)
               and an exact-erf GELU feed-forward network (Section 2, eq. 2,
               with GELU in place of ReLU), with residuals as in Section 3.
               It materialises the full SxS attention matrix per (batch, head)
               and the full SxF FFN intermediate. Forward and backward (the
               backward is the chain rule written out by hand).
``blockwise``  Algorithm 1 of the paper in float64: for each query block,
               online-softmax attention over key/value blocks with running
               max and sum (the carry update of Section 3, Fig. 3), then the
               FFN and residual on that query block. Used to pin the oracle's
               "results do not depend on Bq/Bkv" invariant.
``rows``       The plain definition restricted to a set of query rows: exact
               for every output row it returns, and for every gradient when
               the upstream gradient is zero outside those rows. Used for
               sampled-output parity at full workload sizes.
``bf16_model`` The plain definition with every matrix-multiply operand rounded
               to bfloat16: how far any bf16-operand implementation lands
               from the exact result on a given input (tolerance floor).
``bf16_rows``  ``bf16_model`` restricted to selected query rows, like ``rows``
               (the tolerance floor at full workload sizes).
``xent``       Cross-entropy of a language-model head (Section 3's remark that
               the blockwise scheme applies to the final loss): the plain,
               unblocked logits h W, log-sum-exp, mean token loss and its
               gradients dh, dW.
``dropout``    Masks of the layer's two residual-branch dropouts (the mask the
               paper's memory accounting keeps for the output projection and
               for the FFN output), from Philox4x32-10 written from its
               published definition; ``layer`` applies them when its rate > 0.
``gpt``        A GPT training step (the models of Section 5): token and
               position embedding, L layers of ``layer``, final LayerNorm,
               the ``xent`` head, and an AdamW update.

Every function is pinned by ``tests/test_oracle_*.py`` against brute-force
loops, closed forms, invariants, finite differences and an independent
autograd implementation.
"""
from .layer import (LayerParams, gelu, gelu_grad, layer_norm_fwd, layer_norm_bwd,
                    attention_head, layer_fwd, layer_bwd, params_from_inputs)
from .blockwise import blockwise_attention_head, blockwise_layer_fwd
from .rows import rows_layer_fwd_bwd

__all__ = [
    "LayerParams", "gelu", "gelu_grad", "layer_norm_fwd", "layer_norm_bwd", "attention_head",
    "layer_fwd", "layer_bwd", "params_from_inputs", "blockwise_attention_head",
    "blockwise_layer_fwd", "rows_layer_fwd_bwd",
]
