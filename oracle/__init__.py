"""fp64 CPU oracle for the LoRA-adapted linear layer -- TEST INFRASTRUCTURE.

Only the tests, the package smoke check and the benchmark's CPU-baseline leg
may import this package.  The product path (the HIP library and its Python
binding) never calls it and shares no code with it.

What it computes is the plain definition of the method, evaluated in float64
on the exact decoded bfloat16 inputs:

  Eq. 1 (Section 3, "Model Transfer API"):  output = W0 x + b0 + B A x,
  written row-major over m tokens with the conventional LoRA scale s = alpha/r
  (the configuration of Listing 3 carries LORA_R and LORA_ALPHA; with the
  defaults r = alpha = 16 the scale is 1, exactly Eq. 1):

      U  = X A^T                       [m, r]
      Y  = X W^T + s U B^T             [m, n]     (b0 = 0)

  and its chain-rule backward for the trainable A, B (W0 frozen, so no dW;
  Section 3 names B and A as the trainable weights), for an upstream dY:

      dU = s dY B                      [m, r]
      dX = dY W + dU A                 [m, k]
      dB = s dY^T U                    [n, r]
      dA = dU^T X                      [r, k]

LoRA dropout (Listing 3's LORA_DROPOUT) acts on the adapter's input only:
with a keep mask and rate p, D = keep * X / (1 - p), U = D A^T, and the
backward carries the mask into dX's LoRA term and into dA = dU^T D.

Grouped projections share one input X (query, key and value of an attention
block): each has its own W_g, A_g, B_g and output Y_g, and the input gradient is
the sum dX = sum_g (dY_g W_g + dU_g A_g).

The merge of the adapter into the frozen weight (Eq. 1's second form,
W0 x + B A x = (W0 + B A) x) is W + sign s B A, rounded once to bfloat16
(nearest-even) for the stored result.

The dropout keep mask the library can draw on the device (Philox4x64-10)
is evaluated from the generator's published definition in dropout_rng.py.

Each step is one numpy float64 matrix product; there is no blocking, fusion or
reordering beyond the definition.  The forward and backward are also written
as plain float64 loops over the index definitions in C (lora_loops.c, loaded
by loops.py; its shared library is built by loops.build()): pinned by the same
checks, it is the form the benchmark times as the CPU baseline.  Pins that tie this to the paper and to the
mathematics (merge identity, B = 0 and A = 0 invariants, finite differences,
a hand-worked example, brute-force loops, closed forms) live in
tests/test_oracle_pins.py.
"""
from .lora_oracle import (bf16_bits_to_f64, lora_scale, lora_rank_activation, lora_forward,
                          lora_backward, lora_forward_rows, lora_backward_rows, f64_to_bf16_bits,
                          f64_to_bf16_rne, lora_merged_weight, lora_merge_bf16, dropout_keep,
                          dropped_input, lora_forward_dropout, lora_backward_dropout,
                          lora_group_forward, lora_group_backward)
from .dropout_rng import philox4x64_10, keep_threshold, dropout_keep_philox

__all__ = ["bf16_bits_to_f64", "lora_scale", "lora_rank_activation", "lora_forward",
           "lora_backward", "lora_forward_rows", "lora_backward_rows", "f64_to_bf16_bits",
           "f64_to_bf16_rne", "lora_merged_weight", "lora_merge_bf16", "dropout_keep",
           "dropped_input", "lora_forward_dropout", "lora_backward_dropout",
           "lora_group_forward", "lora_group_backward", "philox4x64_10", "keep_threshold",
           "dropout_keep_philox"]
