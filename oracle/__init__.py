"""CPU oracle for the MoE gate / layout-transform hot path (HetuMoE, arXiv 2203.14685).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously correct
reference written from the paper.  Only the test-suite, the smoke check and the
CPU-baseline leg of the benchmark may import it.  The product library never
calls it, and it shares no code with the HIP path: nothing here imports the
product package and the product package imports nothing from here.

Arithmetic is fp64 on exactly decoded inputs.  bf16 tensors are held as uint16
bit patterns (see :mod:`oracle.bf16`).  Every function cites the passage of the
paper it follows:

* Algorithm 1 (one training step of an MoE layer), steps 1, 2 and 6, and the
  numbered list of Sec. 2 that describes them;
* Eq. 1 (Sec. 3.1, Top1/Top2/Topk gate) and the capacity-factor sentence next
  to it;
* Sec. 3.1 kTop1 (expert prototyping) and Hash Layer paragraphs;
* Sec. 3.2, on the gate (top-k over a (num_tokens, num_experts) input) and
  on the layout transform (tokens of one expert made contiguous);
* the gradient of Eq. 1 that end-to-end training of the layer (Sec. 2) needs,
  and a load-balancing loss (reading R16) for the gates of Sec. 3.1;
* the BASE layer's balanced assignment (Sec. 3.1, the equation of the BASE
  Layer paragraph).

Where the paper is silent the oracle takes one fixed reading, numbered R1,
R2, ...; each is stated at the function that depends on it.

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
against hand-computed cases, brute force, closed forms, library routines or a
published test vector.  The choice of hash (SplitMix64) and of the capacity
formula are readings, not values the paper fixes; the paper prints no worked
example for any step.
"""

from .bf16 import bf16_to_f64, f64_to_bf16, decode, encode
from .gate import (
    GATE_TOPK,
    GATE_KTOP1,
    GATE_HASH,
    GATE_HTOPK,
    capacity,
    logits,
    select,
    gate_weights,
    splitmix64_output,
    hash_ids,
    noisy_logits_f32,
    balanced_hash_table,
    table_hash_ids,
    assign_slots,
    gate,
)
from .layout import dispatch, combine, dispatch_bwd, combine_bwd
from .gate_bwd import gate_dlogits, aux_loss, gate_input_grads
from .base import base_assign, base_weights

__all__ = [
    "bf16_to_f64", "f64_to_bf16", "decode", "encode",
    "GATE_TOPK", "GATE_KTOP1", "GATE_HASH", "GATE_HTOPK", "capacity", "logits", "select",
    "gate_weights", "splitmix64_output", "hash_ids", "noisy_logits_f32", "balanced_hash_table",
    "table_hash_ids", "assign_slots", "gate",
    "dispatch", "combine", "dispatch_bwd", "combine_bwd",
    "gate_dlogits", "aux_loss", "gate_input_grads", "base_assign", "base_weights",
]
