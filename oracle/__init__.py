"""CPU oracle for the structured-dropout LSTM training step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports this package:
only the tests, the smoke check and the CPU-baseline leg of the benchmark do.
It shares no code with the HIP implementation.

Contents
  philox  -- Philox4x64-10 counter-based generator (Salmon et al., SC'11),
             written from that paper's definition.
  masks   -- Case-III structured dropout masks (Sec. 3.1): one keep/drop bit
             per neuron and time step, shared by every row of the batch.
  lstm    -- dense float64 LSTM forward (Eq. 1-6) with the masks applied as
             elementwise multipliers, and back-propagation through time
             (Eq. 7-11) written out by hand.
  embedding -- the embedding-table gradient of a language model's input:
             the layer-0 input gradient rows summed by token id.
  head    -- the output head: pre-FC structured output dropout, the FC
             (vocabulary projection) layer and the softmax cross-entropy
             loss, forward and backward.
  case1   -- the Case-I ("NR+Random") comparator: per-element input
             dropout on every layer, run dense.
"""
from . import philox, masks, lstm, embedding, head, case1  # noqa: F401
