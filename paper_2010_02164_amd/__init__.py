"""streambeam: streaming variable-width batched beam search on MI355X (gfx950).

The search step of Var-Stream (Yang et al., EMNLP 2020, Sec. 3 / Alg. 1) and
its settings Fixed and Var-Batch, as hand-written HIP kernels behind a C ABI
(include/streambeam.h). This package holds the ctypes binding and the build
script; PyTorch only provides device memory and streams.
"""
from .decoder import (Decoder, Hypothesis, decoder_for_workload, group_by_input, inputs_to_device,
                      weights_to_device)

__all__ = ["Decoder", "Hypothesis", "decoder_for_workload", "group_by_input", "inputs_to_device",
           "weights_to_device"]
