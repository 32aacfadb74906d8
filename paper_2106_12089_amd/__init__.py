"""Structured-dropout LSTM training step (forward unroll + BPTT) for AMD
MI355X: hand-written HIP kernels for gfx950 behind a C ABI
(include/lstm_sd.h), with a ctypes binding.

  binding  -- the C ABI, one Python function per entry point
  session  -- device buffers of one workload, allocated with torch
  build    -- hipcc build of liblstm_sd.so
"""
__all__ = ["binding", "session", "build"]
