"""o5: the OpenAI Five LSTM-PPO optimizer step on AMD MI355X (gfx950).

Modules:
  o5     -- ctypes binding of libo5.so (the C ABI declared in include/o5.h)
  step   -- one PPO optimizer step sequenced through the ABI on one stream
  synth  -- seeded synthetic inputs shaped like the paper's workloads
  build  -- hipcc build of libo5.so
"""
__all__ = ["o5", "step", "synth", "build"]
