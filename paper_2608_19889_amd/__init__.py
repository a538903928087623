"""MI355X (gfx950) decoder forward pass: prefill and greedy decode for
Llama/Qwen-style models behind the C ABI of ``include/axon.h``."""
from .axon import Model, AxonError, make_config, make_weights, lib  # noqa: F401
