"""Backbone shapes the library is exercised on (LLaDA-8B and Dream-7B layouts, plus a tiny
one).  The one table of these shapes lives with the seeded inputs (seeded_inputs/spec.py);
any object with the same fields configures a model (api.model_cfg_from)."""
from seeded_inputs.spec import DREAM_7B, LLADA_8B, TINY  # noqa: F401
from seeded_inputs.spec import ModelSpec as ModelConfig  # noqa: F401
