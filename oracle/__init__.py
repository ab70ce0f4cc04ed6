"""CPU fp64 oracle of the MeBP checkpointed LoRA training step.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import it. The product path (the C-ABI library and its
Python binding) never imports, calls or links anything here, and this package imports
nothing from the product path. See ``mebp_oracle`` for what is computed and why.
"""
from .mebp_oracle import *  # noqa: F401,F403
from . import mebp_oracle  # noqa: F401
