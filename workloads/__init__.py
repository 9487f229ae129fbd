"""Seeded synthetic inputs for the grammar-mask workloads.

This package only produces inputs: grammar texts, token vocabularies (byte
spellings), schema lexicons and prefix byte strings cut from random sentences
of the language.  It holds none of the masking arithmetic; both the CPU oracle
and the GPU path consume what it produces.
"""

from .configs import Workload, make_workload, grammar_text, GRAMMAR_DIR  # noqa: F401
