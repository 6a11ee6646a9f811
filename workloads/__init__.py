"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark."""
from .gen import *  # noqa: F401,F403
from .gen import random_bf16, random_scores, random_selection, random_selection_h  # noqa: F401
