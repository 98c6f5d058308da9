"""Seeded synthetic inputs shared by the CPU oracle and the GPU library.

Input description and generation only: loop nests, dependency triples, trip
tables and tensors.  No synchronization arithmetic lives here."""
from .program import *  # noqa: F401,F403
from .configs import *  # noqa: F401,F403
