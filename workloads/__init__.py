"""Seeded synthetic inputs shared by the HIP path's tests/bench and the oracle's tests."""
from .gen import *  # noqa: F401,F403
