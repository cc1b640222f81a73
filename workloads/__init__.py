"""Seeded synthetic workloads for the expand / batch / gather path.

This package only draws inputs: child counts, record lengths, terminal
states, ready orders and record bytes.  It holds no step of the method
itself; both the CPU oracle and the HIP library are fed from it.
"""
from .gen import *  # noqa: F401,F403
