"""Seeded synthetic optimizer-step windows (routing-replay stand-ins).

This module only draws inputs: per-sample lengths and per-sample, per-layer
logical-expert routing counts, plus the planner knobs that go with each
window.  It holds none of the planner's arithmetic, so both the CPU oracle and
the HIP path may consume what it produces.
"""
from .windows import (WINDOWS, Window, make_window, make_tiny_random,
                      anneal_temperatures, window_problem)

__all__ = ["WINDOWS", "Window", "make_window", "make_tiny_random",
           "anneal_temperatures", "window_problem"]
