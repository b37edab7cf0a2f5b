"""The proportional prefill-cap controller, Eq. 2 (Sec. 3.1), float64.

After a guarded cycle -- one in which at least one request was decoding and a
prefill shared the cycle -- the cap is rescaled by target over observed
latency, quantised down to a multiple of 128 tokens, and clamped:

    c_next = clamp(floor_128(c * T / L_obs), c_min, c_max)

A longer-than-target observation shrinks the next chunk, a shorter one grows
it (Sec. 3.1).  When no request is decoding the controller returns to
``c_initial`` and isolated prefill is not capped (Sec. 3.1; caps apply to
running chunked prefills and newly admitted prompts only while a decoder is
active, Sec. 3.2).  The evaluated constants are T = 80 ms, c_initial = 3072,
c_min = 1024, c_max = 6144 (Sec. 3.1).

``floor_128`` is read as ``128 * floor(x / 128)``; the paper's observability
example (3072 at 57.51 ms -> 4224) fixes floor rather than round or ceil.
"""
from __future__ import annotations

import math

UNCAPPED = -1


def floor_quantum(x: float, quantum: int = 128) -> int:
    return int(quantum * math.floor(x / quantum))


def next_cap(cap: int, target_ms: float, observed_ms: float, c_min: int, c_max: int,
             quantum: int = 128) -> int:
    """Eq. 2 for one update."""
    if not (math.isfinite(observed_ms) and observed_ms > 0.0):
        raise ValueError("observed latency must be finite and positive")
    x = cap * target_ms / observed_ms
    return min(max(floor_quantum(x, quantum), c_min), c_max)


class Controller:
    """Controller state with the guard and reset rules."""

    def __init__(self, target_ms: float, c_initial: int, c_min: int, c_max: int,
                 quantum: int = 128):
        if not (0 < c_min <= c_initial <= c_max) or quantum <= 0 or not target_ms > 0:
            raise ValueError("bad controller parameters")
        self.target_ms = float(target_ms)
        self.c_initial, self.c_min, self.c_max, self.quantum = c_initial, c_min, c_max, quantum
        self.cap = c_initial

    def step(self, num_decoding_next: int, last_was_guarded: bool, observed_ms: float) -> int:
        """Update after an executed cycle; return the next cap (UNCAPPED if no decoder)."""
        if last_was_guarded:
            self.cap = next_cap(self.cap, self.target_ms, observed_ms, self.c_min, self.c_max,
                                self.quantum)
        if num_decoding_next == 0:
            self.cap = self.c_initial
            return UNCAPPED
        return self.cap
