"""Plant plausible mistakes in a copy of the attention oracle; the pins must catch each one.

Every mutant is a textual edit of the oracle's own source, executed on the CPU
as a throw-away module.  A mutant that passes every pin would mean the pins
cannot tell that mistake from the definition.
"""
import inspect
import types

import pytest

from oracle import attention as oa

from _attention_pins import ALL_CHECKS

MUTANTS = {
    "interleaved GQA heads": ("kh = h // g", "kh = h % hkv"),
    "top-left causal alignment": ("pos0 = n - q_len", "pos0 = 0"),
    "mask one key short": ("<= positions[:, None]", "< positions[:, None]"),
    "no causal mask": ("s = np.where(visible, s, -np.inf)", "s = s"),
    "missing softmax scale": ("s = scale * (", "s = ("),
    "no max subtraction": ("w = np.exp(s - m)", "w = np.exp(s)"),
    "keys used as values": ("(w @ v[:, kh, :])", "(w @ k[:, kh, :])"),
    "missing normalisation": ("/ w.sum(axis=1, keepdims=True)", ""),
    "query head for key head": ("@ k[:, kh, :].T", "@ k[:, h % hkv, :].T"),
}


def _mutant(old, new):
    src = inspect.getsource(oa)
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod.attention_sequence


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    impl = _mutant(*MUTANTS[name])
    failures = 0
    for check in ALL_CHECKS:
        try:
            check(impl)
        except Exception:  # assertion, overflow, shape error: all count as caught
            failures += 1
    assert failures >= 1, f"mutant '{name}' passed every pin"


def test_unmutated_source_passes_every_pin():
    impl = _mutant("kh = h // g", "kh = h // g")
    for check in ALL_CHECKS:
        check(impl)
