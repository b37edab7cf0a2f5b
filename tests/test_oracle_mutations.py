"""Plant plausible mistakes in a copy of the attention oracle; the pins must catch each one.

Every mutant is a textual edit of the oracle's own source, executed on the CPU
as a throw-away module.  A mutant that passes every pin would mean the pins
cannot tell that mistake from the definition.
"""
import inspect
import types

import pytest

from oracle import attention as oa

from _attention_pins import ALL_CHECKS, check_rows_brute_force

MUTANTS = {
    "interleaved GQA heads": ("kh = h // g", "kh = h % hkv"),
    "top-left causal alignment": ("pos0 = n - q_len", "pos0 = 0"),
    "rows at the wrong positions": ("pos0 + row_idx)", "row_idx)"),
    "mask one key short": ("<= pos[:, None]", "< pos[:, None]"),
    "no causal mask": ("s = torch.where(visible, s, -math.inf)", "s = s"),
    "missing softmax scale": ("s = scale * (", "s = ("),
    "no max subtraction": ("w = torch.exp(s - m)", "w = torch.exp(s)"),
    "keys used as values": ("(w @ v_heads[kh])", "(w @ k_heads[kh])"),
    "missing normalisation": ("/ w.sum(dim=1, keepdim=True)", ""),
    "query head for key head": ("@ k_heads[kh].T", "@ k_heads[h % hkv].T"),
}


def _mutant(old, new):
    src = inspect.getsource(oa)
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


def _checks(mod):
    return [(c, mod.attention_sequence) for c in ALL_CHECKS] + \
           [(check_rows_brute_force, mod.attention_rows)]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    mod = _mutant(*MUTANTS[name])
    failures = 0
    for check, impl in _checks(mod):
        try:
            check(impl)
        except Exception:  # assertion, overflow, shape error: all count as caught
            failures += 1
    assert failures >= 1, f"mutant '{name}' passed every pin"


def test_unmutated_source_passes_every_pin():
    mod = _mutant("kh = h // g", "kh = h // g")
    for check, impl in _checks(mod):
        check(impl)
