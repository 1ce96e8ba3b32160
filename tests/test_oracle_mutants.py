"""Plant plausible mistakes in a copy of the oracle and check that the pins catch each one.

Every mutant is a one-line edit of ``oracle/attention.py`` (dropped term,
wrong sign, wrong index, wrong operand, off-by-one mask). Mistakes are planted
only in this in-memory copy, on the CPU.
"""

import os
import types

import pytest

from tests import oracle_pins as pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "attention.py")

MUTANTS = {
    "dropped_normalisation": ("o = (w @ v) / z[:, None]\n    lse = m[:, 0] + np.log(z)\n    return o, lse\n\n\ndef attend_range",
                              "o = (w @ v)\n    lse = m[:, 0] + np.log(z)\n    return o, lse\n\n\ndef attend_range"),
    "dropped_lse_term": ("lse = m[:, 0] + np.log(z)\n    return o, lse\n\n\ndef attend_range",
                         "lse = m[:, 0]\n    return o, lse\n\n\ndef attend_range"),
    "dropped_scale": ("s = np.float64(np.float32(scale)) * (q @ k.T)          # [R, L]",
                      "s = (q @ k.T)          # [R, L]"),
    "value_operand_is_key": ("o = (w @ v) / z[:, None]\n    lse = m[:, 0] + np.log(z)\n    return o, lse\n\n\ndef attend_range",
                             "o = (w @ k) / z[:, None]\n    lse = m[:, 0] + np.log(z)\n    return o, lse\n\n\ndef attend_range"),
    "causal_off_by_one": ("t[None, :] <= limits[:, None]", "t[None, :] < limits[:, None] + (limits[:, None] == 0)"),
    "extend_prefix_off_by_one": ("prefix = kv - n\n", "prefix = kv - n - 1\n"),
    "extend_row_order_head_major": ("limits = np.repeat(prefix + np.arange(i0, i1), r)",
                                    "limits = np.tile(prefix + np.arange(i0, i1), r)"),
    "page_index_modulo": ("page = int(block_row[t // page_size])", "page = int(block_row[(t // page_size) % 2])"),
    "kv_head_ignored": ("out[t:t + take] = kv_to_f64(pages[page, :take, g, :])",
                        "out[t:t + take] = kv_to_f64(pages[page, :take, 0, :])"),
    "fp8_exponent_bias": ("(e - 7).astype(np.int64)", "(e - 8).astype(np.int64)"),
    "fp8_subnormal_exponent": ("sub = np.ldexp(m / 8.0, -6)", "sub = np.ldexp(m / 8.0, -7)"),
    "fp8_sign_dropped": ("return sign * val", "return val"),
    "fp8_scale_ignored": ("out *= np.float64(head_scale[g])", "out *= 1.0"),
    "fp8_scale_wrong_head": ("out *= np.float64(head_scale[g])", "out *= np.float64(head_scale[0])"),
    "gqa_modulo_mapping": ("o, l = attend(qf[b, g * r:(g + 1) * r], k, v, scale)\n            out[b, g * r:(g + 1) * r] = o\n            lse[b, g * r:(g + 1) * r] = l",
                           "o, l = attend(qf[b, g::hkv], k, v, scale)\n            out[b, g::hkv] = o\n            lse[b, g::hkv] = l"),
    "merge_weight_sign": ("w = np.exp(ls - m)", "w = np.exp(m - ls)"),
    "merge_unnormalised": ("out[n, hh] = (w[:, None] * o_parts[n, :s_count, hh]).sum(axis=0) / z",
                           "out[n, hh] = (w[:, None] * o_parts[n, :s_count, hh]).sum(axis=0)"),
    "tail_token_dropped": ("take = min(page_size, length - t)\n        out[t:t + take]",
                           "take = min(page_size, length - t)\n        take = max(1, take - (take < page_size))\n        out[t:t + take]"),
}


def _mutant_module(name):
    old, new = MUTANTS[name]
    with open(SRC) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    mod = types.ModuleType(f"oracle_mutant_{name}")
    exec(compile(src.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    mod = _mutant_module(name)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except Exception as exc:  # AssertionError, or a shape error the mistake causes
            caught.append((pin.__name__, type(exc).__name__))
    assert caught, f"no pin detects mutant {name}"
