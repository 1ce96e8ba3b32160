"""Plant plausible mistakes in a copy of the oracle and check that the pins catch each one.

Every mutant is a one-line edit of one file of the oracle (dropped term,
wrong sign, wrong index, wrong operand, off-by-one mask or position, wrong
rounding). The pins receive a whole copy of the oracle package carrying that
one edit, so every function they call exists. Mistakes are planted only in
this in-memory copy, on the CPU.
"""

import os
import sys
import types

import pytest

from tests import oracle_pins as pins

ORACLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")
MODULES = ("attention", "kv_append")       # in import order

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


APPEND_MUTANTS = {
    "append_position_off_by_one": ("t = int(kv_lens[b]) - n + i\n", "t = int(kv_lens[b]) - n + i - (i > 0)\n"),
    "append_v_rows_into_k": ("kp[page, t % page_size] = k_rows[q0 + i]", "kp[page, t % page_size] = v_rows[q0 + i]"),
    "encode_ties_away_from_zero": ("((d_hi == d_lo) & (hi % 2 == 0))", "(d_hi == d_lo)"),
    "encode_overflow_to_nan": ("code = np.where(nan, np.uint8(0x7F), code)",
                               "code = np.where(nan | (np.abs(x.ravel()) > 464), np.uint8(0x7F), code)"),
    "quantise_multiplies_by_scale": ("q = (x / s).astype(np.float32)", "q = (x * s).astype(np.float32)"),
    "quantise_via_reciprocal": ("q = (x / s).astype(np.float32)", "q = (x * (np.float32(1) / s)).astype(np.float32)"),
}
SITES = {**{k: ("attention", *v) for k, v in MUTANTS.items()}, **{k: ("kv_append", *v) for k, v in APPEND_MUTANTS.items()}}


def _mutant_oracle(name):
    """A copy of the oracle package with the one edit of mutant ``name``."""
    where, old, new = SITES[name]
    pkg_name = f"oracle_mutant_{name}"
    pkg = types.ModuleType(pkg_name)
    pkg.__path__ = []
    sys.modules[pkg_name] = pkg
    try:
        for mod_name in MODULES:
            with open(os.path.join(ORACLE, mod_name + ".py")) as f:
                src = f.read()
            if mod_name == where:
                assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
                src = src.replace(old, new)
            mod = types.ModuleType(f"{pkg_name}.{mod_name}")
            mod.__package__ = pkg_name
            sys.modules[mod.__name__] = mod
            exec(compile(src, f"<mutant {name}: {mod_name}>", "exec"), mod.__dict__)
            for k, v in mod.__dict__.items():
                if not k.startswith("_"):
                    setattr(pkg, k, v)
    finally:
        for k in [k for k in sys.modules if k == pkg_name or k.startswith(pkg_name + ".")]:
            del sys.modules[k]
    return pkg


def test_mutant_copies_are_complete():
    """Each mutant copy offers every public function of the oracle (so a pin cannot be
    'caught' by a missing attribute)."""
    import oracle

    want = {k for k in dir(oracle) if not k.startswith("_") and callable(getattr(oracle, k))}
    for name in (sorted(MUTANTS)[0], sorted(APPEND_MUTANTS)[0]):
        have = {k for k in dir(_mutant_oracle(name)) if callable(getattr(_mutant_oracle(name), k))}
        assert want <= have, want - have


@pytest.mark.parametrize("name", sorted(SITES))
def test_pins_catch_mutant(name):
    mod = _mutant_oracle(name)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except Exception as exc:  # AssertionError, or a shape error the mistake causes
            caught.append((pin.__name__, type(exc).__name__))
    assert caught, f"no pin detects mutant {name}"
    assert all(kind != "AttributeError" for _, kind in caught), caught
