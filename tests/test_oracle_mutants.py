"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pin suite catches every one of them.

Each mutant is a one-place textual change of ``oracle/rc_oracle.c``: a wrong
constant, shift, index, operand, operator, order or chaining rule.  The copy
is compiled with gcc into a temporary library; the real oracle is untouched.
"""
import os
import subprocess

import pytest

import oracle
import oracle_pins as P

MUTANTS = {
    "fmix_const": ("h *= 0x85EBCA6Bu;", "h *= 0x85EBCA6Du;"),
    "fmix_shift13": ("h ^= h >> 13;", "h ^= h >> 15;"),
    "fmix_last_shift_dropped": ("    h ^= h >> 16;\n    return h;", "    return h;"),
    "rotr_not_rotl": ("return (x << k) | (x >> (32u - k));", "return (x >> k) | (x << (32u - k));"),
    "rot_mod_dropped": ("k = k % 32u;", "k = k % 33u;"),
    "route_cdf_strict": ("if (route_cdf[k] <= o)", "if (route_cdf[k] < o)"),
    "route_cdf_short": ("for (k = 0u; k + 1u < n_routes; ++k)", "for (k = 1u; k + 1u < n_routes; ++k)"),
    "route_mod_off": ("return o % n_routes;", "return (o + 1u) % n_routes;"),
    "decide_mask": ("return (h & 0xFFFFu) < thr ? 1u : 0u;", "return (h & 0x7FFFu) < thr ? 1u : 0u;"),
    "decide_le": ("return (h & 0xFFFFu) < thr ? 1u : 0u;", "return (h & 0xFFFFu) <= thr ? 1u : 0u;"),
    "decide_high_half": ("return (h & 0xFFFFu) < thr ? 1u : 0u;", "return (h >> 16) < thr ? 1u : 0u;"),
    "decide_no_step": ("rc_oracle_fmix32(s0 ^ o ^ step);", "rc_oracle_fmix32(s0 ^ o);"),
    "decide_no_outcome": ("rc_oracle_fmix32(s0 ^ o ^ step);", "rc_oracle_fmix32(s0 ^ step);"),
    "mask_no_wplus1": ("* (w + 1u));", "* w);"),
    "mask_mod8": ("(w % 16u)", "(w % 8u)"),
    "mask_add_not_xor": ("return x ^ (table[r * 16u + (w % 16u)] * (w + 1u));",
                         "return x + (table[r * 16u + (w % 16u)] * (w + 1u));"),
    "rot_by_r": ("return rc_oracle_rotl(x, r + 1u) + o;", "return rc_oracle_rotl(x, r) + o;"),
    "rot_xor_outcome": ("return rc_oracle_rotl(x, r + 1u) + o;", "return rc_oracle_rotl(x, r + 1u) ^ o;"),
    "branches_swapped": ("    if (d)\n        return x ^", "    if (!d)\n        return x ^"),
    "decide_on_word1": ("taken[s - b] = rc_oracle_decide(state[s], o, step, decide_thr);",
                        "taken[s - b] = rc_oracle_decide(state[ld + s], o, step, decide_thr);"),
    "step_not_advanced": ("uint32_t step = step0 + t;", "uint32_t step = step0;"),
    "not_taken_first": ("next_taken = b;\n            next_not = b + n1;",
                        "next_not = b;\n            next_taken = b + (e - b - n1);"),
    "tool_column_swapped": ("eff_tool[slice + slot] = table[r * 16u + d] % 8u;",
                            "eff_tool[slice + slot] = table[r * 16u + (1u - d)] % 8u;"),
    "tool_mod16": ("eff_tool[slice + slot] = table[r * 16u + d] % 8u;",
                   "eff_tool[slice + slot] = table[r * 16u + d] % 16u;"),
    "payload_shifted": ("state[(size_t)q * ld + s];", "state[(size_t)(q + 1u) * ld + s];"),
    "chain_raw_word": ("outcome[s] = rc_oracle_fmix32(state[s]);", "outcome[s] = state[s];"),
    "chain_not_updated": ("outcome[s] = rc_oracle_fmix32(state[s]);", "(void)0;"),
    "count_not_taken": ("n_taken[(size_t)t * n_cohorts + c] = n1;",
                        "n_taken[(size_t)t * n_cohorts + c] = (e - b) - n1;"),
    "sid_relative": ("eff_sid[slice + slot] = s;", "eff_sid[slice + slot] = s - b;"),
    "slice_unshifted": ("size_t slice = (size_t)t * ld;", "size_t slice = 0;"),
    "floor_bit_shifted": ("return (bits[(size_t)t * dwords + s / 32u] >> (s % 32u)) & 1u;",
                          "return (bits[(size_t)t * dwords + s / 32u] >> ((s + 1u) % 32u)) & 1u;"),
    "floor_row_stride": ("return (bits[(size_t)t * dwords + s / 32u] >> (s % 32u)) & 1u;",
                         "return (bits[(size_t)t * (dwords - 1u) + s / 32u] >> (s % 32u)) & 1u;"),
    "floor_dwords_floor": ("const uint32_t dwords = (ld + 31u) / 32u;", "const uint32_t dwords = ld / 32u + 1u;"),
    "floor_inverted": ("taken[s - b] = bit_of(forced, dwords, t, s);",
                       "taken[s - b] = 1u - bit_of(forced, dwords, t, s);"),
    "floor_ignored": ("        if (forced)\n", "        if (0)\n"),
    "record_step_zero": ("uint32_t *word = &record[(size_t)t * dwords + s / 32u];",
                         "uint32_t *word = &record[s / 32u];"),
}


def _pins_all_pass(orc):
    for pin in P.QUICK_PINS:
        pin(orc)
    P.pin_brute_force_cohorts(orc)
    P.pin_brute_force_tiny(orc, quick=True)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) >= 1, "mutation anchor not found: %s" % name
    mutated = src.replace(old, new, 1)
    path = tmp_path / ("mut_%s.c" % name)
    path.write_text(mutated)
    lib = str(tmp_path / ("libmut_%s.so" % name))
    oracle.build(force=True, src=str(path), out=lib)
    orc = oracle.Oracle(lib)
    with pytest.raises(AssertionError):
        _pins_all_pass(orc)


def test_unmutated_copy_passes(tmp_path):
    path = tmp_path / "copy.c"
    path.write_text(open(oracle.SRC).read())
    lib = str(tmp_path / "libcopy.so")
    oracle.build(force=True, src=str(path), out=lib)
    _pins_all_pass(oracle.Oracle(lib))
