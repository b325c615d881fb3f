"""The pins are strong enough: each planted mistake in a copy of the oracle fails one.

Every mutant is a plausible slip (an off-by-one, a dropped term, a wrong sign,
a reversed tie-break).  The mutated copy is compiled into a temporary
directory on the CPU; the real oracle is untouched.
"""
import inspect

import pytest

import test_oracle_pins as pins
from oracle import SRC_PATH, Oracle, build

MUTANTS = {
    "frontier_tie_by_insertion_order": (
        "while (p < *fs && f[p].key < key) ++p;",
        "while (p < *fs && (f[p].key >> 32) <= (key >> 32)) ++p;"),
    "frontier_keeps_L_minus_1": (
        "if (p >= L) return;", "if (p + 1 >= L) return;"),
    "beam_takes_W_plus_1": (
        "for (uint32_t i = 0; i < fs && nb < W; ++i)", "for (uint32_t i = 0; i < fs && nb <= W; ++i)"),
    "beam_only_scans_first_W": (
        "for (uint32_t i = 0; i < fs && nb < W; ++i)", "for (uint32_t i = 0; i < fs && i < W; ++i)"),
    "u8_distance_drops_last_dim": (
        "for (uint32_t d = 0; d < D; ++d) {\n        int64_t t",
        "for (uint32_t d = 0; d + 1 < D; ++d) {\n        int64_t t"),
    "f32_distance_wrong_sign": (
        "float t = a[d] - b[d];", "float t = a[d] + b[d];"),
    "f32_distance_fused": (
        "float sq = t * t;\n        acc = acc + sq;", "acc = __builtin_fmaf(t, t, acc);"),
    "medoid_truncates_mean": (
        "c[d] = (uint8_t)((s + n / 2) / n);", "c[d] = (uint8_t)(s / n);"),
    "medoid_tie_to_larger_id": (
        "uint32_t dd = orc_dist_u8(c, x + i * D, D);\n            if (dd < bd)",
        "uint32_t dd = orc_dist_u8(c, x + i * D, D);\n            if (dd <= bd)"),
    "degree_off_by_one": (
        "if (deg > ix->R) deg = ix->R;", "if (deg > ix->R) deg = ix->R;\n            if (deg) --deg;"),
    "no_visited_check": (
        "if (v >= ix->n || w->in_v[v]) continue;", "if (v >= ix->n) continue;"),
    "pack_does_not_compact": (
        "if (u != ORC_NO_EDGE) store_u32(adj + 4 + 4 * deg++, u);",
        "store_u32(adj + 4 + 4 * j, u); if (u != ORC_NO_EDGE) deg++;"),
    "vectors_first_unpadded_block_base": (
        "return page + ix->records_per_page * V + i * (ix->record_bytes - V);",
        "return page + ix->records_per_page * vec_bytes(ix->dtype, ix->D) + i * (ix->record_bytes - V);"),
    "insert_keeps_stale_flag": (
        "f[p].expanded = 0;", ""),
}


def _pin_calls():
    """(name, callable(orc)) for every pin test in test_oracle_pins."""
    calls = []
    for name, fn in inspect.getmembers(pins, inspect.isfunction):
        if not name.startswith("test_"):
            continue
        marks = getattr(fn, "pytestmark", [])
        params = [m for m in marks if m.name == "parametrize"]
        if not params:
            calls.append((name, lambda o, fn=fn: fn(o)))
            continue
        argname, values = params[0].args[0], params[0].args[1]
        for v in values:
            calls.append((f"{name}[{v}]", lambda o, fn=fn, a=argname, v=v: fn(o, **{a: v})))
    return calls


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_mutant_is_caught(mutant, tmp_path):
    old, new = MUTANTS[mutant]
    src = SRC_PATH.read_text()
    assert src.count(old) == 1, f"mutation site for {mutant} not unique"
    (tmp_path / "m.c").write_text(src.replace(old, new))
    orc = Oracle(build(tmp_path / "m.c", tmp_path / "libm.so"))
    caught = []
    for name, call in _pin_calls():
        try:
            call(orc)
        except (AssertionError, RuntimeError, ValueError):
            caught.append(name)
            break
    assert caught, f"no pin fails for mutant {mutant}"
