"""Plant plausible mistakes in a copy of the C oracle and check that the pin
suite (test_oracle_pins.py) rejects every one of them.

Each mutant is compiled from a text edit of kvx_oracle.c into a temporary
library and the pins run against it in a child process (a mutant that reads or
writes out of bounds may crash the child; that also counts as caught).
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "kvx_oracle.c")

GATHER_KV = "const uint8_t* base = (const uint8_t*)(kv == 0 ? k[l] : v[l]);"
SCATTER_KV = "uint8_t* base = (uint8_t*)(kv == 0 ? k[l] : v[l]);"

MUTANTS = {
    "gather_swaps_k_and_v": (GATHER_KV, GATHER_KV.replace("k[l] : v[l]", "v[l] : k[l]")),
    "scatter_swaps_k_and_v": (SCATTER_KV, SCATTER_KV.replace("k[l] : v[l]", "v[l] : k[l]")),
    "layer_index_not_rebased": ("out + c * S + ((l - l0) * 2 + kv)", "out + c * S + (l * 2 + kv)"),
    "kv_major_instead_of_layer_major": ("out + c * S + ((l - l0) * 2 + kv) * Tc",
                                        "out + c * S + (kv * (l1 - l0) + (l - l0)) * Tc"),
    "block_index_ignores_chunk_stride": ("const int64_t id = bt[c * bpc + j];\n          move_slab(s, kv, out",
                                         "const int64_t id = bt[c + j];\n          move_slab(s, kv, out"),
    "chunk_stride_counts_all_layers": ("const int64_t S = (l1 - l0) * 2 * chunk_tokens * row;",
                                       "const int64_t S = l1 * 2 * chunk_tokens * row;"),
    "last_chunk_strided_as_full": ("((l - l0) * 2 + kv) * Tc * row + j * slab,\n                    (uint8_t*)base",
                                   "((l - l0) * 2 + kv) * chunk_tokens * row + j * slab,\n                    (uint8_t*)base"),
    "scatter_block_off_by_one": ("base + id * slab, 0);", "base + (id ^ 1) * slab, 0);"),
    "hnd_token_head_swapped": ("if (s->layout == KVO_LAYOUT_HND) return ((h * BS + t) * D + d) * e;",
                               "if (s->layout == KVO_LAYOUT_HND) return ((t * H + h) * D + d) * e;"),
    "paged_attn_v_dim_token_swapped": ("if (kv == 1) return ((h * D + d) * BS + t) * e;",
                                       "if (kv == 1) return ((h * BS + t) * D + d) * e;"),
    "paged_attn_k_split_swapped": ("return (((h * (D / x) + d / x) * BS + t) * x + d % x) * e;",
                                   "return (((h * (D / x) + d % x) * BS + t) * x + d / x) * e;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) >= 1, f"mutation anchor for {name} not found"
    mutated = text.replace(old, new, 1)
    c = tmp_path / "mutant.c"
    c.write_text(mutated)
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-o", str(lib), str(c)], check=True)
    env = dict(os.environ, KVX_ORACLE_LIB=str(lib), KVX_NO_AUTOBUILD="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"pins did not catch mutant {name}:\n{r.stdout[-2000:]}"


# ---- the break-even oracle (Python): text edits of oracle/breakeven.py, loaded
# as a module and run through the oracle pins of test_breakeven.py in-process.

BE_SRC = os.path.join(ROOT, "oracle", "breakeven.py")
BE_MUTANTS = {
    "pays_not_strict": ("return g(P) + f(D - P) < f(D)", "return g(P) + f(D - P) <= f(D)"),
    "suffix_recompute_dropped": ("return g(P) + f(D - P) < f(D)", "return g(P) < f(D)"),
    "max_io_copy_sign": ("return f(D) - (g(D) - copy(D))", "return f(D) - g(D) - copy(D)"),
    "threshold_first_crossing": ("if all(g(y) < f(y) for y in grid if y >= x):",
                                 "if g(x) < f(x):"),
    "no_segment_walk": ("    while i < n - 2 and x > tokens[i + 1]:\n        i += 1\n", ""),
    "extrapolation_clamped": ("    return y0 + slope * (x - x0)",
                              "    return y0 + slope * (min(max(x, tokens[0]), tokens[-1]) - x0)"),
    "prefix_grid_starts_at_zero": ("for P in range(granularity, D + 1, granularity):",
                                   "for P in range(0, D + 1, granularity):"),
    "gate_declines_empty_loads": ("return [lb == 0 or lb * block_size >= gate_tokens",
                                  "return [lb * block_size >= gate_tokens"),
    "rate_in_binary_gigabytes": ("x * bytes_per_token / (restore_GBps * 1e9)",
                                 "x * bytes_per_token / (restore_GBps * 2**30)"),
    "rate_transfer_dropped": ("return lambda x: non_transfer(x) + x * bytes_per_token",
                              "return lambda x: non_transfer(x) + 0 * bytes_per_token"),
    "required_without_copy_credit": ("    budget = max_io(f, g, copy, D)\n",
                                     "    budget = f(D) - g(D)\n"),
}


@pytest.mark.parametrize("name", sorted(BE_MUTANTS))
def test_breakeven_pins_reject_mutant(name, tmp_path, monkeypatch):
    import importlib.util

    old, new = BE_MUTANTS[name]
    text = open(BE_SRC).read()
    assert text.count(old) >= 1, f"mutation anchor for {name} not found"
    path = tmp_path / "breakeven_mutant.py"
    path.write_text(text.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location("breakeven_mutant", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    try:
        import test_breakeven as tb
    finally:
        sys.path.pop(0)
    monkeypatch.setattr(tb, "ob", mod)
    caught = False
    pins = [(tb.test_oracle_curve_interpolates_and_extrapolates, ()),
            (tb.test_oracle_special_cases, ()), (tb.test_oracle_exact_tie_does_not_pay, ()),
            (tb.test_oracle_brute_force_frontier_is_minimal, ())]
    pins += [(tb.test_oracle_linear_closed_forms, case) for case in tb.LINES]
    pins += [(tb.test_oracle_hit_from_rate_closed_forms, case) for case in tb.RATES]
    for fn, args in pins:
        try:
            fn(*args)
        except Exception:
            caught = True
            break
    assert caught, f"break-even pins did not catch mutant {name}"


# ---- the prefix / step-plan oracle (Python): text edits of oracle/prefix.py,
# run through the oracle pins of test_step_plan.py in-process.

PREFIX_SRC = os.path.join(ROOT, "oracle", "prefix.py")
PREFIX_MUTANTS = {
    "chunk_keyed_by_first_block": ("out.append((keys[last], last - first + 1))",
                                   "out.append((keys[first], last - first + 1))"),
    "chunk_block_count_full": ("out.append((keys[last], last - first + 1))",
                               "out.append((keys[last], bpc))"),
    "dedupe_last_occurrence": ("return [seen.setdefault(k, i) for i, k in enumerate(keys)]",
                               "return [max(j for j, q in enumerate(keys) if q == k) for k in keys]"),
    "lookup_skips_misses": ("        if key not in cached:\n            break\n        n += 1",
                            "        if key in cached:\n            n += 1"),
    "gate_counts_resident_chunks": ("        if not resident[key]:\n            load[ri] += nb",
                                    "        load[ri] += nb"),
    "declined_request_restores": ("if not resident[key] and loads[ri] and key not in index_of:",
                                  "if not resident[key] and key not in index_of:"),
    "recompute_counted_once": ("            states.append((\"recompute\",))\n            recompute += nb",
                               "            states.append((\"recompute\",))\n"
                               "            recompute += nb if (ri, k) == next((c[0], c[1]) for c in chunks if c[2] == key) else 0"),
    "offload_chunk_index_global": ("            offload.append((ri, c, nb, obt, first_new))",
                                   "            offload.append((ri, len(offload), nb, obt, first_new))"),
}


@pytest.mark.parametrize("name", sorted(PREFIX_MUTANTS))
def test_prefix_pins_reject_mutant(name, tmp_path, monkeypatch):
    import importlib

    old, new = PREFIX_MUTANTS[name]
    text = open(PREFIX_SRC).read()
    assert text.count(old) >= 1, f"mutation anchor for {name} not found"
    pkg = tmp_path / "oracle_mut"
    pkg.mkdir()
    (pkg / "__init__.py").write_text("")
    (pkg / "breakeven.py").write_text(open(os.path.join(ROOT, "oracle", "breakeven.py")).read())
    (pkg / "prefix.py").write_text(text.replace(old, new, 1))
    sys.path.insert(0, str(tmp_path))
    try:
        mod = importlib.import_module("oracle_mut.prefix")
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        import test_step_plan as tsp
    finally:
        while str(tmp_path) in sys.path:
            sys.path.remove(str(tmp_path))
        if os.path.join(ROOT, "tests") in sys.path:
            sys.path.remove(os.path.join(ROOT, "tests"))
    monkeypatch.setattr(tsp, "op", mod)
    caught = False
    pins = [(tsp.test_oracle_reproduces_paper_example, ()),
            (tsp.test_oracle_lookup_stops_at_first_miss, ()),
            (tsp.test_oracle_chunk_identity_golden, ()),
            (tsp.test_oracle_plan_step_golden, (0,)), (tsp.test_oracle_plan_step_golden, (1,))]
    for fn, args in pins:
        try:
            fn(*args)
        except Exception:
            caught = True
            break
    for m in [m for m in sys.modules if m.startswith("oracle_mut")]:
        del sys.modules[m]
    assert caught, f"prefix pins did not catch mutant {name}"
