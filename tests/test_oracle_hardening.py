"""Hardening of the CPU oracle itself (CPU only, no GPU):

- the pins run against a build of oracle.c with AddressSanitizer and
  UndefinedBehaviorSanitizer, which must report nothing (and which does report
  a planted out-of-bounds read, so the check is live);
- each of a list of plausible mistakes, planted in a copy of oracle.c, makes at
  least one pin fail.  Mistakes in which particular subset a key draws are not
  in the list: that choice follows the library's written rule and is pinned by
  the device comparison, not by the paper ("parity unpinned")."""
import os
import subprocess
import sys

import pytest

from conftest import ROOT

sys.path.insert(0, ROOT)
import oracle  # noqa: E402

SRC = os.path.join(ROOT, "oracle", "oracle.c")
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")
SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all"]
SAN_EXIT = 86


def run_pins(lib_path, sanitized=False, stop_first=False):
    env = dict(os.environ, **{oracle.LIB_ENV: lib_path})
    if sanitized:
        asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                              text=True, check=True).stdout.strip()
        env.update(LD_PRELOAD=asan, ASAN_OPTIONS=f"detect_leaks=0:exitcode={SAN_EXIT}",
                   UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:exitcode={SAN_EXIT}")
    cmd = [sys.executable, "-m", "pytest", PINS, "-q", "--capture=sys", "-p", "no:cacheprovider"]
    if stop_first:
        cmd.append("-x")
    return subprocess.run(cmd, capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)


def planted(tmp_path, name, old, new, extra=()):
    """oracle.c with `old` (which must occur exactly once) replaced by `new`,
    built into a library of its own."""
    src = open(SRC).read()
    assert src.count(old) == 1, f"{name}: the text to replace must occur exactly once"
    path = tmp_path / f"{name}.c"
    path.write_text(src.replace(old, new))
    return oracle.compile_oracle(str(tmp_path / f"lib{name}.so"), src=str(path),
                                 extra=("-Wno-error", *extra))


def test_pins_pass_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    lib = oracle.compile_oracle(str(tmp_path / "liboracle_san.so"), extra=SAN_FLAGS)
    r = run_pins(lib, sanitized=True)
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, \
        r.stderr[-3000:]
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]


def test_sanitizer_build_reports_a_planted_overflow(tmp_path):
    # sorting one element past the end of Floyd's output array
    lib = planted(tmp_path, "overflow", "qsort(out, (size_t)f, sizeof(int64_t), cmp_i64);",
                  "qsort(out, (size_t)f + 1, sizeof(int64_t), cmp_i64);", extra=SAN_FLAGS)
    r = run_pins(lib, sanitized=True, stop_first=True)
    assert r.returncode == SAN_EXIT and "heap-buffer-overflow" in r.stderr, r.stderr[-3000:]


# (name, text in oracle.c, the planted mistake)
MUTANTS = [
    ("mix64_shift", "z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;",
     "z = (z ^ (z >> 31)) * 0xBF58476D1CE4E5B9ULL;"),
    ("splitmix_first_output", "return or_mix64(state + OR_GAMMA * (i + 1));",
     "return or_mix64(state + OR_GAMMA * i);"),
    ("key_drops_hop", "return or_mix64(batch_state ^ (((uint64_t)(uint32_t)k << 32) | "
                      "(uint64_t)(uint32_t)v));",
     "return or_mix64(batch_state ^ (uint64_t)(uint32_t)v);"),
    ("below_by_modulo", "return (uint64_t)(p >> 64);", "return h % m;"),
    ("floyd_range_drops_plus_one",
     "(int64_t)or_below(or_splitmix_nth(key, (uint64_t)i), (uint64_t)(j + 1));",
     "(int64_t)or_below(or_splitmix_nth(key, (uint64_t)i), (uint64_t)j);"),
    ("floyd_no_collision_rule", "out[i] = seen ? j : t;", "out[i] = t;"),
    ("new_frontier_rule_resamples_seeds", "front_begin = layered ? 0 : front_end;",
     "front_begin = 0;"),
    ("layered_frontier_only_new", "front_begin = layered ? 0 : front_end;",
     "front_begin = front_end;"),
    ("new_nodes_not_sorted", "qsort(fresh, (size_t)nfresh, sizeof(int32_t), cmp_i32);", ""),
    ("new_nodes_not_deduplicated_against_batch",
     "if (local[cand_nbr[c]] < 0) fresh[nfresh++] = cand_nbr[c];",
     "fresh[nfresh++] = cand_nbr[c];"),
    ("edge_endpoints_transposed",
     "es[e] = (int32_t)cand_src[c];\n        ed[e] = local[cand_nbr[c]];",
     "ed[e] = (int32_t)cand_src[c];\n        es[e] = local[cand_nbr[c]];"),
    ("edge_neighbour_not_relabelled", "ed[e] = local[cand_nbr[c]];", "ed[e] = cand_nbr[c];"),
    ("union_not_deduplicated", "if (i == 0 || all[i] != all[i - 1]) {", "{"),
    ("packed_rows_ignore_cache",
     "if (cache_slot[nodes[(int64_t)b * node_stride + j]] < 0) ++rows;", "++rows;"),
    ("packed_chunk_not_sorted", "qsort(pb, (size_t)cnt, sizeof(int32_t), cmp_i32);", ""),
    ("address_table_sign", "cache_slot[u] >= 0 ? -(cache_slot[u] + 1)",
     "cache_slot[u] >= 0 ? -(cache_slot[u])"),
    ("assembly_cache_row_off_by_one",
     "src = (const char *)cache + (int64_t)(-(int64_t)l - 1) * row_bytes;",
     "src = (const char *)cache + (int64_t)(-(int64_t)l - 2 < 0 ? 0 : -(int64_t)l - 2) "
     "* row_bytes;"),
    ("frequency_ties_by_descending_id", "  return (x > y) - (x < y);\n}\n\nint or_cache",
     "  return (x < y) - (x > y);\n}\n\nint or_cache"),
    ("frequency_counts_every_node_once", "count[u] += 1;", "count[u] = 1;"),
    ("minhash_keeps_maximum", "if (h < s) s = h;", "if (s == INF || h > s) s = h;"),
    ("minhash_ignores_membership",
     "if (find_i32(set[i], node_count[i], v) < 0) continue;", ""),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(tmp_path, name, old, new):
    r = run_pins(planted(tmp_path, name, old, new), stop_first=True)
    assert r.returncode == 1 and "failed" in r.stdout, \
        f"{name}: no pin failed\n{r.stdout[-2000:]}{r.stderr[-2000:]}"
