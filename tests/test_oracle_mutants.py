"""The oracle's pins catch plausible mistakes.  Each case copies the oracle's
source, plants one mistake (a wrong constant, an off-by-one, a dropped term,
a swapped operand, a broken tie rule ...), builds it and runs the oracle's
CPU pin tests against that build, which must fail.  An unmodified copy built
the same way must pass, so the failures come from the planted mistakes."""
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# cheapest first: with -x most mistakes stop the run early
PIN_FILES = ["tests/test_oracle_sim.py", "tests/test_oracle_sage.py",
             "tests/test_oracle_pipeline.py", "tests/test_oracle_pins.py"]

# (name, text in oracle/ggref.cpp, replacement)
MUTANTS = [
    ("philox multiplier", "kPhiloxM0 = 0xD2511F53u", "kPhiloxM0 = 0xD2511F55u"),
    ("philox nine rounds", "for (int round = 0; round < 10; ++round)",
     "for (int round = 0; round < 9; ++round)"),
    ("philox Weyl constants swapped", "k0 += kWeyl0;\n      k1 += kWeyl1;",
     "k0 += kWeyl1;\n      k1 += kWeyl0;"),
    ("philox output words crossed", "const uint32_t y0 = hi1 ^ x1 ^ k0;",
     "const uint32_t y0 = hi0 ^ x1 ^ k0;"),
    ("bounded map off by one", "return ((uint64_t)r * bound) >> 32;",
     "return ((uint64_t)r * (bound - 1)) >> 32;"),
    ("floyd inserts j - 1", "      chosen.insert(j);\n", "      chosen.insert(j - 1);\n"),
    ("floyd draw range short by one", "(uint64_t)(d - k + i + 1));", "(uint64_t)(d - k + i));"),
    ("frontiers not nested", "std::vector<int32_t> next = frontier[b][l];",
     "std::vector<int32_t> next;"),
    ("degree test off by one", "        if (d <= k) {\n          for (int64_t p = 0; p < d; ++p)",
     "        if (d < k) {\n          for (int64_t p = 0; p < d; ++p)"),
    ("hot set keeps local nodes",
     "if (ggref_owner(part, u) != part->local_owner) remote.push_back(u);", "remote.push_back(u);"),
    ("hot set ties by larger id", "    std::stable_sort(uf.begin(), uf.end(),",
     "    std::reverse(uf.begin(), uf.end());\n    std::stable_sort(uf.begin(), uf.end(),"),
    ("relative budget rounds down", "n_hot = (U * hot_num + hot_den - 1) / hot_den;",
     "n_hot = (U * hot_num) / hot_den;"),
    ("buckets not stable",
     "  for (int64_t i = 0; i < hot_count; ++i) {\n    const int32_t m = ggref_owner(part, hot_ids[i]);\n    bucket_ids",
     "  for (int64_t i = hot_count - 1; i >= 0; --i) {\n    const int32_t m = ggref_owner(part, hot_ids[i]);\n    bucket_ids"),
    ("stage slot off by one", "      slot_of[u] = (int32_t)s;\n    }", "      slot_of[u] = (int32_t)s + 1;\n    }"),
    ("stage delta counts retained rows", "if (old < 0) ++stats->delta_rows[m];",
     "if (old >= 0) ++stats->delta_rows[m];"),
    ("stage request counts rows", "stats->requests[m] = stats->rows[m] > 0 ? 1 : 0;",
     "stats->requests[m] = stats->rows[m];"),
    ("stage clears before reading old slots",
     "  for (int64_t s = 0; s < total; ++s) old_slot[(size_t)s] = before[bucket_ids[s]];\n  for (int64_t i = 0; i < clear_count; ++i) slot_of[clear_ids[i]] = -1;",
     "  for (int64_t i = 0; i < clear_count; ++i) slot_of[clear_ids[i]] = -1;\n  for (int64_t s = 0; s < total; ++s) old_slot[(size_t)s] = before[bucket_ids[s]];"),
    ("in-place delta takes the highest free slots",
     "for (int64_t s = 0; s < cache_rows; ++s)\n    if (!used[(size_t)s]) free_slots.push_back(s);",
     "for (int64_t s = cache_rows - 1; s >= 0; --s)\n    if (!used[(size_t)s]) free_slots.push_back(s);"),
    ("in-place staging requests retained rows", "        ++stats->retained;\n        continue;",
     "        ++stats->retained;\n        ++stats->rows[m];\n        continue;"),
    ("in-place staging ignores the previous slots", "if (s >= 0) used[(size_t)s] = 1;",
     "(void)s;"),
    ("in-place rows left uncached counted as fetched",
     "        slot_of[u] = -1;\n        short_of_slots = true;\n        continue;",
     "        slot_of[u] = -1;\n        short_of_slots = true;\n        ++stats->rows[m];\n        continue;"),
    ("in-place staging stops at the first row without a slot",
     "        short_of_slots = true;\n        continue;", "        short_of_slots = true;\n        break;"),
    ("miss request counts rows", "stats->miss_requests[m] = miss[m].empty() ? 0 : 1;",
     "stats->miss_requests[m] = (int64_t)miss[m].size();"),
    ("slot 0 treated as a miss", "} else if (slot_of[u] >= 0) {", "} else if (slot_of[u] > 0) {"),
    ("simulator drops the initiation term",
     "energy = energy + (c->eps_init[m] + c->eps_row[m] * xm);",
     "energy = energy + (c->eps_row[m] * xm);"),
    ("simulator sums owner durations", "if (tm > slowest) slowest = tm;", "slowest += tm;"),
    ("simulator never updates the cache", "    cache = hot;   //", "    //"),
    ("simulator misses against the previous cache",
     "std::set_difference(remote.begin(), remote.end(), hot.begin(), hot.end(),",
     "std::set_difference(remote.begin(), remote.end(), cache.begin(), cache.end(),"),
    ("sage swaps self and neighbour weights",
     "const double ws = ly.w_self[(size_t)c * dout + o], wn = ly.w_neigh[(size_t)c * dout + o];",
     "const double ws = ly.w_neigh[(size_t)c * dout + o], wn = ly.w_self[(size_t)c * dout + o];"),
    ("sage transposes the weights",
     "const double ws = ly.w_self[(size_t)c * dout + o], wn = ly.w_neigh[(size_t)c * dout + o];",
     "const double ws = ly.w_self[(size_t)(o * d + c) % ((size_t)d * dout)], wn = ly.w_neigh[(size_t)c * dout + o];"),
    ("sage mean over the fan-out", "            mean[(size_t)c] /= cnt;", "            mean[(size_t)c] /= k;"),
    ("sage ReLU on every layer", "if (ly.relu && y < 0) y = 0;", "if (y < 0) y = 0;"),
    ("fp16 exponent bias off by one", "std::ldexp((double)(1024 + man), exp - 25)",
     "std::ldexp((double)(1024 + man), exp - 24)"),
]


def _build(tmp, text):
    with open(os.path.join(tmp, "ggref.cpp"), "w") as f:
        f.write(text)
    shutil.copy(os.path.join(ROOT, "oracle", "ggref.h"), tmp)
    lib = os.path.join(tmp, "libggref.so")
    subprocess.run(["g++", "-O1", "-std=c++17", "-ffp-contract=off", "-shared", "-fPIC",
                    os.path.join(tmp, "ggref.cpp"), "-o", lib], check=True,
                   capture_output=True)
    return lib


def _run_pins(lib):
    env = dict(os.environ, GGREF_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", *PIN_FILES, "-x", "-q", "-m", "not gpu",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True,
                       text=True)
    return r.returncode, r.stdout[-2000:]


def _case(item):
    name, old, new = item
    src = open(os.path.join(ROOT, "oracle", "ggref.cpp")).read()
    if name is not None:
        assert src.count(old) == 1, f"{name}: the text to mutate occurs {src.count(old)} times"
        src = src.replace(old, new)
    tmp = tempfile.mkdtemp(prefix="ggmut_")
    try:
        rc, out = _run_pins(_build(tmp, src))
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    return name, rc, out


def test_planted_mistakes_fail_the_pins():
    cases = [(None, None, None)] + MUTANTS
    with cf.ThreadPoolExecutor(max_workers=6) as ex:
        results = list(ex.map(_case, cases))
    control = results[0]
    assert control[1] == 0, "unmodified oracle copy fails its pins:\n" + control[2]
    survivors = [(name, rc, out) for name, rc, out in results[1:] if rc != 1]
    assert not survivors, "mistakes the pins did not catch: " + ", ".join(
        f"{n} (exit {rc})" for n, rc, _ in survivors)
