"""The oracle's pins must catch plausible mistakes: each mutant below plants one in a
copy of the oracle source (CPU only), and at least one pin test has to fail on it."""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, original text, mutated text, pin modules expected to catch it)
MUTANTS = [
    ("count_interval_off_by_one", "i < offsets[j + 1]; ++i", "i <= offsets[j + 1] && i < n; ++i", "count_admit"),
    ("kb_floor_not_ceil", "num / q_num + (num % q_num != 0)", "num / q_num", "count_admit"),
    ("admit_fit_strict", "if (used + k > C) break;", "if (used + k >= C) break;", "count_admit"),
    ("admit_skip_not_stop", "if (used + k > C) break;", "if (used + k > C) continue;", "count_admit"),
    ("admit_tie_key_desc", "return p->b < q->b ? -1 : 1;", "return p->b > q->b ? -1 : 1;", "count_admit"),
    ("admit_cold_sign", "*cold = n_window - carried;", "*cold = carried;", "count_admit"),
    ("lpt_tie_high_index", "L[r] < L[best]", "L[r] <= L[best]", "lpt"),
    ("lpt_no_cold_init", "double init = (double)cold / (double)R;\n    for (uint32_t r = 0; r < R; ++r) L[r] = init;\n"
     "    uint32_t off = 0;\n    for (uint32_t a = 0; a < A; ++a) {\n        uint32_t k = adm_k[a];",
     "double init = 0.0 * (double)cold;\n    for (uint32_t r = 0; r < R; ++r) L[r] = init;\n"
     "    uint32_t off = 0;\n    for (uint32_t a = 0; a < A; ++a) {\n        uint32_t k = adm_k[a];", "lpt"),
    ("lpt_job_not_split", "counts_row[adm_keys[a]] / (double)k;", "counts_row[adm_keys[a]] * 1.0;", "lpt"),
    ("fmix_shift", "x ^= x >> 13;", "x ^= x >> 15;", "hash_route"),
    ("hash_seed_mix", "^ 0x9E3779B9u", "^ 0x9E3779B1u", "hash_route"),
    ("p2c_prefers_d2_on_tie", "L[d2] < L[d1] ? d2 : d1", "L[d2] <= L[d1] ? d2 : d1", "hash_route"),
    ("p2c_draws_swapped", "(h & 0xFFFFu) * R) >> 16);\n            uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);\n            dest[i]",
     "(h >> 16) * R) >> 16);\n            uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);\n            dest[i]", "hash_route"),
    ("live_p2c_draws_swapped", "(h & 0xFFFFu) * R) >> 16);\n            uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);\n            d = load",
     "(h >> 16) * R) >> 16);\n            uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);\n            d = load", "live"),
    ("member_pick_low_half", "(uint64_t)(h >> 16) * k) >> 16", "(uint64_t)(h & 0xFFFFu) * k) >> 16", "hash_route"),
    ("live_no_increment", "        load[d] += 1;", "        ;", "live"),
    ("live_member_tie_high", "(load[m] == load[d] && m < d)", "(load[m] == load[d] && m > d)", "live"),
    ("live_p2c_prefers_d2_on_tie", "d = load[d2] < load[d1] ? d2 : d1;", "d = load[d2] <= load[d1] ? d2 : d1;", "live"),
    ("live_member_most_loaded", "if (load[m] < load[d] ||", "if (load[m] > load[d] ||", "live"),
    ("hash_picks_largest", "if (best < 0 || u < ubest) {", "if (best < 0 || u > ubest) {", "ablation"),
    ("hash_ignores_destination", "return cro_fmix32(cro_fmix32(b ^ t) ^ r);", "return cro_fmix32(cro_fmix32(b ^ t));",
     "ablation"),
    ("hash_ignores_key", "return cro_fmix32(cro_fmix32(b ^ t) ^ r);", "return cro_fmix32(cro_fmix32(t) ^ r);",
     "ablation"),
    ("hash_no_charge", "double x = (double)counts_row[b] / (double)k;", "double x = 0.0 * (double)counts_row[b];",
     "ablation"),
    ("replay_hit_not_refreshed", "memmove(row + 1, row, sizeof(uint32_t) * pos);", ";", "replay"),
    ("replay_no_hit_prefix", "s[3] += prefix_len[b];", ";", "replay"),
    ("replay_prefill_on_hit", "s[2] += prefix_len[b];\n            uint32_t keep", "uint32_t keep", "replay"),
    ("replay_evict_mru", "uint32_t keep = used[d] < W ? used[d] : W - 1;", "uint32_t keep = used[d] < W ? used[d] : 0;", "replay"),
]


def _run_mutant(td, name, old, new, mod):
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/absent: {name}"
    c = os.path.join(td, f"{name}.c")
    so = os.path.join(td, f"lib{name}.so")
    open(c, "w").write(src.replace(old, new))
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared", c, "-o", so])
    env = dict(os.environ, CR_ORACLE_LIB=so, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", f"test_oracle_{mod}.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    return name, mod, r.returncode, r.stdout[-1500:]


def test_every_mutant_is_caught():
    with tempfile.TemporaryDirectory() as td:
        with ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 2)) as ex:
            results = list(ex.map(lambda m: _run_mutant(td, *m), MUTANTS))
    survivors = [(n, mod, out) for n, mod, rc, out in results if rc == 0]
    assert not survivors, "mutants survived their pins: " + "; ".join(f"{n} ({mod})" for n, mod, _ in survivors)
