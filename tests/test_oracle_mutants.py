"""Plant plausible mistakes in copies of the oracle source (on the CPU) and
check that the pins catch every one of them.  Each mutant is compiled to a
temporary library and its pins run in a child process, so a mutant that
crashes also counts as caught."""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))

MUTANTS = {
    "causal_excludes_diagonal": ("const int last_visible = L - Q + i;", "const int last_visible = L - Q + i - 1;"),
    "causal_sees_next_draft": ("const int last_visible = L - Q + i;", "const int last_visible = L - Q + i + 1;"),
    "no_causal_mask": ("if (hi > last_visible + 1)\n        hi = last_visible + 1;", ""),
    "gqa_interleaved": ("const int g = h / G;\n    const int last_visible = L - Q + i;          /* inclusive */",
                        "const int g = h % pr->Hkv;\n    const int last_visible = L - Q + i;          /* inclusive */"),
    "page_index_mod": ("int64_t page = pr->page_table[(size_t)b * pr->max_pages + t / pr->P];\n        int slot = t % pr->P;\n        double acc",
                       "int64_t page = pr->page_table[(size_t)b * pr->max_pages + t % pr->P];\n        int slot = t % pr->P;\n        double acc"),
    "slot_from_page": ("int slot = t % pr->P;\n        double acc", "int slot = (t / pr->P) % pr->P;\n        double acc"),
    "scale_dropped": ("s[t - lo] = pr->scale * acc;", "s[t - lo] = acc;"),
    "scale_squared": ("s[t - lo] = pr->scale * acc;", "s[t - lo] = pr->scale * pr->scale * acc;"),
    "max_sign_flipped": ("s[t - lo] = exp(s[t - lo] - m);", "s[t - lo] = exp(m - s[t - lo]);"),
    "not_normalised": ("o[d] /= l;\n    *lse", "o[d] /= 1.0;\n    *lse"),
    "pool_slot_head_transposed": ("return (((size_t)p * (size_t)Hkv + (size_t)g) * (size_t)P + (size_t)u) * (size_t)D + (size_t)d;",
                                  "return (((size_t)p * (size_t)P + (size_t)u) * (size_t)Hkv + (size_t)g) * (size_t)D + (size_t)d;"),
    "q_row_head_transposed": ("return (((size_t)b * (size_t)Qmax + (size_t)i) * (size_t)Hq + (size_t)h) * (size_t)D + (size_t)d;",
                              "return (((size_t)b * (size_t)Hq + (size_t)h) * (size_t)Qmax + (size_t)i) * (size_t)D + (size_t)d;"),
    "values_read_from_keys": ("o[d] += s[t - lo] * widen_bf16(pr->vp[", "o[d] += s[t - lo] * widen_bf16(pr->kp["),
    "lse_missing_log_sum": ("*lse = m + log(l);", "*lse = m;"),
    "merge_weight_sign": ("double w = exp(lse - M);", "double w = exp(M - lse);"),
    "merge_not_normalised": ("out[(size_t)r * D + d] /= wsum;", "out[(size_t)r * D + d] /= 1.0;"),
    "bf16_widen_shift": ("uint32_t u = ((uint32_t)bits) << 16;", "uint32_t u = ((uint32_t)bits) << 15;"),
    "first_key_skipped": ("int lo = t_begin < 0 ? 0 : t_begin;", "int lo = t_begin < 1 ? 1 : t_begin;"),
    "last_dim_skipped": ("for (int d = 0; d < pr->D; d++) {\n            double qv", "for (int d = 0; d < pr->D - 1; d++) {\n            double qv"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(oracle.SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    mpath = tmp_path / "mutant.c"
    mpath.write_text(src.replace(old, new))
    so = oracle.build(str(mpath), str(tmp_path / "libmutant.so"))
    env = dict(os.environ, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, os.path.join(HERE, "oracle_pins.py"), so],
                       capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode != 0, f"mutant {name} passed every pin"
