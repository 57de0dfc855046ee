"""The oracle's pins must reject plausible mistakes.

Each case plants one mistake in a temporary copy of oracle.c (on the CPU), builds
it, and runs the pin suite against it (the decode pins, or the multi-token pins for
mistakes in the multi-token entry point); at least one pin must fail.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "dropped_scale": ("s[(int64_t)i * L + t] = a->scale * dot;", "s[(int64_t)i * L + t] = dot;"),
    "flipped_exponent_sign": ("si[t] = exp(si[t] - m);", "si[t] = exp(m - si[t]);"),
    "shifted_slot": ("int slot = t % P;\n    if (pid", "int slot = (t + 1) % P;\n    if (pid"),
    "transposed_scale_index": ("(double)a->k_scale[(int64_t)pid * a->num_kv_heads + g]",
                               "(double)a->k_scale[(int64_t)g * a->num_pages + pid]"),
    "missing_normalisation": ("for (int j = 0; j < d; ++j) o[j] /= z;", ""),
    "wrong_fp8_bias": ("mag = ldexp(1.0 + (double)m / 8.0, e - 7);", "mag = ldexp(1.0 + (double)m / 8.0, e - 8);"),
    "ignored_head_map": ("if (a->kv_head_of_q[h] == g) heads[nh++] = h;",
                         "if (h % a->num_kv_heads == g) heads[nh++] = h;"),
    "dropped_last_token": ("for (int t = 0; t < L; ++t) {\n    int pid = a->block_table[(int64_t)b * a->max_pages_per_seq + t / P];\n    int slot = t % P;\n    int64_t base",
                           "for (int t = 0; t < L - 1; ++t) {\n    int pid = a->block_table[(int64_t)b * a->max_pages_per_seq + t / P];\n    int slot = t % P;\n    int64_t base"),
    "bf16_low_half": ("uint32_t u = (uint32_t)bits << 16;", "uint32_t u = (uint32_t)bits << 15;"),
    # multi-token queries
    "causal_limit_one_early": ("const int pos = seq_lens[b] - n + i;", "const int pos = seq_lens[b] - n + i - 1;"),
    "causal_limit_one_late": ("(orc_unit){b, g, pos + 1,", "(orc_unit){b, g, pos + 2 > seq_lens[b] ? pos + 1 : pos + 2,"),
    "query_rows_reversed": ("(int64_t)q_start[b] + i}", "(int64_t)q_start[b] + (n - 1 - i)}"),
    "chunk_at_sequence_start": ("const int pos = seq_lens[b] - n + i;", "const int pos = i;"),
}
MULTI = {"causal_limit_one_early", "causal_limit_one_late", "query_rows_reversed", "chunk_at_sequence_start"}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    src = open(os.path.join(ROOT, "oracle", "oracle.c")).read()
    old, new = MUTANTS[name]
    assert old in src, "mutation site moved; update the pattern"
    shutil.copytree(os.path.join(ROOT, "oracle"), tmp_path / "oracle",
                    ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    (tmp_path / "oracle" / "oracle.c").write_text(src.replace(old, new, 1))
    (tmp_path / "tests").mkdir()
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tmp_path / "tests" / "golden")
    suite = "test_oracle_multi.py" if name in MULTI else "test_oracle.py"
    for f in (suite, "conftest.py"):
        shutil.copy(os.path.join(ROOT, "tests", f), tmp_path / "tests" / f)
    os.symlink(os.path.join(ROOT, "paper_2607_09207_amd"), tmp_path / "paper_2607_09207_amd")
    env = dict(os.environ, PYTHONPATH=str(tmp_path))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "tests/" + suite],
                       cwd=tmp_path, capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 1 and "failed" in r.stdout, r.stdout[-2000:]
