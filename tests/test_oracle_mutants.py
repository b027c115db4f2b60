"""Each plausible mistake planted in a copy of the oracle's C source must be
caught by at least one pin (CPU only).

A mutant is built from the oracle source with one text substitution, loaded in
a child process, and the pins are run against it; the child must fail (an
assertion, an error code, or a crash all count as caught).  Mistakes modelled
on the paper's bug taxonomy are included: a bonus token taken from the draft
(DSD), rejected window entries kept in the cache (BSP), positions that ignore
the padding, a cache that is not shifted, and Algorithm 3's all-accept case.
"""
import os
import subprocess
import sys
import tempfile
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parent.parent
SRC = ROOT / "oracle" / "specdec_oracle.c"

MUTANTS = {
    "argmax_ties_to_last": ("if (x > best_v) {", "if (x >= best_v) {"),
    "argmax_ignores_nan": ("if (isnan(x)) return v;", ""),
    "bf16_widen_wrong_shift": ("(uint32_t)h << 16", "(uint32_t)h << 15"),
    # (a slip in the f16 exponent bias or subnormal scale keeps the order of all
    # values, so no argmax can observe it: stochastic verification, which uses
    # the values, must)
    "f16_mantissa_bit": ("(m | 0x400)", "(m | 0x200)"),
    "f16_exponent_bias": ("e - 25);", "e - 24);"),
    "f16_subnormal_scale": ("v = ldexp((double)m, -24);", "v = ldexp((double)m, -23);"),
    "f16_sign_dropped": ("return sign ? -v : v;", "(void)sign;\n  return v;"),
    "all_accept_reads_as_zero": ("int32_t j = k;", "int32_t j = 0;"),
    "bonus_from_draft": ("if (bonus) bonus[i] = tokens[(int64_t)i * (k + 1) + j];",
                         "if (bonus) bonus[i] = (j < k) ? draft[(int64_t)i * k + j] : tokens[(int64_t)i * (k + 1) + j];"),
    "width_without_pending_entry": ("int32_t a = n_acc[i] + 1;\n    if (c + a > Lp)",
                                    "int32_t a = n_acc[i];\n    if (c + a > Lp)"),
    "offset_sign": ("int32_t delta = (Lp - L) - a;", "int32_t delta = a - (Lp - L);"),
    "window_start_off_by_one": ("const int32_t L = W_in - (k + 1);\n  for (int32_t i = 0; i < B; ++i)\n    if (pad_in[i] < 0",
                                "const int32_t L = W_in - k;\n  for (int32_t i = 0; i < B; ++i)\n    if (pad_in[i] < 0"),
    # rejected window entries kept in place of accepted ones (the last a_i window
    # columns appended instead of the first a_i)
    "keeps_rejected_entries": ("for (int32_t j = L; j < L + a; ++j, ++n)",
                               "for (int32_t j = L + (k + 1 - a); j < L + k + 1; ++j, ++n)"),
    "unpad_skips_first_entry": ("for (int32_t j = pad_in[i]; j < L; ++j, ++n)", "for (int32_t j = pad_in[i] + (pad_in[i] < L); j < L; ++j, ++n)"),
    "no_shift": ("memcpy(d + (int64_t)p_new * D, row,", "memcpy(d + (int64_t)(p_new > pad_in[i] ? pad_in[i] : p_new) * D, row,"),
    "pads_not_cleared": ("for (int64_t j = 0; j < p_new; ++j)\n            memset(d + j * D, 0, sizeof(uint16_t) * D);",
                         "for (int64_t j = 0; j < p_new; ++j)\n            (void)j;"),
    "mask_off_by_one": ("uint8_t m = (j >= pad_out[i]) ? 1 : 0;", "uint8_t m = (j > pad_out[i]) ? 1 : 0;"),
    "positions_from_one": ("pos[(int64_t)i * pm_cap + j] = count - 1 > 0 ? count - 1 : 0;",
                           "pos[(int64_t)i * pm_cap + j] = count;"),
    "token_row_drops_pending": ("for (int32_t j = pad_in[i]; j <= L; ++j) row[n++]",
                                "for (int32_t j = pad_in[i]; j < L; ++j) row[n++]"),
    "token_row_without_bonus": ("for (int32_t r = 0; r < a; ++r) row[n++]", "for (int32_t r = 0; r + 1 < a; ++r) row[n++]"),
    "token_row_pads_zero": ("s_out[(int64_t)i * s_out_stride + j] = pad_id;", "s_out[(int64_t)i * s_out_stride + j] = 0;"),
    "token_row_appends_row0": ("row[n++] = tokens[(int64_t)i * (k + 1) + r];", "row[n++] = tokens[r];"),
    "gather_pads_not_cleared": ("for (int64_t j = 0; j < p; ++j) memset(d + j * D, 0, sizeof(uint16_t) * D);", ""),
    "gather_right_aligned_to_cap": ("const int32_t p = Lb - n;", "const int32_t p = (int32_t)batch_cap - n;"),
    "gather_drops_pending_token": ("for (int32_t j = 0; j <= n; ++j)\n      batch_tok", "for (int32_t j = 0; j < n; ++j)\n      batch_tok"),
    "scatter_drops_last_entry": ("sizeof(uint16_t) * (size_t)(n + a) * D);", "sizeof(uint16_t) * (size_t)(n + a - 1) * D);"),
    "scatter_ignores_padding": ("memcpy(d, s + (int64_t)pads[i] * D,", "memcpy(d, s,"),
    "scatter_overwrites_pending": ("trow[n + 1 + r] = tokens", "trow[n + r] = tokens"),
    "scatter_len_without_bonus": ("len[slot[i]] = n + a;", "len[slot[i]] = n + a - 1;"),
    "scatter_batch_row_at_width": ("batch_tok[(int64_t)i * btok_stride + Lb + 1 + r]", "batch_tok[(int64_t)i * btok_stride + Lb + r]"),
    "positions_raw_column": ("pos[(int64_t)i * pm_cap + j] = count - 1 > 0 ? count - 1 : 0;",
                             "pos[(int64_t)i * pm_cap + j] = j;"),
    # stochastic verification (speculative sampling)
    "sample_ratio_inverted": ("if ((double)u_accept[(int64_t)i * k + r] * qx < px) continue;",
                              "if ((double)u_accept[(int64_t)i * k + r] * px < qx) continue;"),
    "sample_residual_is_target": ("w[v] = p[v] > q[v] ? p[v] - q[v] : 0.0;", "w[v] = p[v];"),
    "sample_residual_reversed": ("w[v] = p[v] > q[v] ? p[v] - q[v] : 0.0;", "w[v] = q[v] > p[v] ? q[v] - p[v] : 0.0;"),
    "sample_temperature_ignored": ("p[v] = exp((logit_at(row, dtype, v) - m) / T);",
                                   "p[v] = exp(logit_at(row, dtype, v) - m);"),
    "sample_temperature_multiplies": ("p[v] = exp((logit_at(row, dtype, v) - m) / T);",
                                      "p[v] = exp((logit_at(row, dtype, v) - m) * T);"),
    "sample_bonus_from_previous_row": ("softmax_row((const char*)logits + ((int64_t)i * (k + 1) + k) * V * eb",
                                       "softmax_row((const char*)logits + ((int64_t)i * (k + 1) + k - 1) * V * eb"),
    "sample_correction_uses_accept_uniform": ("x_out = sample_by_inversion(w, V, (double)u_sample[i]);",
                                              "x_out = sample_by_inversion(w, V, (double)u_accept[(int64_t)i * k + r]);"),
    "sample_draft_logits_of_target": ("softmax_row((const char*)draft_logits + ((int64_t)i * k + r) * V * eb",
                                      "softmax_row((const char*)logits + ((int64_t)i * (k + 1) + r) * V * eb"),
    "sample_accepted_tokens_not_drafts": ("r < acc ? draft[(int64_t)i * k + r] :", "r < acc ? (int32_t)x_out :"),
    # rollback (Family A) and variable-length rollback (Family B)
    "rollback_ignores_minimum": ("if (n_acc[i] < m) m = n_acc[i];", "m = n_acc[i];"),
    "rollback_bonus_from_own_count": ("bonus_out[i] = tokens[(int64_t)i * (k + 1) + m];",
                                      "bonus_out[i] = tokens[(int64_t)i * (k + 1) + n_acc[i]];"),
    "rollback_keeps_padding": ("pad_out[i] = pad_in[i] + ((Lp - L) - (m + 1));", "pad_out[i] = pad_in[i];"),
    "varlen_keep_without_bonus": ("const int64_t keep = (int64_t)cu_in[i + 1] - cu_in[i] - (k - n_acc[i]);",
                                  "const int64_t keep = (int64_t)cu_in[i + 1] - cu_in[i] - (k - n_acc[i]) - 1;"),
    "varlen_offsets_not_cumulative": ("cu_out[i + 1] = cu_out[i] + (int32_t)keep;", "cu_out[i + 1] = (int32_t)keep;"),
    "varlen_positions_from_one": ("for (int64_t t = 0; t < keep; ++t) pos[cu_out[i] + t] = t;",
                                  "for (int64_t t = 0; t < keep; ++t) pos[cu_out[i] + t] = t + 1;"),
    "varlen_source_at_output_offset": ("T_cap * row + (int64_t)cu_in[i] * row;", "T_cap * row + (int64_t)cu_out[i] * row;"),
}

# Plausible slips in the scheduler (oracle/exspec.py), caught by the
# scheduling properties or by the output-equivalence loops.
EXSPEC_SRC = ROOT / "oracle" / "exspec.py"
PY_MUTANTS = {
    "reuse_after_ragged_round": ("uniform = len({int(x) for x in n_acc}) == 1", "uniform = True"),
    "window_unbounded": ("if self.active[s]][: self.W]", "if self.active[s]]"),
    "fallback_takes_last": ("chosen = win[:B]", "chosen = win[-B:]"),
    "grouping_skipped": ("if chosen is not None:\n            lens", "if False:\n            lens"),
    "no_length_sort": ("sort_by_length: bool = True", "sort_by_length: bool = False"),
    "reuse_ignores_finished": ("if self.prev is not None and all(self.active[s] for s in self.prev)",
                               "if self.prev is not None"),
    "length_without_bonus": ("a = int(n_acc[i]) + 1", "a = int(n_acc[i])"),
    # the bucket choice of the same-length grouping
    "bucket_tie_to_longer": ("key=lambda b: (len(b), -self.len[b[0]])", "key=lambda b: (len(b), self.len[b[0]])"),
    "oldest_bucket_rule_dropped": ("if len(first) >= B:", "if False:"),
    "largest_bucket_is_first_found": ("best = max(big, key=lambda b: (len(b), -self.len[b[0]]))", "best = big[0]"),
}

PY_RUNNER = r"""
import sys
sys.path.insert(0, {root!r})
import oracle, oracle.exspec as ex
exec(compile(open({src!r}).read(), "exspec_mutant", "exec"), ex.__dict__)
from tests import pins
failed = []
for pin in pins.ALL_PINS:
    try:
        pin(None)
    except Exception as e:
        failed.append(pin.__name__)
print("FAILED_PINS", failed)
sys.exit(1 if failed else 0)
"""

RUNNER = r"""
import sys
sys.path.insert(0, {root!r})
import oracle
from tests import pins
o = oracle.Oracle({lib!r})
failed = []
for pin in pins.ALL_PINS:
    try:
        pin(o)
    except Exception as e:
        failed.append(pin.__name__)
print("FAILED_PINS", failed)
sys.exit(1 if failed else 0)
"""


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = SRC.read_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/present"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", str(mutated), "-o", str(lib), "-lm"],
                   check=True, capture_output=True)
    r = subprocess.run([sys.executable, "-c", RUNNER.format(root=str(ROOT), lib=str(lib))],
                       capture_output=True, text=True, timeout=600, cwd=str(ROOT))
    assert r.returncode != 0, f"mutant {name} survived every pin:\n{r.stdout[-2000:]}\n{r.stderr[-2000:]}"


@pytest.mark.parametrize("name", sorted(PY_MUTANTS))
def test_scheduler_mutant_is_caught(name, tmp_path):
    old, new = PY_MUTANTS[name]
    src = EXSPEC_SRC.read_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/present"
    mutated = tmp_path / "exspec_mutant.py"
    mutated.write_text(src.replace(old, new))
    r = subprocess.run([sys.executable, "-c", PY_RUNNER.format(root=str(ROOT), src=str(mutated))],
                       capture_output=True, text=True, timeout=600, cwd=str(ROOT))
    assert r.returncode != 0, f"mutant {name} survived every pin:\n{r.stdout[-2000:]}\n{r.stderr[-2000:]}"
