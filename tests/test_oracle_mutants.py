"""The pins are strong enough: each plausible mistake planted in a copy of the
oracle (on the CPU) must make at least one pin fail.

Every mutant is one textual edit of oracle/pcomoe_oracle.c, compiled into a
temporary library; the real oracle is never modified.
"""
import os
import subprocess
import sys

import pytest

import oracle

TESTS = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(TESTS)
SRC = os.path.join(os.path.dirname(oracle.__file__), "pcomoe_oracle.c")

MUTANTS = {
    "tie_to_higher_id": ("if (best < 0 || l[e] > l[best])", "if (best < 0 || l[e] >= l[best])"),
    "softmax_unshifted_numerator": ("p[a] = exp((double)l[ids[a]] - top) / s;",
                                    "p[a] = exp((double)l[ids[a]]) / s;"),
    "diagonal_not_forced": ("if (a == b || mask[(int64_t)ids[a] * n + ids[b]])",
                            "if (mask[(int64_t)ids[a] * n + ids[b]])"),
    "mask_transposed": ("if (a == b || mask[(int64_t)ids[a] * n + ids[b]])",
                        "if (a == b || mask[(int64_t)ids[b] * n + ids[a]])"),
    "src_cond_not_normalised": ("beta[a * k + b] = prod / src;", "beta[a * k + b] = prod;"),
    "src_sum_wrong_index": ("if (b64 >> (a * k + b) & 1) src += p[b];",
                            "if (b64 >> (a * k + b) & 1) src += p[a];"),
    "global_uses_src": ("else beta[a * k + b] = prod / global;", "else beta[a * k + b] = prod / src;"),
    "offsets_shifted": ("cursor[e + 1] += 1;", "cursor[e] += 1;"),
    "row_slot_reversed": ("row_slot[r] = a;", "row_slot[r] = k - 1 - a;"),
    "silu_sign": ("return v / (1.0 + exp(-v));", "return v / (1.0 + exp(v));"),
    "gate_up_swapped": ("U[f] = silu(g) * u;", "U[f] = silu(u) * g;"),
    "down_transposed": ("for (int f = 0; f < F; ++f) s += elem(wd, dtype, row + f) * z[f];",
                        "for (int f = 0; f < F; ++f) s += elem(wd, dtype, w_off + (int64_t)f * H + m) * z[f];"),
    "down_uses_source_expert": ("projection(dtype, w_down, (int64_t)ids[b] * H * F, H, F, Ua, P);",
                                "projection(dtype, w_down, (int64_t)ids[a] * H * F, H, F, Ua, P);"),
    "path_sum_overwrites": ("for (int m = 0; m < H; ++m) y[m] += beta[a * k + b] * P[m];",
                            "for (int m = 0; m < H; ++m) y[m] = beta[a * k + b] * P[m];"),
    "beta_transposed": ("for (int m = 0; m < H; ++m) y[m] += beta[a * k + b] * P[m];",
                        "for (int m = 0; m < H; ++m) y[m] += beta[b * k + a] * P[m];"),
    "bf16_widening": ("uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 16;",
                      "uint32_t bits = (uint32_t)((const uint16_t*)base)[i] << 8;"),
    "x_row_dropped": ("double xv = elem(x, dtype, x_off + h);", "double xv = elem(x, dtype, h);"),
    "reuse_wrong_source": ("const double* Ua = U + (reuse ? (int64_t)a * F : 0);",
                           "const double* Ua = U + (reuse ? (int64_t)b * F : 0);"),
    # scored routing
    "score_bias_transposed": ("return fmaf(lambda, gt[j], gb[i] + bias[(int64_t)i * n + j]);",
                              "return fmaf(lambda, gt[j], gb[i] + bias[(int64_t)j * n + i]);"),
    "score_target_prior_on_source": ("return fmaf(lambda, gt[j], gb[i] + bias[(int64_t)i * n + j]);",
                                     "return fmaf(lambda, gt[i], gb[i] + bias[(int64_t)i * n + j]);"),
    "score_product_rounded_first": ("return fmaf(lambda, gt[j], gb[i] + bias[(int64_t)i * n + j]);",
                                    "return (float)(lambda * gt[j]) + (gb[i] + bias[(int64_t)i * n + j]);"),
    "score_base_on_target": ("return fmaf(lambda, gt[j], gb[i] + bias[(int64_t)i * n + j]);",
                             "return fmaf(lambda, gt[j], gb[j] + bias[(int64_t)i * n + j]);"),
    "scored_mask_ignored": ("if (i != j && !mask[(int64_t)i * n + j]) continue;   /* outside A */",
                            "if (0) continue;"),
    "scored_diagonal_not_forced": ("if (i != j && !mask[(int64_t)i * n + j]) continue;   /* outside A */",
                                   "if (!mask[(int64_t)i * n + j]) continue;"),
    "scored_tie_to_higher": ("if (bi < 0 || s > bs) { bi = i; bj = j; bs = s; }",
                             "if (bi < 0 || s >= bs) { bi = i; bj = j; bs = s; }"),
    "scored_beta_unnormalised": ("for (int r = 0; r < K; ++r) beta[r] = exp((double)score[r] - top) / sum;",
                                 "for (int r = 0; r < K; ++r) beta[r] = exp((double)score[r] - top);"),
    "scored_beta_linear": ("for (int r = 0; r < K; ++r) beta[r] = exp((double)score[r] - top) / sum;",
                           "for (int r = 0; r < K; ++r) beta[r] = 1.0 / K;"),
    "group_bits_transposed": ("b64 |= (uint64_t)1 << (a * K + b);", "b64 |= (uint64_t)1 << (b * K + a);"),
    "group_targets_unsorted": ("if (G[q] < v) pos = q + 1; }", "pos = q + 1; }"),
    "scored_down_uses_source": ("projection(dtype, w_down, (int64_t)tgt[r] * H * F, H, F, Ui, P);",
                                "projection(dtype, w_down, (int64_t)src[r] * H * F, H, F, Ui, P);"),
    "scored_reuse_wrong_slot": ("Ui = U + (int64_t)slot * F;", "Ui = U;"),
    "permute_var_offsets_shifted": ("cursor[e + 1]++;", "cursor[e]++;"),
    "permute_var_slot_reversed": ("row_slot[r] = (int32_t)a;", "row_slot[r] = (int32_t)(K - 1 - a);"),
    "router_weight_transposed": ("s += elem(x, dtype, t * H + h) * elem(w_router, dtype, (int64_t)e * H + h);",
                                 "s += elem(x, dtype, t * H + h) * elem(w_router, dtype, (int64_t)h * n + e);"),
    "router_drops_last_feature": ("            for (int h = 0; h < H; ++h)\n                s += elem(x, dtype, t * H + h)",
                                  "            for (int h = 0; h < H - 1; ++h)\n                s += elem(x, dtype, t * H + h)"),
    "permute_var_stale_slot": ("if (a >= counts[t]) { row_of[t * K + a] = -1; continue; }",
                               "if (a >= counts[t]) { row_of[t * K + a] = 0; continue; }"),
}


def _run_pins_on(src_text: str, name: str, tmp_path) -> int:
    mut_src = tmp_path / "mutant.c"
    mut_src.write_text(src_text)
    so = str(tmp_path / f"libmut_{name}.so")
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-w", "-o", so,
                    str(mut_src), "-lm"], check=True)
    # run the pins in a child process: a mutant may also crash, which counts as caught
    code = ("import sys, oracle, pins\n"
            f"L = oracle.lib({so!r})\n"
            "for pin in pins.ALL_PINS:\n"
            "    try:\n"
            "        pin(L)\n"
            "    except Exception as e:\n"
            "        print('caught by', pin.__name__, str(e)[:100]); sys.exit(3)\n"
            "sys.exit(0)\n")
    env = dict(os.environ, PYTHONPATH=os.pathsep.join([ROOT, TESTS]))
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                       timeout=300)
    return r.returncode


def test_unmutated_oracle_passes_harness(tmp_path):
    """Control: the same harness on the unmodified source passes every pin."""
    assert _run_pins_on(open(SRC).read(), "control", tmp_path) == 0


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    before, after = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(before) == 1, f"mutation site for {name} not unique in the oracle"
    assert _run_pins_on(src.replace(before, after), name, tmp_path) != 0, \
        f"mutant {name} survived every pin"
