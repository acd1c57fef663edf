"""The pins must have teeth: plant plausible mistakes in copies of the CPU
oracle (on the CPU only) and require that some pin in test_oracle_pins fails
for every one of them. The real oracle is restored afterwards."""
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

# (name, original text, mutated text) -- each a mistake one could make when
# transcribing the paper's definitions.
MUTATIONS = [
    ("gen staleness sign flipped", "S += c - (int64_t)v;", "S += (int64_t)v - c;"),
    ("mask tag not excluded", "if (v == -1)\n                continue;            /* non-generated token */",
     "if (v == -2)\n                continue;"),
    ("masked tokens counted in T", "continue;            /* non-generated token */",
     "{ T += 1; continue; }"),
    ("waiting term dropped", "score_out[i] = wait_term + gen_term;", "score_out[i] = gen_term;"),
    ("waiting staleness sign flipped", "double K_wait = (double)((int64_t)V - c);",
     "double K_wait = (double)(c - (int64_t)V);"),
    ("K_gen operands transposed", "double K_gen = (T > 0) ? (double)S / (double)T : 0.0;",
     "double K_gen = (T > 0) ? (double)T / ((double)S + 1.0) : 0.0;"),
    ("phi numerator transposed", "F = (double)A / (double)(A + B);", "F = (double)B / (double)(A + B);"),
    ("ECDF strict instead of <=", "if (window[k] <= prefix[i])", "if (window[k] < prefix[i])"),
    ("gamma ignored on complement", "int64_t B = ipow(W - a, gamma);", "int64_t B = ipow(W - a, 1);"),
    ("F weight applied to waiting term", "double wait_term = w_wait * K_wait;\n        double gen_term = F * K_gen;",
     "double wait_term = w_wait * F * K_wait;\n        double gen_term = K_gen;"),
    ("EMA coefficients swapped", "double r_hat = beta * (*r_hat_inout) + (1.0 - beta) * r;",
     "double r_hat = (1.0 - beta) * (*r_hat_inout) + beta * r;"),
    ("rate normalised by target", "double x = (double)(N - N_tar) / denom;",
     "double x = (double)(N - N_tar) / (double)(N_tar > 1 ? N_tar : 1);"),
    ("budget floors instead of rounding", "b = (int64_t)nearbyint(rc * (double)N);", "b = (int64_t)floor(rc * (double)N);"),
    ("no zero budget at target, no cap", "if (N > N_tar) {\n        double rc = r_hat < r_max ? r_hat : r_max;\n"
     "        b = (int64_t)nearbyint(rc * (double)N);   /* default mode: ties to even */\n"
     "        if (b > N - N_tar)\n            b = N - N_tar;",
     "{\n        double rc = r_hat < r_max ? r_hat : r_max;\n        b = (int64_t)nearbyint(rc * (double)N);"),
    ("surplus cap missing", "        if (b > N - N_tar)\n            b = N - N_tar;\n", ""),
    ("max rejection cap missing", "double rc = r_hat < r_max ? r_hat : r_max;", "double rc = r_hat;"),
    ("select ties to the higher id", "return (a < b) ? -1 : (a > b);", "return (a > b) ? -1 : (a < b);"),
    ("select ascending", "if (sa > sb)\n        return -1;\n    if (sa < sb)\n        return 1;",
     "if (sa < sb)\n        return -1;\n    if (sa > sb)\n        return 1;"),
    ("select off by one", "for (int64_t r = 0; r < budget; r++)", "for (int64_t r = 1; r < budget; r++)"),
    ("compact writes source offsets", "offsets_out[k] = pos;\n        kept_ids_out[k]",
     "offsets_out[k] = offsets[i];\n        kept_ids_out[k]"),
    ("compact copies from packed position", "(const char *)cols_in[c] + (size_t)offsets[i] * e",
     "(const char *)cols_in[c] + (size_t)pos * e"),
    ("validate checks tag against V", "if (v < 0 || v > c)", "if (v < 0 || v > V)"),
    ("group mean divides by size + 1", "sum / (double)(hi - lo) : 0.0", "sum / (double)(hi - lo + 1) : 0.0"),
    ("group sum skips first member", "for (int64_t i = lo; i < hi; i++)\n            sum = sum + score[i];",
     "for (int64_t i = lo + 1; i < hi; i++)\n            sum = sum + score[i];"),
    ("group sum reads one past", "sum = sum + score[i];", "sum = sum + score[i < hi - 1 ? i + 1 : i];"),
    ("empty group scores nonzero", ": 0.0;\n    }\n    return ORC_OK;", ": 1.0;\n    }\n    return ORC_OK;"),
    ("group expand inverted", "keep_out[i] = group_keep[g] ? 1 : 0;", "keep_out[i] = group_keep[g] ? 0 : 1;"),
    ("group expand off by one group", "keep_out[i] = group_keep[g] ? 1 : 0;",
     "keep_out[i] = group_keep[g + 1 < n_groups ? g + 1 : g] ? 1 : 0;"),
    ("group offsets end unchecked", "if (group_offsets[0] != 0 || group_offsets[n_groups] != n)",
     "if (group_offsets[0] != 0)"),
    ("stream quantile rank rounds down", "int64_t k = (int64_t)ceil(p * (double)cnt);",
     "int64_t k = (int64_t)floor(p * (double)cnt);"),
    ("stream quantile of the rate, not its complement", "double p = 1.0 - rate;", "double p = rate;"),
    ("stream rate not capped", "double rate = r_hat < r_max ? r_hat : r_max;", "double rate = r_hat;"),
    ("stream rejects ties with the cutoff", "if (score[i] > kappa) {", "if (score[i] >= kappa) {"),
    ("stream window ignores min observations", "if (cnt >= window_min && cnt > 0 && rate > 0.0) {",
     "if (cnt > 0 && rate > 0.0) {"),
    ("stream draw runs one past the batch", "for (int64_t i = 0; i < n && retained < batch_size; i++) {",
     "for (int64_t i = 0; i < n && retained <= batch_size; i++) {"),
    ("stream window takes only retained scores", "        ring[head] = score[i];\n        head = (head + 1) % cap;",
     "        if (status_out[i] != 1) continue;\n        ring[head] = score[i];\n        head = (head + 1) % cap;"),
    ("prefix score signed, not absolute", "sum = sum + fabs(d);", "sum = sum + d;"),
    ("prefix cap ignored", "if (m == cap)\n                break;", "if (m == cap + 1000000)\n                break;"),
    ("prefix masked tokens counted", "if (tags && tags[t] == -1)\n                continue;                /* non-generated token */",
     "if (tags && tags[t] == -2)\n                continue;"),
    ("prefix minimum not applied", "(m >= min_tokens && m > 0) ? sum / (double)m : NAN;", "(m > 0) ? sum / (double)m : NAN;"),
    ("prefix mean over the span length", "sum / (double)m : NAN;",
     "sum / (double)(prefix_offsets[i + 1] - prefix_offsets[i]) : NAN;"),
    ("stale-k strict comparison", "keep_out[i] = (lag_sum <= k * T) ? 1 : 0;", "keep_out[i] = (lag_sum < k * T) ? 1 : 0;"),
    ("stale-k lag from completion, not current version", "lag_sum += (int64_t)V - (int64_t)tags[t];",
     "lag_sum += (int64_t)completion[i] - (int64_t)tags[t];"),
    ("stale-k empty trajectory admitted always", "keep_out[i] = (wait <= k) ? 1 : 0;", "keep_out[i] = 1;"),
    ("stale-k masked tokens counted", "            if (tags[t] == -1)\n                continue;\n            lag_sum",
     "            if (tags[t] == -2)\n                continue;\n            lag_sum"),
    ("diagnostics bins closed on the right", "while (!(m[q] < e[bin]))", "while (!(m[q] <= e[bin]))"),
    ("diagnostics classes swapped", "int cls = keep[i] ? 1 : 0;", "int cls = keep[i] ? 0 : 1;"),
    ("diagnostics K_gen over all tokens", "m[1] = (T > 0) ? (double)S / (double)T : 0.0;",
     "m[1] = (T > 0) ? (double)S / (double)(offsets[i + 1] - offsets[i]) : 0.0;"),
    ("diagnostics totals miss T", "tot[3] += T;", "tot[3] += S;"),
    ("window power guard removed", "if (W > 0 && !window_power_fits(W, gamma))", "if (0)"),
    ("window power guard computed without overflow check", "if (W > 0 && !window_power_fits(W, gamma))",
     "if (W > 0 && (double)ipow(W, gamma) >= 9007199254740992.0)"),
    ("window power guard takes one factor too many", "for (int k = 0; k < g; k++) {\n        if (W != 0",
     "for (int k = 0; k <= g; k++) {\n        if (W != 0"),
    ("stream window misses the newest entry", "sorted[t] = ring[(head - cnt + t + cap) % cap];",
     "sorted[t] = ring[(head - cnt + t + cap - 1) % cap];"),
]

from tests import test_oracle_group_pins as group_pins
from tests import test_oracle_stream_pins as stream_pins
from tests import test_oracle_prefix_pins as prefix_pins
from tests import test_oracle_diag_pins as diag_pins

PIN_FUNCS = [getattr(m, n) for m in (pins, group_pins, stream_pins, prefix_pins, diag_pins) for n in dir(m)
             if n.startswith("test_") and callable(getattr(m, n))]


def _run_pins():
    failed = []
    for f in PIN_FUNCS:
        try:
            f()
        except (Exception, pytest.fail.Exception) as e:   # assertion, oracle error, hypothesis, pytest.raises
            failed.append((f.__name__, type(e).__name__))
    return failed


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new, tmp_path):
    src = open(oracle._SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    mut = tmp_path / "mut.c"
    mut.write_text(src.replace(old, new))
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
                           "-o", str(so), str(mut), "-lm"])
    real = oracle._load()
    oracle._lib = oracle.load_library(str(so))
    try:
        failed = _run_pins()
    finally:
        oracle._lib = real
    assert failed, "no pin caught the planted mistake: " + name


def test_unmutated_oracle_passes_all_pins():
    assert _run_pins() == []
