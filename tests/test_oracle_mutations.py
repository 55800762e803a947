"""The oracle's pins bite: each plausible mistake planted in a copy of the
oracle (on the CPU) makes at least one pin fail.

Every mutation below is a one-place edit of oracle/opd_oracle.c: a dropped
term, a flipped sign, a sum for a mean, the wrong advantage or weight, a
wrong normaliser, an off-by-one rank, a reversed tie order.  The mutated
copy is built into a temporary library, and the pin modules
(tests/test_oracle_*pins.py) run against it in a child process; they must
fail (exit status 1, test failures).  A control run of the unmutated source
through the same harness must pass, so a failure is the mutation's."""
import os
import shutil
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "opd_oracle.c")
HDR = os.path.join(ROOT, "oracle", "opd_oracle.h")
PINS = [os.path.join(HERE, f) for f in ("test_oracle_pins.py", "test_oracle_cache_pins.py",
                                        "test_oracle_coverage_pins.py",
                                        "test_oracle_diag_pins.py")]

# (name, text in opd_oracle.c, replacement)
MUTATIONS = [
    ("topk_reverse_grad_drops_D",
     "gamma * pt * ((log_pt - log_qt) - kl)", "gamma * pt * (log_pt - log_qt)"),
    ("topk_forward_grad_sign",
     "gamma * (pt - qt)", "gamma * (qt - pt)"),
    ("topk_teacher_not_renormalised",
     "const double log_qt = tau[i] - logZq;          /* log q~(a_i) */",
     "const double log_qt = tau[i];          /* log q~(a_i) */"),
    ("mc_sum_for_mean",
     "  c /= (double)M;\n  *loss = -c;", "  *loss = -c;"),
    ("mc_old_advantage_for_theta",
     "const double A = tau[i] - logp;    /* A_theta(a_i, s) */",
     "const double A = tau[i] - beta[i];    /* A_theta(a_i, s) */"),
    ("mc_no_importance_ratio",
     "    const double rho = exp(logp - beta[i]);\n    c += rho * A;",
     "    const double rho = 1.0;\n    c += rho * A;"),
    ("mc_grad_spike_sign",
     "grad[ids[i]] -= gamma * rho * A / (double)M;", "grad[ids[i]] += gamma * rho * A / (double)M;"),
    ("clip_tie_counts_as_clipped",
     "if (!clip || unclipped <= clipped) {", "if (!clip || unclipped < clipped) {"),
    ("clip_range_upper_bound",
     "    const double rho_bar = fmin(fmax(rho, 1.0 - eps), 1.0 + eps);\n    const double unclipped",
     "    const double rho_bar = fmin(fmax(rho, 1.0 - eps), 1.0 + 2.0 * eps);\n    const double unclipped"),
    ("no_is_loss_without_log_p",
     "total += A * logp;", "total += A;"),
    ("dense_reverse_grad_drops_D",
     "grad[j] = p != 0.0 ? gamma * p * ((logp - logq) - kl) : 0.0;",
     "grad[j] = p != 0.0 ? gamma * p * (logp - logq) : 0.0;"),
    ("dense_forward_log_ratio_flipped",
     "w * (logq - logp)", "w * (logp - logq)"),
    ("truncated_reverse_drops_plus_one",
     "mass += exp(logp) * (logp - tau[i] + 1.0);", "mass += exp(logp) * (logp - tau[i]);"),
    ("log_partition_drops_max",
     "  return m + log(s);", "  return log(s);"),
    ("sample_first_index_at_or_above_u",
     "if (F[j] > ui) {", "if (F[j] >= ui) {"),
    ("topk_ties_by_higher_index",
     "return a->j < b->j ? -1 : (a->j > b->j ? 1 : 0);",
     "return a->j > b->j ? -1 : (a->j < b->j ? 1 : 0);"),
    ("coverage_teacher_mass_rescaled",
     "    sq += exp(tau[i]);\n  }\n  *zp = sp;", "    sq += exp(tau[i] - L);\n  }\n  *zp = sp;"),
    ("diag_variance_biased",
     "  return ss / (n - 1);", "  return ss / n;"),
    ("diag_quantile_rank_floor",
     "int64_t r = (int64_t)ceil(q * (double)n);", "int64_t r = (int64_t)floor(q * (double)n);"),
]

CHILD = r"""
import sys
sys.path.insert(0, %(root)r)
sys.path.insert(0, %(tests)r)
import oracle
oracle._LIB_PATH = %(lib)r
import pytest
sys.exit(pytest.main(["-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"] + %(pins)r))
"""


def run_pins(tmp_path, source):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    src = tmp_path / "opd_oracle.c"
    src.write_text(source)
    shutil.copy(HDR, tmp_path / "opd_oracle.h")
    lib = str(tmp_path / "liboracle.so")
    build = subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", lib, str(src), "-lm"],
                           capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    child = CHILD % {"root": ROOT, "tests": HERE, "lib": lib, "pins": PINS}
    env = dict(os.environ, OMP_NUM_THREADS="4")
    return subprocess.run([sys.executable, "-c", child], capture_output=True, text=True,
                          timeout=900, cwd=str(tmp_path), env=env)


def test_control_unmutated_oracle_passes_the_pins(tmp_path):
    run = run_pins(tmp_path, open(SRC).read())
    assert run.returncode == 0, run.stdout[-3000:]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_a_planted_mistake_fails_a_pin(tmp_path, name, old, new):
    source = open(SRC).read()
    assert source.count(old) >= 1, "mutation %s no longer applies" % name
    run = run_pins(tmp_path, source.replace(old, new, 1))
    assert run.returncode == 1, "%s: pins exit %d\n%s" % (name, run.returncode, run.stdout[-3000:])
