"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a wrong
divisor, a flipped sign, an off-by-one boundary, a wrong constant, a swapped
comparison), builds it, and runs the pin suite (tests/test_oracle_pins.py)
against that build in a subprocess.  At least one pin must fail for every
planted mistake; the pins named here are among those that do.  CPU only: the
mistakes live in the oracle's copy, never in the library.
"""
import os
import re
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle.oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

# (name, original text, planted text, a pin expected to catch it)
MUTATIONS = [
    ("variance divided by K-1",
     "        var_out[tau] = acc / (double)K;\n    }\n#pragma omp parallel for schedule(static)",
     "        var_out[tau] = acc / (double)(K - 1);\n    }\n#pragma omp parallel for schedule(static)",
     "test_variance_identity_in_long_double"),
    ("replica mean divided by K-1",
     "        xbar[j] = s / (double)K;\n    }\n#pragma omp parallel for schedule(dynamic, 1)",
     "        xbar[j] = s / (double)(K - 1);\n    }\n#pragma omp parallel for schedule(dynamic, 1)",
     "test_average_broadcasts_mean_and_is_idempotent"),
    ("gradient noise with the wrong sign",
     "double g = h[j] * (xk[j] - xs[j]) + pb->sigma * z;",
     "double g = h[j] * (xk[j] - xs[j]) - pb->sigma * z;",
     "test_exact_rational_run_bounds_rounding"),
    ("weight decay with the wrong sign",
     "double d = g + pb->weight_decay * xk[j];",
     "double d = g - pb->weight_decay * xk[j];",
     "test_noise_free_run_is_heavy_ball_closed_form"),
    ("momentum with dampening",
     "vk[j] = pb->momentum * vk[j] + d;",
     "vk[j] = pb->momentum * vk[j] + (1.0 - pb->momentum) * d;",
     "test_noise_free_run_is_heavy_ball_closed_form"),
    ("step taken along +v",
     "xk[j] = xk[j] - gamma * vk[j];",
     "xk[j] = xk[j] + gamma * vk[j];",
     "test_noise_free_run_is_heavy_ball_closed_form"),
    ("momentum averaged at every sync",
     "if (pb->avg_momentum && v) {",
     "if (v) {",
     "test_sync_variance_matches_closed_form"),
    ("growth band compares the wrong way",
     "} else if (S < pb->thr_lo * gamma * st->C2) {",
     "} else if (S > pb->thr_lo * gamma * st->C2) {",
     "test_controller_band_keeps_period"),
    ("C2 keeps the last sample, not the running mean",
     "st->C2 += (S / gamma - st->C2) / (double)st->nC2;",
     "st->C2 = S / gamma;",
     "test_controller_sampling_phase_keeps_p_and_averages"),
    ("period allowed to reach 0",
     "if (st->p > 1) st->p -= 1;",
     "st->p -= 1;",
     "test_controller_huge_variance_clamps_period_at_one"),
    ("period growth ignores the cap",
     "if (pb->p_max <= 0 || st->p < pb->p_max) st->p += 1;",
     "st->p += 1;",
     "test_controller_period_cap"),
    ("sync one step late",
     "return st->cnt >= st->p;",
     "return st->cnt > st->p;",
     "test_sync_counts_match_paper"),
    ("first LR decay one step late",
     "if (t >= pb->total_steps / 2) g *= 0.1;",
     "if (t > pb->total_steps / 2) g *= 0.1;",
     "test_learning_rate_step_decay_matches_paper"),
    ("cosine LR without the half",
     "return pb->lr0 * 0.5 * (1.0 + cos(ORC_PI * (double)t / N));",
     "return pb->lr0 * (1.0 + cos(ORC_PI * (double)t / N));",
     "test_learning_rate_cosine_special_points"),
    ("Box-Muller angle in the wrong function",
     "*z0 = radius * cos(2.0 * ORC_PI * u2);",
     "*z0 = radius * sin(2.0 * ORC_PI * u2);",
     "test_box_muller_special_values"),
    ("Box-Muller radius without the factor 2",
     "double radius = sqrt(-2.0 * log(u1));",
     "double radius = sqrt(-log(u1));",
     "test_normals_are_standard_normal"),
    ("Philox multiplier typo",
     "PH_M0 = 0xD2511F53u",
     "PH_M0 = 0xD2511F55u",
     "test_philox_known_answers"),
    ("curvature uniform instead of log-uniform",
     "h[j] = exp(log(pb->h_lo) + u * (log(pb->h_hi) - log(pb->h_lo)));",
     "h[j] = pb->h_lo + u * (pb->h_hi - pb->h_lo);",
     "test_problem_data_laws"),
    ("mean trajectory driven by the summed noise",
     "double zbar = zsum[j] / (double)pb->K;",
     "double zbar = zsum[j];",
     "test_mean_trajectory_is_schedule_independent"),
]


def _failed_pins(name, old, new, tmp):
    src = open(O._SRC).read()
    assert src.count(old) == 1, f"{name}: the original text must occur exactly once"
    tag = re.sub(r"\W+", "_", name)
    path = os.path.join(tmp, f"orc_{tag}.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = O.build_oracle(path, os.path.join(tmp, f"liborc_{tag}.so"))
    env = dict(os.environ, ADPSGD_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(HERE, "test_oracle_pins.py"),
                        "-q", "-rf", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    failed = set(re.findall(r"^FAILED \S+::(\w+)", r.stdout, re.M))
    return r.returncode, failed, r.stdout[-3000:]


@pytest.mark.slow
def test_every_planted_oracle_mistake_fails_a_pin():
    with tempfile.TemporaryDirectory(prefix="orc_mut_") as tmp:
        with ThreadPoolExecutor(max_workers=4) as ex:
            results = list(ex.map(lambda m: _failed_pins(m[0], m[1], m[2], tmp), MUTATIONS))
    missed = []
    for (name, _, _, pin), (rc, failed, tail) in zip(MUTATIONS, results):
        if rc == 0 or not failed:
            missed.append(f"{name}: no pin failed\n{tail}")
        elif pin not in failed:
            missed.append(f"{name}: {pin} did not fail (failed: {sorted(failed)})")
    assert not missed, "\n".join(missed)
