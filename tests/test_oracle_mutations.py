"""The oracle's pins catch plausible mistakes (CPU).

Each case plants one mistake in a scratch copy of the oracle (Python or C), rebuilds the copy's C
part and runs tests/test_oracle_pins.py against it: some pin must fail. The mistakes are ones a
reading of the paper could plausibly make: a rounding rule, a constant of the method, a region
boundary of NITRO-ReLU or its backward, an operand or index of a block's back-propagation, a
rate of IntegerSGD, the orientation of a convolution tap. Nothing here touches a GPU or the
library; the copies live under pytest's temporary directory and run in parallel subprocesses.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PY = "oracle/oracle.py"
C = "oracle/nitro_oracle.c"

# (name, what the mistake misreads, file, text, replacement); each text occurs once
MUTATIONS = [
    ("inner_relu_grad_layer", "ReLU' of an inner layer taken at its own z* instead of the layer below (section 3.3)",
     PY, "nitro_relu_grad(dx, rec.layers[j - 1].zs,", "nitro_relu_grad(dx, rec.layers[j].zs,"),
    ("head_rate", "output layer updated with gamma^fw instead of gamma^lr (Eq. 6 applies to forward layers)",
     PY, "new_w[h] = integer_sgd(self.w[h], step.head_dw, hp.gamma_inv,",
     "new_w[h] = integer_sgd(self.w[h], step.head_dw, hp.gamma_fw,"),
    ("trunc_as_floor", "rounding toward zero computed as the floor macro (the truncation of section 3.3.3's text)",
     PY, "return np.sign(a) * (np.abs(a) // b)", "return a // b"),
    ("one_hot_31", "one-hot target value 31 instead of 32 (section 3.3.4, Appendix A)",
     PY, "y[np.arange(labels.shape[0]), labels] = 32", "y[np.arange(labels.shape[0]), labels] = 31"),
    ("af_2_5", "amplification factor 2^5 G instead of 2^6 G (Eq. 6)",
     PY, "return (1 << 6) * G", "return (1 << 5) * G"),
    ("pool_last_max", "2x2 max-pool picking the last maximum of a window",
     PY, "    idx = np.argmax(v, axis=3)                # numpy returns the first occurrence of the maximum",
     "    idx = 3 - np.argmax(v[:, :, :, ::-1, :], axis=3)"),
    ("sf_k_not_k2", "conv scaling factor with K instead of K^2 (section 3.2.1)",
     PY, "return (1 << 8) * k * k * c_prev", "return (1 << 8) * k * c_prev"),
    ("relu_mu_64", "NITRO-ReLU mean with segment mean 64 instead of 63 (section 3.2.2)",
     PY, "int(idiv(-127, 2 * alpha_inv, mode)), 63, 127]", "int(idiv(-127, 2 * alpha_inv, mode)), 64, 127]"),
    ("relu_grad_leaky_bound", "backward leaky region without z* = -127",
     PY, "out = np.where((zs < 0) & (zs >= -127), slope, out)", "out = np.where((zs < 0) & (zs > -127), slope, out)"),
    ("relu_grad_pass_bound", "backward pass region without z* = 127",
     PY, "out = np.where((zs >= 0) & (zs <= 127), delta, 0)", "out = np.where((zs >= 0) & (zs < 127), delta, 0)"),
    ("sgd_decay_sign", "weight decay added instead of subtracted (Alg. 1)",
     PY, "return check_int32(w - (idiv(dw, gamma_inv, mode) + decay), \"updated weights\")",
     "return check_int32(w - (idiv(dw, gamma_inv, mode) - decay), \"updated weights\")"),
    ("learning_sf_from_g", "learning layer scaled by 2^8 G instead of 2^8 d (section 3.2.1)",
     PY, "nitro_scaling(z, scaling_factor_linear(w_lr.shape[1]), mode), \"yhat\")",
     "nitro_scaling(z, scaling_factor_linear(w_lr.shape[0]), mode), \"yhat\")"),
    ("loss_grad_sign", "RSS gradient y - yhat instead of yhat - y (Eq. 4)",
     PY, "return np.asarray(yhat, dtype=np.int64) - one_hot32(labels, G)",
     "return one_hot32(labels, G) - np.asarray(yhat, dtype=np.int64)"),
    ("learning_pool_width_first", "learning-pool window halving the width first",
     PY, "if (turn_h and can_h) or not can_w:", "if (not turn_h and can_h) or not can_w:"),
    ("relu_clamp_128", "NITRO-ReLU clamping negatives at -128 instead of -127 (section 3.2.2)",
     PY, "neg = idiv(np.maximum(zs, -127), alpha_inv, mode) - mu", "neg = idiv(np.maximum(zs, -128), alpha_inv, mode) - mu"),
    ("eta_is_lambda", "decay divisor lambda instead of gamma lambda (Alg. 1)",
     PY, "eta = gamma_inv * lambda_inv if eta_inv < 0 else eta_inv", "eta = lambda_inv if eta_inv < 0 else eta_inv"),
    ("forward_rate", "forward layers updated with gamma instead of AF gamma (Eq. 6)",
     PY, "new_w[k] = integer_sgd(self.w[k], rec.dw[j], hp.gamma_fw,",
     "new_w[k] = integer_sgd(self.w[k], rec.dw[j], hp.gamma_inv,"),
    ("dropout_threshold", "dropout threshold on a 31-bit scale",
     PY, "return (p_ppm << 32) // 1000000", "return (p_ppm << 31) // 1000000"),
    ("relu_pos_clamp_126", "NITRO-ReLU clamping positives at 126",
     PY, "pos = np.minimum(zs, 127) - mu", "pos = np.minimum(zs, 126) - mu"),
    ("relu_grad_slope", "leaky segment's gradient not divided by alpha_inv",
     PY, "slope = delta if ste else idiv(delta, alpha_inv, mode)", "slope = delta"),
    ("conv_fwd_flipped", "forward as a convolution (flipped taps) instead of a correlation",
     C, "                        int hh = h + r - 1;\n                        if (hh < 0 || hh >= H) continue;\n"
        "                        for (int s = 0; s < 3; s++) {\n                            int ww = w + s - 1;\n"
        "                            if (ww < 0 || ww >= W) continue;\n"
        "                            const int8_t *xp = x + (((int64_t)n * H + hh) * W + ww) * C;\n"
        "                            const int32_t *wp",
     "                        int hh = h - r + 1;\n                        if (hh < 0 || hh >= H) continue;\n"
     "                        for (int s = 0; s < 3; s++) {\n                            int ww = w - s + 1;\n"
     "                            if (ww < 0 || ww >= W) continue;\n"
     "                            const int8_t *xp = x + (((int64_t)n * H + hh) * W + ww) * C;\n"
     "                            const int32_t *wp"),
    ("conv_dx_unflipped", "input gradient without the adjoint's flipped taps",
     C, "int ho = h - r + 1;", "int ho = h + r - 1;"),
    ("conv_dw_col_flipped", "weight gradient with the column tap flipped",
     C, "                            int ww = w + s - 1;\n                            if (ww < 0 || ww >= W) continue;\n"
        "                            const int8_t *xp = x + (((int64_t)n * H + hh) * W + ww) * C;\n"
        "                            int64_t *op",
     "                            int ww = w - s + 1;\n                            if (ww < 0 || ww >= W) continue;\n"
     "                            const int8_t *xp = x + (((int64_t)n * H + hh) * W + ww) * C;\n"
     "                            int64_t *op"),
]


def _run(base: str, mutation) -> tuple:
    name, _, f, old, new = mutation
    d = os.path.join(base, name)
    for sub in ("tests", "oracle", "paper_2407_11698_amd"):
        shutil.copytree(os.path.join(ROOT, sub), os.path.join(d, sub),
                        ignore=shutil.ignore_patterns("__pycache__", "*.so", "csrc"))
    p = os.path.join(d, f)
    s = open(p).read()
    if s.count(old) != 1:
        return False, "the text to replace occurs %d times" % s.count(old)
    open(p, "w").write(s.replace(old, new))
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "tests/test_oracle_pins.py", "-q", "-x",
                        "-p", "no:cacheprovider"], cwd=d, env=env, stdout=subprocess.PIPE,
                       stderr=subprocess.STDOUT, text=True, timeout=600)
    failed = [l for l in r.stdout.splitlines() if l.startswith("FAILED") or l.startswith("ERROR")]
    return r.returncode != 0, (failed[0] if failed else r.stdout.strip().splitlines()[-1])


# the control: an unchanged copy (the text replaced by itself) passes every pin, so a mutant's
# failure comes from its mistake and not from the copying
CONTROL = ("unchanged", "nothing", PY, "return (1 << 6) * G", "return (1 << 6) * G")


@pytest.fixture(scope="module")
def outcomes(tmp_path_factory):
    base = str(tmp_path_factory.mktemp("mutants"))
    cases = MUTATIONS + [CONTROL]
    with ThreadPoolExecutor(max_workers=max(1, min(6, (os.cpu_count() or 2) - 1))) as ex:
        res = list(ex.map(lambda m: _run(base, m), cases))
    return {m[0]: r for m, r in zip(cases, res)}


@pytest.mark.slow
def test_unchanged_copy_passes(outcomes):
    failed, detail = outcomes[CONTROL[0]]
    assert not failed, "an unchanged copy of the oracle fails its pins: %s" % detail


@pytest.mark.slow
@pytest.mark.parametrize("mutation", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(outcomes, mutation):
    caught, detail = outcomes[mutation[0]]
    assert caught, "a copy of the oracle with this mistake passes every pin (%s): %s" % (mutation[1], detail)
