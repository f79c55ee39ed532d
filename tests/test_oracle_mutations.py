"""Each plausible mistake planted in a copy of the oracle must make a pin test fail.

The mutated copy lives in a temporary directory placed first on the import path of a
fresh pytest process; the real oracle is never modified.  CPU only.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_TESTS = [os.path.join(ROOT, "tests", f) for f in
             ("test_oracle_fusion.py", "test_oracle_head.py", "test_oracle_accept.py",
              "test_oracle_sampling.py", "test_oracle_adaptive.py")]

MUTATIONS = {
    "prior_sign": ("f = f - weighted(beta, prior)", "f = f + weighted(beta, prior)"),
    "drop_short": ("f = f + weighted(alpha, short_row)", "f = f + 0.0 * np.asarray(short_row, dtype=F64)"),
    "zero_weight_as_product": ("    if w == 0:\n        return np.zeros_like(x)\n", ""),
    "zero_weight_masks_all": ("        return np.zeros_like(x)\n", "        return np.where(np.isneginf(x), x, 0.0)\n"),
    "tie_highest_index": ("return int(np.argmax(np.asarray(fused, dtype=np.float32)))",
                          "a = np.asarray(fused, dtype=np.float32); return int(len(a) - 1 - np.argmax(a[::-1]))"),
    "gate_swap_rz": ("r = sigmoid(gi[:H] + gh[:H])", "r = sigmoid(gi[H:2 * H] + gh[H:2 * H])"),
    "update_swap": ("return (1.0 - z) * n + z * h", "return z * n + (1.0 - z) * h"),
    "reset_on_sum": ("n = np.tanh(gi[2 * H:] + r * gh[2 * H:])", "n = np.tanh(r * (gi[2 * H:] + gh[2 * H:]))"),
    "silu_as_sigmoid": ("return x * sigmoid(x)", "return sigmoid(x)"),
    "no_rank_activation": ("rho = silu(self.w_rank @ h)", "rho = self.w_rank @ h"),
    "no_feedback": ("            u = res.token\n", "            u = int(last_token[b])\n"),
    "lse_no_shift": ("return float(m + np.log(np.sum(np.exp(x - m))))",
                     "return float(m + np.log(np.sum(np.exp(x))))"),
    "score_norm_drop_wlong": ("norm = float(weighted(w_long, lse_l))", "norm = float(lse_l)"),
    "logprob_wrong_lse": ("logprob=float(scaled[tok] - lse_f)", "logprob=float(scaled[tok] - lse_l)"),
    "gap_top1_only": ("return float(top[1] - top[0])", "return float(top[1])"),
    "accept_off_by_one": ("while a < B and draft[b, a] == target[b, a]",
                          "while a < B - 1 and draft[b, a] == target[b, a]"),
    "tau_no_bonus": ("return np.asarray(accepted) + 1", "return np.asarray(accepted)"),
    "literal_row_index": ("if first_row_long_only and j == 0:", "if first_row_long_only and j == 1:"),
    "prior_no_smoothing": ("c = np.asarray(counts, dtype=F64) + F64(smoothing)",
                           "c = np.asarray(counts, dtype=F64) + F64(0.0)"),
    "state_carried_across_rows": ("                state, s = head.step(state, u)",
                                  "                state, s = head.step(head.init_state(), u)"),
    "gain_ratio_denominator": ("(tau_dels - tau_base) / (tau_joint - tau_base)",
                               "(tau_dels - tau_base) / (tau_joint)"),
    "philox_multiplier_swap": ("p0 = np.uint64(PHILOX_M0) * c[0]", "p0 = np.uint64(PHILOX_M1) * c[0]"),
    "philox_no_key_bump": ("k0 = (k0 + np.uint64(PHILOX_W0)) & m", "k0 = k0 & m"),
    "gumbel_single_log": ("return -np.log(-np.log(uniforms_row(seed, b, j, V)))",
                          "return -np.log(uniforms_row(seed, b, j, V))"),
    "temperature_ignored": ("scaled = fused / F64(temperature)", "scaled = fused"),
    "entropy_sign": ("return float(-np.sum(p[keep] * logp[keep]))", "return float(np.sum(p[keep] * logp[keep]))"),
    "entropy_over_v": ("return long_entropy(long_row) / np.log(F64(V))", "return long_entropy(long_row) / F64(V)"),
    "maxprob_unnormalised": ("return (1.0 - long_max_prob(long_row)) / (1.0 - 1.0 / F64(V))",
                             "return 1.0 - long_max_prob(long_row)"),
    "gate_unclamped": ("return float(min(1.0, max(0.0, (F64(u) - h_lo) / (F64(h_hi) - h_lo))))",
                       "return float((F64(u) - h_lo) / (F64(h_hi) - h_lo))"),
    "gate_alpha_only": ("_at(beta, j) * gf,", "_at(beta, j),"),
    "gate_of_first_sequence": ("float(gates[b, j])", "float(gates[0, j])"),
    "uniform_no_half": ("return ((x >> np.uint64(9)).astype(F64) + 0.5) * 2.0 ** -23",
                        "return ((x >> np.uint64(9)).astype(F64)) * 2.0 ** -23"),
}


def _run_pins(tmp_path, old=None, new=None):
    src = open(os.path.join(ROOT, "oracle", "dels_oracle.py")).read()
    pkg = tmp_path / "oracle"
    shutil.copytree(os.path.join(ROOT, "oracle"), pkg,
                    ignore=shutil.ignore_patterns("__pycache__", "*.so", "*.o"))
    if old is not None:
        assert src.count(old) >= 1, "mutation anchor not found"
        src = src.replace(old, new)
    # a sentinel proves the copy (not the real oracle) is the one imported
    (pkg / "dels_oracle.py").write_text(src + "\nMUTANT_COPY = True\n")
    env = dict(os.environ, PYTHONPATH=f"{tmp_path}{os.pathsep}{ROOT}",
               PYTHONDONTWRITEBYTECODE="1")
    check = subprocess.run([sys.executable, "-c", "import oracle.dels_oracle as O; print(O.MUTANT_COPY)"],
                           cwd=tmp_path, env=env, capture_output=True, text=True, timeout=120)
    assert check.stdout.strip() == "True", check.stderr
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "-m", "not gpu", *PIN_TESTS],
                          cwd=tmp_path, env=env, capture_output=True, text=True, timeout=600)


def test_unmutated_copy_passes(tmp_path):
    proc = _run_pins(tmp_path)
    assert proc.returncode == 0, proc.stdout[-2000:]


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_mutation(name, tmp_path):
    old, new = MUTATIONS[name]
    proc = _run_pins(tmp_path, old, new)
    assert proc.returncode != 0, f"mutation {name} survived the pins:\n{proc.stdout[-2000:]}"
