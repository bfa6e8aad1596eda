"""The oracle's pins must catch plausible mistakes.  Each case plants one error
into a temporary copy of the oracle (on the CPU only) and runs the pin suite
against that copy; the suite has to fail."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, original text, planted mistake)
MUTATIONS = [
    ("lut_sign", "e = q[m * dsub + j] - C[m, :, j]", "e = q[m * dsub + j] + C[m, :, j]"),
    ("lut_drops_weight", "acc = acc + w[m * dsub + j] * (e * e)", "acc = acc + (e * e)"),
    ("lut_wrong_subdim", "w[m * dsub + j] * (e * e)", "w[m * dsub] * (e * e)"),
    ("delta_wrong_index", "delta = delta + alpha[m, t] * W[m, t]", "delta = delta + alpha[t % M, m % r] * W[m, t]"),
    ("delta_dropped", "C[m] = C_pq[m] + delta", "C[m] = C_pq[m]"),
    ("adc_transposed", "d = d + lut[m][codes[ids, m]].astype(dtype)", "d = d + lut[m][codes[m % codes.shape[0], ids % codes.shape[1]]].astype(dtype)"),
    ("topk_tie_larger_id", "order = np.lexsort((ids, d))[:k]", "order = np.lexsort((-ids, d))[:k]"),
    ("filter_closed_hi", "mask &= (a >= lo) & (a < hi)", "mask &= (a >= lo) & (a <= hi)"),
    ("bitmap_msb_first", "(idx & 31).astype(np.uint32)", "(31 - (idx & 31)).astype(np.uint32)"),
    ("softplus_plain_exp", "y[~big] = np.log1p(np.exp(x[~big]))", "y[~big] = np.exp(x[~big])"),
    ("fnv_wrong_order", "h ^= byte\n        h = (h * _FNV_PRIME) & _MASK64", "h = (h * _FNV_PRIME) & _MASK64\n        h ^= byte"),
    ("alpha_single_row", "for r_i in rows:", "for r_i in rows[:1]:"),
    ("fingerprint_no_clauses", "out.append(struct.pack(\"<iqq\", int(col), int(lo), int(hi)))", "pass"),
    ("exact_abs_not_square", "        d = d + e * e\n", "        d = d + np.abs(e)\n"),
    ("exact_drops_last_dim", "    for j in range(x.shape[1]):\n        e = x[ids, j]", "    for j in range(x.shape[1] - 1):\n        e = x[ids, j]"),
    ("sdc_encode_last_minimum", "        codes[m] = int(np.argmin(acc))          # first minimum", "        codes[m] = int(K - 1 - np.argmin(acc[::-1]))"),
    ("sdc_table_transposed_subspace", "            e = C[m, :, j][:, None] - C[m, :, j][None, :]", "            e = C[m, :, j][:, None] - C[(m + 1) % M, :, j][None, :]"),
    ("sdc_lut_data_row", "    lut = T[np.arange(T.shape[0]), codes]", "    lut = T[np.arange(T.shape[0]), (codes + 1) % T.shape[1]]"),
    ("reconstruct_wrong_subspace", "    return np.concatenate([C[m][codes[:, m]] for m in range(M)], axis=1)", "    return np.concatenate([C[m][codes[:, (m + 1) % M]] for m in range(M)], axis=1)"),
    ("hash_mask_not_modulus", "rows.append(splitmix64(key ^ salt) % n_rows)",
     "rows.append(splitmix64(key ^ salt) & (n_rows - 1))"),
    ("hash_salt_seed_xor_index", "salt = splitmix64((hash_seed + i) & _MASK64)",
     "salt = splitmix64((hash_seed ^ i) & _MASK64)"),
    ("exact_query_index_shift", "        e = x[ids, j].astype(dtype) - q[j]", "        e = x[ids, j].astype(dtype) - q[(j + 1) % q.shape[0]]"),
]


# Planted mistakes in the training oracle, caught by its own pins.
TRAIN_MUTATIONS = [
    ("train_anchor_factor", "(lam * 2.0 / (M * K * d) / nq)", "(lam / (M * K * d) / nq)"),
    ("train_table_grad_sign", 'g_delta = g_lut[:, :, None] * (-2.0 * wm * f["e"])',
     'g_delta = g_lut[:, :, None] * (2.0 * wm * f["e"])'),
    ("train_positive_share", 'g_s = f["p"] - f["pos"] / f["n_pos"]', 'g_s = f["p"] - f["pos"]'),
    ("train_alpha_wrong_direction", 'g_alpha = np.einsum("mcj,mtcj->mt", g_delta, W.astype(np.float64)).reshape(M * r)',
     'g_alpha = np.einsum("mcj,mtcj->tm", g_delta, W.astype(np.float64)).reshape(M * r)'),
    ("train_bank_first_row_only", 'for row in f["rows"]:', 'for row in f["rows"][:1]:'),
    ("train_wz_no_softplus_slope", "g_wz[i] = g_w * _sigmoid(np.asarray(w_z, dtype=np.float64))", "g_wz[i] = g_w"),
    ("train_temperature_dropped", "g_dist = -g_s / tau / nq", "g_dist = -g_s / nq"),
]


# Planted mistakes in the predicate-encoder oracle, caught by its pins.
ENCODER_MUTATIONS = [
    ("enc_softmax_over_queries", "A = _softmax_rows((Q[:, sl] @ K[:, sl].T) / np.sqrt(dtype(dh)))",
     "A = _softmax_rows((K[:, sl] @ Q[:, sl].T) / np.sqrt(dtype(dh))).T"),
    ("enc_unscaled_scores", "A = _softmax_rows((Q[:, sl] @ K[:, sl].T) / np.sqrt(dtype(dh)))",
     "A = _softmax_rows(Q[:, sl] @ K[:, sl].T)"),
    ("enc_heads_share_values", "O[:, sl] = A @ V[:, sl]", "O[:, sl] = A @ V[:, :dh]"),
    ("enc_attention_residual_dropped", 'X = X + O @ f("Wo") + f("bo")', 'X = O @ f("Wo") + f("bo")'),
    ("enc_ffn_without_relu", 'Hd = np.maximum(Z @ f("W1") + f("b1"), dtype(0))', 'Hd = Z @ f("W1") + f("b1")'),
    ("enc_layer_norm_without_eps", "np.sqrt(var + dtype(LN_EPS))", "np.sqrt(var)"),
    ("enc_summary_token_last", 'z = layer_norm(X[0], enc["lnf_g"]', 'z = layer_norm(X[-1], enc["lnf_g"]'),
    ("enc_bounds_swapped", "rows.append(ce[int(cl[0])] + a * fw[0] + b * fw[1] + fb)",
     "rows.append(ce[int(cl[0])] + b * fw[0] + a * fw[1] + fb)"),
    ("enc_bounds_unclipped", "a = min(max((float(lo) - off) * sc, -1.0), 2.0)", "a = (float(lo) - off) * sc"),
]


def _run_pins_on_copy(tmp_path, old, new, target="ifvs_oracle.py", pins="test_oracle_pins.py"):
    src = os.path.join(ROOT, "oracle", target)
    text = open(src).read()
    assert old in text, f"mutation text {old!r} no longer applies; update it"
    dst = tmp_path / "oracle"
    shutil.copytree(os.path.join(ROOT, "oracle"), dst,
                    ignore=shutil.ignore_patterns("__pycache__"))
    (dst / target).write_text(text.replace(old, new, 1))
    tests = tmp_path / "tests"
    tests.mkdir()
    shutil.copy(os.path.join(ROOT, "tests", pins), tests)
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tests / "golden")
    # The copy comes first on the path; the seeded input generators come
    # from the repository (they hold none of the oracle's arithmetic).
    env = dict(os.environ, PYTHONPATH=os.pathsep.join([str(tmp_path), ROOT]), PYTHONDONTWRITEBYTECODE="1")
    proc = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                           str(tests / pins)],
                          cwd=tmp_path, env=env, capture_output=True, text=True, timeout=300)
    return proc


def test_unmutated_copy_passes(tmp_path):
    old = MUTATIONS[0][1]
    proc = _run_pins_on_copy(tmp_path, old, old)
    assert proc.returncode == 0, proc.stdout[-2000:]


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new):
    proc = _run_pins_on_copy(tmp_path, old, new)
    assert proc.returncode == 1, f"planted mistake {name} went unnoticed:\n{proc.stdout[-2000:]}"


def test_unmutated_train_copy_passes(tmp_path):
    old = TRAIN_MUTATIONS[0][1]
    proc = _run_pins_on_copy(tmp_path, old, old, "ifvs_train_oracle.py", "test_oracle_train.py")
    assert proc.returncode == 0, proc.stdout[-2000:]


@pytest.mark.parametrize("name,old,new", TRAIN_MUTATIONS, ids=[m[0] for m in TRAIN_MUTATIONS])
def test_train_pins_catch_planted_mistake(tmp_path, name, old, new):
    proc = _run_pins_on_copy(tmp_path, old, new, "ifvs_train_oracle.py", "test_oracle_train.py")
    assert proc.returncode == 1, f"the training pins did not catch {name}:\n{proc.stdout[-2000:]}"


def test_unmutated_encoder_copy_passes(tmp_path):
    old = ENCODER_MUTATIONS[0][1]
    proc = _run_pins_on_copy(tmp_path, old, old, "ifvs_encoder_oracle.py", "test_oracle_encoder.py")
    assert proc.returncode == 0, proc.stdout[-2000:]


@pytest.mark.parametrize("name,old,new", ENCODER_MUTATIONS, ids=[m[0] for m in ENCODER_MUTATIONS])
def test_encoder_pins_catch_planted_mistake(tmp_path, name, old, new):
    proc = _run_pins_on_copy(tmp_path, old, new, "ifvs_encoder_oracle.py", "test_oracle_encoder.py")
    assert proc.returncode == 1, f"the encoder pins did not catch {name}:\n{proc.stdout[-2000:]}"
