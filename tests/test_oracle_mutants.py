"""Plant plausible mistakes in copies of the oracle and check that the pins
in test_oracle.py catch every one (CPU only; the real oracle is untouched)."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "oracle.cpp")

# (name, exact text in oracle.cpp, replacement)
MUTANTS = [
    ("bias_dropped", "        acc += b[n];\n        s += std::fabs(b[n]);\n      }\n      Y[m * N + n] = acc;",
     "        s += std::fabs(b[n]);\n      }\n      Y[m * N + n] = acc;"),
    ("fwd_weight_transposed", "        double p = X[m * K + k] * W[n * K + k];\n        acc += p;\n        s += std::fabs(p);\n      }\n      if (b) {\n        acc += b[n];\n        s += std::fabs(b[n]);\n      }\n      Y[m * N + n]",
     "        double p = X[m * K + k] * W[k * N + n];\n        acc += p;\n        s += std::fabs(p);\n      }\n      if (b) {\n        acc += b[n];\n        s += std::fabs(b[n]);\n      }\n      Y[m * N + n]"),
    ("dx_sign_flipped", "        double p = g * W[n * K + k];\n        acc[k] += p;",
     "        double p = g * W[n * K + k];\n        acc[k] -= p;"),
    ("dw_upstream_index_swapped", "      double g = dY[m * N + n];\n      for (int64_t k = 0; k < K; ++k) {\n        double p = g * X[m * K + k];",
     "      double g = dY[(m % N) * N + (n % M)];\n      for (int64_t k = 0; k < K; ++k) {\n        double p = g * X[m * K + k];"),
    ("db_off_by_one_row", "    for (int64_t m = 0; m < M; ++m) {\n      acc += dY[m * N + n];",
     "    for (int64_t m = 1; m < M; ++m) {\n      acc += dY[m * N + n];"),
    ("S_without_abs", "        acc += p;\n        s += std::fabs(p);\n      }\n      if (b) {",
     "        acc += p;\n        s += p;\n      }\n      if (b) {"),
    ("broadcast_batch_not_clamped",
     "  for (int i = 0; i < p.nbatch; ++i) off = off * opbatch[i] + (opbatch[i] == 1 ? 0 : idx[i]);",
     "  for (int i = 0; i < p.nbatch; ++i) off = off * opbatch[i] + (opbatch[i] == 1 ? 0 : idx[i] % 2);"),
    ("grad_skips_broadcast_sum", "        for (int64_t bi = 0; bi < nbatch; ++bi) {\n          if (amap[bi] != ai) continue;",
     "        for (int64_t bi = 0; bi < nbatch; ++bi) {\n          if (amap[bi] != ai || bi != amap[bi] * (nbatch / (nabatch ? nabatch : 1))) continue;"),
    ("reduce_keeps_wrong_axis", "    for (int d = 0; d < nout_dims; ++d) j = j * pin[d] + (pin[d] == 1 ? 0 : idx[d]);",
     "    for (int d = 0; d < nout_dims; ++d) j = j * pin[d] + (pin[d] == 1 ? 0 : idx[d] % pin[d]);\n    if (nout_dims > 1 && pin[0] == 1) continue;"),
    ("broadcast_rule_accepts_mismatch", "    else return OR_ERR_SHAPE;\n    out[n - 1 - i] = d;",
     "    else d = da > db ? da : db;\n    out[n - 1 - i] = d;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/found"
    mutated = tmp_path / "oracle_mut.cpp"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mut.so"
    subprocess.run(["g++", "-std=c++17", "-O1", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
                    "-o", str(lib), str(mutated)], check=True)
    env = dict(os.environ, MT_ORACLE_LIB_OVERRIDE=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the oracle pins:\n{r.stdout[-2000:]}"


# planted mistakes in oracle/nn.py, caught by test_oracle_nn.py
NN_SRC = os.path.join(ROOT, "oracle", "nn.py")
MUTANTS_NN = [
    ("gelu_tanh_approximation", "        return z * normal_cdf(z)\n",
     "        return 0.5 * z * (1.0 + np.tanh(0.7978845608028654 * (z + 0.044715 * z ** 3)))\n"),
    ("gelu_grad_drops_pdf_term", "        return normal_cdf(z) + z * normal_pdf(z)\n",
     "        return normal_cdf(z)\n"),
    ("relu_grad_one_at_zero", "        return (z > 0).astype(np.float64)\n",
     "        return (z >= 0).astype(np.float64)\n"),
    ("sigmoid_grad_sign", "        return s * (1.0 - s)\n", "        return s * (1.0 + s)\n"),
    ("tanh_grad_not_squared", "        return 1.0 - t * t\n", "        return 1.0 - t\n"),
    ("act_bwd_evaluates_grad_at_output", "    dZ = dH * act_grad(kind, Z)\n",
     "    dZ = dH * act_grad(kind, act(kind, Z))\n"),
    ("db_skips_first_row", "    for m in range(Z.shape[0]):   # rows in ascending order\n",
     "    for m in range(1, Z.shape[0]):\n"),
    ("mse_sum_not_mean", "    L = float(np.sum(d * d)) / N if N else 0.0\n",
     "    L = float(np.sum(d * d)) if N else 0.0\n"),
    ("mse_grad_missing_two", "    dP = 2.0 * d / N if N else d.copy()\n", "    dP = d / N if N else d.copy()\n"),
    ("sgd_weight_decay_sign", "    v_new = momentum * v + g + weight_decay * theta\n",
     "    v_new = momentum * v + g - weight_decay * theta\n"),
    ("sgd_steps_with_old_velocity", "    theta_new = theta - lr * v_new\n", "    theta_new = theta - lr * v\n"),
    ("adam_no_first_debias", "    bc1 = 1.0 - beta1 ** t\n", "    bc1 = 1.0\n"),
    ("adam_eps_inside_root", "    denom = np.sqrt(vhat) + eps\n", "    denom = np.sqrt(vhat + eps)\n"),
    ("rmsprop_eps_outside_root", "    scale = 1.0 / np.sqrt(v_new + eps)\n",
     "    scale = 1.0 / (np.sqrt(v_new) + eps)\n"),
    ("rmsprop_average_weights_swapped", "    v_new = alpha * v + (1.0 - alpha) * g * g\n",
     "    v_new = (1.0 - alpha) * v + alpha * g * g\n"),
    ("mlp_dW1_skips_activation", "    dW1, _ = _dense.linear_bwd_dw(dZ1, X)\n",
     "    dW1, _ = _dense.linear_bwd_dw(dH1, X)\n"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS_NN, ids=[m[0] for m in MUTANTS_NN])
def test_nn_pins_catch_mutant(tmp_path, name, old, new):
    src = open(NN_SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/found"
    mutated = tmp_path / "nn_mut.py"
    mutated.write_text(src.replace(old, new))
    env = dict(os.environ, MT_ORACLE_NN_OVERRIDE=str(mutated), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_nn.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the oracle pins:\n{r.stdout[-2000:]}"


# planted mistakes in the convolution part of oracle/oracle.cpp, caught by test_oracle_conv.py
MUTANTS_CONV = [
    ("conv_padding_sign", "  double acc = 0.0, s = 0.0;\n  for (int64_t ci = 0; ci < c.C; ++ci)\n    for (int64_t u = 0; u < c.KH; ++u)\n      for (int64_t v = 0; v < c.KW; ++v) {\n        const int64_t h = i * c.sh + u - c.ph,",
     "  double acc = 0.0, s = 0.0;\n  for (int64_t ci = 0; ci < c.C; ++ci)\n    for (int64_t u = 0; u < c.KH; ++u)\n      for (int64_t v = 0; v < c.KW; ++v) {\n        const int64_t h = i * c.sh + u + c.ph,"),
    ("conv_kernel_flipped", "        const double p = w[((co * c.C + ci) * c.KH + u) * c.KW + v] *\n                         x[((n * c.C + ci) * c.H + h) * c.W + xx];",
     "        const double p = w[((co * c.C + ci) * c.KH + (c.KH - 1 - u)) * c.KW + v] *\n                         x[((n * c.C + ci) * c.H + h) * c.W + xx];"),
    ("conv_dx_ignores_stride_phase", "        if (ti < 0 || tj < 0 || ti % c.sh || tj % c.sw) continue;",
     "        if (ti < 0 || tj < 0) continue;"),
    ("conv_dw_kernel_axes_swapped", "        const int64_t h = i * c.sh + u - c.ph, xx = j * c.sw + v - c.pw;\n        if (h < 0 || h >= c.H || xx < 0 || xx >= c.W) continue;\n        const double p = dy[((n * c.CO + co) * c.HO + i) * c.WO + j] *",
     "        const int64_t h = i * c.sh + v - c.ph, xx = j * c.sw + u - c.pw;\n        if (h < 0 || h >= c.H || xx < 0 || xx >= c.W) continue;\n        const double p = dy[((n * c.CO + co) * c.HO + i) * c.WO + j] *"),
    ("conv_db_skips_first_image", "    for (int64_t n = 0; n < c.N; ++n)\n      for (int64_t i = 0; i < c.HO; ++i)\n        for (int64_t j = 0; j < c.WO; ++j) {\n          const double g",
     "    for (int64_t n = 1; n < c.N; ++n)\n      for (int64_t i = 0; i < c.HO; ++i)\n        for (int64_t j = 0; j < c.WO; ++j) {\n          const double g"),
    ("conv_output_size_floor_off", "  c.HO = (c.H + 2 * c.ph - c.KH) / c.sh + 1;", "  c.HO = (c.H + 2 * c.ph - c.KH + c.sh - 1) / c.sh + 1;"),
    ("conv_bias_dropped", "  if (b) {\n    acc += b[co];\n    s += std::fabs(b[co]);\n  }\n  *out = acc;",
     "  if (b) {\n    s += std::fabs(b[co]);\n  }\n  *out = acc;"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS_CONV, ids=[m[0] for m in MUTANTS_CONV])
def test_conv_pins_catch_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/found"
    mutated = tmp_path / "oracle_mut.cpp"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "liboracle_mut.so"
    subprocess.run(["g++", "-std=c++17", "-O1", "-fopenmp", "-ffp-contract=off", "-fPIC", "-shared",
                    "-o", str(lib), str(mutated)], check=True)
    env = dict(os.environ, MT_ORACLE_LIB_OVERRIDE=str(lib), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(HERE, "test_oracle_conv.py")], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"mutant {name} survived the oracle pins:\n{r.stdout[-2000:]}"
