"""Planted mistakes in the oracle, each of which the CPU suite must catch.

Not a test module (pytest does not collect it): a check of the pins
themselves.  Every entry plants one plausible mistake in a copy of the
tree -- a wrong constant, index, sign, operand order or definition in the
random stream, the model, the estimator, the updates or the schedule --
builds that copy's oracle and runs ``pytest -m "not gpu" -x`` on it.  The
oracle is pinned where every planted mistake makes some test fail.

    python tests/oracle_mutants.py            # all of them (about 8 minutes)
    python tests/oracle_mutants.py ID ...     # the named ones
    python tests/oracle_mutants.py --list
"""
import os
import shutil
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
C = "oracle/soma_oracle.c"
PL = "oracle/plateau.py"

# (id, file, text, replacement, the mistake)
MUTANTS = [
    ('philox_9_rounds', C, 'round < 10; ++round',
     'round < 9; ++round',
     'Philox: nine rounds'),
    ('philox_weyl', C, 'k1 += PHILOX_W1;',
     'k1 += PHILOX_W0;',
     'Philox: wrong Weyl increment of k1'),
    ('philox_key_word', C, '(uint32_t)(p1 >> 32) ^ x1 ^ k0;',
     '(uint32_t)(p1 >> 32) ^ x1 ^ k1;',
     'Philox: wrong key word in a round'),
    ('bm_words_swapped', C, 'float lnu = oracle_ln_u24((wa >> 8) + 1u);\n  float r = sqrtf(-2.0f * lnu);\n  float c, s;\n  oracle_sincos_2pi_u24(wb >> 8, &c, &s);',
     'float lnu = oracle_ln_u24((wb >> 8) + 1u);\n  float r = sqrtf(-2.0f * lnu);\n  float c, s;\n  oracle_sincos_2pi_u24(wa >> 8, &c, &s);',
     'Box-Muller: radius and angle words swapped'),
    ('bm_cos_sin_swapped', C, '*za = r * c;\n  *zb = r * s;',
     '*za = r * s;\n  *zb = r * c;',
     'Box-Muller: cos and sin outputs swapped'),
    ('bm_radius_factor', C, 'sqrtf(-2.0f * lnu)',
     'sqrtf(-1.0f * lnu)',
     'Box-Muller: radius sqrt(-ln u) instead of sqrt(-2 ln u)'),
    ('ln_coefficient', C, 'q = fmaf(s2, q, 1.0f / 5.0f);',
     'q = fmaf(s2, q, 1.0f / 6.0f);',
     'ln series: a wrong coefficient'),
    ('ln_scale', C, 'const float n = (float)(e - 24);',
     'const float n = (float)(e - 23);',
     'ln: wrong exponent offset'),
    ('sincos_quadrant', C, 'case 1: c = -sn; s = cs;  break;',
     'case 1: c = sn; s = cs;  break;',
     'sincos: wrong sign in one quadrant'),
    ('sin_coefficient_index', C, 'sp = fmaf(r2, sp, g_sin_c[1]);',
     'sp = fmaf(r2, sp, g_sin_c[2]);',
     'sin series: wrong coefficient index'),
    ('stream_counter_words', C, 'uint32_t ctr[4] = {(uint32_t)q, pair, (uint32_t)step, (uint32_t)(q >> 32)};',
     'uint32_t ctr[4] = {(uint32_t)q, (uint32_t)step, pair, (uint32_t)(q >> 32)};',
     'Gaussian stream: pair and step counter words swapped'),
    ('stream_quad_lane', C, '    out[i] = z[k & 3];\n  }\n}\n\n/* Rademacher',
     '    out[i] = z[(k + 1) & 3];\n  }\n}\n\n/* Rademacher',
     'Gaussian stream: wrong element of the quad'),
    ('rad_word_index', C, 'w[(k >> 4) & 3]',
     'w[(k >> 2) & 3]',
     'Rademacher: wrong word of the block'),
    ('rad_sign_lost', C, 'return (field >> 1) ? sgn : 0.0f;',
     'return (field >> 1) ? 1.0f : 0.0f;',
     'sparse Rademacher: sign dropped'),
    ('rad_dense_uses_sparse', C, 'if (law == 2) return sgn;',
     'if (law == 3) return sgn;',
     'dense Rademacher drawn from the sparse law'),
    ('lstm_gates_f_g_swapped', C, 'double fg = sigmoid(a[H + u]);\n        double gg = tanh(a[2 * H + u]);',
     'double fg = sigmoid(a[2 * H + u]);\n        double gg = tanh(a[H + u]);',
     'LSTM: gate blocks f and g swapped'),
    ('lstm_cell_i_f_swapped', C, 'cl[u] = fg * cl[u] + ig * gg;\n        hl[u] = og * tanh(cl[u]);\n      }\n      for (int u = 0; u < H; ++u) x[u] = hl[u];',
     'cl[u] = ig * cl[u] + fg * gg;\n        hl[u] = og * tanh(cl[u]);\n      }\n      for (int u = 0; u < H; ++u) x[u] = hl[u];',
     'LSTM: input and forget gates swapped in the cell'),
    ('lstm_h_no_tanh', C, 'hl[u] = og * tanh(cl[u]);\n      }\n      for (int u = 0; u < H; ++u) x[u] = hl[u];',
     'hl[u] = og * cl[u];\n      }\n      for (int u = 0; u < H; ++u) x[u] = hl[u];',
     'LSTM: h = o c (tanh dropped)'),
    ('lstm_recurrent_columns', C, 'for (int k = 0; k < H; ++k) acc += wr[xin + k] * hl[k];',
     'for (int k = 0; k < H; ++k) acc += wr[k] * hl[k];',
     'LSTM: recurrent product reads the input columns'),
    ('lstm_no_recurrence', C, 'for (int k = 0; k < H; ++k) acc += wr[xin + k] * hl[k];',
     '',
     'LSTM: recurrent term dropped'),
    ('lstm_layer_input', C, 'for (int u = 0; u < H; ++u) x[u] = hl[u];\n      xin = H;',
     'xin = H;',
     'stacked LSTM: layer l+1 reads the embedding, not h'),
    ('ce_target_index', C, 'total += log(se) + mx - logits[seq[t + 1]];',
     'total += log(se) + mx - logits[seq[t]];',
     'cross entropy: target is the current byte'),
    ('ce_max_dropped', C, 'total += log(se) + mx - logits[seq[t + 1]];',
     'total += log(se) - logits[seq[t + 1]];',
     'cross entropy: max shift not added back'),
    ('ce_mean_over_T', C, 'return total / ((double)B * (double)(T - 1));',
     'return total / ((double)B * (double)T);',
     'loss: mean over B T instead of B (T-1)'),
    ('embedding_next_byte', C, 'const double *erow = emb + (size_t)seq[t] * E;',
     'const double *erow = emb + (size_t)seq[t + 1] * E;',
     'embedding of the target byte'),
    ('head_offset', C, 'const double *head = w + off_layer(c, L);',
     'const double *head = w + off_layer(c, L - 1);',
     'head read from the wrong offset'),
    ('ln_eps', C, '#define LN_EPS 1e-5',
     '#define LN_EPS 1e-6',
     'LayerNorm epsilon 1e-6'),
    ('ln_unbiased_var', C, '  var /= d;',
     '  var /= (d - 1);',
     'LayerNorm: unbiased variance'),
    ('gelu_tanh', C, 'return 0.5 * u * (1.0 + erf(u / sqrt(2.0)));',
     'return 0.5 * u * (1.0 + tanh(0.7978845608028654 * (u + 0.044715 * u * u * u)));',
     'GELU: tanh approximation'),
    ('body_residual_dropped', C, 'for (int k = 0; k < d; ++k) x[k] += hl[k];                 /* residual */\n      layer_norm(x, g2, d, n);                                   /* MLP sublayer */\n      for (int r = 0; r < 4 * d; ++r) {',
     'for (int k = 0; k < d; ++k) x[k] = hl[k];                 /* residual */\n      layer_norm(x, g2, d, n);                                   /* MLP sublayer */\n      for (int r = 0; r < 4 * d; ++r) {',
     'body: LSTM sublayer residual dropped'),
    ('body_mlp_gain', C, 'layer_norm(x, g2, d, n);                                   /* MLP sublayer */\n      for (int r = 0; r < 4 * d; ++r) {',
     'layer_norm(x, g1, d, n);                                   /* MLP sublayer */\n      for (int r = 0; r < 4 * d; ++r) {',
     'body: MLP LayerNorm uses the LSTM gain'),
    ('delta_pre_ln', C, 'for (int k = 0; k < d; ++k) dE[(size_t)v * d + k] += pv * n[k];',
     'for (int k = 0; k < d; ++k) dE[(size_t)v * d + k] += pv * x[k];',
     'delta rule: pre-LayerNorm x instead of f'),
    ('delta_no_onehot', C, 'const double pv = exp(logits[v] - mx) / se - (v == y ? 1.0 : 0.0);\n        for (int k = 0; k < d; ++k)',
     'const double pv = exp(logits[v] - mx) / se;\n        for (int k = 0; k < d; ++k)',
     'delta rule: one-hot term dropped'),
    ('wide_pout_transposed', C, 'acc += n[k] * Pout[(size_t)k * dE_ + q];',
     'acc += n[k] * Pout[(size_t)q * d + k];',
     'wide body: P_out read transposed'),
    ('wide_pin_transposed', C, 'acc += Pin[(size_t)k * dE_ + q] * ey[q];',
     'acc += Pin[(size_t)q * d + k] * ey[q];',
     'wide body: P_in read transposed'),
    ('wide_gain_order', C, 'const double *g1 = gains + 2 * (size_t)l * d, *g2 = g1 + d;',
     'const double *g2 = gains + 2 * (size_t)l * d, *g1 = g2 + d;',
     'wide body: gains g1 and g2 swapped'),
    ('gain_law', C, 'c->probe == 1 && body_is_gain(c, k)) ? 2 : c->probe;',
     'c->probe == 2 && body_is_gain(c, k)) ? 2 : c->probe;',
     'gains not dense under the sparse law'),
    ('gain_positions', C, 'return r < d || (r >= d + 8 * d * d && r < 2 * d + 8 * d * d);',
     'return r < d;',
     'body: g2 not counted as a gain'),
    ('update_sign', C, 'theta_out[i] = (float)((double)theta[k] - (double)lr * g);',
     'theta_out[i] = (float)((double)theta[k] + (double)lr * g);',
     'SGD: update sign flipped'),
    ('update_lr_dropped', C, 'theta_out[i] = (float)((double)theta[k] - (double)lr * g);',
     'theta_out[i] = (float)((double)theta[k] - g);',
     'SGD: lr dropped'),
    ('update_wrong_direction', C, 'probe_quad(law_of(c, k & ~(int64_t)3), seed, step, (uint32_t)j, (uint64_t)k >> 2, z);\n      g += coef[j]',
     'probe_quad(law_of(c, k & ~(int64_t)3), seed, step, (uint32_t)(P - 1 - j), (uint64_t)k >> 2, z);\n      g += coef[j]',
     'update: coefficient j paired with direction P-1-j'),
    ('update_wrong_step', C, 'probe_quad(law_of(c, k & ~(int64_t)3), seed, step, (uint32_t)j, (uint64_t)k >> 2, z);\n      g += coef[j]',
     'probe_quad(law_of(c, k & ~(int64_t)3), seed, step + 1, (uint32_t)j, (uint64_t)k >> 2, z);\n      g += coef[j]',
     'update: probes of the next step'),
    ('coef_no_half', C, 'cf[(size_t)e * P + j] = diff / (2.0 * (double)eps[e] * (double)P);',
     'cf[(size_t)e * P + j] = diff / ((double)eps[e] * (double)P);',
     'coefficient: factor 2 dropped'),
    ('coef_sign', C, 'diff = L[((size_t)e * P + j) * 2 + 0] - L[((size_t)e * P + j) * 2 + 1];',
     'diff = L[((size_t)e * P + j) * 2 + 1] - L[((size_t)e * P + j) * 2 + 0];',
     'coefficient: L- - L+'),
    ('coef_divides_by_P_not_D', C, 'cf[(size_t)e * P + j] = diff / (2.0 * (double)eps[e] * (double)P);',
     'cf[(size_t)e * P + j] = diff / (2.0 * (double)eps[e] * (double)Pb);',
     'accumulation: divides by P instead of A P'),
    ('accum_one_batch', C, 'bytes + ((size_t)(j / Pb) * N + e) * bstride);',
     'bytes + ((size_t)(0) * N + e) * bstride);',
     'accumulation: every direction on batch 0'),
    ('summed_misses_expert', C, 'for (int e2 = 0; e2 < N; ++e2)\n          diff +=',
     'for (int e2 = 0; e2 + 1 < N; ++e2)\n          diff +=',
     'summed loss: last expert left out'),
    ('summed_uses_first_eps', C, 'cf[(size_t)e * P + j] = diff / (2.0 * (double)eps[e] * (double)P);',
     'cf[(size_t)e * P + j] = diff / (2.0 * (double)eps[0] * (double)P);',
     "per-expert radius: expert 0's eps for all"),
    ('separability_seed', C, 'oracle_apply_update(c, theta + (size_t)e * d, seeds[e], step,',
     'oracle_apply_update(c, theta + (size_t)e * d, seeds[0], step,',
     "update regenerates expert 0's probes for every expert"),
    ('mask_ignored', C, 'const uint32_t m = c->perturb_mask ? c->perturb_mask : 7u;',
     'const uint32_t m = 7u;',
     'mask ignored'),
    ('mask_group_boundary', C, '(k < off_layer(c, c->n_layers) ? 1 : 2)',
     '(k <= off_layer(c, c->n_layers) ? 1 : 2)',
     'mask: first head weight counted in the LSTM group'),
    ('mask_update_ignored', C, 'if (!coord_perturbed(c, k)) {          /* masked: no estimate, no update */',
     'if (0) {          /* masked: no estimate, no update */',
     'mask not applied to the update'),
    ('adam_no_bias_correction', C, '(m1 / bc1) / (sqrt(v1 / bc2) + delta)',
     'm1 / (sqrt(v1) + delta)',
     'Adam: bias correction dropped'),
    ('adam_no_decay', C, 'const double g = gh + lambda * th;',
     'const double g = gh;',
     'Adam: weight decay dropped'),
    ('adam_v_not_squared', C, '(1.0 - beta2) * g * g;',
     '(1.0 - beta2) * g * (g > 0 ? g : -g) * 0.5;',
     'Adam: second moment wrong'),
    ('adam_delta_inside', C, '(sqrt(v1 / bc2) + delta)',
     'sqrt(v1 / bc2 + delta)',
     'Adam: delta inside the square root'),
    ('param_count', C, 'if (c->arch == 1) return c->n_layers * body_block(c->hidden) + c->hidden;',
     'if (c->arch == 1) return c->n_layers * body_block(c->hidden) + 2 * c->hidden;',
     'body parameter count off by d'),
    ('head_delta_mean', C, 'for (size_t i = 0; i < (size_t)VOCAB * d; ++i) grad[i] *= inv;',
     '',
     'delta rule: sum instead of mean'),
    ('plateau_threshold', PL, 'if float(v) < float(self.best[e]) - float(self.threshold):',
     'if float(v) < float(self.best[e]):',
     'plateau: threshold ignored'),
    ('plateau_patience', PL, 'if self.since[e] >= self.patience:',
     'if self.since[e] > self.patience:',
     'plateau: decays one update late'),
    ('plateau_floor', PL, 'return min(x, max(f32(x * self.factor), self.floor))',
     'return max(f32(x * self.factor), self.floor)',
     'plateau: a rate below the floor is raised'),
    ('plateau_eps_kept', PL, '                self.eps[e] = self._decay(self.eps[e])\n',
     '',
     'plateau: eps not decayed'),
    ('plateau_since_kept', PL, '                self.eps[e] = self._decay(self.eps[e])\n                self.since[e] = 0\n',
     '                self.eps[e] = self._decay(self.eps[e])\n',
     'plateau: counter not restarted after a decay'),
]

SKIP_DIRS = {".git", "_work", "gpurun_out", "__pycache__", ".pytest_cache", "profiles"}


def plant(dst, mutant):
    mid, rel, old, new, _ = mutant
    path = os.path.join(dst, rel)
    with open(path) as f:
        text = f.read()
    if text.count(old) != 1:
        raise SystemExit("%s: the text to replace occurs %d times in %s" % (mid, text.count(old), rel))
    with open(path, "w") as f:
        f.write(text.replace(old, new))


def run_one(mutant, workdir):
    dst = os.path.join(workdir, mutant[0])
    shutil.copytree(ROOT, dst, ignore=lambda d, names: [n for n in names if n in SKIP_DIRS])
    plant(dst, mutant)
    env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
    b = subprocess.run([sys.executable, "-c", "import oracle; oracle.build(force=True)"], cwd=dst, env=env,
                       capture_output=True, text=True)
    if b.returncode != 0:
        return "BUILD FAILED"
    t = subprocess.run([sys.executable, "-m", "pytest", "tests", "-x", "-q", "-m", "not gpu"], cwd=dst, env=env,
                       capture_output=True, text=True, timeout=900)
    shutil.rmtree(dst, ignore_errors=True)
    if t.returncode == 0:
        return "SURVIVED"
    first = next((ln for ln in t.stdout.splitlines() if ln.startswith(("FAILED", "ERROR"))), "")
    return "caught: " + first.split(" - ")[0]


def main(argv):
    if "--list" in argv:
        for m in MUTANTS:
            print("%-28s %s" % (m[0], m[4]))
        return 0
    chosen = [m for m in MUTANTS if not argv or m[0] in argv]
    survived = []
    with tempfile.TemporaryDirectory(prefix="oracle_mutants_") as work:
        for m in chosen:
            res = run_one(m, work)
            print("%-28s %s" % (m[0], res), flush=True)
            if not res.startswith("caught"):
                survived.append(m[0])
    print("%d planted, %d caught" % (len(chosen), len(chosen) - len(survived)))
    return 1 if survived else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
