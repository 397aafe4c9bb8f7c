"""The pins catch planted slips: each case changes one line of a copy of the oracle's C source (a sign,
an index, an offset, a constant, a dropped term) and runs the pins that should notice; at least one of
them must fail.  Nothing here runs on the GPU, and the repository's own oracle is never modified.

Each case builds its own oracle copy with gcc and runs one pin file with -x, so the whole module takes
a minute or two on the CPU.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PINS = "tests/test_oracle_pins.py"
KAPPA = "tests/test_oracle_kappa_causal.py"
SNIS = "tests/test_oracle_snis.py"
BWD = "tests/test_oracle_backward.py"

# (pin file, original line fragment, planted slip); each fragment occurs exactly once in the source
MUTATIONS = [
    # Algorithm 1: propagation, random search, tie rule, random numbers
    (PINS, "int64_t r = nb / P->Wk - ox;", "int64_t r = nb / P->Wk + ox;"),
    (PINS, "static const int jumps[4] = {8, 4, 2, 1};", "static const int jumps[4] = {4, 4, 2, 1};"),
    (PINS, "return sa > sb || (sa == sb && ia < ib);", "return sa > sb || (sa == sb && ia > ib);"),
    (PINS, "int64_t u = st->cur / P->Wk, v = st->cur % P->Wk;",
     "int64_t u = J_prev[g] / P->Wk, v = J_prev[g] % P->Wk;"),
    (PINS, "D /= 2;", "D = D / 2 + (D > 2);"),
    (PINS, "uint32_t w_row = w[2 * (k % 2)], w_col = w[2 * (k % 2) + 1];",
     "uint32_t w_row = w[2 * (k % 2) + 1], w_col = w[2 * (k % 2)];"),
    (PINS, "k0 += PHILOX_WEYL_A;", "k0 += PHILOX_WEYL_B;"),
    (PINS, "int64_t u = pick_in_range(w[0], 0, Hk - 1);", "int64_t u = pick_in_range(w[0], 0, Wk - 1);"),
    (PINS, "for (int jj = 0; jj < 4; ++jj) {", "for (int jj = 0; jj < 3; ++jj) {"),
    # the near-tie flag that decides which GPU map differences are excused
    (PINS, "if (fabs(sc - st->best) <= P->tie_rel * scale) st->tie = 1;", "st->tie = 1;"),
    (PINS, "if (fabs(sc - st->best) <= P->tie_rel * scale) st->tie = 1;",
     "if (fabs(sc - st->best) <= 10 * P->tie_rel * scale) st->tie = 1;"),
    (PINS, "if (idx != st->cur && st->best != -INFINITY) {", "if (st->best != -INFINITY) {"),
    (PINS, "double scale = a > st->best_abs ? a : st->best_abs;",
     "double scale = fabs(sc) > fabs(st->best) ? fabs(sc) : fabs(st->best);"),
    (PINS, "static const int dirs[4][2] = {{-1, 0}, {1, 0}, {0, -1}, {0, 1}};",
     "static const int dirs[4][2] = {{-1, 0}, {1, 0}, {0, -1}, {0, -1}};"),
    # Algorithm 2: window edges, scale, softmax
    (PINS, "int64_t r = u + a, col = v + c;", "int64_t r = u + a, col = v + c + 1;"),  # window off centre
    (PINS, "double w = exp(scale * dot", "double w = exp(dot"),
    (PINS, "if (sc > m) m = sc;", "if (sc > m) m = sc + 0.5;"),
    # several matches and causal masking
    (KAPPA, "if (cheb < P->sep) return 0;", "if (cheb <= P->sep) return 0;"),
    (KAPPA, "if ((P->flags & OR_CAUSAL) && idx > g % plane) return 0;",
     "if ((P->flags & OR_CAUSAL) && idx >= g % plane) return 0;"),
    (KAPPA, "uint32_t ctr[4] = {(uint32_t)g, 0u, 0u, (uint32_t)n_prev};",
     "uint32_t ctr[4] = {(uint32_t)g, 0u, 0u, 0u};"),
    (KAPPA, "idx = pick_in_range(w[0], 0, g % plane);", "idx = pick_in_range(w[0], 0, g % plane + 1);"),
    (KAPPA, "for (int64_t f = 0; f < e && !seen; ++f) seen = in_window(r, col, J[f * n + g], Wk, b);",
     "for (int64_t f = 0; f < e && !seen; ++f) seen = 0;"),
    # importance sampling
    (SNIS, "return a / (double)kappa * local + (1.0 - a) / (double)(Hk * Wk);",
     "return a * local + (1.0 - a) / (double)(Hk * Wk);"),
    (SNIS, "if (r == 0) return offset_cdf(-centre, m);", "if (r == 0) return offset_pmf(-centre, m);"),
    (SNIS, "if (r == len - 1) return offset_cdf(centre - (len - 1), m);",
     "if (r == len - 1) return offset_cdf(len - 1 - centre, m);"),
    (SNIS, "return choose(2 * m, (int)(delta + m)) / ldexp(1.0, 2 * m);",
     "return choose(2 * m, (int)(delta + m)) / ldexp(1.0, 2 * m + 1);"),
    (SNIS, "if ((int)(w[0] >> 16) < alpha_q16(alpha)) {", "if ((int)(w[0] >> 16) >= alpha_q16(alpha)) {"),
    (SNIS, "const int64_t e = pick_in_range(w[1], 0, kappa - 1);", "const int64_t e = 0;"),
    (SNIS, "r = modes[e] / Wk + (popcount32(w[2] & mask) - m);", "r = modes[e] / Wk + (popcount32(w[2] & mask) - m + 1);"),
    (SNIS, "c = modes[e] % Wk + (popcount32(w[3] & mask) - m);", "c = modes[e] % Wk + (popcount32(w[2] & mask) - m);"),
    (SNIS, "lw[t] = a - log(snis_density(qm, kappa, Hk, Wk, radius, alpha, js[t]));", "lw[t] = a;"),
    (SNIS, "const double wn = exp(lw[t] - mx) / s1;", "const double wn = exp(lw[t] - mx);"),
    (SNIS, "if (ess) ess[i] = s2 > 0.0 ? s1 * s1 / s2 : 0.0;", "if (ess) ess[i] = s2 > 0.0 ? s1 / s2 : 0.0;"),
    (SNIS, "if (js[t] > last) {", "if (js[t] >= last) {"),
    (SNIS, "const double a = scale * dot(q, Ks + js[t] * d, d);", "const double a = dot(q, Ks + js[t] * d, d);"),
    (SNIS, "for (int e = 0; e < dv; ++e) vr[e] += wn * wn * (v[e] - o[e]) * (v[e] - o[e]);",
     "for (int e = 0; e < dv; ++e) vr[e] += wn * (v[e] - o[e]) * (v[e] - o[e]);"),
    (SNIS, "const uint32_t ctr[4] = {(uint32_t)g, (uint32_t)t, 0u, OR_SNIS_TAG};",
     "const uint32_t ctr[4] = {(uint32_t)g, 0u, (uint32_t)t, OR_SNIS_TAG};"),
    (SNIS, "static int alpha_q16(double alpha) { return (int)floor(alpha * 65536.0 + 0.5); }",
     "static int alpha_q16(double alpha) { return (int)floor(alpha * 65535.0 + 0.5); }"),
    # backward of the attend step
    (BWD, "dQ[g * d + e] += scale * ds * k[e];", "dQ[g * d + e] += ds * k[e];"),
    (BWD, "gK[keys[j] * d + e] += scale * ds * q[e];", "gK[keys[j] * d + e] += scale * ds * k[e];"),
    (BWD, "const double ds = p[j] * (dp[j] - D);", "const double ds = p[j] * dp[j];"),
    (BWD, "for (int e = 0; e < dv; ++e) gV[keys[j] * dv + e] += p[j] * go[e];",
     "for (int e = 0; e < dv; ++e) gV[keys[j] * dv + e] += go[e];"),
    (BWD, "            D += p[j] * dp[j];", "            D += dp[j];"),
    (BWD, "            p[j] /= l;", "            p[j] /= l + 1e-3;"),
]


@pytest.mark.parametrize("pins,old,new", MUTATIONS, ids=[f"{i:02d}-{os.path.basename(m[0])[12:-3]}"
                                                         for i, m in enumerate(MUTATIONS)])
def test_pins_catch_planted_slip(tmp_path, pins, old, new):
    for part in ("oracle", "scram_inputs", "tests"):
        shutil.copytree(os.path.join(ROOT, part), tmp_path / part,
                        ignore=shutil.ignore_patterns("*.so", "__pycache__"))
    shutil.copy(os.path.join(ROOT, "pytest.ini"), tmp_path)
    src_path = tmp_path / "oracle" / "scram_oracle.c"
    src = src_path.read_text()
    assert src.count(old) == 1, f"the line to mutate is not in the oracle exactly once: {old!r}"
    src_path.write_text(src.replace(old, new))
    env = dict(os.environ, OMP_NUM_THREADS=os.environ.get("OMP_NUM_THREADS", "4"))
    r = subprocess.run([sys.executable, "-m", "pytest", pins, "-x", "-q", "-m", "not gpu", "-p", "no:cacheprovider"],
                       cwd=tmp_path, capture_output=True, text=True, timeout=600, env=env)
    tail = "\n".join(r.stdout.strip().splitlines()[-3:])
    assert r.returncode == 1, f"planted slip not caught by {pins} (pytest exit {r.returncode}):\n{new}\n{tail}"
