"""Plants plausible mistakes in copies of the oracle's C source (CPU only).

Each mutant is compiled to a temporary library and run against the pin suite
in a child process; every mutant must fail at least one pin. This shows the
pins would catch a dropped term, a wrong sign, index or normalisation.
"""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTANTS = [
    ("scale 1/d instead of 1/sqrt(d)", "const double scale = 1.0 / sqrt((double)d);",
     "const double scale = 1.0 / (double)d;"),
    ("unbiased variance", "  var /= c_z;", "  var /= (c_z - 1);"),
    ("eps outside the square root", "const double inv = 1.0 / sqrt(var + eps);",
     "const double inv = 1.0 / (sqrt(var) + eps);"),
    ("mean not subtracted", "const double xhat = (load_elem(z, dtype, off + c) - mu) * inv;",
     "const double xhat = load_elem(z, dtype, off + c) * inv;"),
    ("gate dropped", "out_row[h * d + e] = g_row[h * d + e] * (num / den);",
     "out_row[h * d + e] = (num / den);"),
    ("bias subtracted", "logit[j - k0] = dot * scale + bias_row[j * n_heads + h];",
     "logit[j - k0] = dot * scale - bias_row[j * n_heads + h];"),
    ("mask ignored", "if (mask && !mask[j]) {", "if (0) {"),
    ("key head offset dropped", "dot += q_row[h * d + e] * k[j * hd + h * d + e];",
     "dot += q_row[h * d + e] * k[j * hd + e];"),
    ("value head offset dropped", "num += exp(logit[j] - mx) * v[j * (int64_t)n_heads * d + h * d + e];",
     "num += exp(logit[j] - mx) * v[j * (int64_t)n_heads * d + e];"),
    ("merge without rescale", "*l = a * *l + b * lb;", "*l = *l + lb;"),
    ("chunk start without min", "*start = p * q + (p < r ? p : r);", "*start = p * q + p;"),
    ("sigmoid sign", "return 1.0 / (1.0 + exp(-x));", "return 1.0 / (1.0 + exp(x));"),
    ("beta dropped", "+ (beta ? beta[c] : 0.0);", "+ 0.0;"),
    ("gamma dropped", "ln[c] = (gamma ? gamma[c] : 1.0) * xhat", "ln[c] = 1.0 * xhat"),
    ("projection bias dropped", "b_out[h] = acc + (b_b ? b_b[h] : 0.0);", "b_out[h] = acc;"),
    ("linear transposed", "acc += w[(int64_t)o * n_in + c] * x[t * n_in + c];",
     "acc += w[(int64_t)(c % n_out) * n_in + (o % n_in)] * x[t * n_in + c];"),
    ("blocked partial not rescaled",
     "for (int e = 0; e < d; ++e) acc[e] = a * acc[e] + b * accb[e];",
     "for (int e = 0; e < d; ++e) acc[e] = acc[e] + accb[e];"),
    ("sparse empty slot read as atom 0", "const int32_t j = nbr[r * k + t];",
     "const int32_t j = nbr[r * k + t] < 0 ? 0 : nbr[r * k + t];"),
    ("sparse pair slice of slot 0", "pair_bias(p_rows, p_dtype, (r * k + t) * (int64_t)c_ap,",
     "pair_bias(p_rows, p_dtype, (r * k) * (int64_t)c_ap,"),
    ("sparse value of the query atom", "accb[e] += w * vv[(int64_t)nbr[r * k + t] * hd + h * d + e];",
     "accb[e] += w * vv[(int64_t)i * hd + h * d + e];"),
    ("sparse block filter overlaps", "j < bstart || j >= bstart + bsize) continue;",
     "j < bstart || j > bstart + bsize) continue;"),
    ("sparse gate dropped", "out[r * hd + h * d + e] = sigmoid(gp[h * d + e]) * o;",
     "out[r * hd + h * d + e] = o;"),
    ("sparse query from key weights", "oracle_linear(1, c_atom, hd, ai, w_q, q);",
     "oracle_linear(1, c_atom, hd, ai, w_k, q);"),
    ("knn ties by larger index", "return a.d2 < b.d2 || (a.d2 == b.d2 && a.j < b.j);",
     "return a.d2 < b.d2 || (a.d2 == b.d2 && a.j > b.j);"),
    ("knn distance summed in another order", "const float s = xx + yy;\n  return s + zz;",
     "const float s = yy + zz;\n  return xx + s;"),
    ("knn group mode inverted", "if (group_mode == 1 && group_c[j] != group_q[r]) continue;",
     "if (group_mode == 1 && group_c[j] == group_q[r]) continue;"),
    ("knn merge drops the second list", "      if (idx_b[r * k + t] >= 0) {", "      if (0) {"),
    ("knn block offset lost", "keys[n].j = c_index0 + j;", "keys[n].j = j;"),
    ("transition silu without the input", "h[u] = a / (1.0 + exp(-a)) * b;", "h[u] = 1.0 / (1.0 + exp(-a)) * b;"),
    ("transition gate on the other branch", "h[u] = a / (1.0 + exp(-a)) * b;", "h[u] = b / (1.0 + exp(-b)) * a;"),
    ("transition residual dropped", "out[p * c_z + c] = x[c] + t;", "out[p * c_z + c] = t;"),
    ("transition beta dropped", "((x[c] - mu) * inv) + (beta ? beta[c] : 0.0);", "((x[c] - mu) * inv);"),
    ("scatter mean divides by the token count + 1",
     "out[t * c + k] = cnt[t] > 0 ? out[t * c + k] / (double)cnt[t] : 0.0;",
     "out[t * c + k] = cnt[t] > 0 ? out[t * c + k] / (double)(cnt[t] + 1) : 0.0;"),
    ("scatter mean keeps the last atom only", "for (int k = 0; k < c; ++k) out[t * c + k] += load_elem(a, dtype, i * c + k);",
     "for (int k = 0; k < c; ++k) out[t * c + k] = load_elem(a, dtype, i * c + k);"),
    ("scatter mean drops the last token", "if (t < 0 || t >= n_tokens) continue;",
     "if (t < 0 || t >= n_tokens - 1) continue;"),
    ("transition w3 transposed", "t += w3[(int64_t)c * hidden + u] * h[u];",
     "t += w3[(int64_t)(u % c_z) * hidden + (c % hidden)] * h[u];"),
]

RUNNER = r"""
import ctypes, sys
sys.path.insert(0, {root!r}); sys.path.insert(0, {tests!r})
import oracle
oracle._lib = oracle._configure(ctypes.CDLL({lib!r}))
import oracle_pins
for pin in oracle_pins.ALL_PINS:
    try:
        pin()
    except Exception as exc:
        print("KILLED_BY", pin.__name__, type(exc).__name__)
        sys.exit(0)
print("SURVIVED")
"""


def _run(mutant, tmp):
    name, old, new = mutant
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation anchor not found: {name}"
    path = os.path.join(tmp, "m_%d" % abs(hash(name)))
    with open(path + ".c", "w") as f:
        f.write(src.replace(old, new))
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", path + ".c", "-lm",
                           "-o", path + ".so"])
    env = dict(os.environ, OMP_NUM_THREADS="2")
    p = subprocess.run([sys.executable, "-c", RUNNER.format(root=ROOT, tests=HERE, lib=path + ".so")],
                       capture_output=True, text=True, timeout=600, env=env)
    # a crash also counts as detection, but report it
    return name, p.returncode, p.stdout.strip().splitlines()[-1:] if p.stdout.strip() else [p.stderr[-200:]]


def test_every_mutant_fails_a_pin():
    with tempfile.TemporaryDirectory() as tmp, ThreadPoolExecutor(4) as ex:
        results = list(ex.map(lambda m: _run(m, tmp), MUTANTS))
    survivors = [(n, rc, out) for n, rc, out in results if rc == 0 and out and out[-1] == "SURVIVED"]
    assert not survivors, survivors
