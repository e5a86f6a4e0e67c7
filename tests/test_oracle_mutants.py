"""The oracle's pins must catch plausible mistakes.

Each case below plants one mistake in a copy of the oracle's C source (a
dropped term, a wrong sign, a swapped or transposed index, an off-by-one),
builds it, and runs tests/pin_battery.py against that build in a child
process: the battery must report a failure.  The unmodified source must pass.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "qcnn_oracle.c")

# (function, text to replace, replacement, what the mistake is)
MUTANTS = [
    ("qo_conv_lut", "codes[(((size_t)t * dk + ky) * dk + kx) * M + m]",
     "codes[(((size_t)t * dk + kx) * dk + ky) * M + m]", "kernel offsets ky/kx swapped in the code index"),
    ("qo_conv_lut", "int xi = xo * stride - pad + kx;", "int xi = xo * stride + pad + kx;", "padding sign"),
    ("qo_conv_lut", "int yi = yo * stride - pad + ky;", "int yi = yo - pad + ky;", "stride dropped on rows"),
    ("qo_conv_lut", "if (xi < 0 || xi >= W) continue;", "if (xi < 1 || xi >= W) continue;",
     "off-by-one at the left border"),
    ("qo_conv_lut", "for (int m = 0; m < M; ++m) {", "for (int m = 1; m < M; ++m) {", "first subspace dropped"),
    ("qo_conv_lut",
     "if (bias) { s += (double)bias[t]; a += fabs((double)bias[t]); }\n          if (relu && s < 0.0) s = 0.0;",
     "if (relu && s < 0.0) s = 0.0;\n          if (bias) { s += (double)bias[t]; a += fabs((double)bias[t]); }",
     "ReLU applied before the bias"),
    ("qo_conv_lut", "if (alut) a += alut[o];", "if (alut) a += lut[o];", "bound sums signed terms"),
    ("qo_lut", "for (int j = 0; j < Csp; ++j) {", "for (int j = 1; j < Csp; ++j) {", "dropped term of the inner product"),
    ("qo_lut", "(double)x[((size_t)n * Cs + (size_t)m * Csp + j) * HW + p]",
     "(double)x[((size_t)n * Cs + (size_t)m + j) * HW + p]", "wrong subspace channel offset"),
    ("qo_lut", "(double)D[((size_t)m * K + k) * Csp + j]", "(double)D[((size_t)m * Csp + j) * K + k]",
     "codebook transposed"),
    ("qo_lut", "s += term;", "s -= term;", "sign of the table entry"),
    ("qo_fc_lut", "int k = codes[(size_t)t * M + m];", "int k = codes[(size_t)m * Ct + t];", "FC codes transposed"),
    ("qo_fc_lut", "(double)x[(size_t)n * Cs + (size_t)m * Csp + j]", "(double)x[(size_t)m * Csp + j]",
     "FC image index dropped"),
    ("qo_conv_direct", "What[(((size_t)t * Cs + (size_t)m * Csp + j) * dk + ky) * dk + kx]",
     "What[(((size_t)t * Cs + (size_t)m * Csp + j) * dk + kx) * dk + ky]", "rebuilt kernel transposed"),
    ("qo_conv_points", "int xi = xo * stride - pad + kx;", "int xi = xo * stride - pad + ky;", "point: kx read as ky"),
    ("qo_fc_direct", "for (int c = 0; c < Cs; ++c) s +=", "for (int c = 0; c < Cs - 1; ++c) s +=", "FC last input dropped"),
    ("qo_maxpool", "if (v > best) best = v;", "if (v < best || best == -INFINITY) best = v;", "min instead of max"),
    ("pq_dist", "* dk * dk) + p]", "* dk) + p]", "quantizer: sub-vector stride over kernel positions"),
    ("pq_dist", "d += diff * diff;", "d += fabs(diff);", "quantizer: distance not squared"),
    ("qo_pq_assign", "if (d < bd) { bd = d; best = k; }", "if (d <= bd) { bd = d; best = k; }",
     "quantizer: ties to the highest index"),
    ("qo_pq_assign", "for (int k = 1; k < K; ++k) {", "for (int k = 1; k < K - 1; ++k) {",
     "quantizer: last sub-codeword never considered"),
    ("qo_pq_assign", "s += bd;", "s += sqrt(bd);", "quantizer: objective not squared"),
    ("qo_pq_distances", "if (d < bd) bd = d;", "if (d > bd) bd = d;", "quantizer check: largest distance as the minimum"),
    ("qo_pq_distances", "Dm + (size_t)codes[i] * Csp);", "Dm + (size_t)codes[i]);", "quantizer check: code stride"),
    ("qo_pq_update", "int k = codes[((size_t)t * P + p) * M + m];", "int k = codes[((size_t)p * Ct + t) * M + m];",
     "quantizer: update reads the codes transposed"),
    ("qo_pq_update", "/ (double)cnt[k])", "/ (double)(cnt[k] + 1))", "quantizer: mean divided by count + 1"),
    ("qo_pq_update", ": D_in[o];", ": 0.0f;", "quantizer: unused sub-codeword zeroed"),
    ("qo_pq_kmeans", "for (int it = 0; it <= iters && !e; ++it) {", "for (int it = 0; it < iters && !e; ++it) {",
     "quantizer: no final assignment"),
    ("qo_pack_codes", "<< (q % 8));", "<< (7 - q % 8));", "packed codes: most significant bit first in a byte"),
    ("qo_pack_codes", "const long long q = i * b + j;", "const long long q = (n - 1 - i) * b + j;",
     "packed codes: codes stored in reverse order"),
    ("qo_code_bits", "while ((1 << b) < K) ++b;", "while ((2 << b) <= K) ++b;",
     "packed codes: floor(log2 K) bits"),
    ("qo_unpack_codes", "v |= ((in[q / 8] >> (q % 8)) & 1) << j;", "v |= ((in[q / 8] >> (q % 8)) & 1) << (b - 1 - j);",
     "packed codes: value bits reversed on unpack"),
]


def _mutate(src: str, func: str, old: str, new: str) -> str:
    for ret in ("int", "float", "double"):
        start = src.find("%s %s(" % (ret, func))
        if start >= 0:
            break
    assert start >= 0, func
    end = src.index("\n}\n", start)
    body = src[start:end]
    assert old in body, (func, old)
    return src[:start] + body.replace(old, new, 1) + src[end:]


def _battery(lib: str) -> subprocess.CompletedProcess:
    return subprocess.run([sys.executable, os.path.join(ROOT, "tests", "pin_battery.py"), lib],
                          capture_output=True, text=True, timeout=300)


def _build(src_text: str, tmp_path, name: str) -> str:
    c = tmp_path / (name + ".c")
    so = tmp_path / (name + ".so")
    c.write_text(src_text)
    subprocess.check_call(["gcc", "-O1", "-std=c99", "-fPIC", "-shared", "-o", str(so), str(c), "-lm"])
    return str(so)


def test_unmodified_oracle_passes(tmp_path):
    lib = _build(open(SRC).read(), tmp_path, "orig")
    r = _battery(lib)
    assert r.returncode == 0, r.stdout + r.stderr


@pytest.mark.parametrize("mut", MUTANTS, ids=[m[3] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, mut):
    func, old, new, what = mut
    lib = _build(_mutate(open(SRC).read(), func, old, new), tmp_path, "mut")
    r = _battery(lib)
    assert r.returncode == 1 and "FAILED" in r.stdout, "mutant survived: %s\n%s%s" % (what, r.stdout, r.stderr)


# Mistakes planted in a copy of the error-correction oracle (oracle/ec.py,
# Eq. (8)-(12)); the module copy is loaded on its own and the battery's EC
# checks must flag each one.
EC_SRC = os.path.join(ROOT, "oracle", "ec.py")
EC_MUTANTS = [
    ("Dm[k] = solve_normal(G, P[:, Lk].sum(axis=1)) / Lk.sum()",
     "Dm[k] = solve_normal(G, P[:, Lk].sum(axis=1))", "sub-codebook: sum not divided by |L_k|"),
    ("cost = q[:, None] - 2.0 * (Dm @ P)", "cost = q[:, None] - (Dm @ P)", "assignment: cross term not doubled"),
    ("codes_m = np.argmin(cost, axis=0)", "codes_m = np.argmax(cost, axis=0)", "assignment: argmax"),
    ("R = T - Y + old", "R = T - Y", "residual keeps the subspace's own contribution"),
    ("for _ in range(inner):\n        for k in range(K):",
     "for _ in range(inner):\n        for k in range(K - 1):", "last sub-codeword never updated"),
    ("P = Sm.T @ R ", "P = Sm.T @ (R - R.mean(axis=0)) ", "residual centred"),
    ("if A[j, j] <= PIVOT_REL * scale or A[j, j] <= 0.0:", "if A[j, j] < 0.0:", "dead directions not dropped"),
    ("Y = Y - old + Sm @ D[m][codes[:, m]].T", "Y = Y + Sm @ D[m][codes[:, m]].T",
     "response not updated correctly after a subspace"),
]


def _ec_module(text, tmp_path, name):
    import importlib.util
    path = tmp_path / (name + ".py")
    path.write_text(text)
    spec = importlib.util.spec_from_file_location(name, str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_unmodified_ec_passes(tmp_path):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    mod = _ec_module(open(EC_SRC).read(), tmp_path, "ec_orig")
    bad = [n for n, ok in pin_battery.ec_checks(np.random.Generator(np.random.PCG64(11)), mod) if not ok]
    assert not bad, bad


@pytest.mark.filterwarnings("ignore::RuntimeWarning")  # some mutants divide by a zero pivot
@pytest.mark.parametrize("mut", EC_MUTANTS, ids=[m[2] for m in EC_MUTANTS])
def test_ec_pins_catch_mutant(tmp_path, mut):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    old, new, what = mut
    src = open(EC_SRC).read()
    assert old in src, old
    mod = _ec_module(src.replace(old, new, 1), tmp_path, "ec_mut")
    try:
        res = pin_battery.ec_checks(np.random.Generator(np.random.PCG64(11)), mod)
        survived = all(ok for _, ok in res)
    except Exception:  # a crash is a caught mistake too
        survived = False
    assert not survived, "mutant survived: " + what


# Mistakes planted in a copy of the conv error-correction oracle
# (oracle/ec_conv.py, App. B); each entry is a list of replacements.
ECC_SRC = os.path.join(ROOT, "oracle", "ec_conv.py")
ECC_MUTANTS = [
    ([("for p in other:", "for p in range(P):")], "Q takes out every position, its own too"),
    ([("A = s[:, :, mine[c], :].sum(axis=2)", "A = s[:, :, np.flatnonzero(mine[c])[:1], :].sum(axis=2)")],
     "only the first position of a channel on sub-codeword k fitted"),
    ([("    for k in range(K):\n        mine = codes_m == k", "    Dz = Dm.copy()\n    for k in range(K):\n        mine = codes_m == k"),
      ("Q -= s[:, :, p, :] @ Dm[codes_m[c, p]]", "Q -= s[:, :, p, :] @ Dz[codes_m[c, p]]")],
     "codebook update not sequential (old sub-codewords in Q)"),
    ([("if q != p:", "if True:")], "P takes out the position being assigned"),
    ([("    for p in range(P):\n        for c in range(Ct):", "    cz = codes_m.copy()\n    for p in range(P):\n        for c in range(Ct):"),
      ("Pp -= s[:, :, q, :] @ Dm[codes_m[c, q]]", "Pp -= s[:, :, q, :] @ Dm[cz[c, q]]")],
     "assignment update not sequential (old codes in P)"),
    ([("codes_m[c, p] = int(np.argmin(err))", "codes_m[c, p] = int(np.argmax(err))")], "assignment: argmax"),
    ([("Sp[:, :, pad:pad + H, pad:pad + W] = Sm", "Sp[:, :, :H, :W] = Sm")], "padding ignored"),
    ([("s[:, :, ky * dk + kx, :] = win", "s[:, :, kx * dk + ky, :] = win")], "kernel positions transposed"),
    ([("R = Tf - Y + old", "R = Tf - Y")], "residual keeps the subspace's own contribution"),
    ([("for _ in range(inner):\n        update_codebook(s, R, Dm, codes_m)\n",
       "for _ in range(inner):\n")], "codebook never updated"),
]


def test_unmodified_ec_conv_passes(tmp_path):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    mod = _ec_module(open(ECC_SRC).read(), tmp_path, "ecc_orig")
    bad = [n for n, ok in pin_battery.ec_conv_checks(np.random.Generator(np.random.PCG64(13)), mod) if not ok]
    assert not bad, bad


@pytest.mark.filterwarnings("ignore::RuntimeWarning")
@pytest.mark.parametrize("mut", ECC_MUTANTS, ids=[m[1] for m in ECC_MUTANTS])
def test_ec_conv_pins_catch_mutant(tmp_path, mut):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    reps, what = mut
    src = open(ECC_SRC).read()
    for old, new in reps:
        assert old in src, old
        src = src.replace(old, new, 1)
    mod = _ec_module(src, tmp_path, "ecc_mut")
    try:
        res = pin_battery.ec_conv_checks(np.random.Generator(np.random.PCG64(13)), mod)
        survived = all(ok for _, ok in res)
    except Exception:  # a crash is a caught mistake too
        survived = False
    assert not survived, "mutant survived: " + what


# Mistakes planted in a copy of the multi-layer oracle (oracle/ec_network.py).
ECN_SRC = os.path.join(ROOT, "oracle", "ec_network.py")
ECN_MUTANTS = [
    ([("        out.append(lin.astype(np.float32))\n",
       "        out.append((lin + (0.1 if spec.get('bias') is not None else 0.0)).astype(np.float32))\n")],
     "T shifted (bias folded in)"),
    ([("        lin = dense_linear(ho, spec)                              # M1",
       "        lin = dense_linear(np.maximum(ho, 0.0), spec)                              # M1"),
      ("            ho = O.maxpool(ho, spec[\"k\"], spec[\"s\"]).astype(np.float32)\n",
       "            ho = -O.maxpool(ho, spec[\"k\"], spec[\"s\"]).astype(np.float32)\n")],
     "original network's pool output negated"),
    ([("        if spec[\"relu\"]:\n            lin = np.maximum(lin, 0.0)", "        if False:\n            lin = np.maximum(lin, 0.0)")],
     "original network without ReLU"),
    ([("            ho = O.maxpool(ho, spec[\"k\"], spec[\"s\"]).astype(np.float32)\n", "")],
     "original network skips the pool"),
    ([("relu=spec[\"relu\"]).astype(np.float32)", "relu=False).astype(np.float32)")],
     "quantized network without ReLU after a conv"),
    ([("            S = hq\n", "            S = np.abs(hq - 0.05)\n")], "conv S is not the quantized activations"),
]


@pytest.mark.filterwarnings("ignore::RuntimeWarning")
@pytest.mark.parametrize("mut", ECN_MUTANTS, ids=[m[1] for m in ECN_MUTANTS])
def test_ec_network_pins_catch_mutant(tmp_path, mut):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    reps, what = mut
    src = open(ECN_SRC).read()
    for old, new in reps:
        assert old in src, old
        src = src.replace(old, new, 1)
    mod = _ec_module(src, tmp_path, "ecn_mut")
    try:
        res = pin_battery.ec_network_checks(np.random.Generator(np.random.PCG64(17)), mod)
        survived = all(ok for _, ok in res)
    except Exception:  # a crash is a caught mistake too
        survived = False
    assert not survived, "mutant survived: " + what


def test_unmodified_ec_network_passes(tmp_path):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    mod = _ec_module(open(ECN_SRC).read(), tmp_path, "ecn_orig")
    bad = [n for n, ok in pin_battery.ec_network_checks(np.random.Generator(np.random.PCG64(17)), mod) if not ok]
    assert not bad, bad


# Mistakes planted in a copy of the oracle's network composition
# (oracle/oracle.py, network()): the copy runs on the same C oracle library and
# the battery's network checks must flag each one.
NET_SRC = os.path.join(ROOT, "oracle", "oracle.py")
NET_MUTANTS = [
    ('fc_lut(h32.reshape(h32.shape[0], -1), D,',
     'fc_lut(np.ascontiguousarray(h32.transpose(0, 2, 3, 1) if h32.ndim == 4 else h32)'
     '.reshape(h32.shape[0], -1), D,', "flatten in NHWC order"),
    ('h = maxpool(h32, L["k"], L["s"])', 'h = h32', "pool skipped"),
    ('relu = bool(L["relu"]) and not absolute', 'relu = False', "ReLU dropped"),
    ('D = np.abs(L["D"]) if absolute else L["D"]', 'D = L["D"]', "absolute network keeps signed codebooks"),
    ('h = np.abs(x) if absolute else x', 'h = x', "absolute network keeps signed inputs"),
]


def _net_module(text, tmp_path, name):
    here = '_HERE = os.path.dirname(os.path.abspath(__file__))'
    assert here in text
    return _ec_module(text.replace(here, "_HERE = %r" % os.path.join(ROOT, "oracle"), 1), tmp_path, name)


def test_unmodified_network_passes(tmp_path):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    mod = _net_module(open(NET_SRC).read(), tmp_path, "net_orig")
    bad = [n for n, ok in pin_battery.network_checks(np.random.Generator(np.random.PCG64(5)), mod) if not ok]
    assert not bad, bad


@pytest.mark.parametrize("mut", NET_MUTANTS, ids=[m[2] for m in NET_MUTANTS])
def test_network_pins_catch_mutant(tmp_path, mut):
    import numpy as np
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import pin_battery
    old, new, what = mut
    src = open(NET_SRC).read()
    assert old in src, old
    mod = _net_module(src.replace(old, new, 1), tmp_path, "net_mut")
    try:
        res = pin_battery.network_checks(np.random.Generator(np.random.PCG64(5)), mod)
        survived = all(ok for _, ok in res)
    except Exception:  # a crash is a caught mistake too
        survived = False
    assert not survived, "mutant survived: " + what
