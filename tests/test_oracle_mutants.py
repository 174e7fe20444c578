"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a scratch copy of oracle/speechkv_oracle.c (on
the CPU, in a temporary directory), runs tests/test_oracle_pins.py against that
copy, and requires at least one pin to fail.  The real oracle is never touched.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = {
    "gate sign flipped": ("s += (u ? u[(size_t)g * D + e] : 0.0) * k[e];",
                          "s -= (u ? u[(size_t)g * D + e] : 0.0) * k[e];"),
    "window dated one frame late": ("return last < P + T - 1 ? last : P + T - 1;",
                                    "return last + 1 < P + T - 1 ? last + 1 : P + T - 1;"),
    "window dated one frame early": ("return last < P + T - 1 ? last : P + T - 1;",
                                     "return last - 1 < P + T - 1 ? last - 1 : P + T - 1;"),
    "GQA heads interleaved": ("int g = h / group;\n      int nW", "int g = h % Hkv;\n      int nW"),
    "logit scale dropped": ("z[c] = scale * s;\n          if", "z[c] = s;\n          if"),
    "suffix read one row early": ("RAW(k_raw, P[b] + T[b] + m)", "RAW(k_raw, P[b] + T[b] + m - 1)"),
    "values pooled uniformly": ("vs += alpha[j] * RAW(v_raw, first + j)[e];",
                                "vs += RAW(v_raw, first + j)[e] / n;"),
    "short last window dropped": ("return (T + weff - 1) / weff;", "return T / weff;"),
    "row cannot see its own key": ("visible_from(c, P[b], T[b], nW, weff, mask_mode) > p",
                                   "visible_from(c, P[b], T[b], nW, weff, mask_mode) >= p"),
    "window-start mask late": ("if (mode == 1) return P + i * weff;",
                               "if (mode == 1) return P + i * weff + 1;"),
    "layer l0 left uncompressed": ("return layer >= l0 ? w : 1;", "return layer > l0 ? w : 1;"),
    "lse without the max": ("if (l) *l = m + log(sum);", "if (l) *l = log(sum);"),
    "decode GQA interleaved": ("int g = h / group;\n      int len = clen[b];",
                               "int g = h % Hkv;\n      int len = clen[b];"),
    "decode drops last key": ("for (int c = 0; c < len; ++c) {\n        const double* k = k_hat",
                              "for (int c = 0; c < len - 1; ++c) {\n        const double* k = k_hat"),
}

# Mistakes in the gradients, caught by tests/test_oracle_bwd_pins.py.
BWD_MUTANTS = {
    "bwd softmax mean dropped": ("double dz = pi[c] * (dpi[c] - mean);",
                                 "double dz = pi[c] * dpi[c];"),
    "bwd dq without scale": ("gq[e] += scale * dz * k[e];", "gq[e] += dz * k[e];"),
    "bwd dk^ from the wrong operand": ("gk[e] += scale * dz * qr[e];", "gk[e] += scale * dz * go[e];"),
    "bwd dv^ weighted by dz": ("gv[e] += pi[c] * go[e];", "gv[e] += dz * go[e];"),
    "bwd heads of another group": ("for (int h = g * group; h < (g + 1) * group; ++h) {",
                                   "for (int h = g; h < Hq; h += Hkv) {"),
    "bwd mask off by one": ("if (visible_from(c, P[b], T[b], nW, weff, mask_mode) > p) continue;",
                            "if (visible_from(c, P[b], T[b], nW, weff, mask_mode) >= p) continue;"),
    "bwd dk misses the logit path": (
        "dk[e] = alpha[j] * gk[e] + ds * (u ? u[(size_t)g * D + e] : 0.0);",
        "dk[e] = alpha[j] * gk[e];"),
    "bwd dalpha ignores values": ("d += gk[e] * k[e] + gv[e] * v[e];", "d += gk[e] * k[e];"),
    "bwd du sign flipped": ("du[(size_t)g * D + e] += ds * k[e];", "du[(size_t)g * D + e] -= ds * k[e];"),
    "bwd gate Jacobian without mean": ("double ds = alpha[j] * (dalpha[j] - mean);",
                                       "double ds = alpha[j] * dalpha[j];"),
    "bwd suffix gradient one row early": ("memcpy(RAW(dk_raw, P[b] + T[b] + m), HAT(dk_hat, P[b] + nW + m),",
                                          "memcpy(RAW(dk_raw, P[b] + T[b] + m - 1), HAT(dk_hat, P[b] + nW + m),"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS) + sorted(BWD_MUTANTS))
def test_planted_mistake_is_caught(name, tmp_path):
    before, after = MUTANTS[name] if name in MUTANTS else BWD_MUTANTS[name]
    pins = "tests/test_oracle_pins.py" if name in MUTANTS else "tests/test_oracle_bwd_pins.py"
    src = open(os.path.join(ROOT, "oracle", "speechkv_oracle.c")).read()
    assert src.count(before) >= 1, "mutation site not found"
    skip = shutil.ignore_patterns("__pycache__", "*.so", "*.tmp")
    shutil.copytree(os.path.join(ROOT, "oracle"), tmp_path / "oracle", ignore=skip)
    shutil.copytree(os.path.join(ROOT, "tests"), tmp_path / "tests", ignore=skip)
    (tmp_path / "oracle" / "speechkv_oracle.c").write_text(src.replace(before, after, 1))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        pins], cwd=tmp_path, capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 1 and " failed" in r.stdout, r.stdout[-2000:]
