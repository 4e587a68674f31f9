"""Meta-test: the oracle's pins are discriminating.  Each case plants one
plausible mistake (a dropped term, a wrong sign, a swapped index, = instead of
+=, a backward that runs where Lemma 1 says it must not) in a copy of the oracle source, builds it on the CPU, and runs the pin
suite against it: at least one pin must fail."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "mpipe_ref.cpp")

MUTATIONS = {
    "rope_sign": ("v[j + half] = x2 * cs + x1 * sn;", "v[j + half] = x2 * cs - x1 * sn;"),
    "ln_unbiased_variance": ("var /= (T)n;", "var /= (T)(n - 1);"),
    "attention_no_scale": ("sc[j] = dot * scale;", "sc[j] = dot;"),
    "merge_window_order": ("row_of(tau, 2 * hb + q / 2, 2 * wb + q % 2, gh, gw)",
                           "row_of(tau, 2 * hb + q % 2, 2 * wb + q / 2, gh, gw)"),
    "ln_bwd_dropped_term": ("dx[i] = rstd[r] * (dy[i] * g[i] - s1 - xh * s2);",
                            "dx[i] = rstd[r] * (dy[i] * g[i] - s1);"),
    "attention_bwd_no_delta": ("const T ds = p[j] * (dp[j] - delta);",
                               "const T ds = p[j] * dp[j];"),
    "gelu_grad_sign": ("return Phi + u * phi;", "return Phi - u * phi;"),
    "residual_grad_dropped": ("for (size_t i = 0; i < dHm.size(); ++i) dHm[i] += dH[i];", ""),
    "bias_grad_assigned": ("db[n] += s;", "db[n] = s;"),
    # merger-only trainability: the block backward must not run, the merger's own
    # LayerNorm affine gradients must
    "merger_only_runs_blocks": [("  if (merger_only) return 0;\n", ""),
                                ("if (!dM || merger_only) { Layer<T> empty;", "if (!dM) { Layer<T> empty;")],
    "merger_only_skips_merger_ln": ("  layernorm_bwd(dZ.data(), H.data(), P(MG + 0),",
                                    "  if (merger_only) return 0;\n  layernorm_bwd(dZ.data(), H.data(), P(MG + 0),"),
    "qk_transposed_head": ("const T* kj = k + (size_t)(a + j) * ld + (size_t)hd * d;\n        T dot = 0;\n        for (int e = 0; e < d; ++e) dot += qi[e] * kj[e];",
                           "const T* kj = k + (size_t)(a + j) * ld + (size_t)((hd + 1) % heads) * d;\n        T dot = 0;\n        for (int e = 0; e < d; ++e) dot += qi[e] * kj[e];"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    edits = MUTATIONS[name]
    src = open(SRC).read()
    for a, b in (edits if isinstance(edits, list) else [edits]):
        assert a in src, f"mutation anchor for {name} no longer present in the oracle source"
        src = src.replace(a, b, 1)
    mut = tmp_path / "m.cpp"
    mut.write_text(src)
    lib = tmp_path / "liboracle_mut.so"
    subprocess.run(["g++", "-O1", "-std=c++17", "-fPIC", "-shared", "-fopenmp",
                    "-I", os.path.join(ROOT, "oracle"), "-o", str(lib), str(mut)], check=True)
    env = dict(os.environ, MPIPE_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_oracle_merger_mode.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode != 0, f"no pin caught the planted mistake '{name}'"
    assert "failed" in r.stdout
