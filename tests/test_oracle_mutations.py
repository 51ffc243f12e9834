"""The oracle's pins must catch plausible mistakes.  Each case compiles a copy
of the oracle with one planted error and runs the pin suite against it in a
subprocess; the suite has to fail.  Everything runs on the CPU."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

MUTANTS = {
    "rmsnorm_gain_dropped": (" * (double)orc_bf16_to_f32(g[i]));", ");"),
    "rmsnorm_eps_outside_sqrt": ("sqrt(ss / (double)d + (double)eps)", "(sqrt(ss / (double)d) + (double)eps)"),
    "rope_sign": ("u[i] = (float)(a * c - b * s);", "u[i] = (float)(a * c + b * s);"),
    "rope_theta_exponent": ("-2.0 * (double)i / (double)head_dim", "-1.0 * (double)i / (double)head_dim"),
    "attention_scale_dropped": ("s[j] = dot * scale;", "s[j] = dot;"),
    "attention_excludes_self": ("pos + 1, hd, o + hh * hd);", "pos > 0 ? pos : 1, hd, o + hh * hd);"),
    "gqa_mapping_modulo": ("int g = hh / G;", "int g = hh % Hkv;"),
    "residual_dropped": ("orc_gemv(lin(L, 3), lin_scale(L, 3), m->wfmt, d, H * hd, o, y);\n"
                         "    for (int i = 0; i < d; ++i) x[i] = (float)((double)x[i] + (double)y[i]);",
                         "orc_gemv(lin(L, 3), lin_scale(L, 3), m->wfmt, d, H * hd, o, y);\n"
                         "    for (int i = 0; i < d; ++i) x[i] = y[i];"),
    "swiglu_swapped": ("orc_silu((double)gt[i]) * (double)up[i]", "orc_silu((double)up[i]) * (double)gt[i]"),
    "int8_scale_dropped": ("acc *= (double)orc_fp16_to_f32(scale[n]);", ""),
    "gemv_transposed": ("acc += (double)orc_bf16_to_f32(row[k]) * (double)x[k];",
                        "acc += (double)orc_bf16_to_f32(((const uint16_t*)w)[((size_t)k * (size_t)n_out"
                        " + (size_t)n) % ((size_t)n_out * (size_t)n_in)]) * (double)x[k];"),
    "argmax_last_tie": ("if (x[i] > x[best]) best = i;", "if (x[i] >= x[best]) best = i;"),
    "kv_truncated_not_rounded": ("  u += 0x7fffu + lsb;\n", "  (void)lsb;\n"),
    "value_not_key_rope": ("for (int g = 0; g < Hkv; ++g) orc_rope(k + g * hd, hd, pos, m->rope_base);",
                           "for (int g = 0; g < Hkv; ++g) orc_rope(v + g * hd, hd, pos, m->rope_base);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation anchor not found: " + name
    mpath = tmp_path / "oracle_mut.c"
    mpath.write_text(src.replace(old, new))
    so = tmp_path / "liboracle_mut.so"
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-I",
                           os.path.join(ROOT, "oracle"), "-o", str(so), str(mpath), "-lm"])
    env = dict(os.environ, AIO_ORACLE_LIB=str(so), OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 1, "planted mistake %s was not caught:\n%s" % (name, r.stdout[-2000:])
