"""Planted mistakes in the oracle.

Each entry below alters the C oracle in one plausible way (a dropped term, a
wrong sign, norm, index, word, order or rounding).  The test writes the
altered copy to a scratch directory, points the oracle loader at it
(DQGAN_ORACLE_DIR) and runs the oracle's pin tests in a child process: every
alteration must make at least one pin fail.  This is what shows that the pins
tie the oracle to the paper (Algorithm 2, Definition 1, Theorem 1, equation
qsgd, Appendix A, Appendix B) rather than to itself.  CPU only.
"""
import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "dqgan_oracle.c")
# the oracle's pins (the sanitizer run of those same pins builds its own copy)
PIN_FILES = sorted(f for f in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py"))
                   if not f.endswith("test_oracle_sanitized.py"))

# (name, what the mistake is, [(original text, altered text), ...]); each
# original text must occur in the oracle source, and its first occurrence is
# replaced.
MUTATIONS = [
    ("ef_drop_e", "EF accumulate without the residual",
     [("p[i] = eg + e[i];", "p[i] = eg;")]),
    ("ef_fma", "EF accumulate as one fused multiply-add",
     [("        float eg = eta * g[i];\n        p[i] = eg + e[i];", "        p[i] = fmaf(eta, g[i], e[i]);")]),
    ("l1_no_mean", "sign scale = the L1 norm instead of its mean",
     [("return (float)(sum / (double)n);", "return (float)sum;")]),
    ("l2_no_sqrt", "quantizer scale = squared norm",
     [("return (float)sqrt(sum);", "return (float)sum;")]),
    ("l2_as_l1", "quantizer scale = L1 norm",
     [("sum += (double)p[i] * (double)p[i];", "sum += fabs((double)p[i]);")]),
    ("linf_signed", "max norm over signed values",
     [("        float a = fabsf(p[i]);\n        if (a > mx) mx = a;", "        float a = p[i];\n        if (a > mx) mx = a;")]),
    ("sign_flip", "scaled sign with the sign reversed",
     [("float q = neg ? -scale : scale;", "float q = neg ? scale : -scale;")]),
    ("sign_of_zero", "sign by comparison (-0 treated as +0)",
     [("int neg = signbit(p[i]) ? 1 : 0;", "int neg = (p[i] < 0.0f) ? 1 : 0;")]),
    ("sign_residual_reversed", "sign residual p-hat - p",
     [("e_out[i] = p[i] - q;", "e_out[i] = q - p[i];")]),
    ("qsgd_residual_reversed", "quantizer residual p-hat - p",
     [("        phat[i] = q;\n        e_out[i] = p[i] - q;\n    }\n}\n\n/* Top-k",
       "        phat[i] = q;\n        e_out[i] = q - p[i];\n    }\n}\n\n/* Top-k")]),
    ("qsgd_round_inverted", "round up with probability 1 - frac",
     [("((u < frac) ? 1 : 0)", "((u > frac) ? 1 : 0)")]),
    ("qsgd_nearest", "deterministic nearest level before the random step",
     [("float l = floorf(r);", "float l = rintf(r);")]),
    ("qsgd_step_reciprocal", "decode step as the reciprocal of s / sigma",
     [("step = su / fs;", "step = 1.0f / inv;")]),
    ("qsgd_no_range", "s / sigma evaluated unscaled for tiny norms (overflows: every level s)",
     [("if (sigma < 0x1.0p-64f) {", "if (sigma < 0.0f) {")]),
    ("qsgd_inf_norm", "a norm of +inf quantized like a finite one (p-hat = 0 * inf)",
     [("if (!(sigma > 0.0f) || !(sigma <= FLT_MAX)) return 0;", "if (!(sigma > 0.0f)) return 0;")]),
    ("qsgd_range_not_undone", "tiny-norm p-hat left in the scaled range",
     [("float mag = ((float)level * step) * down;", "float mag = (float)level * step;")]),
    ("decode_range_not_undone", "server decodes tiny-norm levels without scaling back",
     [("float mag = ((float)levels[i] * step) * down;", "float mag = (float)levels[i] * step;")]),
    ("qsgd_segment_counter", "every segment restarts the random counter at 0",
     [("oracle_qsgd_encode(n, a, p + a, sc, D->levels,", "oracle_qsgd_encode(n, 0, p + a, sc, D->levels,")]),
    ("philox_word", "uniform from the wrong output word",
     [("uint32_t word = out[i & 3];", "uint32_t word = out[(i >> 2) & 3];")]),
    ("philox_key", "second key word advanced by the first Weyl constant",
     [("k1 += PHILOX_W1;", "k1 += PHILOX_W0;")]),
    ("philox_counter", "worker and iteration swapped in the counter",
     [("{(uint32_t)block, (uint32_t)m, t, (uint32_t)(block >> 32)}",
       "{(uint32_t)block, t, (uint32_t)m, (uint32_t)(block >> 32)}")]),
    ("philox_rounds", "seven rounds instead of ten",
     [("round < 10", "round < 7")]),
    ("uniform_bits", "uniform from 23 bits",
     [("(float)(word >> 8) * 0x1.0p-24f", "(float)(word >> 9) * 0x1.0p-24f")]),
    ("topk_tie", "ties to the higher index",
     [("return (x->idx < y->idx) ? -1 : 1;", "return (x->idx > y->idx) ? -1 : 1;")]),
    ("topk_signed", "top-k by signed value, not magnitude",
     [("float a = fabsf(v);", "float a = v;")]),
    ("topk_idx_unsorted", "indices sent in selection order",
     [("qsort(idx, (size_t)k, sizeof(uint32_t), idx_cmp);", "")]),
    ("topk_residual", "top-k leaves the residual at p on the kept set",
     [("e_out[i] = p[i] - p[i];", "e_out[i] = p[i];")]),
    ("pack_msb_first", "bit fields packed and unpacked high to low",
     [("words[i / per] |= f << (uint32_t)(b * (i % per));",
       "words[i / per] |= f << (uint32_t)(b * (per - 1 - i % per));"),
      ("fields[i] = (uint16_t)((words[i / per] >> (uint32_t)(b * (i % per))) & mask);",
       "fields[i] = (uint16_t)((words[i / per] >> (uint32_t)(b * (per - 1 - i % per))) & mask);")]),
    ("decode_sign_flip", "server decodes the sign plane reversed",
     [("phat[i] = signs[i] ? -scale : scale;", "phat[i] = signs[i] ? scale : -scale;")]),
    ("decode_step", "server decodes levels with s + 1 steps",
     [("if (kind == 1 && qsgd_range(scale, &up, &down)) step = (scale * up) / (float)s;",
       "if (kind == 1 && qsgd_range(scale, &up, &down)) step = (scale * up) / (float)(s + 1);")]),
    ("mbit_split_mask", "m-bit split keeps the sign bit in the level",
     [("uint16_t mask = (uint16_t)((1u << (mbits - 1)) - 1u);", "uint16_t mask = (uint16_t)((1u << mbits) - 1u);")]),
    ("linf_flag_ignored", "the quantizer ignores the max-norm flag",
     [("else if (D->norm == 3) sc = oracle_scale_linf(n, p + a);",
       "else if (D->norm == 4) sc = oracle_scale_linf(n, p + a);")]),
    ("server_order", "server sum in descending worker order",
     [("float S = phat[i];\n        for (int32_t m = 1; m < M; ++m) S = S + phat[(int64_t)m * ld + i];",
       "float S = phat[(int64_t)(M - 1) * ld + i];\n        for (int32_t m = M - 2; m >= 0; --m) S = S + phat[(int64_t)m * ld + i];"),
      ("    for (int32_t m = 0; m < M; ++m) {\n        const float *g", "    for (int32_t m = M - 1; m >= 0; --m) {\n        const float *g"),
      ("if (m == 0) for (int64_t i = 0; i < d; ++i) S[i] = dec[i];",
       "if (m == M - 1) for (int64_t i = 0; i < d; ++i) S[i] = dec[i];")]),
    ("server_reciprocal", "average as the sum times fl(1/M)",
     [("qhat[i] = S / (float)M;", "qhat[i] = S * (1.0f / (float)M);"),
      ("qhat[i] = S[i] / (float)M;", "qhat[i] = S[i] * (1.0f / (float)M);")]),
    ("omd_sign", "OMD update adds the average",
     [("w[i] = w[i] - qhat[i];", "w[i] = w[i] + qhat[i];")]),
    ("wx_without_e", "evaluation point without the second error compensation",
     [("float x = eg + e[i];", "float x = eg;")]),
    ("wx_from_old_w", "evaluation point from w_{t-1}",
     [("    oracle_omd_update(d, qhat, W);\n    for (int32_t m = 0; m < M; ++m)\n"
       "        oracle_extrapolate(d, eta, W, G + (int64_t)m * ld, E + (int64_t)m * ld, WX + (int64_t)m * ld);",
       "    for (int32_t m = 0; m < M; ++m)\n"
       "        oracle_extrapolate(d, eta, W, G + (int64_t)m * ld, E + (int64_t)m * ld, WX + (int64_t)m * ld);\n"
       "    oracle_omd_update(d, qhat, W);")]),
    ("mbit_sign_bit", "m-bit code with the sign one bit too high",
     [("((uint32_t)bits[i] << (mbits - 1))", "((uint32_t)bits[i] << mbits)")]),
    ("mbit_levels", "m-bit quantizer with 2^(m-1) levels",
     [("int32_t mlevels = mbits ? (1 << (mbits - 1)) - 1 : 0;", "int32_t mlevels = mbits ? (1 << (mbits - 1)) : 0;")]),
]


def _altered_source(edits):
    with open(ORACLE_SRC) as f:
        src = f.read()
    for old, new in edits:
        assert old in src, "planted-mistake entry no longer matches the oracle source: %r" % old[:60]
        src = src.replace(old, new, 1)
    return src


def _run_one(entry, scratch):
    name, _, edits = entry
    d = os.path.join(scratch, name)
    os.makedirs(d)
    with open(os.path.join(d, "dqgan_oracle.c"), "w") as f:
        f.write(_altered_source(edits))
    env = dict(os.environ, DQGAN_ORACLE_DIR=d)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu"]
                       + PIN_FILES, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return name, r.returncode, (r.stdout + r.stderr)[-1500:]


def test_planted_mistake_entries_apply():
    for name, _, edits in MUTATIONS:
        assert _altered_source(edits) != _altered_source([]), name


def test_every_planted_mistake_fails_a_pin(tmp_path):
    assert PIN_FILES
    scratch = str(tmp_path)
    with concurrent.futures.ThreadPoolExecutor(max_workers=4) as ex:
        results = list(ex.map(lambda e: _run_one(e, scratch), MUTATIONS))
    shutil.rmtree(scratch, ignore_errors=True)
    # pytest exit status 1 = some test failed; 0 would mean the mistake went
    # unnoticed; anything else (collection error, crash) is not a pin failure
    bad = [(n, rc, out) for n, rc, out in results if rc != 1]
    assert not bad, "\n\n".join("%s: pytest exit %d\n%s" % b for b in bad)
