"""The CPU oracle, pinned (CPU only).

See ``oracle_pins.py`` for what each pin checks.  The mutation test below
plants plausible mistakes in copies of the oracle's C source (sign, index,
operand, scale, rounding, packing) and requires each copy to fail a pin, so
the pins are shown to have teeth.
"""
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle
from oracle import brute

import oracle_pins as P


@pytest.mark.parametrize("pin", P.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(orc, pin):
    pin(orc)


# ---------------------------------------------------- the numpy twin, pinned

def test_brute_attention_is_sdpa():
    rng = np.random.default_rng(20)
    q, k, v = rng.standard_normal((3, 2, 3, 21, 128))
    out, p = brute.attention_np(q, k, v)
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v)).numpy()
    assert np.allclose(out, want, atol=1e-12)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-14)


def test_brute_nearest_bf16_is_torch_on_float32():
    rng = np.random.default_rng(21)
    x = (rng.standard_normal(5000) * np.exp2(rng.integers(-60, 60, 5000))).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(brute.nearest_bf16(x.astype(np.float64)), want)


def test_brute_positions_grid():
    pos = brute.grid_positions(2 + 2 * 3 * 4, 2, 3, 4)
    assert (pos[:2] == -1).all()
    assert tuple(pos[2]) == (0, 0, 0) and tuple(pos[3]) == (0, 0, 1)
    assert tuple(pos[2 + 4]) == (0, 1, 0) and tuple(pos[2 + 12]) == (1, 0, 0)
    assert tuple(pos[-1]) == (1, 2, 3)


def test_oracle_rejects_bad_arguments(orc):
    q = np.zeros((1, 1, 4, 128), np.uint16)
    with pytest.raises(ValueError):
        orc.attn_rows(q, q, q, 2, 2, 2)            # grid larger than the sequence
    with pytest.raises(ValueError):
        orc.attn_rows(q, q, q, 1, 1, 1, rows=np.array([4]))   # row out of range
    with pytest.raises(TypeError):
        orc.attn_rows(q.astype(np.float32), q, q, 1, 1, 1)


# ------------------------------------------------------------ mutation test

_NORM_THEN_ROTATE = """  if (gamma) {
    rms_normalize(dst, D, gamma, eps);
    changed = 1;
  }
  int pt, ph, pw;
  if (use_rope && token_position(n, N, T, Hl, Wl, &pt, &ph, &pw)) {
    rotate_vector(dst, D, dt, dh, dw, base, pt, ph, pw);
    changed = 1;
  }
"""
_ROTATE_THEN_NORM = """  int pt, ph, pw;
  if (use_rope && token_position(n, N, T, Hl, Wl, &pt, &ph, &pw)) {
    rotate_vector(dst, D, dt, dh, dw, base, pt, ph, pw);
    changed = 1;
  }
  if (gamma) {
    rms_normalize(dst, D, gamma, eps);
    changed = 1;
  }
"""

MUTANTS = [
    ("rotation turns the wrong way",
     "x[off + 2 * i] = re * c - im * s;\n      x[off + 2 * i + 1] = re * s + im * c;",
     "x[off + 2 * i] = re * c + im * s;\n      x[off + 2 * i + 1] = -re * s + im * c;"),
    ("frequency exponent over the whole head dim",
     "pow(base, -2.0 * i / (double)d)", "pow(base, -2.0 * i / (double)D)"),
    ("frequency index off by one",
     "pow(base, -2.0 * i / (double)d)", "pow(base, -2.0 * (i + 1) / (double)d)"),
    ("axis chunks not advanced", "    off += d;\n", "\n"),
    ("rotary split ignored (default widths)", "    int d = widths[a];", "    int d = a ? 3 * D / 8 : D / 4;"),
    ("h/w raster swapped", "*ph = (int)((r / Wl) % Hl);", "*ph = (int)(r % Hl);"),
    ("prefix tokens rotated", "if (n < nt) return 0;", "if (n < 0) return 0;"),
    ("softmax scale dropped", "s[j] = dot * scale;", "s[j] = dot;"),
    ("exponent sign flipped", "double p = exp(s[j] - m);", "double p = exp(m - s[j]);"),
    ("normaliser dropped", "(float)(acc[d] / l)", "(float)(acc[d])"),
    ("keys used as values", "const double* vj = J->vd + (int64_t)j * D;",
     "const double* vj = J->khat + (int64_t)j * D;"),
    ("ties rounded away from zero",
     "if (rem > 0.5 || (rem == 0.5 && fmod(fl, 2.0) != 0.0)) fl += 1.0;\n  double r = fl * quantum;",
     "if (rem >= 0.5) fl += 1.0;\n  double r = fl * quantum;"),
    ("rotated q/k not rounded to bf16", "  if (contract && changed)\n", "  if (0)\n"),
    ("dot product skips the last dim", "for (int d = 0; d < D; ++d) dot += qhat[d] * kj[d];",
     "for (int d = 0; d < D - 1; ++d) dot += qhat[d] * kj[d];"),
    # QK normalization
    ("norm: mean over the head dim dropped", "sqrt(ss / (double)D + eps)", "sqrt(ss + eps)"),
    ("norm: eps outside the root", "1.0 / sqrt(ss / (double)D + eps)",
     "1.0 / (sqrt(ss / (double)D) + eps)"),
    ("norm: square root missing", "1.0 / sqrt(ss / (double)D + eps)", "1.0 / (ss / (double)D + eps)"),
    ("norm: weights not applied", "x[d] = x[d] * inv * gamma[d];", "x[d] = x[d] * inv;"),
    ("norm: weights reversed", "x[d] * inv * gamma[d]", "x[d] * inv * gamma[D - 1 - d]"),
    ("norm: applied after the rotation", _NORM_THEN_ROTATE, _ROTATE_THEN_NORM),
    ("norm: prefix tokens skipped", "  if (gamma) {\n    rms_normalize",
     "  if (gamma && n >= (int64_t)N - (int64_t)T * Hl * Wl) {\n    rms_normalize"),
    ("norm: keys not normalised", "J->base, J->kside.rope, J->contract, J->kside.gamma, J->eps);",
     "J->base, J->kside.rope, J->contract, NULL, J->eps);"),
    # FP8 E4M3 output codes
    ("e4m3: ties rounded away from zero", "if (rem > 0.5 || (rem == 0.5 && ((int64_t)fl & 1))) fl += 1.0;",
     "if (rem >= 0.5) fl += 1.0;"),
    ("e4m3: subnormal quantum halved", "if (e < -6) e = -6;", "if (e < -7) e = -7;"),
    ("e4m3: exponent bias 8", "((e + 7) << 3)", "((e + 8) << 3)"),
    ("e4m3: no saturation", "if (a >= 448.0) return sign | 0x7e;", "if (a >= 480.0) return sign | 0x7f;"),
    # block-sparse routing and attention
    ("sparse: sample standard deviation", "sqrt(var / (double)nkb)", "sqrt(var / (double)(nkb - 1))"),
    ("sparse: threshold below the mean", "mu + tau * sqrt", "mu - tau * sqrt"),
    ("sparse: prefix sink dropped", "const int sink = (int64_t)J * kblk < nt;", "const int sink = 0;"),
    ("sparse: prefix queries not dense", "const int dense = (int64_t)I * qblk < nt;", "const int dense = 0;"),
    ("sparse: best block not kept", "dense || sink || J == best || s[J] > t", "dense || sink || s[J] > t"),
    ("sparse: key blocks summed, not averaged", "kbar[J * D + d] /= (double)keys;", "(void)keys;"),
    ("sparse: mask ignored", "if (keep && !keep[j / J->kblk]) s[j] = -INFINITY;", "(void)keep;"),
    # block-INT8 QKV records
    ("records: scale needs 127 s > max", "if (127.0 * ue5m3_value((uint8_t)mid) >= amax) past = mid;",
     "if (127.0 * ue5m3_value((uint8_t)mid) > amax) past = mid;"),
    ("records: scale rounded down", "if (127.0 * ue5m3_value((uint8_t)mid) >= amax) past = mid;",
     "if (127.0 * ue5m3_value((uint8_t)(mid + 1)) > amax) past = mid;"),
    ("records: codes tie away from zero",
     "if (rem > 0.5 || (rem == 0.5 && fmod(fl, 2.0) != 0.0)) fl += 1.0;\n  if (fl > 127.0)",
     "if (rem >= 0.5) fl += 1.0;\n  if (fl > 127.0)"),
    ("records: codes truncated", "double y = x / s;", "double y = trunc(x / s);"),
    ("records: codes reach -128", "if (fl < -127.0) fl = -127.0;", "if (fl < -128.0) fl = -128.0;"),
    ("records: scale slots group-major", "r[REC_SCALES + 4 * p + g] = sc;", "r[REC_SCALES + 3 * g + p] = sc;"),
    ("records: head-major record order",
     "        uint8_t* r = rec + (((int64_t)b * N + n) * H + h) * REC_BYTES;",
     "        uint8_t* r = rec + (((int64_t)b * H + h) * N + n) * REC_BYTES;"),
    ("records: decode truncated to bf16",
     "x[d] = double_to_bf16((double)(int8_t)r[128 * p + d] * s);",
     "{ float f = (float)((double)(int8_t)r[128 * p + d] * s); uint32_t u; memcpy(&u, &f, 4);"
     " x[d] = (uint16_t)(u >> 16); }"),
    ("ue5m3: exponent bias 16", "return ldexp(8.0 + m, e - 18);", "return ldexp(8.0 + m, e - 19);"),
    ("ue5m3: subnormals read as normals", "if (e == 0) return ldexp((double)m, -17);",
     "if (e == 0) return ldexp(8.0 + m, -18);"),
    ("out records: group max over 16 values",
     "for (int d = 32 * g; d < 32 * g + 32; ++d) amax = fmax(amax, fabs(xr[d]));",
     "for (int d = 32 * g; d < 32 * g + 16; ++d) amax = fmax(amax, fabs(xr[d]));"),
    ("out records: scales one slot late", "o[128 + g] = sc;", "o[129 + g] = sc;"),
    # queries and keys of different lengths
    ("key count taken from the queries", "for (int j = 0; j < Nkv; ++j) {\n    const double* kj",
     "for (int j = 0; j < Nkv && j < J->qs.N; ++j) {\n    const double* kj"),
]


@pytest.mark.parametrize("name,find,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, find, repl):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "solref.c")).read()
    assert src.count(find) == 1, "mutation anchor not found: %s" % name
    path = tmp_path / "solref_mut.c"
    path.write_text(src.replace(find, repl))
    lib = tmp_path / "libsolref_mut.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", str(path), "-o",
                    str(lib), "-lm"], check=True)
    mutant = oracle.Oracle(str(lib))
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(mutant)
        except AssertionError:
            failed.append(pin.__name__)
    assert failed, "no pin caught: %s" % name
