"""Mutation check of the oracle's pins (no GPU): each case plants one
plausible mistake in a copy of oracle.c (a dropped term, a wrong sign, a
swapped operand, an off-by-one, a wrong constant, a different rounding),
builds it, and runs the pin suite against it.  Every mutant must fail at
least one pin; the unmutated copy must pass them all."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PIN_FILES = ["tests/test_oracle_pins.py", "tests/test_golden.py"]
FLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fno-math-errno",
         "-fexcess-precision=standard", "-fPIC", "-shared"]

# (name, text to find, replacement); each text must occur in oracle.c
MUTANTS = [
    ("no weight decay", "const float w_decayed = w * sc->decay;", "const float w_decayed = w;"),
    ("update sign flipped", "const float w_next = w_decayed - delta;", "const float w_next = w_decayed + delta;"),
    ("beta2 used for m", "const float m_keep = sc->beta1 * m_prev;", "const float m_keep = sc->beta2 * m_prev;"),
    ("1-beta1 used for v", "const float v_push = sc->omb2 * grad_sq;", "const float v_push = sc->omb1 * grad_sq;"),
    ("g instead of g^2", "const float grad_sq = grad * grad;", "const float grad_sq = grad;"),
    ("eps inside the root", "const float root = sqrtf(v_next);", "const float root = sqrtf(v_next + sc->eps);"),
    ("no bias correction of the step", "out->step_size = (float)(lr / (1.0 - b1_pow));",
     "out->step_size = (float)lr;"),
    ("bias2 from beta1", "out->rs_bc2 = (float)(1.0 / sqrt(1.0 - b2_pow));",
     "out->rs_bc2 = (float)(1.0 / sqrt(1.0 - b1_pow));"),
    ("one power too many", "for (uint64_t t = 0; t < step; t++) {", "for (uint64_t t = 0; t <= step; t++) {"),
    ("decay from lr alone", "out->decay = (float)(1.0 - lr * wd);", "out->decay = (float)(1.0 - wd);"),
    ("ties away from zero", "if (dropped > half || (dropped == half && (kept & 1u) != 0u)) {",
     "if (dropped >= half) {"),
    ("bf16 truncates", "kept = kept + 1u;", "kept = kept;"),
    ("splitmix shift 30 -> 31", "z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;",
     "z = (z ^ (z >> 31)) * 0xBF58476D1CE4E5B9ull;"),
    ("splitmix without gamma", "uint64_t z = x + 0x9E3779B97F4A7C15ull;", "uint64_t z = x;"),
    ("m tag in bit 55", "sum += oracle_splitmix64((uint64_t)f32_bits(m[i]) ^ (index | (1ull << 56)));",
     "sum += oracle_splitmix64((uint64_t)f32_bits(m[i]) ^ (index | (1ull << 55)));"),
    ("index off by one", "        const uint64_t index = first_index + i;\n        sum += oracle_splitmix64((uint64_t)f32_bits(p[i])",
     "        const uint64_t index = first_index + i + 1;\n        sum += oracle_splitmix64((uint64_t)f32_bits(p[i])"),
    ("words sign-extended", "sum += oracle_splitmix64((uint64_t)f32_bits(p[i]) ^ (index | (0ull << 56)));",
     "sum += oracle_splitmix64((uint64_t)(int64_t)(int32_t)f32_bits(p[i]) ^ (index | (0ull << 56)));"),
    ("v dropped from the digest", "sum += oracle_splitmix64((uint64_t)f32_bits(v[i]) ^ (index | (2ull << 56)));",
     ""),
    ("bf16 digest tag 2", "sum += oracle_splitmix64((uint64_t)b[i] ^ (index | (3ull << 56)));",
     "sum += oracle_splitmix64((uint64_t)b[i] ^ (index | (2ull << 56)));"),
    ("zeroed gradient is -0", "g[i] = 0.0f;", "g[i] = -0.0f;"),
    ("guard compares values", "if (f32_bits(g[i]) != 0u) {", "if (g[i] != 0.0f) {"),
    ("bf16 state m truncated", "m[i] = oracle_bf16_rne(f32_bits(mm));", "m[i] = (uint16_t)(f32_bits(mm) >> 16);"),
    ("bf16 state digest tag swap", "sum += oracle_splitmix64((uint64_t)m[i] ^ (index | (1ull << 56)));",
     "sum += oracle_splitmix64((uint64_t)m[i] ^ (index | (2ull << 56)));"),
]


def _build(tmp_path, text, name):
    src = tmp_path / f"{name}.c"
    src.write_text(text)
    lib = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", *FLAGS, "-I", os.path.join(ROOT, "oracle"), "-o", str(lib), str(src), "-lm"],
                   check=True)
    return lib


def _pins_pass(lib):
    env = dict(os.environ, PACT_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PIN_FILES],
                       cwd=ROOT, env=env, capture_output=True, text=True)
    return r.returncode == 0, r.stdout[-400:]


def test_unmutated_copy_passes(tmp_path):
    ok, out = _pins_pass(_build(tmp_path, open(SRC).read(), "clean"))
    assert ok, out


@pytest.mark.parametrize("name,find,repl", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, find, repl):
    text = open(SRC).read()
    assert text.count(find) == 1, f"mutation site not unique: {name}"
    ok, out = _pins_pass(_build(tmp_path, text.replace(find, repl), "mutant"))
    assert not ok, f"the pins did not catch: {name}"
