"""Mutation check of the oracle's pins (no GPU): each case plants one
plausible mistake in a copy of the oracle -- in oracle.c (a dropped term, a
wrong sign, a swapped operand, an off-by-one, a wrong constant, a different
rounding) or in the segment walkers of oracle/__init__.py (a segment given
another segment's hyperparameters, a segment digested at the wrong flat
index) -- and runs the pin suite against it.  Only tests/test_oracle_pins.py
runs: the stored oracle-written digests under tests/golden/ would trip on
almost any change and so cannot show that the pins themselves bite.  Every
mutant must fail at least one pin; the unmutated copies must pass them all."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
PIN_FILES = ["tests/test_oracle_pins.py"]
PY_SRC = os.path.join(ROOT, "oracle", "__init__.py")
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


def _pins_pass(basetemp, lib=None, root=ROOT):
    env = dict(os.environ)
    if lib is not None:
        env["PACT_ORACLE_LIB"] = str(lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        f"--basetemp={basetemp}", *PIN_FILES],
                       cwd=root, env=env, capture_output=True, text=True)
    return r.returncode == 0, r.stdout[-400:]


# (name, text to find, replacement); each text must occur in oracle/__init__.py
PY_MUTANTS = [
    ("walker gives every segment the first hyper set", "bf16[sl], hypers[hi], step,", "bf16[sl], hypers[0], step,"),
    ("walker digests each segment at the shard start", "global_offset + off)\n        per.append(d)",
     "global_offset)\n        per.append(d)"),
    ("walker ignores the shard's global offset", "global_offset + off)\n        per.append(d)",
     "off)\n        per.append(d)"),
    ("read-only walker drops the segment offset", "v[sl], global_offset + off))",
     "v[sl], global_offset))"),
]


def _tree_with_oracle_init(tmp_path, init_text):
    """A copy of the repository made of symlinks, except oracle/__init__.py,
    which holds `init_text`: the pins then import that oracle module."""
    root = tmp_path / "root"
    root.mkdir()
    for name in os.listdir(ROOT):
        if name in ("oracle", ".git", "_work", "gpurun_out", ".pytest_cache", "__pycache__"):
            continue
        os.symlink(os.path.join(ROOT, name), root / name)
    od = root / "oracle"
    od.mkdir()
    for name in os.listdir(os.path.join(ROOT, "oracle")):
        if name not in ("__init__.py", "__pycache__"):
            os.symlink(os.path.join(ROOT, "oracle", name), od / name)
    (od / "__init__.py").write_text(init_text)
    return root


# every case: (id, kind, text to find or None, replacement)
CASES = ([("clean oracle.c", "c", None, None)] + [(n, "c", f, r) for n, f, r in MUTANTS]
         + [("clean walker", "py", None, None)] + [(n, "py", f, r) for n, f, r in PY_MUTANTS])


@pytest.fixture(scope="module")
def outcomes(tmp_path_factory):
    """Runs the pin suite once per case, several cases at a time (each in its
    own process with its own oracle); returns {id: (pins passed, tail)}."""
    def run(case):
        name, kind, find, repl = case
        src = SRC if kind == "c" else PY_SRC
        text = open(src).read()
        if find is not None:
            if text.count(find) != 1:
                return None
            text = text.replace(find, repl)
        d = tmp_path_factory.mktemp("case")
        if kind == "c":
            return _pins_pass(d / "pytest", lib=_build(d, text, "oracle_case"))
        return _pins_pass(d / "pytest", root=_tree_with_oracle_init(d, text))

    with ThreadPoolExecutor(max(1, min(6, os.cpu_count() or 1))) as ex:
        return dict(zip([c[0] for c in CASES], ex.map(run, CASES)))


@pytest.mark.parametrize("name", ["clean oracle.c", "clean walker"])
def test_unmutated_copy_passes(outcomes, name):
    ok, out = outcomes[name]
    assert ok, out


@pytest.mark.parametrize("name", [c[0] for c in CASES if c[2] is not None])
def test_mutant_is_caught(outcomes, name):
    assert outcomes[name] is not None, f"mutation site not unique: {name}"
    ok, out = outcomes[name]
    assert not ok, f"the pins did not catch: {name}"
