"""The oracle's pins reject a broken oracle.

Each case copies oracle/bsref.c, plants one plausible mistake in the copy (a
wrong rounding, sign, index, bit order, dropped term or transposed operand),
builds it with the oracle's own gcc command line, and runs the oracle pin
tests (test_oracle_*.py, CPU only) against that build in a subprocess: at
least one pin must fail.  The unmodified copy, built the same way, must pass
them all, so a failure comes from the planted mistake and not from the
harness.  Every mistake keeps the copy's memory accesses in bounds.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from oracle import bsref  # noqa: E402

PIN_TESTS = ["tests/test_oracle_worked.py", "tests/test_oracle_quantize_pack.py",
             "tests/test_oracle_conv_dense.py", "tests/test_oracle_encodings.py"]

# (name, original text of bsref.c, planted replacement)
MUTANTS = [
    ("round_half_up",
     "float r = rintf(product);", "float r = floorf(product + 0.5f);"),
    ("saturate_below_top_code",
     "v = (uint8_t)qmax;", "v = (uint8_t)(qmax - 1);"),
    ("bipolar_zero_is_minus_one",
     "q[i] = (x[i] >= 0.0f) ? 1 : 0;", "q[i] = (x[i] > 0.0f) ? 1 : 0;"),
    ("signed_saturates_one_high",
     "                v = smin;", "                v = smin + 1;"),
    ("pack_msb_first",
     "word |= bit << u;", "word |= bit << (31 - u);"),
    ("pack_planes_reversed",
     "uint32_t bit = ((uint32_t)q[r * k + e] >> b) & 1u;",
     "uint32_t bit = ((uint32_t)q[r * k + e] >> (bits - 1 - b)) & 1u;"),
    ("pack_tail_takes_next_row",
     "                    if (e < k) {\n                        uint32_t bit",
     "                    if (e < k || (e == k && r + 1 < rows)) {\n"
     "                        uint32_t bit"),
    ("pack_ex_inner_reversed",
     "uint8_t v = q[(o * k + e) * inner + i];",
     "uint8_t v = q[(o * k + e) * inner + (inner - 1 - i)];"),
    ("bipolar_levels_negated",
     "level = 2 * bit - 1;", "level = 1 - 2 * bit;"),
    ("signed_top_plane_positive",
     "level = -bit;", "level = bit;"),
    ("plane_weights_reversed",
     "v += level * ((int64_t)1 << j);",
     "v += level * ((int64_t)1 << (bits - 1 - j));"),
    ("padding_added_not_subtracted",
     "int64_t ih = y * p->stride_h - p->pad_h + r;",
     "int64_t ih = y * p->stride_h + p->pad_h + r;"),
    ("width_uses_height_stride",
     "int64_t iw = x * p->stride_w - p->pad_w + s;",
     "int64_t iw = x * p->stride_h - p->pad_w + s;"),
    ("filter_flipped",
     "wts + ((o * p->kh + r) * p->kw + s) * p->wbits * cw;",
     "wts + ((o * p->kh + (p->kh - 1 - r)) * p->kw + (p->kw - 1 - s)) *"
     " p->wbits * cw;"),
    ("conv_drops_channel_0",
     "for (int64_t c = 0; c < p->c; ++c)", "for (int64_t c = 1; c < p->c; ++c)"),
    ("dense_drops_term_0",
     "for (int64_t c = 0; c < k; ++c)", "for (int64_t c = 1; c < k; ++c)"),
    ("output_size_rounds_up",
     "*oh = (int32_t)(eh / p->stride_h + 1);",
     "*oh = (int32_t)((eh + p->stride_h - 1) / p->stride_h + 1);"),
    ("dense_ignores_activation_encoding",
     "sum += code_value(avec, kw, abits, aenc, c) *",
     "sum += code_value(avec, kw, abits, BSREF_UNIPOLAR, c) *"),
]


def build_copy(tmp_path, mutation=None):
    src_dir = os.path.join(ROOT, "oracle")
    for f in ("bsref.c", "bsref.h"):
        shutil.copy(os.path.join(src_dir, f), tmp_path / f)
    if mutation is not None:
        old, new = mutation
        text = (tmp_path / "bsref.c").read_text()
        assert text.count(old) == 1, "mutation site not unique: %r" % old
        (tmp_path / "bsref.c").write_text(text.replace(old, new))
    lib = str(tmp_path / "libbsref_copy.so")
    bsref.compile_to(str(tmp_path / "bsref.c"), lib)
    return lib


def run_pins(lib):
    env = dict(os.environ, BSREF_LIBRARY=lib)
    r = subprocess.run(
        [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
         "-m", "not gpu and not slow"] + PIN_TESTS,
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout + r.stderr


def test_unmodified_copy_passes_the_pins(tmp_path):
    rc, out = run_pins(build_copy(tmp_path))
    assert rc == 0, out[-2000:]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(tmp_path, name, old, new):
    rc, out = run_pins(build_copy(tmp_path, (old, new)))
    assert rc == 1 and "failed" in out, \
        "mutant %s survived the pins:\n%s" % (name, out[-2000:])
