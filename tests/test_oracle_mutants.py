"""Mutation check of the oracle's pins.

Each mutant plants one plausible mistake in a copy of ``oracle/`` (a dropped
term, a wrong sign, index, constant or tie rule, a swapped operand) and runs
the oracle pin tests (``tests/test_oracle_*.py``) against the copy; at least
one pin must fail for every mutant.  The unmutated copy must pass (the
control).  Nothing here touches the repository's own ``oracle/``; mutants
live in a temporary directory, on the CPU.
"""

import glob
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, file under oracle/, exact text, replacement); the text must occur
# exactly once in the file.
MUTANTS = [
    # formats: grids, tie rules, bf16 rounding
    ("e2m1_tie_odd", "formats.py", "tie_goes_up = (j + 1) % 2 == 0", "tie_goes_up = (j + 1) % 2 == 1"),
    ("e4m3_subnormal_exponent", "formats.py", "mag = man * 2.0 ** -9", "mag = man * 2.0 ** -10"),
    ("e2m1_exponent_bias", "formats.py", "mag = (1.0 + man / 2.0) * 2.0 ** (exp - 1)",
     "mag = (1.0 + man / 2.0) * 2.0 ** (exp - 2)"),
    ("e4m3_tie_odd", "formats.py", "on_tie & ((below + 1) % 2 == 0)", "on_tie & ((below + 1) % 2 == 1)"),
    ("bf16_truncates", "formats.py", "np.rint(np.ldexp(m, 8))", "np.floor(np.ldexp(m, 8))"),
    ("range_4_not_6", "formats.py", "NVFP4_RANGE = E2M1_MAX * E4M3_MAX", "NVFP4_RANGE = 4.0 * E4M3_MAX"),
    # quant: scale rule, sign, packing, zero scales, amax, dequantization
    ("scale_over_4", "quant.py", "rne_index_sorted(amax_b * g, 6.0, E4M3_GRID)",
     "rne_index_sorted(amax_b * g, 4.0, E4M3_GRID)"),
    ("sign_from_less_than", "quant.py", "sign = np.signbit(x).astype(np.int64)",
     "sign = (x < 0).astype(np.int64)"),
    ("nibbles_swapped", "quant.py", "(codes[:, 0::2] | (codes[:, 1::2] << 4))",
     "(codes[:, 1::2] | (codes[:, 0::2] << 4))"),
    # (with S = 0 the codes are forced to 0; dividing by a tiny stand-in for
    # S instead lets |x| G / S round to non-zero codes)
    ("zero_scale_keeps_codes", "quant.py",
     "den = np.where(zero_scale, 1.0, s)[:, :, None]\n    mag = rne_index(ax * g, den, E2M1_GRID)\n"
     "    mag[np.broadcast_to(zero_scale[:, :, None], mag.shape)] = 0",
     "den = np.where(zero_scale, 2.0 ** -12, s)[:, :, None]\n    mag = rne_index(ax * g, den, E2M1_GRID)"),
    ("amax_with_sign_bit", "quant.py", "mag = (x_bits & np.uint16(0x7FFF)).max()", "mag = x_bits.max() & 0x7FFF"),
    ("dequant_multiplies_g", "quant.py", "return v / g if g != 0.0", "return v * g if g != 0.0"),
    ("decode_sign_bit", "quant.py", "np.where(codes & 8, -mag, mag)", "np.where(codes & 4, -mag, mag)"),
    ("g_off_by_one_ulp", "quant.py", "g = np.float32(NVFP4_RANGE / amax)",
     "g = np.nextafter(np.float32(NVFP4_RANGE / amax), np.float32(np.inf))"),
    # gemm: segment scales, the tolerance bound, the exact form
    ("abs_bound_drops_alpha", "gemm.py", "return (a @ w.T) * np.abs(alpha)[None, :]", "return (a @ w.T)"),
    ("abs_bound_drops_abs", "gemm.py", "a = np.abs(decode_unscaled(a_packed, a_scales))",
     "a = decode_unscaled(a_packed, a_scales)"),
    ("alpha_of_segment_0", "gemm.py", "float(np.float32(g_w_seg[s]))", "float(np.float32(g_w_seg[0]))"),
    ("exact_scale_2_19", "gemm.py", "acc.astype(np.float64) * 2.0 ** -20", "acc.astype(np.float64) * 2.0 ** -19"),
    ("exact_scale_operand", "gemm.py", "(E4M3_GRID[scales] * 512.0)", "(E4M3_GRID[scales] * 256.0)"),
    ("gemm_transposed_block", "gemm.py", 'np.einsum("mbi,nbi->mnb", ea, ew)', 'np.einsum("mbi,nbi->mnb", ea, ew[:, :, ::-1])'),
    # norm: where eps enters, mean vs sum, gamma
    ("eps_outside_sqrt", "norm.py", "x / np.sqrt(ms + float(np.float32(eps)))[:, None]",
     "x / (np.sqrt(ms) + float(np.float32(eps)))[:, None]"),
    ("eps_times_10", "norm.py", "np.sqrt(ms + float(np.float32(eps)))", "np.sqrt(ms + 10.0 * float(np.float32(eps)))"),
    ("sum_not_mean", "norm.py", "ms = np.mean(x * x, axis=1)", "ms = np.sum(x * x, axis=1)"),
    ("gamma_dropped", "norm.py", "[:, None] * g[None, :]", "[:, None]"),
    # harmonize: direction of the shared scale, direction of the fold
    ("shared_is_max", "harmonize.py", "np.float32(pos.min())", "np.float32(pos.max())"),
    ("fold_inverted", "harmonize.py", "out[a:b] = rne_index_sorted(num, g, E4M3_GRID)",
     "out[a:b] = rne_index_sorted(E4M3_GRID[scales[a:b].astype(np.int64)] * g, gs, E4M3_GRID)"),
    # gates (Eq. 1)
    ("sigmoid_flipped", "gates.py", "np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))",
     "np.where(x >= 0, e / (1.0 + e), 1.0 / (1.0 + e))"),
    ("a_log_not_exponentiated", "gates.py", "-np.exp(np.asarray(a_log, dtype=np.float64))",
     "-np.asarray(a_log, dtype=np.float64)"),
    ("dt_bias_subtracted", "gates.py", "y[:, h:] + np.asarray(dt_bias", "y[:, h:] - np.asarray(dt_bias"),
]


def _stage(tmp, mutant):
    """A minimal tree in tmp: the (mutated) oracle, its pin tests and the
    input helpers they use."""
    shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(tmp, "oracle"),
                    ignore=shutil.ignore_patterns("__pycache__"))
    os.makedirs(os.path.join(tmp, "tests"))
    for f in ["__init__.py", "conftest.py", "bruteforce.py"] + \
            [os.path.basename(p) for p in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py"))
             if not p.endswith("test_oracle_mutants.py")]:
        shutil.copy(os.path.join(ROOT, "tests", f), os.path.join(tmp, "tests", f))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), os.path.join(tmp, "tests", "golden"))
    os.makedirs(os.path.join(tmp, "paper_2609_04098_amd"))
    for f in ["__init__.py", "synth.py"]:
        shutil.copy(os.path.join(ROOT, "paper_2609_04098_amd", f), os.path.join(tmp, "paper_2609_04098_amd", f))
    shutil.copy(os.path.join(ROOT, "pytest.ini"), os.path.join(tmp, "pytest.ini"))
    if mutant is not None:
        _, fname, old, new = mutant
        path = os.path.join(tmp, "oracle", fname)
        text = open(path).read()
        assert text.count(old) == 1, "mutant text must occur once in %s: %r" % (fname, old)
        open(path, "w").write(text.replace(old, new))


def _pins_pass(mutant):
    tmp = tempfile.mkdtemp(prefix="oracle_mutant_")
    try:
        _stage(tmp, mutant)
        env = dict(os.environ, PYTHONDONTWRITEBYTECODE="1")
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "tests"],
                           cwd=tmp, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, timeout=600)
        return r.returncode == 0, r.stdout.decode(errors="replace")[-2000:]
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


def test_mutant_texts_are_unique():
    for name, fname, old, _ in MUTANTS:
        text = open(os.path.join(ROOT, "oracle", fname)).read()
        assert text.count(old) == 1, name


def test_every_mutant_fails_a_pin():
    with ThreadPoolExecutor(max_workers=4) as ex:
        control = ex.submit(_pins_pass, None)
        results = list(ex.map(_pins_pass, MUTANTS))
    ok, out = control.result()
    assert ok, "the unmutated oracle copy must pass its pins:\n" + out
    survivors = [m[0] for m, (passed, _) in zip(MUTANTS, results) if passed]
    assert not survivors, "mutants no pin catches: %s" % survivors
