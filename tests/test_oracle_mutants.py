"""The oracle's pins have teeth: each plausible mistake planted in a copy of
the oracle source (on the CPU only) makes at least one pin test fail."""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "uq_oracle.c")
PIN_TESTS = [os.path.join(ROOT, "tests", f) for f in (
    "test_oracle_philox.py", "test_oracle_scale.py", "test_oracle_index.py",
    "test_oracle_quantize.py", "test_oracle_aggregate.py", "test_oracle_randk.py")]

MUTANTS = {
    "philox multiplier": ("0xD2511F53u * (uint64_t)x0", "0xD2511F55u * (uint64_t)x0"),
    "philox key schedule": ("k1 += 0xBB67AE85u;", "k1 += 0xBB67AE84u;"),
    "word halves reused": ("unsigned shift = (j / 4) * 16;", "unsigned shift = (j % 2) * 16;"),
    "L1 instead of L2": ("s = s + x * x;", "s = s + fabs(x);"),
    "sum instead of max": ("best = sumsq[m];", "best += sumsq[m];"),
    "missing 1/M": ("deq[k] = W / ((float)M * scales[k]);", "deq[k] = W / scales[k];"),
    "strict scale rule": ("if (x <= s0) {", "if (x < s0) {"),
    "sharing by max": ("if (kstar_scratch[i] < idx[i])", "if (kstar_scratch[i] > idx[i])"),
    "reversed coin": ("l + (r < t ? 1 : 0)", "l + (r > t ? 1 : 0)"),
    "lost sign": ("(int8_t)(vi < 0.0f ? -mag : mag)", "(int8_t)(vi < 0.0f ? mag : -mag)"),
    "truncated level": ("float p = x - lf;", "float p = x - lf; p = p * 0.5f;"),
    "dequant ignores index": ("out[i] = (float)sum[i] * deq[k];", "out[i] = (float)sum[i] * deq[0];"),
    "worker not in counter": ("(uint32_t)(block >> 32), worker, 0u", "(uint32_t)(block >> 32), 0u, 0u"),
    "randk largest keys": ("out[j] = keys[j].idx;", "out[j] = keys[d - 1 - j].idx;"),
    "randk low word reused": ("        ctr[3] = 3u;\n        orc_philox4x32_10(ctr, key, out);\n        lo[j]",
                              "        ctr[3] = 2u;\n        orc_philox4x32_10(ctr, key, out);\n        lo[j]"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name!r} not unique"
    with tempfile.TemporaryDirectory() as tmp:
        c = os.path.join(tmp, "mutant.c")
        so = os.path.join(tmp, "libmutant.so")
        open(c, "w").write(src.replace(old, new))
        subprocess.run(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math",
                        "-shared", "-fPIC", c, "-o", so, "-lm"], check=True)
        env = dict(os.environ, UQ_ORACLE_LIB=so)
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            *PIN_TESTS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
        assert r.returncode == 1, f"mutant {name!r} survived the pins:\n{r.stdout[-2000:]}"
