"""The fp64 oracle against its pins, and the pins against planted mistakes.

The mutants are copies of the oracle's C source with one plausible mistake
each, compiled on the CPU into a temporary directory; every mutant must fail
at least one pin."""
from __future__ import annotations

import os
import subprocess

import pytest

import oracle
from tests import oracle_pins

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


@pytest.fixture(scope="module")
def orc():
    return oracle.get()


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


# (description, exact source text, replacement)
MUTANTS = [
    ("scale dropped", "s[j] = scale * dot;", "s[j] = dot;"),
    ("scale 1/d", "const double scale = 1.0 / sqrt((double)d);",
     "const double scale = 1.0 / (double)d;"),
    ("max shift not undone in lse", "const double L = m + log(l);", "const double L = log(l);"),
    ("values read from keys", "const float* vj = v + j * row_stride;",
     "const float* vj = k + j * row_stride;"),
    ("head index ignored for keys", "k + IDX4(b, 0, h, 0, Nk, H, d)", "k + IDX4(b, 0, 0, 0, Nk, H, d)"),
    ("query row not offset", "attention_row(q + IDX4(b, i, h, 0, Nq, H, d)",
     "attention_row(q + IDX4(b, 0, h, 0, Nq, H, d)"),
    ("lse stored transposed", "if (lse) lse[(b * H + h) * nrows + r] = row_lse;",
     "if (lse) lse[(b * nrows + r) * H + h] = row_lse;"),
    ("merge weight sign", "const double w = exp((double)lses[r][lidx] - L);",
     "const double w = exp(L - (double)lses[r][lidx]);"),
    ("merge uses max only", "const double L = M + log(sum);", "const double L = M;"),
    ("merge drops last partial", "for (int32_t r = 0; r < n; ++r) {\n            const double w",
     "for (int32_t r = 0; r < n - 1; ++r) {\n            const double w"),
    ("update writes K into V plane", "fresh_v[IDX4(b, i, h, c, len, H, d)];",
     "fresh_k[IDX4(b, i, h, c, len, H, d)];"),
    ("patch skips its update", "int rc = xo_patch_update(kv_buf, off, len,",
     "int rc = xo_patch_update(kv_buf, off, 0,"),
    ("every range takes the first fresh rows", "const int64_t src = IDX4(b, base + i, h, c, F, H, d);",
     "const int64_t src = IDX4(b, i, h, c, F, H, d);"),
    ("last range not stored", "    for (int32_t r = 0; r < nr; ++r) {\n        for (int64_t b = 0; b < B; ++b)",
     "    for (int32_t r = 0; r < nr - 1; ++r) {\n        for (int64_t b = 0; b < B; ++b)"),
    ("ranged step attends over the fresh rows only",
     "return xo_attention(q, kv_buf, kv_buf + plane, B, Nq, N, H, d, rows, nrows, out, lse);",
     "return xo_attention(q, fresh_k, fresh_v, B, Nq, F, H, d, rows, nrows, out, lse);"),
    ("stage keys projected with Wq", "sk += (double)xr[c] * (double)wk[c * HD + n];",
     "sk += (double)xr[c] * (double)wq[c * HD + n];"),
    ("stage attends over stale keys", "            kr[n] = sk;\n", "            (void)sk;\n"),
    ("stage output projection uses Wo transposed", "acc += orow[n] * (double)wo[n * C + c];",
     "acc += orow[n] * (double)wo[(c * HD + n) % (HD * C)];"),
    ("stage skips the output projection rows past the first",
     "for (int64_t t = 0; t < B * nrows; ++t) {\n        const double* orow",
     "for (int64_t t = 0; t < (B * nrows > 0 ? 1 : 0); ++t) {\n        const double* orow"),
]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(tmp_path, name, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, f"mutation anchor not unique: {name}"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib = tmp_path / "libmutant.so"
    oracle.build(str(mutated), str(lib))
    orc = oracle.Oracle(str(lib))
    failures = []
    for pin in oracle_pins.PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError):
            failures.append(pin.__name__)
    assert failures, f"no pin caught the planted mistake: {name}"
