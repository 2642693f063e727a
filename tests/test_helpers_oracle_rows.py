"""The chunked all-rows oracle helper used by the full-size parity tests gives
the same fp64 outputs as the oracle on one multi-layer pool holding every row
(CPU only)."""

import numpy as np

import synth
from helpers import Case, oracle_rows


def test_oracle_rows_equals_one_pool_oracle():
    lens = [300, 1, 17, 0, 64, 999]
    case = Case(3, 8, 2, 64, "bf16", lens, seed=31, layer=2, value_scale=0.3)
    want = case.oracle_out()
    for chunk in (1 << 20, 400, 1):            # one chunk, several, one row each
        got = oracle_rows(31, range(len(lens)), lens, 2, case.q, 2, 64, "bf16", 0.3, chunk_tokens=chunk)
        assert np.array_equal(got, want)


def test_oracle_rows_kv_override():
    lens = [50, 40]
    case = Case(1, 4, 1, 64, "f32", lens, seed=32)
    k, v = case.kv[1]
    k, v = k.copy(), v.copy()
    v[7] += 3.0
    case.kv[1] = (k, v)
    got = oracle_rows(32, [0, 1], lens, 0, case.q, 1, 64, "f32", 1.0, kv_override={1: (k, v)})
    assert np.array_equal(got, case.oracle_out())
