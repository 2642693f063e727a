"""The accounting closed forms against numbers the paper prints (CPU only)."""

import json
import math
import os

import pytest

from paper_2609_25782_amd import accounting as acc

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def g(key):
    return GOLD[key]["value"]


def test_capacity_reproduces_165_and_3900_sessions():
    """(192 - 56.8) GiB / 0.82 GiB = 164.9 -> 165; with 3 TiB of HBF: 3,911 -> about 3,900
    (Sec. IV, Capacity and latency)."""
    hbm_only = acc.sessions_per_device(g("hbm_gib") * acc.GIB, g("weights_gib") * acc.GIB,
                                       g("mean_resident_gib") * acc.GIB)
    with_hbf = acc.sessions_per_device(g("hbm_gib") * acc.GIB, g("weights_gib") * acc.GIB,
                                       g("mean_resident_gib") * acc.GIB, g("hbf_tib") * acc.TIB)
    assert round(hbm_only) == g("sessions_hbm_only")
    assert abs(with_hbf - g("sessions_with_hbf")) / g("sessions_with_hbf") < 0.01
    assert round(with_hbf / hbm_only) == 24          # "24x more concurrent sessions" (abstract)


def test_peak_context_bytes():
    per_token = acc.kv_bytes_per_token(48, 4, 128, 2)
    assert per_token == g("kv_bytes_per_token")
    assert abs(g("peak_context_tokens") * per_token / acc.GIB - g("peak_context_gib")) < 0.01


def test_read_power_matches_the_printed_savings():
    """The hot set of N_a=48 (about 96 GiB incl. weights) read every 14 ms is the rate
    whose HBF-vs-HBM energy difference gives about 950 W at 20 pJ/bit, 7.6 kW per 8-GPU
    node, and 2.1-12.2 kW per node over 8-30 pJ/bit (Sec. IV, Read energy)."""
    rate = g("hot_set_gib_na48") * acc.GIB / (g("tbt_ms_na48") * 1e-3)
    hbm = g("hbm_pj_per_bit")
    saving = acc.read_power_watts([rate], [20.0]) - acc.read_power_watts([rate], [hbm])
    assert abs(saving - g("power_saving_w_per_device_at_20pj")) / 950 < 0.06
    assert abs(8 * saving / 1e3 - g("power_saving_kw_per_node_at_20pj")) < 0.5
    lo, hi = g("hbf_pj_per_bit_range")
    node = [8 * (acc.read_power_watts([rate], [e]) - acc.read_power_watts([rate], [hbm])) / 1e3
            for e in (lo, hi)]
    assert abs(node[0] - g("power_saving_kw_per_node_range")[0]) < 0.2
    assert abs(node[1] - g("power_saving_kw_per_node_range")[1]) < 0.7


def test_eq1_lifetime_closed_form():
    """Eq. (1) by hand: 3 TiB x 1e5 cycles at 1 GiB/s with WAF 1.02 is
    3 * 1024 * 1e5 / 1.02 seconds = 9.55 years; doubling the write rate halves it."""
    c, n, waf = g("hbf_tib") * acc.TIB, g("pe_cycles"), g("waf")
    t1 = acc.flash_lifetime_years(c, n, acc.GIB, waf)
    assert abs(t1 - 3 * 1024 * 1e5 / 1.02 / acc.SECONDS_PER_YEAR) < 1e-9
    assert abs(t1 - 9.55) < 0.01
    assert abs(acc.flash_lifetime_years(c, n, 2 * acc.GIB, waf) - t1 / 2) < 1e-9
    assert acc.flash_lifetime_years(c, n, 0.0, waf) == math.inf
    # the inverse: the write rate that lasts the 5-year warranty (Sec. IV, Endurance)
    r5 = acc.write_rate_for_lifetime(c, n, 5.0, waf)
    assert abs(acc.flash_lifetime_years(c, n, r5, waf) - 5.0) < 1e-9
