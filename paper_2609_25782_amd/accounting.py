"""Closed-form accounting of the hot-cold hierarchy (paper Sec. II and IV).

These are the formulas the paper states or uses to turn simulated traffic into
its headline quantities; the replay driver feeds them measured pool counters.

* Flash lifetime, Eq. (1): T_life = C * N_PE / (R_W * WAF), with C the tier
  capacity, N_PE the rated program/erase cycles, R_W the application write rate
  and WAF the write-amplification factor (Sec. II, "High bandwidth flash").
* Read power: each tier's read rate times its energy per bit (Sec. IV,
  Methodology: HBF swept over 8-30 pJ/bit against about 3.5 pJ/bit for HBM).
* Sessions per device: the KV capacity left after the weights divided by the
  mean resident footprint of an agent (Sec. IV, "Capacity and latency").
"""

from __future__ import annotations

GIB = 1024 ** 3
TIB = 1024 ** 4
SECONDS_PER_YEAR = 365.25 * 24 * 3600


def flash_lifetime_years(capacity_bytes: float, pe_cycles: float, write_bytes_per_s: float,
                         waf: float) -> float:
    """Eq. (1): years until the rated P/E budget is spent (inf with no writes)."""
    if write_bytes_per_s <= 0:
        return float("inf")
    return capacity_bytes * pe_cycles / (write_bytes_per_s * waf) / SECONDS_PER_YEAR


def write_rate_for_lifetime(capacity_bytes: float, pe_cycles: float, years: float, waf: float) -> float:
    """Eq. (1) solved for the write rate that spends the budget in `years`."""
    return capacity_bytes * pe_cycles / (years * SECONDS_PER_YEAR * waf)


def read_power_watts(rates_bytes_per_s, energies_pj_per_bit) -> float:
    """Sum over tiers of read rate x energy per bit."""
    return sum(r * 8.0 * e * 1e-12 for r, e in zip(rates_bytes_per_s, energies_pj_per_bit))


def sessions_per_device(memory_bytes: float, weight_bytes: float, footprint_bytes: float,
                        extra_tier_bytes: float = 0.0) -> float:
    """KV capacity (fast tier minus weights, plus any capacity tier) over the mean
    resident footprint of one agent."""
    return (memory_bytes - weight_bytes + extra_tier_bytes) / footprint_bytes


def kv_bytes_per_token(num_layers: int, num_kv_heads: int, head_dim: int, elt_bytes: int) -> int:
    return 2 * num_layers * num_kv_heads * head_dim * elt_bytes
