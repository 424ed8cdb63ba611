"""Energy-per-token arithmetic of the benchmark's energy figures (CPU only).

The report states training energy in MWh per 500 billion tokens (Section 3,
Tables 5 and 6).  report() turns a measured loop (calls, seconds, joules) into
average power, joules per token and that unit; these tests pin it with hand
computed values and the unit identities it rests on."""
import math

import pytest

from paper_2510_02483_amd import energy


def test_report_hand_example():
    # 10 calls of 1000 tokens in 2 s drawing 2400 J: 1200 W, 0.24 J per token;
    # 500e9 tokens x 0.24 J = 1.2e11 J = 1.2e11 / 3.6e9 MWh = 33.333 MWh
    out = energy.report(10, 2.0, 2400.0, 1000)
    assert out["calls"] == 10 and out["seconds"] == 2.0
    assert out["joules"] == 2400.0
    assert out["avg_power_w"] == 1200.0
    assert math.isclose(out["joules_per_token"], 0.24, rel_tol=1e-12)
    assert out["mwh_per_500b_tokens"] == pytest.approx(33.3333, abs=1e-4)


def test_report_units():
    # one joule per token is 500e9 J per 500e9 tokens = 500e9 / 3.6e9 MWh
    out = energy.report(1, 1.0, 8192.0, 8192)
    assert out["joules_per_token"] == 1.0
    assert out["mwh_per_500b_tokens"] == pytest.approx(500e9 / 3.6e9, abs=1e-4)
    # MWh per 500B tokens scales linearly with joules and inversely with tokens
    a = energy.report(3, 1.5, 900.0, 4096)
    b = energy.report(3, 1.5, 1800.0, 4096)
    c = energy.report(6, 1.5, 1800.0, 4096)
    assert b["mwh_per_500b_tokens"] == pytest.approx(2 * a["mwh_per_500b_tokens"], rel=1e-3)
    assert c["mwh_per_500b_tokens"] == pytest.approx(a["mwh_per_500b_tokens"], rel=1e-3)


def test_report_block_bench_magnitude():
    # a 1235 W draw at 1.45 M tokens/s is 0.85 mJ per token and 0.119 MWh per 500B tokens
    tokens_per_s = 1.447e6
    out = energy.report(100, 1.0, 1235.0, int(tokens_per_s / 100))
    assert out["joules_per_token"] == pytest.approx(1235.0 / tokens_per_s, rel=1e-4)
    assert out["mwh_per_500b_tokens"] == pytest.approx(1235.0 / tokens_per_s * 500e9 / 3.6e9, rel=1e-3)


@pytest.mark.parametrize("joules", [None, 0.0, -5.0])
def test_report_without_reading(joules):
    out = energy.report(4, 1.0, joules, 100)
    assert out["calls"] == 4
    assert out["joules"] is None and out["avg_power_w"] is None
    assert out["joules_per_token"] is None and out["mwh_per_500b_tokens"] is None


def test_mean_clock_skips_invalid_readings():
    # per-XCD samples; "N/A", 0xFFFF and None mark readings the firmware did not fill
    samples = [[2000, 2100, "N/A", 65535], [1900, None, 2000, 2000]]
    assert energy.mean_clock_mhz(samples) == pytest.approx((2000 + 2100 + 1900 + 2000 + 2000) / 5, abs=0.05)
    assert energy.mean_clock_mhz([]) is None
    assert energy.mean_clock_mhz([["N/A"], [65535]]) is None
