"""The measured-ceiling calls of librkcalib on an MI355X: plausible against the published
peaks (int32 VALU 256 CU x 64 lanes x 2.4 GHz; HBM 8 TB/s)."""
import pytest

from paper_2307_01236_amd import calib

pytestmark = pytest.mark.gpu


def test_valu_rate_near_nominal_peak():
    """k_valu runs exactly 2 VALU instructions per step (SQ_INSTS_VALU per wave =
    16 x iterations + 17, profiles/valu_ceiling_k_valu.md), so its rate cannot pass the
    nominal peak by more than the clock allows: runs measure 97-105% of 39.32 T."""
    r = calib.valu_int32_rate(1 << 12)
    assert 0.5 * 39.32e12 < r < 1.08 * 39.32e12, r


def test_copy_bandwidth_below_hbm_peak():
    bw = calib.copy_bandwidth(1 << 28)
    assert 1e12 < bw < 8.0e12, bw


def test_read_bandwidth_below_hbm_peak():
    bw = calib.read_bandwidth(1 << 28)
    assert 1e12 < bw < 8.0e12, bw
