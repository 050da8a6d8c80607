"""Pins of the oracle's staging accounting against the paper's printed numbers.

The oracle's live trace of the window loop (Eq. 1 over the windows of §2
"Bounded installation") is evaluated at the paper's own chunk size and plan
lengths and compared with the values the paper reports (fixture
tests/golden/paper_law.json, each entry with its section or table).
"""

import json
import os

import pytest

import oracle

with open(os.path.join(os.path.dirname(__file__), "golden", "paper_law.json")) as f:
    LAW = json.load(f)

C = LAW["chunk_bytes_mtp_off"]["value"]
MIB = 1 << 20


def test_rws_flat_across_clean_sweep():
    """Prop. 1: at W = 32 the peak does not depend on N (appendix table)."""
    W = LAW["clean_sweep"]["W"]
    for tokens, objects, mib in LAW["clean_sweep"]["rows"]:
        peak = oracle.peak_live_staging(objects, W, C)
        assert peak == LAW["rws_w32_bytes"]["value"]
        assert peak == mib * MIB


@pytest.mark.parametrize("W,mib", LAW["w_sweep_256k"]["rows"])
def test_window_law(W, mib):
    """Eq. 5: M_L1(W) = W x c with zero residual at W in {8,16,32,64}."""
    assert oracle.peak_live_staging(LAW["w_sweep_256k"]["n_chunks"], W, C) == mib * MIB


@pytest.mark.parametrize("n,peak", LAW["whole_plan_peaks"]["rows"])
def test_whole_plan_peak(n, peak):
    """Eq. 2: legacy whole-plan (W = 0) staging is the whole plan."""
    assert oracle.peak_live_staging(n, 0, C) == peak


def test_live_units_never_exceed_W():
    """Eq. 3 on the trace itself, for ragged last windows too."""
    for n in (1, 31, 32, 33, 95, 2047):
        for W in (1, 8, 32, 64):
            tr = oracle.live_trace(oracle.plan_windows(n, W), 1)
            assert max(tr) == min(W, n)
            assert len(oracle.plan_windows(n, W)) == -(-n // W)


def test_external_over_staging_ratio_and_growth():
    ext = dict((n, b) for n, b in LAW["external_bytes"]["rows"])
    rws = oracle.peak_live_staging(2047, 32, C)
    ratio = ext[2047] / rws
    assert round(ratio, LAW["external_to_staging_ratio"]["digits"]) == LAW["external_to_staging_ratio"]["value"]
    assert ext[2047] / ext[128] == LAW["growth_factor"]["value"]
    # Theta(|S|): external bytes grow linearly with the number of chunk objects
    per_obj = {b // n for n, b in ext.items()}
    assert len(per_obj) == 1 and all(b % n == 0 for n, b in ext.items())


def test_mtp_on_law():
    c_mtp = LAW["mtp_on_rws_w32_bytes"]["value"] // 32
    assert oracle.peak_live_staging(2047, 32, c_mtp) == LAW["mtp_on_rws_w32_bytes"]["value"]
    assert LAW["mtp_on_rws_w32_bytes"]["value"] == 507.625 * MIB
