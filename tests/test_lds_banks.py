"""The LDS bank model (paper_1909_02765_amd.lds_banks) against the hardware
measurements it was fitted to (profiles/lds_bank_probe.json: the lds_probe
kernel under rocprofv3 on one MI355X), and what it says about the kernel's
layouts.  Host only."""
import json
import os

from paper_1909_02765_amd import lds_banks as lb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
MEASURED = json.load(open(os.path.join(ROOT, "profiles", "lds_bank_probe.json")))["passes_per_read"]


def test_model_reproduces_every_measured_b32_and_b64_pattern():
    checked = 0
    for name, width, addrs in lb.probe_patterns():
        if name in MEASURED and width in (1, 2):
            assert lb.model_cost(name, width, addrs) == MEASURED[name], name
            checked += 1
    assert checked >= 150


def test_weights_through_lds_layout_reads_conflict_free():
    """Lane (g, l) at word KKP*l + COT*KKP*g (KKP = 12 or 28; COT*KKP a
    multiple of 64), the kernel's A-operand ds_read_b128: measured 0; the
    earlier layout (rows of CC*KKP + 4 words, channels KKP apart) measured 4."""
    for kkp in (12, 28):
        for plane in (64, 192, 256, 384, 448):
            assert MEASURED[f"b128_l{kkp}_g{plane}"] == 0.0
    assert MEASURED["b128_l388_g12"] == 4.0 and MEASURED["b128_l196_g12"] == 4.0


def test_tight_halo_layouts_cost_at_most_two_passes():
    for (th, tw, s, k, nwp) in lb.TILE_SHAPES:
        hcp, pl = lb.tight_layout(th, tw, s, k)
        costs = lb.b_read_costs(th, tw, s, hcp, pl, nwp)
        assert max(costs) <= 2, (th, tw, s, k, costs)


def test_sixteen_word_rows_of_the_14x14_tile_conflict_for_any_plane_pitch():
    """14-pixel rows in 16-word rows: every full block spans two rows and two
    of its banks hold a word of each of the half-wave's two channels."""
    for pl in range(256, 320):
        costs = lb.b_read_costs(14, 14, 1, 16, pl)
        assert costs[:12] == [2] * 12, pl
    assert lb.b_read_costs(14, 14, 1, 16, 272)[12] == 0
    measured = [MEASURED[f"b32_tile14x14_s1_k3_rule_hcp16_pl272_w0_n{n}"] for n in range(13)]
    assert measured == [2.0] * 12 + [0.0]


def test_model_layouts_measured_conflict_free():
    for name, width, addrs in lb.probe_patterns():
        if "_model_" in name and name in MEASURED:
            assert MEASURED[name] == lb.conflicts_b32(addrs), name
