"""The analytic cost model (Sec. 5, Eqs. (16)-(20)) against every M.S. /
D.S. / C.O. value printed in Tables 2 and 3 and the approximate ratios the
text quotes (Secs. 5.1, 5.3, 6.3)."""
import os

import pytest

from paper_2010_07565_amd import costmodel as cm

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_cost_tables.txt")


def printed_rows():
    rows = []
    for line in open(GOLDEN):
        line = line.split("#")[0].strip()
        if line:
            ds, model, q, val, where = line.split()
            rows.append((ds, model, q, val, where))
    return rows


def matches_printed(x: float, printed: str) -> bool:
    """x shown at the precision of `printed` equals it."""
    if "e" in printed:
        mant = printed.split("e")[0]
        digits = len(mant.split(".")[1]) if "." in mant else 0
        return ("%.*e" % (digits, x)).replace("e+0", "e").replace("e+", "e") == printed
    digits = len(printed.split(".")[1]) if "." in printed else 0
    return "%.*f" % (digits, x) == printed


def test_golden_covers_both_tables():
    rows = printed_rows()
    assert len(rows) == 54
    assert {r[4] for r in rows} == {"Table2", "Table3"}


@pytest.mark.parametrize("ds,model,q,printed,where", printed_rows())
def test_table_entry(ds, model, q, printed, where):
    e = cm.table_entries(cm.DATASETS[ds], model)
    key = {"ms": "ms_kib", "ds": "ds_mib", "co": "co"}[q]
    assert matches_printed(e[key], printed), (ds, model, q, e[key], printed, where)


def test_matches_printed_rejects_neighbours():
    assert matches_printed(2.4995e8, "2.50e8")
    assert not matches_printed(2.4949e8, "2.50e8")
    assert matches_printed(0.4729, "0.47") and not matches_printed(0.4649, "0.47")


def near(x, quoted):
    """The text's "~q x": within one of q (it writes 53.5 as ~53, 58.8 as ~59)."""
    return abs(x - quoted) < 1.0


def test_equation_ratios_quoted_in_the_text():
    cora = cm.DATASETS["cora"]
    # Sec. 5.1: ~31x parameter compression for Cora's first layer (Eq. (16))
    assert near(cm.pc(cora.features), 31)
    # Sec. 5.3: ~59x and ~21x feature-extraction speed-up for Cora's two
    # layers (Eq. (18)), ~53x for the whole 2-layer model
    assert near(cm.s_fe(cora.features), 59)
    assert near(cm.s_fe(cora.hidden), 21)
    r_cora = cm.theoretical_ratios(cora.nodes, cora.edges,
                                   [cora.features, cora.hidden, cora.classes])
    assert near(r_cora["cycle_ops"], 53)
    # Sec. 6.3: ~47x average inference speed-up and ~30x lower memory over
    # the two citation graphs; only ~10x on Reddit (large mean degree)
    pub = cm.DATASETS["pubmed"]
    r_pub = cm.theoretical_ratios(pub.nodes, pub.edges, [pub.features, pub.hidden, pub.classes])
    assert near((r_cora["cycle_ops"] + r_pub["cycle_ops"]) / 2, 47)
    assert near((r_cora["data_size"] + r_pub["data_size"]) / 2, 30)
    red = cm.DATASETS["reddit"]
    r_red = cm.theoretical_ratios(red.nodes, red.edges, [red.features, red.hidden, red.classes])
    assert near(r_red["cycle_ops"], 10)


def test_closed_forms_agree_with_the_counts():
    # Eq. (17) is the per-row form of the D.S. ratio; Eq. (16) the per-layer
    # form of the M.S. ratio; Eq. (18) the feature-extraction C.O. ratio.
    for d in (1, 7, 64, 500, 1433):
        assert cm.dc(d) == pytest.approx(cm.data_size_bytes(10, d, False)
                                         / cm.data_size_bytes(10, d, True))
        assert cm.pc(d) == pytest.approx(cm.model_size_bytes([d, 5], False)
                                         / cm.model_size_bytes([d, 5], True))
        assert cm.s_fe(d) == pytest.approx(cm.cycle_ops(100, 0, [d, 9], False)
                                           / cm.cycle_ops(100, 0, [d, 9], True))
        # Eq. (19) with |E| = N deg / 2, and Eq. (20) as deg -> 0
        n, deg = 1000, 4.0
        assert cm.s_full(d, deg) == pytest.approx(
            cm.cycle_ops(n, n * deg / 2, [d, 9], False) / cm.cycle_ops(n, n * deg / 2, [d, 9], True))
        assert cm.s_full(d, 0.0) == pytest.approx(cm.s_fe(d))


def test_breakdown_shares():
    cora = cm.DATASETS["cora"]
    b = cm.co_breakdown(cora.nodes, cora.edges, [cora.features, cora.hidden, cora.classes])
    assert sum(b.values()) == pytest.approx(1.0)
    assert b["binary"] > 0.8                     # binary operations dominate on Cora
    red = cm.DATASETS["reddit"]
    b = cm.co_breakdown(red.nodes, red.edges, [red.features, red.hidden, red.classes])
    assert b["aggregation"] > 0.8                # aggregation dominates on Reddit
