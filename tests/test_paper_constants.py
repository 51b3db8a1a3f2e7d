"""The paper's figures quoted by the benchmark match the cited fixture
(tests/golden/paper_results_hallusion.txt, from the paper's results table)."""
import os

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load():
    out = {}
    for line in open(os.path.join(GOLDEN, "paper_results_hallusion.txt")):
        if line.strip() and not line.startswith("#"):
            model, temp, sr, tau = line.split()
            out[(model, int(temp))] = (float(sr), float(tau))
    return out


def test_bench_quotes_the_paper_table():
    t = load()
    assert bench.PAPER_TAU == t[("LLaVA-1.5-7B", 0)][1]
    for model, sr in bench.PAPER_SR.items():
        assert sr == t[(model, 0)][0]
    # MSD accepts more per cycle at temperature 0 than at 1 in every quoted row
    for model in ("LLaVA-1.5-7B", "LLaVA-1.5-13B"):
        assert t[(model, 0)][1] > t[(model, 1)][1]
