"""Values the paper fixes, stored under tests/golden with their citations."""
import os
from fractions import Fraction

from oracle import predictor as P

G = os.path.join(os.path.dirname(__file__), "golden")


def rows(name):
    with open(os.path.join(G, name)) as f:
        return [l.split() for l in f if l.strip() and not l.startswith("#")]


def test_peff_uniform_prior_table():
    for n, num, den in rows("peff_uniform_prior.txt"):
        assert abs(P.p_eff(int(n), 0, 8) - float(Fraction(int(num), int(den)))) < 1e-14
        assert abs(P.p_eff(int(n), int(n), 8) - float(Fraction(int(num), int(den)))) < 1e-14


def test_abandon_time_table():
    for tau, n_a in rows("abandon_time.txt"):
        n = 2
        while P.decide(n, 0, 8, 8, float(tau))[0] == P.CONTINUE:
            n += 1
        assert n == int(n_a)


def test_ablation_table_is_the_oracles():
    """tests/golden/ablation_sweeps.txt is exactly what the committed oracle
    writes for the ablation sweeps (the GPU test compares against it)."""
    from tests.golden import make_ablation_table as AB
    assert AB.oracle_lines() == AB.read_golden()
