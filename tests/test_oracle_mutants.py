"""The oracle's pins reject planted mistakes (CPU): each mutant of
oracle/oracle.c named here (tests/oracle_mutants.py builds it into a
temporary directory) must fail the oracle's tests.  These are the mutants
the fast tests reject; the mistakes in the FP16 conversion that only the
exhaustive 2^32 comparison sees are run by hand with
``python tests/oracle_mutants.py``."""
import pytest

from tests import oracle_mutants

FAST = ["normal ties away from zero", "overflow threshold at 65504", "residual sign flipped",
        "lo not scaled", "last k dropped", "elementwise XB before XA",
        "elementwise block folded first", "elementwise drops XB",
        "termwise cross sums added first", "termwise XB accumulates XA",
        "cross-first as (acc + HH_g) + X_g/s", "cross-first without XB"]


@pytest.mark.slow
@pytest.mark.parametrize("name", FAST)
def test_planted_mistake_is_rejected(name, tmp_path):
    killed, test = oracle_mutants.run_mutant(name, str(tmp_path))
    assert killed, f"the oracle's tests accept the mutant {name!r}"
