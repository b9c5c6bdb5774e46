"""Host logic of the prune policies (CPU): each baseline's parameters, the
static layer tables handed to the budget split, and the window rule."""
import numpy as np
import pytest

import oracle
from paper_2511_06029_amd import policies


def test_policy_parameters():
    assert policies.get("h2o").gamma == 1.0 and policies.get("h2o").sink == 0
    assert policies.get("streaming").sink == 4 and policies.get("streaming").window_fills
    assert policies.get("lethe", gamma=0.9).gamma == 0.9
    assert policies.get("lethe-shared").shared and not policies.get("lethe").shared
    with pytest.raises(ValueError):
        policies.get("nope")


def test_uniform_and_sparsity_tables():
    assert policies.get("h2o").sparsity_in(5) == [0.0] * 5
    assert policies.get("lethe").sparsity_in(5) is None


@pytest.mark.parametrize("Ly,beta", [(32, 20.0), (28, 4.0), (2, 10.0)])
def test_pyramid_table_gives_the_progression(Ly, beta):
    """The static table, pushed through the oracle's budget split without
    floors, reproduces PyramidKV's progression to within the split's integer
    rounding."""
    pol = policies.get("pyramid", beta=beta)
    S = np.array(pol.sparsity_in(Ly), np.float32)
    assert S[0] == 0.0 and np.all(np.diff(S) > 0)            # weights fall with depth
    per_layer = 1000
    n = np.full(Ly, 10 * per_layer, np.int32)
    budget, inf = oracle.budget_split(n, S, 0, 0, per_layer * Ly)
    assert not inf and budget.sum() == per_layer * Ly
    prog = np.array(oracle.pyramid_budgets(Ly, per_layer * Ly, beta))
    assert np.all(np.abs(budget - prog) <= 1.0), (budget, prog)


def test_streaming_window_fills_the_budget():
    pol = policies.get("streaming", sink=4)
    assert pol.windows(300, 16) == (296, 4)
    assert pol.windows(3, 16) == (0, 4)
    assert policies.get("h2o").windows(300, 16) == (16, 0)


def test_per_layer_budget_floor():
    assert policies.per_layer_budget(0.4, 2560) == 1024
    assert policies.per_layer_budget(0.3, 16640) == 4992
    assert policies.per_layer_budget(0.25, 3) == 0
