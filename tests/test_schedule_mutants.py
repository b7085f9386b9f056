"""Plant plausible mistakes in the schedule reference (oracle/daso_schedule.py)
by editing one expression of its source, and check that a pin of
tests/test_schedule.py fails for each.  CPU only."""
import inspect
import textwrap

import pytest

from oracle import daso_schedule as O
from tests import test_schedule as pins

# (original expression, planted mistake, pins expected to catch it)
MUTANTS = [
    ("max(1, cfg.B_init // 4)", "max(1, cfg.B_init // 2)", [pins.test_initial_wait_is_a_quarter_of_B]),
    ("newB, newW = cfg.B_init, W0", "newB, newW = B, W", [pins.test_plateaus_halve_B_and_W_down_to_one_then_reset]),
    ("max(1, W // 2)", "max(1, W)", [pins.test_plateaus_halve_B_and_W_down_to_one_then_reset]),
    ("max(1, B // 2)", "max(1, B - 1)", [pins.test_plateaus_halve_B_and_W_down_to_one_then_reset]),
    ("arrive = t + W", "arrive = t + W + 1",
     [pins.test_cycling_exchanges_every_B_batches_and_merges_W_later]),
    ("if since_start == B:", "if since_start == B + 1:",
     [pins.test_cycling_exchanges_every_B_batches_and_merges_W_later, pins.test_exchange_count_per_cycling_epoch]),
    ("grp = exchanges % g\n                        exchanges += 1", "grp = 0\n                        exchanges += 1",
     [pins.test_global_sync_role_rotates_between_groups]),
    ("plan[\"S\"] = 0", "plan[\"S\"] = W", [pins.test_blocking_phases_synchronise_after_every_batch]),
    ("if flat < cfg.patience:", "if flat < 1:", [pins.test_patience_and_tolerance]),
    ("loss < best - cfg.plateau_rel_tol * abs(best)", "loss < best", [pins.test_patience_and_tolerance]),
]


def _mutated_plan_training(original: str, planted: str):
    src = textwrap.dedent(inspect.getsource(O.plan_training))
    assert src.count(original) >= 1, original
    src = src.replace(original, planted, 1)
    ns = dict(vars(O))
    exec(compile(src, "<mutant>", "exec"), ns)
    return ns["plan_training"]


@pytest.mark.parametrize("original,planted,catchers", MUTANTS, ids=[m[1][:40] for m in MUTANTS])
def test_schedule_pins_catch_planted_mistake(monkeypatch, original, planted, catchers):
    monkeypatch.setattr(O, "plan_training", _mutated_plan_training(original, planted))
    for pin in catchers:
        with pytest.raises(AssertionError):
            pin()
