"""Plant plausible mistakes in the oracle (on the CPU, by monkeypatching) and
check that at least one pin catches each of them."""
import numpy as np
import pytest

from oracle import daso_oracle as O
from tests import test_oracle_pins as pins

F32 = np.float32


def _merge_S_not_2S(xl, stale, S):
    P = len(stale)
    if P == 0:
        return np.array(xl, dtype=np.float32, copy=True)
    a = F32(S) * xl
    for st in stale:
        a = a + O.bf16_widen(st)
    return a / F32(S + P)


def _merge_wrong_denominator(xl, stale, S):
    P = len(stale)
    if P == 0:
        return np.array(xl, dtype=np.float32, copy=True)
    a = F32(2 * S) * xl
    for st in stale:
        a = a + O.bf16_widen(st)
    return a / F32(2 * S + P + 1)


def _merge_drops_last_copy(xl, stale, S):
    P = len(stale)
    if P == 0:
        return np.array(xl, dtype=np.float32, copy=True)
    a = F32(2 * S) * xl
    for st in stale[:-1]:
        a = a + O.bf16_widen(st)
    return a / F32(2 * S + P)


def _avg_drops_replica(grads):
    s = np.array(grads[0], dtype=np.float32, copy=True)
    for r in range(1, len(grads) - 1):
        s = s + grads[r]
    return s / F32(len(grads))


def _avg_divides_by_g_minus_1(grads):
    s = np.array(grads[0], dtype=np.float32, copy=True)
    for r in range(1, len(grads)):
        s = s + grads[r]
    return s / F32(max(len(grads) - 1, 1))


def _bf16_truncates(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    r = (x.view(np.uint32) >> 16).astype(np.uint16)
    r[np.isnan(x)] = 0x7FC0
    return r


def _bf16_ties_away(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x8000)) >> np.uint64(16)).astype(np.uint16)
    r[np.isnan(x)] = 0x7FC0
    return r


def _sgd_wrong_sign(x, m, gbar, lr, mu, wd):
    m_new = (F32(mu) * m) + gbar
    return x + (F32(lr) * m_new), m_new


def _sgd_momentum_misplaced(x, m, gbar, lr, mu, wd):
    m_new = F32(mu) * (m + gbar)
    return x - (F32(lr) * m_new), m_new


def _sgd_ignores_wd(x, m, gbar, lr, mu, wd):
    m_new = (F32(mu) * m) + gbar
    return x - (F32(lr) * m_new), m_new


def _stats_count_nan_only(gbar, xl, x_new):
    g, d, _ = _true_bucket_stats(gbar, xl, x_new)
    return g, d, int(np.count_nonzero(np.isnan(x_new)))


def _stats_sums_in_float32(gbar, xl, x_new):
    g32 = np.asarray(gbar, dtype=np.float32)
    d32 = np.asarray(x_new, dtype=np.float32) - np.asarray(xl, dtype=np.float32)
    _, _, nf = _true_bucket_stats(gbar, xl, x_new)
    return float(np.sum(g32 * g32)), float(np.sum(d32 * d32)), nf


def _stats_abs_not_square(gbar, xl, x_new):
    _, d, nf = _true_bucket_stats(gbar, xl, x_new)
    return float(np.sum(np.abs(np.asarray(gbar, dtype=np.float64)))), d, nf


_true_bucket_stats = O.bucket_stats
_true_global_merge = O.global_merge
_true_fused_sync_step = O.fused_sync_step


def _one_S_for_every_bucket(buckets):
    return [(s, k, buckets[0][2]) for (s, k, _) in buckets]


def _neighbour_bucket_S(buckets):
    nb = len(buckets)
    return [(s, k, buckets[(b + 1) % nb][2]) for b, (s, k, _) in enumerate(buckets)]


def _global_merge_one_S(params, stale, buckets, *a, **k):
    return _true_global_merge(params, stale, _one_S_for_every_bucket(buckets), *a, **k)


def _global_merge_neighbour_S(params, stale, buckets, *a, **k):
    return _true_global_merge(params, stale, _neighbour_bucket_S(buckets), *a, **k)


def _fused_one_S(grads, params, momentum, stale, buckets, *a, **k):
    return _true_fused_sync_step(grads, params, momentum, stale, _one_S_for_every_bucket(buckets), *a, **k)


def _fused_neighbour_S(grads, params, momentum, stale, buckets, *a, **k):
    return _true_fused_sync_step(grads, params, momentum, stale, _neighbour_bucket_S(buckets), *a, **k)


def _merge_zero_S_keeps_local_term(xl, stale, S):
    P = len(stale)
    if P == 0:
        return np.array(xl, dtype=np.float32, copy=True)
    a = F32(2 * S) * np.asarray(xl, dtype=np.float32)
    for st in stale:
        a = a + O.bf16_widen(st)
    return a / F32(2 * S + P)


MUTANTS = [
    ("global_merge", _global_merge_one_S, [pins.test_per_bucket_staleness_matches_exact_rational_eq1]),
    ("global_merge", _global_merge_neighbour_S, [pins.test_per_bucket_staleness_matches_exact_rational_eq1]),
    ("fused_sync_step", _fused_one_S, [pins.test_per_bucket_staleness_matches_exact_rational_eq1]),
    ("fused_sync_step", _fused_neighbour_S, [pins.test_per_bucket_staleness_matches_exact_rational_eq1]),
    ("merge_eq1", _merge_zero_S_keeps_local_term, [pins.test_merge_zero_staleness_ignores_the_local_state]),
    ("merge_eq1", _merge_S_not_2S, [pins.test_merge_gradient_form_appendix,
                                    pins.test_merge_small_integers_match_exact_rational_eq1]),
    ("merge_eq1", _merge_wrong_denominator, [pins.test_merge_weights_sum_to_one,
                                             pins.test_merge_gradient_form_appendix]),
    ("merge_eq1", _merge_drops_last_copy, [pins.test_merge_zero_staleness_is_plain_mean_of_copies]),
    ("local_avg", _avg_drops_replica, [pins.test_local_avg_matches_exact_rational_mean]),
    ("local_avg", _avg_divides_by_g_minus_1, [pins.test_local_avg_close_to_fp64_mean]),
    ("bf16_rne", _bf16_truncates, [pins.test_bf16_golden_encodings,
                                   pins.test_bf16_rne_matches_bruteforce_every_high_half]),
    ("bf16_rne", _bf16_ties_away, [pins.test_bf16_golden_encodings,
                                   pins.test_bf16_rne_matches_torch_cast_on_finite_values]),
    ("sgd_momentum", _sgd_wrong_sign, [pins.test_sgd_matches_torch_optim_sgd]),
    ("sgd_momentum", _sgd_momentum_misplaced, [pins.test_sgd_matches_torch_optim_sgd]),
    ("sgd_momentum", _sgd_ignores_wd, [pins.test_sgd_matches_torch_optim_sgd]),
    ("bucket_stats", _stats_count_nan_only, [pins.test_stats_count_nonfinite]),
    ("bucket_stats", _stats_sums_in_float32, [pins.test_stats_match_exactly_rounded_sums]),
    ("bucket_stats", _stats_abs_not_square, [pins.test_stats_match_exactly_rounded_sums]),
]


@pytest.mark.parametrize("name,mutant,catchers", MUTANTS,
                         ids=[m[1].__name__.lstrip("_") for m in MUTANTS])
def test_pins_catch_planted_mistake(monkeypatch, name, mutant, catchers):
    monkeypatch.setattr(O, name, mutant)
    for pin in catchers:
        with pytest.raises(AssertionError):
            pin()
