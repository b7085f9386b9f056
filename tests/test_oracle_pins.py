"""Pins for the CPU oracle: each check ties the oracle to something other than
itself (the bfloat16 format definition, exact rational arithmetic, closed forms
of the paper's update rules, PyTorch's own SGD, brute force).  No GPU."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import daso_oracle as O

F32 = np.float32
HERE = os.path.dirname(os.path.abspath(__file__))


# ------------------------------------------------------------ helpers
def f32_bits(x):
    return np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)


def from_bits(u):
    return np.ascontiguousarray(u, dtype=np.uint32).view(np.float32)


def frac_to_f32(fr: Fraction) -> np.float32:
    """Exact rational -> nearest binary32 (ties to even), normal range only."""
    if fr == 0:
        return F32(0.0)
    sign = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    # choose e so that 2^23 <= a / 2^(e-23) < 2^24
    while a >= Fraction(2) ** (e + 1):
        e += 1
    while a < Fraction(2) ** e:
        e -= 1
    assert -126 <= e <= 127, "outside the normal range"
    q = a / Fraction(2) ** (e - 23)
    whole, rem = divmod(q.numerator, q.denominator)
    twice = 2 * rem
    if twice > q.denominator or (twice == q.denominator and whole % 2 == 1):
        whole += 1
    return F32(sign * math.ldexp(whole, e - 23))


def bf16_bruteforce(u32: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 by direct comparison of the two neighbours, written from
    the definition: the truncated pattern and the next one up in magnitude are
    the candidates, the nearer wins, a tie picks the even pattern, and the
    pattern past the largest finite value stands for 2^128 (IEEE overflow)."""
    with np.errstate(invalid="ignore"):
        return _bf16_bruteforce(np.asarray(u32, dtype=np.uint32))


def _bf16_bruteforce(u32):
    f = from_bits(u32).astype(np.float64)
    lo = (u32 >> 16).astype(np.uint32)
    hi = lo + 1
    v_lo = np.abs(from_bits(lo << 16).astype(np.float64))
    mag_hi_bits = (hi & 0x7FFF) << 16
    v_hi = np.where((hi & 0x7FFF) == 0x7F80, 2.0 ** 128,
                    np.abs(from_bits(mag_hi_bits.astype(np.uint32)).astype(np.float64)))
    af = np.abs(f)
    d_lo = af - v_lo
    d_hi = v_hi - af
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ((lo & 1) == 1))
    out = np.where(pick_hi, hi, lo).astype(np.uint16)
    nan = np.isnan(f)
    out[nan] = 0x7FC0
    inf = np.isinf(f)
    out[inf] = lo[inf].astype(np.uint16)
    return out


# ------------------------------------------------------------- bf16 pack
def test_bf16_golden_encodings():
    path = os.path.join(HERE, "golden", "bf16_encodings.txt")
    rows = [ln.split() for ln in open(path) if ln.strip() and not ln.startswith("#")]
    assert len(rows) >= 20
    src = np.array([int(r[0], 16) for r in rows], dtype=np.uint32)
    exp = np.array([int(r[1], 16) for r in rows], dtype=np.uint16)
    got = O.bf16_rne(from_bits(src))
    bad = [(rows[i][0], hex(got[i]), rows[i][1]) for i in np.nonzero(got != exp)[0]]
    assert not bad, bad


def _structured_patterns():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x3FFF, 0x4000, 0x7FFE, 0x7FFF, 0x8000, 0x8001,
                     0x8002, 0xBFFF, 0xC000, 0xFFFE, 0xFFFF], dtype=np.uint32)
    rng = np.random.default_rng(7)
    lows = np.concatenate([lows, rng.integers(0, 1 << 16, 6, dtype=np.uint32)])
    return (hi[:, None] | lows[None, :]).ravel()


def test_bf16_rne_matches_bruteforce_every_high_half():
    """Every one of the 65,536 bf16 high halves, each with the discarded halves
    that decide the rounding (0, just below/at/above the tie, extremes) plus
    random ones: 1.2M patterns covering every sign, exponent and mantissa."""
    u = _structured_patterns()
    got = O.bf16_rne(from_bits(u))
    exp = bf16_bruteforce(u)
    bad = np.nonzero(got != exp)[0]
    assert bad.size == 0, [(hex(u[i]), hex(got[i]), hex(exp[i])) for i in bad[:10]]


def test_bf16_rne_matches_bruteforce_random_patterns():
    u = np.random.default_rng(11).integers(0, 1 << 32, 4_000_000, dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(O.bf16_rne(from_bits(u)), bf16_bruteforce(u))


def test_bf16_rne_matches_torch_cast_on_finite_values():
    """Library special case: torch's CPU float->bfloat16 cast is round to
    nearest even; on finite inputs it must agree bit for bit."""
    u = _structured_patterns()
    f = from_bits(u)
    fin = np.isfinite(f)
    want = torch.from_numpy(f[fin].copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.bf16_rne(f[fin]), want)


def test_bf16_widen_is_exact_inverse_on_bf16_values():
    h = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    f = O.bf16_widen(h)
    assert np.array_equal(f32_bits(f) >> 16, h.astype(np.uint32))
    assert np.all((f32_bits(f) & 0xFFFF) == 0)
    keep = ~np.isnan(f)
    assert np.array_equal(O.bf16_rne(f[keep]), h[keep])


# ------------------------------------------------------- local average
def test_local_avg_single_replica_is_identity():
    g0 = np.random.default_rng(0).standard_normal(1000).astype(F32)
    assert np.array_equal(f32_bits(O.local_avg([g0])), f32_bits(g0))


def test_local_avg_matches_exact_rational_mean():
    """Small integer gradients sum exactly in binary32, so the oracle must return
    the exact mean rounded once (one IEEE division), for g = 1..9 including
    non-powers of two where the division is inexact."""
    rng = np.random.default_rng(1)
    for g in range(1, 10):
        G = [rng.integers(-1000, 1000, 64).astype(F32) for _ in range(g)]
        got = O.local_avg(G)
        for j in range(64):
            exact = Fraction(sum(int(G[r][j]) for r in range(g)), g)
            assert got[j] == frac_to_f32(exact), (g, j)


def test_local_avg_close_to_fp64_mean():
    rng = np.random.default_rng(2)
    for g in (2, 3, 4, 7, 8):
        G = [(rng.standard_normal(10000) * 1e-3).astype(F32) for _ in range(g)]
        exact = np.mean(np.stack(G).astype(np.float64), axis=0)
        bound = g * 2.0 ** -24 * np.sum(np.abs(np.stack(G).astype(np.float64)), axis=0) / g + 1e-45
        assert np.all(np.abs(O.local_avg(G) - exact) <= bound)


def test_local_avg_pow2_equals_scaled_sum():
    rng = np.random.default_rng(3)
    G = [rng.standard_normal(5000).astype(F32) for _ in range(8)]
    s = G[0].copy()
    for r in range(1, 8):
        s = s + G[r]
    assert np.array_equal(f32_bits(O.local_avg(G)), f32_bits(s * F32(0.125)))


# ---------------------------------------------------------------- SGD
def test_sgd_first_step_closed_form():
    """From a zero momentum buffer the first step leaves m' = d and
    x_l = x - lr*d (with the buffer's sign of zero aside)."""
    rng = np.random.default_rng(4)
    x = rng.standard_normal(4096).astype(F32)
    d = (rng.standard_normal(4096) * 1e-3).astype(F32)
    xl, m = O.sgd_momentum(x, np.zeros_like(x), d, 0.1, 0.9, 0.0)
    assert np.array_equal(f32_bits(m), f32_bits(d + F32(0)))
    assert np.array_equal(f32_bits(xl), f32_bits(x - F32(0.1) * d))


def test_sgd_matches_torch_optim_sgd():
    """Library special case: torch.optim.SGD (momentum, zero dampening, no
    Nesterov, coupled weight decay) over several steps, within the rounding
    PyTorch's own operation order may introduce."""
    rng = np.random.default_rng(5)
    n = 20000
    x0 = rng.standard_normal(n).astype(F32) * F32(0.02)
    for wd in (0.0, 1e-4):
        p = torch.nn.Parameter(torch.from_numpy(x0.copy()))
        opt = torch.optim.SGD([p], lr=0.1, momentum=0.9, dampening=0, nesterov=False,
                              weight_decay=wd, foreach=False)
        x, m = x0.copy(), np.zeros(n, F32)
        for step in range(5):
            gr = (rng.standard_normal(n) * 1e-3).astype(F32)
            p.grad = torch.from_numpy(gr.copy())
            opt.step()
            x, m = O.sgd_momentum(x, m, gr, 0.1, 0.9, wd)
            ref = p.detach().numpy()
            assert np.max(np.abs(x - ref) / np.maximum(1.0, np.abs(ref))) <= 1e-6, (wd, step)
        buf = opt.state[p]["momentum_buffer"].numpy()
        assert np.max(np.abs(m - buf)) <= 1e-6 * np.max(np.abs(buf))


def test_sgd_unrolled_steps_match_appendix_eq2():
    """With mu = 0 and no weight decay, S steps from x_t give
    x_{t+S} = x_t - eta * sum_k G_k (appendix, minibatch SGD unrolled)."""
    rng = np.random.default_rng(6)
    n = 8000
    x = rng.standard_normal(n).astype(F32) * F32(0.02)
    Gs = [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(6)]
    cur, m = x.copy(), np.zeros(n, F32)
    for G in Gs:
        cur, m = O.sgd_momentum(cur, m, G, 0.1, 0.0, 0.0)
    want = x.astype(np.float64) - 0.1 * np.sum(np.stack(Gs).astype(np.float64), axis=0)
    assert np.max(np.abs(cur - want)) <= 12 * 2.0 ** -24 * 0.2


# ------------------------------------------------------ merge (Eq. 1)
def test_merge_small_integers_match_exact_rational_eq1():
    """Brute force against Eq. (1) in exact rationals: with small integer
    states every partial sum is exact, so only the final division rounds."""
    rng = np.random.default_rng(8)
    for S in range(0, 6):
        for P in range(0, 9):
            if S == 0 and P == 0:
                continue
            xl = rng.integers(-200, 200, 32).astype(F32)
            st = [O.bf16_rne(rng.integers(-200, 200, 32).astype(F32)) for _ in range(P)]
            got = O.merge_eq1(xl, st, S)
            for j in range(32):
                if P == 0:
                    assert got[j] == xl[j]
                    continue
                num = 2 * S * Fraction(int(xl[j])) + sum(Fraction(int(O.bf16_widen(s)[j])) for s in st)
                assert got[j] == frac_to_f32(num / (2 * S + P)), (S, P, j)


def test_merge_weights_sum_to_one():
    """A constant field merges to itself: the local weight 2S/(2S+P) plus P
    copies of weight 1/(2S+P) sum to one (exact for bf16-representable c)."""
    for S in range(0, 9):
        for P in range(1, 33):
            c = O.bf16_widen(O.bf16_rne(np.full(16, 0.7, F32)))
            st = [O.bf16_rne(c)] * P
            got = O.merge_eq1(c, st, S)
            assert np.max(np.abs(got - c)) <= 2.0 ** -24 * 0.7 * 2, (S, P)


def test_merge_identical_bf16_copies_give_local_state_bit_exact():
    rng = np.random.default_rng(9)
    xl = O.bf16_widen(O.bf16_rne(rng.standard_normal(1 << 16).astype(F32) * F32(0.02)))
    for S, P in ((1, 2), (2, 4), (4, 8), (4, 16), (8, 32), (3, 5), (1, 32)):
        st = [O.bf16_rne(xl)] * P
        assert np.array_equal(f32_bits(O.merge_eq1(xl, st, S)), f32_bits(xl)), (S, P)


def test_merge_without_copies_is_identity():
    xl = np.random.default_rng(10).standard_normal(1000).astype(F32)
    for S in (0, 1, 3, 8):
        assert np.array_equal(f32_bits(O.merge_eq1(xl, [], S)), f32_bits(xl))


def test_merge_zero_staleness_is_plain_mean_of_copies():
    """S = 0 (blocking global synchronisation): the local term drops out and
    the merge is the plain average of the P exchanged states."""
    rng = np.random.default_rng(12)
    xl = rng.standard_normal(3000).astype(F32)
    for P in (1, 2, 3, 5, 16):
        st = [O.bf16_rne(rng.standard_normal(3000).astype(F32)) for _ in range(P)]
        want = np.mean(np.stack([O.bf16_widen(s) for s in st]).astype(np.float64), axis=0)
        got = O.merge_eq1(xl, st, 0)
        assert np.max(np.abs(got - want) / np.maximum(np.abs(want), 1e-30)) <= (P + 1) * 2.0 ** -24 * 8


def test_merge_zero_staleness_ignores_the_local_state():
    """S = 0 is the blocking average of the exchanged states (Section 3, warm-up
    and cool-down phases): the local state has weight zero and does not enter,
    so a NaN or infinite local state still gives the exact mean of finite
    copies, and copies that are all -0 average to -0 (an IEEE sum of -0s)."""
    rng = np.random.default_rng(120)
    n = 64
    xl = rng.standard_normal(n).astype(F32)
    xl[0::3] = np.nan
    xl[1::3] = np.inf
    xl[2::6] = -np.inf
    for P in (1, 2, 3, 5):
        ints = [rng.integers(-200, 200, n) for _ in range(P)]
        st = [O.bf16_rne(v.astype(F32)) for v in ints]
        got = O.merge_eq1(xl, st, 0)
        for j in range(n):
            want = frac_to_f32(Fraction(sum(int(v[j]) for v in ints), P))
            assert f32_bits(got[j:j + 1])[0] == f32_bits(np.array([want], F32))[0], (P, j)
    negz = [np.full(n, 0x8000, np.uint16) for _ in range(3)]
    got = O.merge_eq1(xl, negz, 0)
    assert np.all(f32_bits(got) == 0x80000000)


def _per_bucket_case():
    """Small exact case: integers for params, gradients and copies, lr = mu = 1/2
    and a zero momentum buffer, so gbar (half-integers), the local state
    xl = x - gbar/2 (quarter-integers) and every partial sum of Eq. (1) are exact
    binary32 values and only the final division rounds.  The buckets are given
    out of order, with S = 3, 1, 8, 0 and an empty bucket with S = 5."""
    rng = np.random.default_rng(121)
    n, P = 40, 5
    x_i = rng.integers(-64, 65, n)
    g_i = [rng.integers(-64, 65, n) for _ in range(2)]
    c_i = [rng.integers(-200, 201, n) for _ in range(P)]
    buckets = [(24, 9, 3), (0, 10, 1), (10, 0, 5), (33, 7, 8), (10, 14, 0)]
    S_of = np.empty(n, np.int64)
    for (s, k, S) in buckets:
        S_of[s:s + k] = S
    xl = [Fraction(int(x_i[j])) - Fraction(int(g_i[0][j]) + int(g_i[1][j]), 4) for j in range(n)]
    want = []
    for j in range(n):
        S = int(S_of[j])
        num = 2 * S * xl[j] + sum(Fraction(int(c[j])) for c in c_i)
        want.append(frac_to_f32(num / (2 * S + P)))
    return {"x": x_i.astype(F32), "grads": [g.astype(F32) for g in g_i],
            "stale": [O.bf16_rne(c.astype(F32)) for c in c_i], "buckets": buckets,
            "xl": np.array([float(v) for v in xl], F32), "want": np.array(want, F32)}


def test_per_bucket_staleness_matches_exact_rational_eq1():
    """Each element is merged with the S of its own bucket, whatever the order in
    which the buckets are listed: global_merge and fused_sync_step against Eq. (1)
    evaluated exactly, element by element, with that element's bucket's S."""
    c = _per_bucket_case()
    got, wire = O.global_merge(c["xl"], c["stale"], c["buckets"], pack=True)
    assert np.array_equal(f32_bits(got), f32_bits(c["want"]))
    out = O.fused_sync_step(c["grads"], c["x"], np.zeros_like(c["x"]), c["stale"], c["buckets"], 0.5, 0.5, 0.0)
    assert np.array_equal(f32_bits(out["x_local"]), f32_bits(c["xl"]))
    assert np.array_equal(f32_bits(out["params"]), f32_bits(c["want"]))


def test_merge_gradient_form_appendix():
    """Appendix, gradient form of the global synchronisation:
    x_DASO = x_t - alpha (2S sum_{k<S} G_l,k + sum_i G_p,i), alpha = eta/(2S+P),
    where the local state took S steps from x_t and copy i is x_t - eta G_p,i.
    The peer gradients are defined from the bf16 copies so the identity is exact
    in real arithmetic; the oracle's binary32 result must agree to rounding."""
    rng = np.random.default_rng(13)
    n, eta = 4000, 0.1
    for S, P in ((1, 2), (2, 4), (4, 8), (4, 16), (8, 32), (3, 7)):
        xt = (rng.standard_normal(n) * 0.02).astype(F32)
        Gl = [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(S)]
        xl = xt.copy()
        for G in Gl:
            xl = xl - F32(eta) * G
        st = [O.bf16_rne(xt - F32(eta) * (rng.standard_normal(n) * 1e-3).astype(F32)) for _ in range(P)]
        Gp = [(xt.astype(np.float64) - O.bf16_widen(s).astype(np.float64)) / eta for s in st]
        GlS = (xt.astype(np.float64) - xl.astype(np.float64)) / eta  # = sum_k G_l,k exactly
        alpha = eta / (2 * S + P)
        want = xt.astype(np.float64) - alpha * (2 * S * GlS + np.sum(np.stack(Gp), axis=0))
        got = O.merge_eq1(xl, st, S).astype(np.float64)
        assert np.max(np.abs(got - want)) <= (P + 3) * 2.0 ** -24 * 0.1, (S, P)


def test_merge_is_permutation_invariant_and_translation_equivariant():
    """Reordering the copies changes only rounding; shifting the local state and
    every copy by c shifts the merge by c.  Values are multiples of 1/16 below
    16 in magnitude so the shifted copies stay exactly representable in bf16."""
    rng = np.random.default_rng(14)
    xl = (rng.integers(-100, 100, 2000) / 16).astype(F32)
    st = [O.bf16_rne((rng.integers(-100, 100, 2000) / 16).astype(F32)) for _ in range(6)]
    a = O.merge_eq1(xl, st, 2)
    b = O.merge_eq1(xl, st[::-1], 2)
    assert np.max(np.abs(a - b)) <= 2.0 ** -24 * 8
    c = F32(2.0)
    shifted_st = [O.bf16_rne(O.bf16_widen(s) + c) for s in st]
    assert all(np.array_equal(O.bf16_widen(t), O.bf16_widen(s) + c) for s, t in zip(st, shifted_st))
    shifted = O.merge_eq1(xl + c, shifted_st, 2)
    assert np.max(np.abs((shifted - c) - a)) <= 2.0 ** -24 * 16


# ---------------------------------------------------- fused and global
def _small_case(n=4099, g=3, P=5, seed=15):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal(n) * 0.02).astype(F32)
    m = (rng.standard_normal(n) * 1e-3).astype(F32)
    grads = [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(g)]
    stale = [O.bf16_rne(x + (rng.standard_normal(n) * 1e-4).astype(F32)) for _ in range(P)]
    a, b = n // 4, n // 2
    buckets = [(0, a, 1), (a, 7, 0), (a + 7, b, 4), (a + 7 + b, n - (a + 7 + b), 2)]
    return grads, x, m, stale, buckets


def test_fused_equals_composition_of_steps():
    grads, x, m, stale, buckets = _small_case()
    for wd in (0.0, 1e-4):
        out = O.fused_sync_step(grads, x, m, stale, buckets, 0.1, 0.9, wd)
        gbar = O.local_avg(grads)
        xl, m2 = O.sgd_momentum(x, m, gbar, 0.1, 0.9, wd)
        xn, wire = O.global_merge(xl, stale, buckets, pack=True)
        assert np.array_equal(f32_bits(out["params"]), f32_bits(xn))
        assert np.array_equal(f32_bits(out["momentum"]), f32_bits(m2))
        assert np.array_equal(out["wire"], wire)
        assert np.array_equal(out["wire"], O.pack_bf16(xn))
        pre = O.fused_sync_step(grads, x, m, stale, buckets, 0.1, 0.9, wd, flags=O.PACK_PRE_MERGE)
        assert np.array_equal(pre["wire"], O.pack_bf16(xl))


def test_fused_single_replica_no_copies_is_plain_sgd_plus_pack():
    rng = np.random.default_rng(16)
    n = 3001
    x = rng.standard_normal(n).astype(F32)
    m = rng.standard_normal(n).astype(F32)
    G = rng.standard_normal(n).astype(F32)
    out = O.fused_sync_step([G], x, m, [], [(0, n, 3)], 0.1, 0.9, 0.0)
    p = torch.nn.Parameter(torch.from_numpy(x.copy()))
    opt = torch.optim.SGD([p], lr=0.1, momentum=0.9, foreach=False)
    opt.state[p]["momentum_buffer"] = torch.from_numpy(m.copy())
    p.grad = torch.from_numpy(G.copy())
    opt.step()
    ref = p.detach().numpy()
    assert np.max(np.abs(out["params"] - ref) / np.maximum(1, np.abs(ref))) <= 1e-6
    assert np.array_equal(out["wire"], O.pack_bf16(out["params"]))
    assert out["stats"][0][1] == 0.0


def test_stats_match_exactly_rounded_sums():
    grads, x, m, stale, buckets = _small_case(n=2051, seed=17)
    out = O.fused_sync_step(grads, x, m, stale, buckets, 0.1, 0.9, 0.0)
    gbar, xl, xn = out["grad_avg"], out["x_local"], out["params"]
    for b, (s, k, _) in enumerate(buckets):
        gsq = math.fsum(float(v) * float(v) for v in gbar[s:s + k])
        dsq = math.fsum((float(a) - float(c)) ** 2 for a, c in zip(xn[s:s + k], xl[s:s + k]))
        got = out["stats"][b]
        assert abs(got[0] - gsq) <= 1e-12 * max(gsq, 1e-300)
        assert abs(got[1] - dsq) <= 1e-12 * max(dsq, 1e-300)
        assert got[2] == 0


def test_stats_count_nonfinite():
    grads, x, m, stale, buckets = _small_case(n=2051, seed=18)
    grads[1] = grads[1].copy()
    grads[1][[3, 1500]] = np.inf
    x = x.copy()
    x[[10, 2050]] = np.nan
    out = O.fused_sync_step(grads, x, m, stale, buckets, 0.1, 0.9, 0.0)
    counts = [st[2] for st in out["stats"]]
    # n = 2051: buckets [0,512) [512,519) [519,1544) [1544,2051)
    assert counts == [2, 0, 1, 1]  # 3 and 10 in bucket 0; 1500 in bucket 2; 2050 in bucket 3
    assert out["wire"][10] == 0x7FC0


def test_bucket_validation():
    grads, x, m, stale, _ = _small_case(n=100, seed=19)
    for bad in ([(0, 50, 1)], [(0, 60, 1), (50, 50, 1)], [(0, 100, -1)], [(1, 99, 1)]):
        with pytest.raises(ValueError):
            O.fused_sync_step(grads, x, m, stale, bad, 0.1, 0.9)


# ---------------------------------------------------------- fp32 exchange
def test_merge_f32_small_integers_match_exact_rational_eq1():
    """fp32 exchange: integers up to 2^20 are exact binary32 values whose sums
    stay exact, so only the final division rounds (exact rational Eq. (1))."""
    rng = np.random.default_rng(50)
    for S in range(0, 5):
        for P in range(1, 7):
            xl = rng.integers(-(1 << 20), 1 << 20, 16).astype(F32)
            st = [rng.integers(-(1 << 20), 1 << 20, 16).astype(F32) for _ in range(P)]
            got = O.merge_eq1(xl, st, S)
            for j in range(16):
                num = 2 * S * Fraction(int(xl[j])) + sum(Fraction(int(s[j])) for s in st)
                assert got[j] == frac_to_f32(num / (2 * S + P)), (S, P, j)


def test_f32_exchange_equals_bf16_exchange_on_bf16_values():
    """Copies that are exactly bf16 values merge to the same bits whichever way
    they travel; the fp32 wire then holds x' itself."""
    grads, x, m, stale, buckets = _small_case(n=3001, seed=51)
    st32 = [O.bf16_widen(s) for s in stale]
    a = O.fused_sync_step(grads, x, m, stale, buckets, 0.1, 0.9)
    b = O.fused_sync_step(grads, x, m, st32, buckets, 0.1, 0.9, exchange="f32")
    assert np.array_equal(f32_bits(a["params"]), f32_bits(b["params"]))
    assert np.array_equal(f32_bits(b["wire"]), f32_bits(b["params"]))
    pre = O.fused_sync_step(grads, x, m, st32, buckets, 0.1, 0.9, flags=O.PACK_PRE_MERGE, exchange="f32")
    assert np.array_equal(f32_bits(pre["wire"]), f32_bits(pre["x_local"]))
    with pytest.raises(TypeError):
        O.fused_sync_step(grads, x, m, stale, buckets, 0.1, 0.9, exchange="f32")


def test_merge_f32_gradient_form_appendix():
    """The appendix's gradient form, with fp32 copies (no bf16 rounding)."""
    rng = np.random.default_rng(52)
    n, eta = 4000, 0.1
    for S, P in ((1, 2), (4, 8), (8, 32), (3, 7)):
        xt = (rng.standard_normal(n) * 0.02).astype(F32)
        Gl = [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(S)]
        xl = xt.copy()
        for G in Gl:
            xl = xl - F32(eta) * G
        st = [(xt - F32(eta) * (rng.standard_normal(n) * 1e-3).astype(F32)).astype(F32) for _ in range(P)]
        Gp = [(xt.astype(np.float64) - s.astype(np.float64)) / eta for s in st]
        GlS = (xt.astype(np.float64) - xl.astype(np.float64)) / eta
        want = xt.astype(np.float64) - eta / (2 * S + P) * (2 * S * GlS + np.sum(np.stack(Gp), axis=0))
        got = O.merge_eq1(xl, st, S).astype(np.float64)
        assert np.max(np.abs(got - want)) <= (P + 3) * 2.0 ** -24 * 0.1, (S, P)
