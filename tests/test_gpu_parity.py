"""GPU parity: every C-ABI entry point against the CPU oracle on the same seeded
inputs.  The bar: bf16 wire and integer outputs bit-exact; fp32 outputs within
max |err| <= 1e-6 * max(1, |x|), and bit-exact as well, since both sides
evaluate the same binary32 operations in the same order (NaN payloads aside:
a NaN must meet a NaN).  Side-output sums are fp64 reductions in different
orders: relative 1e-10."""
import numpy as np
import pytest
import torch

import paper_2104_05588_amd as daso
from oracle import daso_oracle as O
from workloads import recipes as R
from workloads import generate as Gen

pytestmark = pytest.mark.gpu

F32 = np.float32


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    daso.load()
    yield
    torch.cuda.synchronize()


def announce(*what):
    print("\n[case]", *what, flush=True)


# ---------------------------------------------------------------- helpers
def dev_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=F32)).to("cuda")


def dev_bf16(u16):
    return torch.from_numpy(np.ascontiguousarray(u16, dtype=np.uint16).view(np.int16)).to("cuda")


def host_f32(t):
    return t.detach().cpu().numpy()


def host_u16(t):
    return t.detach().cpu().numpy().view(np.uint16)


def check_f32(got, want, what):
    got = np.asarray(got, dtype=F32)
    want = np.asarray(want, dtype=F32)
    assert got.shape == want.shape, what
    both_nan = np.isnan(got) & np.isnan(want)
    fin = np.isfinite(want) & np.isfinite(got)
    err = np.abs(got[fin].astype(np.float64) - want[fin].astype(np.float64))
    lim = 1e-6 * np.maximum(1.0, np.abs(want[fin].astype(np.float64)))
    over = int(np.count_nonzero(err > lim))
    diff = (got.view(np.uint32) != want.view(np.uint32)) & ~both_nan
    nd = int(np.count_nonzero(diff))
    if over or nd:
        idx = np.nonzero(diff)[0][:6]
        raise AssertionError(f"{what}: {over} elements beyond 1e-6*max(1,|x|), {nd} of {got.size} "
                             f"not bit-identical; first at {idx.tolist()}: got {got[idx].tolist()} "
                             f"want {want[idx].tolist()}")


def check_u16(got, want, what):
    got = np.asarray(got, dtype=np.uint16)
    want = np.asarray(want, dtype=np.uint16)
    diff = got != want
    if diff.any():
        idx = np.nonzero(diff)[0][:6]
        raise AssertionError(f"{what}: {int(diff.sum())} of {got.size} differ; first at {idx.tolist()}: "
                             f"got {[hex(v) for v in got[idx]]} want {[hex(v) for v in want[idx]]}")


def check_stats(got, want, what):
    assert len(got) == len(want), what
    for b, (g, w) in enumerate(zip(got, want)):
        for k in (0, 1):
            if np.isnan(w[k]):
                assert np.isnan(g[k]), (what, b, k, g, w)
            elif np.isinf(w[k]):
                assert g[k] == w[k], (what, b, k, g, w)
            else:
                assert abs(g[k] - w[k]) <= 1e-10 * max(abs(w[k]), 1e-300), (what, b, k, g, w)
        assert g[2] == w[2], (what, b, g, w)


def random_buckets(rng, n, nb, S_choices=(0, 1, 2, 3, 4, 8)):
    """nb buckets with random (mostly unaligned) boundaries tiling [0, n)."""
    if n == 0:
        return [(0, 0, 1)]
    cuts = sorted(set(rng.integers(1, n, size=max(nb - 1, 0)).tolist())) if n > 1 else []
    edges = [0] + cuts + [n]
    bks = [(edges[i], edges[i + 1] - edges[i], int(rng.choice(S_choices))) for i in range(len(edges) - 1)]
    order = rng.permutation(len(bks))  # the ABI takes buckets in any order
    return [bks[i] for i in order]


def random_inputs(rng, n, g, P, specials=False):
    x = (rng.standard_normal(n) * 0.02).astype(F32)
    m = (rng.standard_normal(n) * 1e-3).astype(F32)
    grads = [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(g)]
    stale = [O.bf16_rne(x + (rng.standard_normal(n) * 1e-4).astype(F32)) for _ in range(P)]
    if specials and n:
        vals = np.array([np.nan, np.inf, -np.inf, 1e-40, -1e-41, 3.4e38, -3.4e38, -0.0, 0.0,
                         1.17549435e-38, 2.0 ** -149], dtype=F32)
        for arr in [x, m] + grads:
            k = max(1, n // 50)
            pos = rng.integers(0, n, k)
            arr[pos] = rng.choice(vals, k)
        for i in range(P):
            k = max(1, n // 50)
            pos = rng.integers(0, n, k)
            stale[i][pos] = O.bf16_rne(rng.choice(vals, k))
    return {"params": x, "momentum": m, "grads": grads, "stale": stale}


def run_fused(inp, buckets, lr=0.1, mu=0.9, wd=0.0, flags=0, wire=True, gavg="none", stats=True, f32=False):
    n = inp["params"].shape[0]
    grads = [dev_f32(a) for a in inp["grads"]]
    stale = [(dev_f32 if f32 else dev_bf16)(a) for a in inp["stale"]]
    x = dev_f32(inp["params"])
    m = dev_f32(inp["momentum"])
    w = torch.empty(n, dtype=torch.float32 if f32 else torch.int16, device="cuda") if wire else None
    ga = grads[0] if gavg == "alias" else (torch.empty(n, dtype=torch.float32, device="cuda")
                                           if gavg == "new" else None)
    st = daso.new_stats(len(buckets)) if stats else None
    daso.fused_sync_step(grads, x, m, stale, buckets, lr, mu, wd, w, ga, st, flags)
    torch.cuda.synchronize()
    return {"params": host_f32(x), "momentum": host_f32(m),
            "wire": (host_f32(w) if f32 else host_u16(w)) if wire else None,
            "grad_avg": host_f32(ga) if ga is not None else None,
            "stats": daso.decode_stats(st) if stats else None}


def compare_fused(got, want, what, wire=True, gavg=False, stats=True):
    check_f32(got["params"], want["params"], what + " params")
    check_f32(got["momentum"], want["momentum"], what + " momentum")
    if wire:
        (check_f32 if want["wire"].dtype == F32 else check_u16)(got["wire"], want["wire"], what + " wire")
    if gavg:
        check_f32(got["grad_avg"], want["grad_avg"], what + " grad_avg")
    if stats:
        check_stats(got["stats"], want["stats"], what + " stats")


SIZES = [1, 3, 4, 5, 7, 8, 9, 4095, 4097, 8191, 8192, 8193, 100_003]


# ------------------------------------------------------------------ pack
def test_pack_every_high_half_and_specials():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x4000, 0xC000], dtype=np.uint32)
    u = (hi[:, None] | lows[None, :]).ravel()
    u = np.concatenate([u, np.random.default_rng(1).integers(0, 1 << 32, 1_000_003, dtype=np.uint64)
                        .astype(np.uint32)])
    f = u.view(F32)
    announce("pack_bf16 n=", f.size)
    src = dev_f32(f)
    wire = torch.empty(f.size, dtype=torch.int16, device="cuda")
    daso.pack_bf16(src, wire)
    torch.cuda.synchronize()
    check_u16(host_u16(wire), O.pack_bf16(f), "pack")


def test_pack_every_binary32_pattern():
    """daso_pack_bf16 on all 2^32 binary32 bit patterns, in 32 launches of
    2^27, against the oracle (which the host C check ties to the nearest-value
    definition on every pattern)."""
    chunk = 1 << 27
    wire = torch.empty(chunk, dtype=torch.int16, device="cuda")
    for c in range(32):
        announce("pack_bf16 patterns", hex(c * chunk), "to", hex((c + 1) * chunk - 1))
        bits = torch.arange(c * chunk, (c + 1) * chunk, dtype=torch.int64, device="cuda")
        bits = torch.where(bits >= (1 << 31), bits - (1 << 32), bits).to(torch.int32)
        daso.pack_bf16(bits.view(torch.float32), wire)
        torch.cuda.synchronize()
        del bits
        u = np.arange(c * chunk, (c + 1) * chunk, dtype=np.uint64).astype(np.uint32)
        check_u16(host_u16(wire), O.pack_bf16(u.view(F32)), f"pack patterns chunk {c}")


@pytest.mark.parametrize("n", SIZES)
def test_pack_sizes(n):
    announce("pack_bf16 n=", n)
    f = (np.random.default_rng(n).standard_normal(n) * 3).astype(F32)
    src = dev_f32(f)
    wire = torch.full((n + 8,), 0x1234, dtype=torch.int16, device="cuda")
    daso.pack_bf16(src, wire[:n])
    torch.cuda.synchronize()
    h = host_u16(wire)
    check_u16(h[:n], O.pack_bf16(f), f"pack n={n}")
    assert np.all(h[n:] == 0x1234), "wrote past the end"


# ------------------------------------------------------------ local avg
@pytest.mark.parametrize("g", [1, 2, 3, 4, 5, 7, 8, 16, 64])
def test_local_avg(g):
    rng = np.random.default_rng(100 + g)
    for n in (1, 7, 8193, 100_003):
        announce("local_avg g=", g, "n=", n)
        G = [(rng.standard_normal(n) * 1e-3).astype(F32) for _ in range(g)]
        gd = [dev_f32(a) for a in G]
        out = torch.empty(n + 4, dtype=torch.float32, device="cuda").fill_(7.0)
        daso.local_avg(gd, out[:n])
        torch.cuda.synchronize()
        h = host_f32(out)
        check_f32(h[:n], O.local_avg(G), f"local_avg g={g} n={n}")
        assert np.all(h[n:] == 7.0)
        # in place: every replica's gradients become the average (Figure 2)
        daso.local_avg(gd, gd[0])
        torch.cuda.synchronize()
        check_f32(host_f32(gd[0]), O.local_avg(G), f"local_avg in place g={g} n={n}")


# ---------------------------------------------------------------- merge
@pytest.mark.parametrize("P", [0, 1, 2, 3, 4, 8, 16, 17, 32, 64])
def test_global_merge(P):
    rng = np.random.default_rng(200 + P)
    for n in (1, 9, 4097, 300_001):
        for nb in (1, 5):
            bks = random_buckets(rng, n, nb)
            announce("global_merge P=", P, "n=", n, "buckets=", len(bks))
            x = (rng.standard_normal(n) * 0.02).astype(F32)
            st = [O.bf16_rne(x + (rng.standard_normal(n) * 1e-4).astype(F32)) for _ in range(P)]
            want, wire_want = O.global_merge(x, st, bks, pack=True)
            xd = dev_f32(x)
            wd = torch.empty(n, dtype=torch.int16, device="cuda")
            daso.global_merge(xd, [dev_bf16(s) for s in st], bks, wd)
            torch.cuda.synchronize()
            check_f32(host_f32(xd), want, f"merge P={P} n={n}")
            check_u16(host_u16(wd), wire_want, f"merge wire P={P} n={n}")
            xd2 = dev_f32(x)
            daso.global_merge(xd2, [dev_bf16(s) for s in st], bks, None)
            torch.cuda.synchronize()
            check_f32(host_f32(xd2), want, f"merge no-wire P={P} n={n}")


def test_global_merge_many_buckets():
    """More buckets than one launch carries: the library splits the launches."""
    rng = np.random.default_rng(300)
    n, P = 500_000, 6
    bks = random_buckets(rng, n, 150)
    announce("global_merge many buckets", len(bks))
    x = (rng.standard_normal(n) * 0.02).astype(F32)
    st = [O.bf16_rne(x + (rng.standard_normal(n) * 1e-4).astype(F32)) for _ in range(P)]
    want, wire_want = O.global_merge(x, st, bks, pack=True)
    xd = dev_f32(x)
    wd = torch.empty(n, dtype=torch.int16, device="cuda")
    daso.global_merge(xd, [dev_bf16(s) for s in st], bks, wd)
    torch.cuda.synchronize()
    check_f32(host_f32(xd), want, "merge many")
    check_u16(host_u16(wd), wire_want, "merge many wire")


# ---------------------------------------------------------------- fused
FUSED_CASES = [
    # (seed, n, g, P, nbuckets, wd, flags, gavg)
    (1, 1, 1, 0, 1, 0.0, 0, "none"),
    (2, 7, 4, 2, 1, 0.0, 0, "new"),
    (3, 4097, 4, 8, 3, 0.0, 0, "alias"),
    (4, 8193, 3, 5, 4, 1e-4, 0, "new"),
    (5, 100_003, 8, 32, 6, 0.0, 0, "none"),
    (6, 100_003, 2, 0, 2, 1e-4, daso.DASO_PACK_PRE_MERGE, "new"),
    (7, 65_536, 4, 2, 1, 0.0, daso.DASO_PACK_PRE_MERGE, "none"),
    (8, 300_007, 5, 17, 9, 1e-4, 0, "alias"),
    (9, 123_457, 1, 1, 2, 0.0, 0, "none"),
    (10, 50_001, 64, 64, 3, 0.0, 0, "new"),
    (11, 77_777, 4, 16, 5, 0.0, 0, "none"),
    (12, 12_345, 6, 3, 70, 0.0, 0, "none"),
    # whole blocks of XCD tile runs: 45 streams (runs of 32 tiles), 26 streams (runs of 16)
    (13, 2 * 256 * 1024 + 4_097, 8, 32, 4, 0.0, 0, "none"),
    (14, 5 * 128 * 1024 + 333, 4, 16, 3, 0.0, 0, "new"),
]


@pytest.mark.parametrize("case", FUSED_CASES, ids=[f"s{c[0]}_n{c[1]}_g{c[2]}_P{c[3]}" for c in FUSED_CASES])
def test_fused_random(case):
    seed, n, g, P, nb, wd, flags, gavg = case
    rng = np.random.default_rng(seed)
    bks = random_buckets(rng, n, nb)
    inp = random_inputs(rng, n, g, P)
    announce("fused", case, "buckets", len(bks))
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks,
                             0.1, 0.9, wd, flags)
    got = run_fused(inp, bks, wd=wd, flags=flags, gavg=gavg)
    compare_fused(got, want, f"fused {case}", gavg=gavg != "none")


HYPER_CASES = [
    # (seed, n, g, P, lr, mu, wd, S choices): other optimizer constants, large S
    (31, 40_000, 4, 8, 0.05, 0.5, 5e-4, (0, 4, 12, 100)),
    (32, 40_000, 4, 8, 1e-3, 0.0, 0.0, (1, 3, 1000)),
    (33, 20_001, 8, 32, 1.7, 0.99, 1e-5, (1, 2, 4, 8, 16)),
    (34, 20_001, 3, 7, 0.0, 0.9, 0.0, (0, 5, 999)),
    (35, 9_999, 1, 0, 0.3, 0.95, 1e-2, (0,)),
    (36, 65_536, 2, 4, 0.1, 0.9, 0.0, (2, 6, 30, 62)),
    (37, 30_000, 4, 8, 0.1, 0.9, 0.0, (1 << 20, (1 << 20) - 3, 0)),   # the largest S accepted
]


@pytest.mark.parametrize("case", HYPER_CASES, ids=[f"s{c[0]}_lr{c[4]}_mu{c[5]}" for c in HYPER_CASES])
def test_fused_other_constants_and_large_S(case):
    """lr, mu and wd other than the workloads' (mu = 0, lr = 0 included) and
    staleness up to 1000, with 2S + P both powers of two and not."""
    seed, n, g, P, lr, mu, wd, S_choices = case
    rng = np.random.default_rng(seed)
    bks = random_buckets(rng, n, 5, S_choices)
    inp = random_inputs(rng, n, g, P)
    announce("fused constants", case)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks,
                             lr, mu, wd)
    got = run_fused(inp, bks, lr=lr, mu=mu, wd=wd, gavg="new")
    compare_fused(got, want, f"fused constants {case}", gavg=True)


@pytest.mark.parametrize("g,P", [(4, 32), (8, 2), (8, 4), (8, 8), (8, 16)])
def test_fused_node_shapes(g, P):
    """The compile-time instances for 4- and 8-GPU nodes (g) in groups of 2 to
    32 nodes (P), over several XCD run blocks and a ragged tail."""
    rng = np.random.default_rng(900 + 10 * g + P)
    n = 700_001
    bks = random_buckets(rng, n, 4)
    inp = random_inputs(rng, n, g, P)
    announce("fused node shape g=", g, "P=", P)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9, 1e-4)
    got = run_fused(inp, bks, wd=1e-4, gavg="new")
    compare_fused(got, want, f"node shape g={g} P={P}", gavg=True)


@pytest.mark.parametrize("g,P", [(3, 12), (8, 12), (5, 8), (7, 16), (2, 9), (1, 0), (6, 0), (8, 3)])
def test_fused_other_counts(g, P):
    """Counts between the node shapes: the instances bounded by 4 or 8 replicas
    and 8 or 16 copies (missing streams skipped), and the run-time-count one."""
    rng = np.random.default_rng(970 + 10 * g + P)
    n = 300_007
    bks = random_buckets(rng, n, 3)
    inp = random_inputs(rng, n, g, P)
    announce("fused other counts g=", g, "P=", P)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9, 1e-4)
    got = run_fused(inp, bks, wd=1e-4, gavg="new")
    compare_fused(got, want, f"other counts g={g} P={P}", gavg=True)


@pytest.mark.parametrize("P", [9, 12, 16, 33])
def test_global_merge_other_counts(P):
    rng = np.random.default_rng(990 + P)
    n = 200_003
    bks = random_buckets(rng, n, 3)
    x = (rng.standard_normal(n) * 0.02).astype(F32)
    st = [O.bf16_rne(x + (rng.standard_normal(n) * 1e-4).astype(F32)) for _ in range(P)]
    announce("global_merge other counts P=", P)
    want, wire_want = O.global_merge(x, st, bks, pack=True)
    xd = dev_f32(x)
    wd = torch.empty(n, dtype=torch.int16, device="cuda")
    daso.global_merge(xd, [dev_bf16(s_) for s_ in st], bks, wd)
    torch.cuda.synchronize()
    check_f32(host_f32(xd), want, f"merge P={P}")
    check_u16(host_u16(wd), wire_want, f"merge wire P={P}")


@pytest.mark.parametrize("g,P", [(4, 2), (4, 4), (4, 16), (4, 32), (8, 2), (8, 4), (8, 8), (8, 16)])
def test_fused_node_shapes_f32_exchange(g, P):
    """The fp32-exchange instances for the node shapes, over several XCD run
    blocks and a ragged tail."""
    rng = np.random.default_rng(950 + 10 * g + P)
    n = 700_007
    bks = random_buckets(rng, n, 3)
    inp = random_inputs(rng, n, g, 0)
    inp["stale"] = [(inp["params"] + (rng.standard_normal(n) * 1e-4).astype(F32)).astype(F32) for _ in range(P)]
    announce("fused node shape, fp32 exchange, g=", g, "P=", P)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9,
                             exchange="f32")
    got = run_fused(inp, bks, gavg="new", f32=True)
    compare_fused(got, want, f"node shape f32 g={g} P={P}", gavg=True)


@pytest.mark.parametrize("seed", [21, 22, 23])
def test_fused_special_values(seed):
    """NaN, infinities, subnormals, the largest finite values and signed zeros
    injected into every input stream."""
    rng = np.random.default_rng(seed)
    n, g, P = 20_011, 3, 5
    bks = random_buckets(rng, n, 4)
    inp = random_inputs(rng, n, g, P, specials=True)
    announce("fused specials seed", seed)
    for wd in (0.0, 1e-4):
        want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks,
                                 0.1, 0.9, wd)
        got = run_fused(inp, bks, wd=wd, gavg="new")
        compare_fused(got, want, f"fused specials seed={seed} wd={wd}", gavg=True)
        assert sum(s[2] for s in got["stats"]) > 0


@pytest.mark.parametrize("g,P,f32", [(4, 8, False), (3, 5, False), (9, 40, False), (8, 32, False),
                                     (4, 8, True), (5, 7, True)])
def test_zero_staleness_ignores_a_nonfinite_local_state(g, P, f32):
    """S = 0 (blocking average): a NaN or infinite local state leaves the merged
    value the plain mean of the finite copies; copies that are all -0 give -0.
    Buckets with S = 0 sit next to buckets with S > 0 (whose results do take
    the non-finite local state).  Fused step and the merge entry points, with
    exact, bounded and run-time stream counts, bf16 and fp32 exchange."""
    rng = np.random.default_rng(1000 + 10 * g + P + (5 if f32 else 0))
    n = 9_001
    inp = random_inputs(rng, n, g, P)
    for pos in (rng.integers(0, n, 300), rng.integers(0, n, 300), rng.integers(0, n, 300)):
        inp["params"][pos] = rng.choice(np.array([np.nan, np.inf, -np.inf], F32), pos.size)
    negz = rng.integers(0, n, 40)
    for st in inp["stale"]:
        st[negz] = 0x8000
    if f32:
        inp["stale"] = [O.bf16_widen(s) for s in inp["stale"]]
    bks = [(0, 3000, 0), (3000, 1001, 2), (4001, 5000, 0)]
    announce("S=0 non-finite local state g=", g, "P=", P, "f32=", f32)
    exch = "f32" if f32 else "bf16"
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks,
                             0.1, 0.9, 0.0, exchange=exch)
    zero_s = np.r_[0:3000, 4001:9001]
    assert np.all(np.isfinite(want["params"][zero_s]))
    assert not np.all(np.isfinite(want["x_local"][zero_s]))
    assert np.all(want["params"].view(np.uint32)[negz[negz < 3000]] == 0x80000000)
    got = run_fused(inp, bks, f32=f32)
    compare_fused(got, want, f"S=0 fused g={g} P={P} f32={f32}")
    # the merge entry point on the same local state
    xl = want["x_local"]
    mwant, mwire = O.global_merge(xl, inp["stale"], bks, pack=True, exchange=exch)
    xd = dev_f32(xl)
    wd_ = torch.empty(n, dtype=torch.float32 if f32 else torch.int16, device="cuda")
    daso.global_merge(xd, [(dev_f32 if f32 else dev_bf16)(a) for a in inp["stale"]], bks, wd_)
    torch.cuda.synchronize()
    check_f32(host_f32(xd), mwant, f"S=0 merge P={P} f32={f32}")
    (check_f32 if f32 else check_u16)(host_f32(wd_) if f32 else host_u16(wd_), mwire, f"S=0 merge wire P={P}")


def test_fused_without_optional_outputs():
    rng = np.random.default_rng(31)
    n = 33_333
    bks = random_buckets(rng, n, 3)
    inp = random_inputs(rng, n, 4, 4)
    announce("fused without wire/stats")
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
    got = run_fused(inp, bks, wire=False, stats=False)
    compare_fused(got, want, "fused bare", wire=False, stats=False)


def test_fused_empty_buckets_and_many_launches():
    rng = np.random.default_rng(32)
    n = 400_000
    bks = random_buckets(rng, n, 180) + [(n, 0, 3), (0, 0, 1)]
    inp = random_inputs(rng, n, 2, 3)
    announce("fused empty + many buckets", len(bks))
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
    got = run_fused(inp, bks)
    compare_fused(got, want, "fused many buckets")
    assert got["stats"][-1] == (0.0, 0.0, 0) and got["stats"][-2] == (0.0, 0.0, 0)


def test_binding_launches_on_the_current_stream():
    """With no stream given, the binding passes torch's current stream: the
    default one, or the one a `torch.cuda.stream` context selects."""
    from paper_2104_05588_amd import _lib as L
    announce("binding stream handle")
    side = torch.cuda.Stream()
    assert (L._stream_handle(None).value or 0) == torch.cuda.current_stream().cuda_stream
    with torch.cuda.stream(side):
        assert L._stream_handle(None).value == side.cuda_stream
    assert L._stream_handle(side).value == side.cuda_stream


def test_fused_is_deterministic_and_stream_ordered():
    w = R.workload("resnet18")
    inp = Gen.host_inputs(w)
    bks = [(b.start, b.numel, b.S) for b in w.buckets]
    announce("fused determinism resnet18")
    side = torch.cuda.Stream()
    outs = []
    for _ in range(2):
        grads = [dev_f32(a) for a in inp["grads"]]
        stale = [dev_bf16(a) for a in inp["stale"]]
        x, m = dev_f32(inp["params"]), dev_f32(inp["momentum"])
        wire = torch.empty(w.n, dtype=torch.int16, device="cuda")
        st = daso.new_stats(len(bks))
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            daso.fused_sync_step(grads, x, m, stale, bks, 0.1, 0.9, 0.0, wire, None, st)
            res = (x.clone(), wire.clone(), st.clone())
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        outs.append([host_f32(res[0]).view(np.uint32), host_u16(res[1]), host_f32(res[2])])
    for a, b in zip(outs[0], outs[1]):
        assert np.array_equal(a, b)


# ---------------------------------------------------- workloads, full size
@pytest.mark.parametrize("name", ["tiny", "resnet18", "resnet50", "segnet"])
def test_fused_workload_full(name):
    """Element-by-element parity at the full workload size, in the launch
    configuration the bench times (wire and statistics on)."""
    w = R.workload(name)
    announce("fused workload", name, "n=", w.n, "g=", w.g, "P=", w.P)
    inp = Gen.host_inputs(w)
    bks = [(b.start, b.numel, b.S) for b in w.buckets]
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks,
                             w.lr, w.mu, w.wd)
    got = run_fused(inp, bks, lr=w.lr, mu=w.mu, wd=w.wd)
    del inp
    compare_fused(got, want, f"workload {name}")


def test_fused_gpt_medium_full_size_every_element():
    """The 354.8M-parameter, g=8, P=32 workload (37 buckets, S = 1/2/4/8 by
    bucket) at full size, in the launch configuration the bench times (wire and
    statistics on): inputs are made on the device, the pre-step params and
    momentum are kept, and after the step every bucket's inputs and outputs are
    copied to the host and compared element by element with the oracle run on
    that bucket alone (bit for bit), with the bucket's statistics."""
    import threading
    from concurrent.futures import ThreadPoolExecutor

    w = R.workload("gpt_medium")
    announce("fused gpt_medium full size, every element: n=", w.n, "buckets=", len(w.buckets))
    inp = Gen.device_inputs(w)
    x0, m0 = inp["params"].clone(), inp["momentum"].clone()
    bks = [(b.start, b.numel, b.S) for b in w.buckets]
    wire = torch.empty(w.n, dtype=torch.int16, device="cuda")
    st = daso.new_stats(len(bks))
    daso.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks,
                         w.lr, w.mu, w.wd, wire, None, st)
    torch.cuda.synchronize()
    got_stats = daso.decode_stats(st)

    def check_bucket(b, part):
        want = O.fused_sync_step(part["grads"], part["x0"], part["m0"], part["stale"], [(0, part["k"], part["S"])],
                                 w.lr, w.mu, w.wd)
        what = f"gpt_medium bucket {b} (start {w.buckets[b].start}, {part['k']} elements, S={part['S']})"
        check_f32(part["params"], want["params"], what + " params")
        check_f32(part["momentum"], want["momentum"], what + " momentum")
        check_u16(part["wire"], want["wire"], what + " wire")
        check_stats([got_stats[b]], want["stats"], what + " stats")
        return part["k"]

    # the device-to-host copies run here, the oracle in worker threads (numpy
    # releases the GIL); at most 6 buckets are held on the host at once
    slots = threading.Semaphore(6)
    futures = []
    with ThreadPoolExecutor(8) as ex:
        for b, bk in enumerate(w.buckets):
            sl = slice(bk.start, bk.start + bk.numel)
            slots.acquire()
            part = {"k": bk.numel, "S": bk.S, "grads": [host_f32(t[sl]) for t in inp["grads"]],
                    "stale": [host_u16(t[sl]) for t in inp["stale"]], "x0": host_f32(x0[sl]),
                    "m0": host_f32(m0[sl]), "params": host_f32(inp["params"][sl]),
                    "momentum": host_f32(inp["momentum"][sl]), "wire": host_u16(wire[sl])}

            def job(b=b, part=part):
                try:
                    return check_bucket(b, part)
                finally:
                    slots.release()
            futures.append(ex.submit(job))
        checked = sum(f.result() for f in futures)
    assert checked == w.n


# ------------------------------------------------------------ fp32 exchange
@pytest.mark.parametrize("P", [0, 3, 8, 20])
def test_global_merge_f32(P):
    rng = np.random.default_rng(400 + P)
    for n in (5, 4097, 200_003):
        bks = random_buckets(rng, n, 4)
        announce("global_merge_f32 P=", P, "n=", n)
        x = (rng.standard_normal(n) * 0.02).astype(F32)
        st = [(x + (rng.standard_normal(n) * 1e-4).astype(F32)).astype(F32) for _ in range(P)]
        want, wire_want = O.global_merge(x, st, bks, pack=True, exchange="f32")
        xd = dev_f32(x)
        wd = torch.empty(n, dtype=torch.float32, device="cuda")
        daso.global_merge(xd, [dev_f32(a) for a in st], bks, wd)
        torch.cuda.synchronize()
        check_f32(host_f32(xd), want, f"merge_f32 P={P} n={n}")
        check_f32(host_f32(wd), wire_want, f"merge_f32 wire P={P} n={n}")


F32X_CASES = [
    # (seed, n, g, P, nbuckets, wd, flags)
    (61, 50_001, 4, 8, 3, 0.0, 0),
    (62, 33_333, 3, 5, 4, 1e-4, daso.DASO_PACK_PRE_MERGE),
    (63, 4097, 8, 32, 2, 0.0, 0),
    (64, 262_144, 4, 8, 1, 0.0, daso.DASO_PACK_PRE_MERGE),
    (65, 600_001, 8, 32, 3, 0.0, 0),           # run-time-count instance over whole XCD run blocks
]


@pytest.mark.parametrize("case", F32X_CASES, ids=[f"s{c[0]}_n{c[1]}_g{c[2]}_P{c[3]}" for c in F32X_CASES])
def test_fused_f32_exchange(case):
    seed, n, g, P, nb, wd, flags = case
    rng = np.random.default_rng(seed)
    bks = random_buckets(rng, n, nb)
    inp = random_inputs(rng, n, g, 0, specials=(seed == 62))
    inp["stale"] = [(inp["params"] + (rng.standard_normal(n) * 1e-4).astype(F32)).astype(F32) for _ in range(P)]
    announce("fused f32 exchange", case)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9, wd, flags,
                             exchange="f32")
    got = run_fused(inp, bks, wd=wd, flags=flags, gavg="new", f32=True)
    compare_fused(got, want, f"fused f32 {case}", gavg=True)


def test_fused_seeded_sweep_over_the_argument_space():
    """Seeded random draws over every argument at once: replica and copy counts
    that select the exact, bounded and run-time-count instances, both exchange
    types, the pre-merge pack flag, the wire, grad_avg and statistics each on or
    off, weight decay, S from 0 to 1000, and 1 to 8 buckets in any order over
    sizes that span several tiles with ragged tails."""
    rng = np.random.default_rng(2104_05588)
    for case in range(64):
        g = int(rng.choice([1, 2, 3, 4, 4, 5, 8, 8, 12, 16]))
        P = int(rng.choice([0, 1, 2, 3, 4, 6, 8, 8, 12, 16, 20, 32, 40]))
        f32 = bool(rng.random() < 0.3)
        n = int(rng.integers(1, 70_000))
        nb = int(rng.integers(1, 9))
        flags = daso.DASO_PACK_PRE_MERGE if rng.random() < 0.25 else 0
        wd = float(rng.choice([0.0, 1e-4]))
        lr, mu = float(rng.choice([0.1, 0.05])), float(rng.choice([0.9, 0.0]))
        wire = bool(rng.random() < 0.8)
        stats = bool(rng.random() < 0.7)
        gavg = str(rng.choice(["none", "new", "alias"]))
        bks = random_buckets(rng, n, nb, (0, 1, 2, 3, 4, 7, 1000))
        inp = random_inputs(rng, n, g, 0 if f32 else P)
        if f32:
            inp["stale"] = [(inp["params"] + (rng.standard_normal(n) * 1e-4).astype(F32)).astype(F32)
                            for _ in range(P)]
        what = f"sweep case {case}: n={n} g={g} P={P} f32={f32} buckets={len(bks)} flags={flags} " \
               f"wire={wire} stats={stats} gavg={gavg} wd={wd} lr={lr} mu={mu}"
        announce(what)
        want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, lr, mu, wd,
                                 flags, exchange="f32" if f32 else "bf16")
        got = run_fused(inp, bks, lr=lr, mu=mu, wd=wd, flags=flags, wire=wire, gavg=gavg, stats=stats, f32=f32)
        compare_fused(got, want, what, wire=wire, gavg=gavg != "none", stats=stats)


# ----------------------------------------------------------- edge cases
def test_empty_inputs_launch_nothing():
    announce("n = 0 on every entry point")
    e = torch.empty(0, dtype=torch.float32, device="cuda")
    h = torch.empty(0, dtype=torch.int16, device="cuda")
    daso.local_avg([e, e], e)
    daso.pack_bf16(e, h)
    daso.global_merge(e, [h, h], [(0, 0, 1)], h)
    daso.fused_sync_step([e], e, e.clone(), [h], [(0, 0, 2)], 0.1, 0.9, 0.0, h, None, daso.new_stats(1))
    torch.cuda.synchronize()


def test_fused_beyond_int32_element_count():
    """n = 2^31 + 13 elements (g = 1, P = 1, 37 GB of streams): element offsets
    and tile counts past 32 bits; sampled elements around 2^31 and the ends
    are checked against the oracle one by one."""
    n = (1 << 31) + 13
    announce("fused n =", n)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2104)
    x = torch.randn(n, generator=gen, device="cuda") * 0.02
    m = torch.zeros(n, device="cuda")
    gr = torch.randn(n, generator=gen, device="cuda") * 1e-3
    st = (x + torch.randn(n, generator=gen, device="cuda") * 1e-4).to(torch.bfloat16).view(torch.int16)
    wire = torch.empty(n, dtype=torch.int16, device="cuda")
    cut = (1 << 31) - 5   # bucket boundary just below 2^31, not vector aligned
    bks = [(0, cut, 1), (cut, n - cut, 3)]
    idx = np.unique(np.concatenate([np.arange(0, 16), np.arange(cut - 16, cut + 16), np.arange((1 << 31) - 16,
                                    (1 << 31) + 13), np.random.default_rng(3).integers(0, n, 4096)]))
    it = torch.from_numpy(idx).to("cuda")
    take = lambda t: t.index_select(0, it).cpu().numpy()  # noqa: E731
    s_x, s_m, s_g, s_s = take(x), take(m), take(gr), take(st).view(np.uint16)
    st_dev = daso.new_stats(2)
    daso.fused_sync_step([gr], x, m, [st], bks, 0.1, 0.9, 0.0, wire, None, st_dev)
    torch.cuda.synchronize()
    s_bks, i0 = [], 0
    side = idx >= cut
    for i in range(1, len(idx) + 1):
        if i == len(idx) or side[i] != side[i0]:
            s_bks.append((i0, i - i0, 3 if side[i0] else 1))
            i0 = i
    want = O.fused_sync_step([s_g], s_x, s_m, [s_s], s_bks, 0.1, 0.9)
    check_f32(take(x), want["params"], "n > 2^31 params")
    check_f32(take(m), want["momentum"], "n > 2^31 momentum")
    check_u16(take(wire).view(np.uint16), want["wire"], "n > 2^31 wire")
    got = daso.decode_stats(st_dev)
    assert got[0][2] == 0 and got[1][2] == 0 and got[0][0] > 0 and got[1][1] > 0


@pytest.mark.parametrize("n", [300_001, 60_001], ids=["large_launch", "small_launch"])
def test_fused_step_replays_in_a_hip_graph(n):
    """After a first eager call (which allocates the statistics workspace), the
    fused step can be captured in a graph: every replay, with eager work and
    synchronisations between replays, gives the eager result bit for bit.  The
    eager call of the small launch (at most 64 tiles) sums its statistics in its
    last workgroup, the captured one in the statistics kernel: the same bits."""
    rng = np.random.default_rng(77)
    bks = random_buckets(rng, n, 3)
    inp = random_inputs(rng, n, 4, 8)
    announce("fused step in a HIP graph")
    grads = [dev_f32(a) for a in inp["grads"]]
    stale = [dev_bf16(a) for a in inp["stale"]]
    x0, m0 = dev_f32(inp["params"]), dev_f32(inp["momentum"])
    x, m = x0.clone(), m0.clone()
    wire = torch.empty(n, dtype=torch.int16, device="cuda")
    stats = daso.new_stats(len(bks))
    step = daso.FusedStep(grads, x, m, stale, bks, 0.1, 0.9, 0.0, wire=wire, stats=stats)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                  # eager call on the capturing stream: allocates its workspace
    torch.cuda.synchronize()
    eager = (x.clone(), m.clone(), wire.clone(), stats.clone())
    x.copy_(x0)
    m.copy_(m0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        if rep == 1:
            # a larger eager call on the same stream enlarges the statistics
            # workspace; the graph keeps using the buffer it captured
            big = 100_000_000   # 48,829 tiles: more partials than the first 1 MB workspace holds
            bx, bm = torch.zeros(big, device="cuda"), torch.zeros(big, device="cuda")
            bg = [torch.zeros(big, device="cuda")]
            with torch.cuda.stream(side):
                daso.fused_sync_step(bg, bx, bm, [], [(0, big, 1)], 0.1, 0.9, 0.0, None, None, daso.new_stats(1))
            torch.cuda.synchronize()
            del bx, bm, bg
        x.copy_(x0)
        m.copy_(m0)
        wire.fill_(0)
        stats.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(x.view(torch.int32), eager[0].view(torch.int32)), rep
        assert torch.equal(m.view(torch.int32), eager[1].view(torch.int32)), rep
        assert torch.equal(wire, eager[2]), rep
        assert torch.equal(stats.view(torch.int64), eager[3].view(torch.int64)), rep


def test_buckets_on_concurrent_streams():
    """Bucket-granular use, as when buckets become ready one after another in
    backpropagation: each bucket's fused step runs on its own stream, on views
    of the flat buffers (every tensor starts at a multiple of 8 elements, so the
    views stay 16-byte aligned).  Together they equal one whole-buffer step."""
    w = R.workload("resnet18")
    inp = Gen.host_inputs(w)
    announce("fused step per bucket on", len(w.buckets), "streams")
    grads = [dev_f32(a) for a in inp["grads"]]
    stale = [dev_bf16(a) for a in inp["stale"]]
    x, m = dev_f32(inp["params"]), dev_f32(inp["momentum"])
    wire = torch.empty(w.n, dtype=torch.int16, device="cuda")
    streams = [torch.cuda.Stream() for _ in w.buckets]
    stats = [daso.new_stats(1) for _ in w.buckets]
    torch.cuda.synchronize()
    for bk, s, st in zip(w.buckets, streams, stats):
        sl = slice(bk.start, bk.start + bk.numel)
        with torch.cuda.stream(s):
            daso.fused_sync_step([g[sl] for g in grads], x[sl], m[sl], [t[sl] for t in stale], [(0, bk.numel, bk.S)],
                                 w.lr, w.mu, w.wd, wire[sl], None, st)
    torch.cuda.synchronize()
    bks = [(b.start, b.numel, b.S) for b in w.buckets]
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, w.lr, w.mu, w.wd)
    check_f32(host_f32(x), want["params"], "per-bucket params")
    check_f32(host_f32(m), want["momentum"], "per-bucket momentum")
    check_u16(host_u16(wire), want["wire"], "per-bucket wire")
    check_stats([daso.decode_stats(st)[0] for st in stats], want["stats"], "per-bucket stats")


def test_earlier_hip_error_is_neither_blamed_nor_consumed():
    """A failed HIP call made before (here an impossible hipMalloc) may leave its
    error as the thread's last error: the next library call must still succeed
    (its launches report their own status)."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7")          # the HIP runtime this process already uses
    hip.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    rng = np.random.default_rng(808)
    n = 10_001
    bks = random_buckets(rng, n, 2)
    inp = random_inputs(rng, n, 4, 8)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
    grads = [dev_f32(a) for a in inp["grads"]]
    stale = [dev_bf16(a) for a in inp["stale"]]
    x, m = dev_f32(inp["params"]), dev_f32(inp["momentum"])
    wire = torch.empty(n, dtype=torch.int16, device="cuda")
    st = daso.new_stats(len(bks))
    torch.cuda.synchronize()
    announce("fused step after a failed hipMalloc")
    ptr = ctypes.c_void_p()
    failed = hip.hipMalloc(ctypes.byref(ptr), ctypes.c_size_t(1 << 62))
    assert failed != 0
    daso.fused_sync_step(grads, x, m, stale, bks, 0.1, 0.9, 0.0, wire, None, st)
    hip.hipGetLastError()                               # clear it before torch launches again
    torch.cuda.synchronize()
    got = {"params": host_f32(x), "momentum": host_f32(m), "wire": host_u16(wire), "grad_avg": None,
           "stats": daso.decode_stats(st)}
    compare_fused(got, want, "after a failed hipMalloc")


def test_small_and_large_launches_alternate_on_one_stream():
    """Launches of at most 64 tiles sum their statistics in their last workgroup
    (a counter in the workspace that each leaves at zero), larger ones in a
    second kernel; mixed on one stream, every call's statistics and outputs
    match the oracle."""
    rng = np.random.default_rng(515)
    sizes = [20_000, 130_000, 65_536, 1, 400_000, 131_072, 2_000_003, 9_000]
    for k, n in enumerate(sizes):
        bks = random_buckets(rng, n, int(rng.integers(1, 5)))
        inp = random_inputs(rng, n, 4, 8)
        announce("alternating launch sizes, call", k, "n =", n)
        got = run_fused(inp, bks)
        want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
        compare_fused(got, want, f"alternating launch sizes, call {k} (n = {n})")


def test_tile_order_choice_keeps_results_and_a_pending_error():
    """The first calls of a fused shape alternate between two tile orders and
    time them with events the library polls: every call gives the same bits,
    the order it settles on is one of the two, and while a caller's HIP error
    is pending the polling leaves it in place (neither consumed nor replaced)."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7")
    hip.hipMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t]
    rng = np.random.default_rng(909)
    for n, use_error in ((1_000_003, False), (1_000_013, True)):
        bks = random_buckets(rng, n, 3)
        inp = random_inputs(rng, n, 4, 16)
        announce("tile-order choice n=", n, "pending error:", use_error)
        grads = [dev_f32(a) for a in inp["grads"]]
        stale = [dev_bf16(a) for a in inp["stale"]]
        x0, m0 = dev_f32(inp["params"]), dev_f32(inp["momentum"])
        xs = [x0.clone() for _ in range(8)]
        ms = [m0.clone() for _ in range(8)]
        wires = [torch.empty(n, dtype=torch.int16, device="cuda") for _ in range(8)]
        sts = [daso.new_stats(len(bks)) for _ in range(8)]
        steps = [daso.FusedStep(grads, xs[k], ms[k], stale, bks, 0.1, 0.9, 0.0, wire=wires[k], stats=sts[k])
                 for k in range(8)]
        cfg = steps[0].launch_config()
        rule = cfg["xcd_run_tiles"]
        torch.cuda.synchronize()
        if use_error:
            ptr = ctypes.c_void_p()
            failed = hip.hipMalloc(ctypes.byref(ptr), ctypes.c_size_t(1 << 62))
            assert failed != 0
        for st in steps:
            st()
        if use_error:
            assert hip.hipGetLastError() == failed     # still the caller's error
            assert hip.hipGetLastError() == 0
        torch.cuda.synchronize()
        steps[0]()                                      # polls the samples, now complete
        torch.cuda.synchronize()
        chosen = steps[0].launch_config()["xcd_run_tiles"]
        assert chosen in (rule, 1), (chosen, rule)
        want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
        for k in range(1, 8):
            got = {"params": host_f32(xs[k]), "momentum": host_f32(ms[k]), "wire": host_u16(wires[k]),
                   "grad_avg": None, "stats": daso.decode_stats(sts[k])}
            compare_fused(got, want, f"tile-order choice call {k}")


def test_tile_order_samples_on_two_streams_finishing_out_of_order():
    """After a shape's first call, its six sampled calls alternate between two
    streams; the first stream is kept busy, so the later samples on the second
    one finish first.  A call that polls then must not read the unfinished
    samples' times or leave a HIP error behind; a later poll decides, and every
    call gives the oracle's bits."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so.7")
    rng = np.random.default_rng(919)
    n = 1_000_033
    bks = random_buckets(rng, n, 3)
    inp = random_inputs(rng, n, 4, 16)
    announce("tile-order samples on two streams, n=", n)
    grads = [dev_f32(a) for a in inp["grads"]]
    stale = [dev_bf16(a) for a in inp["stale"]]
    x0, m0 = dev_f32(inp["params"]), dev_f32(inp["momentum"])
    sampled = 1 + 6                       # the unsampled first call, then the samples
    calls = sampled + 2
    xs = [x0.clone() for _ in range(calls)]
    ms = [m0.clone() for _ in range(calls)]
    wires = [torch.empty(n, dtype=torch.int16, device="cuda") for _ in range(calls)]
    sts = [daso.new_stats(len(bks)) for _ in range(calls)]
    steps = [daso.FusedStep(grads, xs[k], ms[k], stale, bks, 0.1, 0.9, 0.0, wire=wires[k], stats=sts[k])
             for k in range(calls)]
    rule = steps[0].launch_config()["xcd_run_tiles"]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    busy = torch.empty(1 << 29, dtype=torch.float32, device="cuda")   # 2 GiB
    torch.cuda.synchronize()
    for k in range(sampled):              # odd calls on the first stream, the last sample on the second
        s = sa if k % 2 == 1 else sb
        with torch.cuda.stream(s):
            if s is sa:
                for i in range(6):        # a few ms of fills ahead of each sample on the first stream
                    busy.fill_(float(i))
            steps[k]()
    sb.synchronize()                      # the second stream's samples are done
    with torch.cuda.stream(sb):
        steps[sampled]()                  # polls while the first stream's samples are still queued
    assert hip.hipPeekAtLastError() == 0
    torch.cuda.synchronize()
    with torch.cuda.stream(sb):
        steps[sampled + 1]()              # polls again: every sample has completed
    torch.cuda.synchronize()
    assert hip.hipGetLastError() == 0
    assert steps[0].launch_config()["xcd_run_tiles"] in (rule, 1)
    del busy
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
    for k in range(calls):
        got = {"params": host_f32(xs[k]), "momentum": host_f32(ms[k]), "wire": host_u16(wires[k]),
               "grad_avg": None, "stats": daso.decode_stats(sts[k])}
        compare_fused(got, want, f"two-stream sampling call {k}")


def test_calls_from_several_host_threads():
    """Four host threads make fused calls with statistics at once, two of them
    on one shared stream: every call must still see its own tile partials (a
    call's step and statistics pass are queued together)."""
    import threading
    rng = np.random.default_rng(707)
    streams = [torch.cuda.Stream() for _ in range(3)]
    owner = [0, 0, 1, 2]                     # thread -> stream
    jobs = []
    for t in range(4):
        for _ in range(12):
            n = int(rng.integers(1_000, 200_000))
            bks = random_buckets(rng, n, int(rng.integers(1, 4)))
            inp = random_inputs(rng, n, 4, 8)
            dev = {"grads": [dev_f32(a) for a in inp["grads"]], "stale": [dev_bf16(a) for a in inp["stale"]],
                   "x": dev_f32(inp["params"]), "m": dev_f32(inp["momentum"]),
                   "wire": torch.empty(n, dtype=torch.int16, device="cuda"), "stats": daso.new_stats(len(bks))}
            jobs.append((t, bks, inp, dev))
    torch.cuda.synchronize()
    announce("fused calls from 4 host threads,", len(jobs), "calls, 2 threads sharing a stream")
    start = threading.Barrier(4)
    errors = []

    def work(t):
        try:
            start.wait()
            for (tt, bks, _, d) in jobs:
                if tt == t:
                    daso.fused_sync_step(d["grads"], d["x"], d["m"], d["stale"], bks, 0.1, 0.9, 0.0, d["wire"],
                                         None, d["stats"], 0, streams[owner[t]])
        except Exception as e:  # reported by the main thread
            errors.append(e)

    th = [threading.Thread(target=work, args=(t,)) for t in range(4)]
    for x in th:
        x.start()
    for x in th:
        x.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for k, (t, bks, inp, d) in enumerate(jobs):
        want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], inp["stale"], bks, 0.1, 0.9)
        got = {"params": host_f32(d["x"]), "momentum": host_f32(d["m"]), "wire": host_u16(d["wire"]),
               "grad_avg": None, "stats": daso.decode_stats(d["stats"])}
        compare_fused(got, want, f"thread {t} call {k}")


@pytest.mark.parametrize("g", [1, 2, 4, 8])
def test_fused_local_step_only(g):
    """P = 0: the local step of a cycling batch without arrivals, with and
    without packing the wire (the batch that starts an exchange)."""
    rng = np.random.default_rng(600 + g)
    n = 70_001
    bks = random_buckets(rng, n, 3)
    inp = random_inputs(rng, n, g, 0)
    announce("fused local step g=", g)
    want = O.fused_sync_step(inp["grads"], inp["params"], inp["momentum"], [], bks, 0.1, 0.9)
    got = run_fused(inp, bks)
    compare_fused(got, want, f"local step g={g}")
    got = run_fused(inp, bks, wire=False, stats=False)
    compare_fused(got, want, f"local step g={g} bare", wire=False, stats=False)


_RUN_ORDER_SCRIPT = r"""
import sys
import numpy as np
import torch
sys.path.insert(0, sys.argv[1])
import paper_2104_05588_amd as daso
torch.cuda.set_device(0)
n, g, P = 1_200_007, int(sys.argv[2]), int(sys.argv[3])
bks = [(0, 500_003, 4), (500_003, n - 500_003, 2)]
gen = torch.Generator(device="cuda")
gen.manual_seed(77)
x = torch.randn(n, generator=gen, device="cuda") * 0.02
m = torch.randn(n, generator=gen, device="cuda") * 1e-3
grads = [torch.randn(n, generator=gen, device="cuda") * 1e-3 for _ in range(g)]
stale = [(x + torch.randn(n, generator=gen, device="cuda") * 1e-4).to(torch.bfloat16).view(torch.int16)
         for _ in range(P)]
outs = []
for k in range(10):  # after its first call a shape samples two tile orders (6 calls), later ones take the chosen one
    xk, mk = x.clone(), m.clone()
    wire = torch.empty(n, dtype=torch.int16, device="cuda")
    st = daso.new_stats(len(bks))
    daso.fused_sync_step(grads, xk, mk, stale, bks, 0.1, 0.9, 0.0, wire, None, st)
    torch.cuda.synchronize()
    outs.append(np.concatenate([xk.cpu().numpy().view(np.uint8), mk.cpu().numpy().view(np.uint8),
                                wire.cpu().numpy().view(np.uint8), st.cpu().numpy().ravel().view(np.uint8)]))
assert all(np.array_equal(o, outs[0]) for o in outs), "calls of one process differ"
sys.stdout.buffer.write(outs[0].tobytes())
"""


@pytest.mark.parametrize("g,P", [(4, 8), (8, 32)])
def test_launch_shape_never_changes_a_result(g, P):
    """DASO_FUSED_RUN_ELEMS, DASO_FUSED_WG_PER_CU and DASO_FUSED_TUNE change only
    which XCD takes which tiles and how many workgroups share a CU: plain order,
    the default runs (chosen per shape from the first calls, or not), longer or
    shorter runs, no occupancy cap and caps of 1 to 3 workgroups per CU all give
    the same bits (2048- and 1024-element tiles)."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    outs = {}
    for run, cap, tune in (("", "", ""), ("0", "0", ""), ("4096", "1", ""), ("65536", "3", ""),
                           ("1048576", "2", ""), ("", "", "0")):
        announce("launch shape g=", g, "P=", P, "DASO_FUSED_RUN_ELEMS =", repr(run), "DASO_FUSED_WG_PER_CU =",
                 repr(cap), "DASO_FUSED_TUNE =", repr(tune))
        env = dict(os.environ, DASO_FUSED_RUN_ELEMS=run, DASO_FUSED_WG_PER_CU=cap, DASO_FUSED_TUNE=tune)
        res = subprocess.run([sys.executable, "-c", _RUN_ORDER_SCRIPT, root, str(g), str(P)], capture_output=True,
                             env=env, timeout=110)
        assert res.returncode == 0, res.stderr.decode()[-2000:]
        outs[(run, cap, tune)] = res.stdout
    base = outs[("", "", "")]
    assert len(base) > 0
    for v, o in outs.items():
        assert o == base, v
