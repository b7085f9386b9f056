"""The C-ABI library without a GPU: it loads, exports every function that
include/daso.h declares, and rejects bad arguments before anything is launched.

The argument checks run on the host before any HIP call, so they can be fed
fake (never dereferenced) device addresses.  These tests only ever pass
arguments that must be rejected; to be certain that nothing is launched on
real hardware with such addresses, they skip when a GPU is visible."""
import ctypes
import os
import re

import pytest

from paper_2104_05588_amd import _lib as L
from paper_2104_05588_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "daso.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        B.build()
    return L.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(daso_\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("daso_local_avg", "daso_pack_bf16", "daso_global_merge", "daso_fused_sync_step",
                     "daso_status_string"):
        assert required in names
    assert set(names) == set(L.EXPORTED)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings_and_version(lib):
    assert lib.daso_abi_version() == 102
    for code in (L.DASO_OK, L.DASO_EINVAL, L.DASO_EALIGN, L.DASO_EALIAS, L.DASO_EHIP, L.DASO_ENOSPACE):
        s = L.status_string(code)
        assert s.startswith("DASO_")
    assert "unknown" in L.status_string(-99)


def test_struct_layouts_match_header(tmp_path):
    """Field offsets and sizes of the binding's ctypes structs equal what a C
    compiler makes of include/daso.h."""
    import subprocess
    fields = {"daso_bucket": [f[0] for f in L.daso_bucket._fields_],
              "daso_bucket_stats": [f[0] for f in L.daso_bucket_stats._fields_],
              "daso_sync_args": [f[0] for f in L.daso_sync_args._fields_],
              "daso_schedule_config": [f[0] for f in L.daso_schedule_config._fields_],
              "daso_batch_plan": [f[0] for f in L.daso_batch_plan._fields_],
              "daso_launch_config": [f[0] for f in L.daso_launch_config._fields_]}
    src = ["#include <stdio.h>", "#include <stddef.h>", '#include "daso.h"', "int main(void) {"]
    for st, names in fields.items():
        src.append(f'  printf("{st} size %zu\\n", sizeof({st}));')
        for f in names:
            src.append(f'  printf("{st} {f} %zu\\n", offsetof({st}, {f}));')
    src.append("  return 0; }")
    c = tmp_path / "layout.c"
    c.write_text("\n".join(src) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include",
                    str(c), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    for line in filter(None, out):
        st, f, v = line.split()
        cls = getattr(L, st)
        want = ctypes.sizeof(cls) if f == "size" else getattr(cls, f).offset
        assert int(v) == want, (st, f, int(v), want)


# ------------------------------------------------------------- validation
def _no_gpu():
    import torch
    if torch.cuda.is_available():
        pytest.skip("argument-check tests use fake device addresses; run them without a GPU")


A = 0x10000000          # fake, 16-byte aligned "device" addresses, never dereferenced
MB = 1 << 20


def ptrs(*xs):
    arr = (ctypes.c_void_p * max(len(xs), 1))()
    for i, x in enumerate(xs):
        arr[i] = x
    return arr


def test_local_avg_rejects(lib):
    _no_gpu()
    f, n = lib.daso_local_avg, 1000
    g4 = ptrs(A, A + MB, A + 2 * MB, A + 3 * MB)
    assert f(g4, 0, A + 8 * MB, n, None) == L.DASO_EINVAL
    assert f(g4, 65, A + 8 * MB, n, None) == L.DASO_EINVAL
    assert f(None, 4, A + 8 * MB, n, None) == L.DASO_EINVAL
    assert f(g4, 4, None, n, None) == L.DASO_EINVAL
    assert f(g4, 4, A + 8 * MB, -1, None) == L.DASO_EINVAL
    assert f(ptrs(A, 0, A + 2 * MB, A + 3 * MB), 4, A + 8 * MB, n, None) == L.DASO_EINVAL
    assert f(g4, 4, A + 8 * MB + 4, n, None) == L.DASO_EALIGN
    assert f(ptrs(A, A + MB + 8, A + 2 * MB, A + 3 * MB), 4, A + 8 * MB, n, None) == L.DASO_EALIGN
    assert f(g4, 4, A + MB + 64, n, None) == L.DASO_EALIAS  # partial overlap with grads[1]
    assert f(g4, 4, A + 8 * MB, 0, None) == L.DASO_OK       # n == 0: no-op


def test_pack_rejects(lib):
    _no_gpu()
    f = lib.daso_pack_bf16
    assert f(A, A + 1008, 1000, None) == L.DASO_EALIAS
    assert f(A, A + 8 * MB + 2, 1000, None) == L.DASO_EALIGN
    assert f(None, A + 8 * MB, 1000, None) == L.DASO_EINVAL
    assert f(A, A + 8 * MB, -5, None) == L.DASO_EINVAL
    assert f(A, A + 8 * MB, 0, None) == L.DASO_OK


def test_global_merge_rejects(lib):
    _no_gpu()
    f, n = lib.daso_global_merge, 1000
    st = ptrs(A + MB, A + 2 * MB)
    ok_b = L.bucket_table([(0, 600, 1), (600, 400, 2)])
    assert f(A, st, 2, L.bucket_table([(0, 600, 1), (601, 399, 2)]), 2, None, n, None) == L.DASO_EINVAL
    assert f(A, st, 2, L.bucket_table([(0, 600, 1), (600, 401, 2)]), 2, None, n, None) == L.DASO_EINVAL
    assert f(A, st, 2, L.bucket_table([(0, 600, -1), (600, 400, 2)]), 2, None, n, None) == L.DASO_EINVAL
    assert f(A, st, 2, L.bucket_table([(0, 1000, 1 << 21)]), 1, None, n, None) == L.DASO_EINVAL
    assert f(A, st, 2, L.bucket_table([(0, 1000, (1 << 20) + 1)]), 1, None, n, None) == L.DASO_EINVAL
    # S = DASO_MAX_S passes the checks; with no GPU here the call then fails in HIP
    assert f(A, st, 2, L.bucket_table([(0, 1000, 1 << 20)]), 1, None, n, None) == L.DASO_EHIP
    assert f(A, st, 2, ok_b, 0, None, n, None) == L.DASO_EINVAL
    bad = L.bucket_table([(0, 1000, 1)])
    bad[0].reserved = 3
    assert f(A, st, 2, bad, 1, None, n, None) == L.DASO_EINVAL
    assert f(A, st, 65, ok_b, 2, None, n, None) == L.DASO_EINVAL
    assert f(A, None, 2, ok_b, 2, None, n, None) == L.DASO_EINVAL
    assert f(A, ptrs(A + 1024, A + 2 * MB), 2, ok_b, 2, None, n, None) == L.DASO_EALIAS
    assert f(A, st, 2, ok_b, 2, A + 2 * MB + 512, n, None) == L.DASO_EALIAS
    assert f(A, st, 2, ok_b, 2, A + 3 * MB + 2, n, None) == L.DASO_EALIGN
    assert f(A + 4, st, 2, ok_b, 2, None, n, None) == L.DASO_EALIGN


def _args(n=1000, g=2, P=2):
    a = L.daso_sync_args()
    keep = [ptrs(*[A + r * MB for r in range(g)]), ptrs(*[A + (10 + i) * MB for i in range(P)]),
            L.bucket_table([(0, n, 2)])]
    a.n, a.g, a.P = n, g, P
    a.grads, a.stale = keep[0], keep[1]
    a.params, a.momentum = A + 20 * MB, A + 21 * MB
    a.wire, a.grad_avg, a.stats = A + 22 * MB, None, None
    a.buckets, a.nbuckets = keep[2], 1
    a.lr, a.mu, a.weight_decay, a.flags = 0.1, 0.9, 0.0, 0
    return a, keep


@pytest.mark.parametrize("entry", ["daso_fused_sync_step", "daso_fused_sync_step_noalloc"])
def test_fused_rejects(lib, entry):
    _no_gpu()
    f = getattr(lib, entry)
    assert f(None, None) == L.DASO_EINVAL

    def rc(**kw):
        a, keep = _args()
        for k, v in kw.items():
            setattr(a, k, v)
        return f(ctypes.byref(a), None)

    assert rc(g=0) == L.DASO_EINVAL
    assert rc(P=-1) == L.DASO_EINVAL
    assert rc(flags=4) == L.DASO_EINVAL
    assert rc(params=None) == L.DASO_EINVAL
    assert rc(momentum=A + 21 * MB + 4) == L.DASO_EALIGN
    assert rc(stats=A + 30 * MB + 4) == L.DASO_EALIGN
    assert rc(momentum=A + 20 * MB + 16) == L.DASO_EALIAS        # params / momentum overlap
    assert rc(wire=A + 21 * MB + 64) == L.DASO_EALIAS            # wire inside momentum
    assert rc(wire=A + 10 * MB) == L.DASO_EALIAS                 # wire on a stale copy
    assert rc(params=A + MB + 32) == L.DASO_EALIAS               # params inside grads[1]
    assert rc(grad_avg=A + 11 * MB) == L.DASO_EALIAS             # grad_avg on a stale copy
    assert rc(grad_avg=A + MB + 16) == L.DASO_EALIAS             # partial overlap with grads[1]
    assert rc(grad_avg=A + 20 * MB) == L.DASO_EALIAS             # grad_avg on params
    assert rc(stats=A + 22 * MB) == L.DASO_EALIAS                # stats on the wire
    assert rc(nbuckets=0) == L.DASO_EINVAL
    assert rc(n=0) == L.DASO_OK
    # fp32 exchange: the copies and the wire move to stale_f32 / wire_f32
    st32 = ptrs(A + 10 * MB, A + 14 * MB)
    assert rc(flags=L.DASO_EXCHANGE_F32) == L.DASO_EINVAL                        # stale still set
    assert rc(stale_f32=st32) == L.DASO_EINVAL                                   # without the flag
    assert rc(flags=L.DASO_EXCHANGE_F32, stale=None, wire=None,
              stale_f32=st32, wire_f32=A + 10 * MB + 2000) == L.DASO_EALIAS     # wire inside copy 0 (4 B/elem)
    assert rc(flags=L.DASO_EXCHANGE_F32, stale=None, wire=None,
              stale_f32=st32, wire_f32=A + 30 * MB + 8) == L.DASO_EALIGN
    assert rc(flags=L.DASO_EXCHANGE_F32, stale=None, wire=None, n=0, stale_f32=st32) == L.DASO_OK


def test_noalloc_rejects_statistics_beyond_its_scratch(lib):
    """daso_fused_sync_step_noalloc keeps a 256-byte counter, the statistics
    partials (24 bytes per tile) and the 65-entry table of a launch in its fixed
    16 MiB array: 699,029 tiles fit, one more is DASO_ENOSPACE before any HIP call.  g = 1, P = 0 runs
    2048-element tiles.  Without statistics there is no limit; with room the
    call goes on to HIP, which fails here without a GPU."""
    _no_gpu()
    f = lib.daso_fused_sync_step_noalloc
    GB8 = 8 << 30
    assert L.DASO_ENOSPACE == -5 and "DASO_ENOSPACE" in L.status_string(L.DASO_ENOSPACE)
    fit = 699_029

    def rc(n, stats=True, nb=1):
        a = L.daso_sync_args()
        keep = [ptrs(A), L.bucket_table([(0, n, 1)] if nb == 1 else [(0, n - 5, 1), (n - 5, 5, 2)])]
        a.n, a.g, a.P = n, 1, 0
        a.grads, a.stale = keep[0], None
        a.params, a.momentum, a.wire = A + GB8, A + 2 * GB8, A + 3 * GB8
        a.stats = A + 4 * GB8 if stats else None
        a.buckets, a.nbuckets = keep[1], nb
        a.lr, a.mu = 0.1, 0.9
        return f(ctypes.byref(a), None)

    assert (256 + 24 * fit + 65 * 4) <= (16 << 20) < 256 + 24 * (fit + 1) + 65 * 4
    assert rc(fit * 2048 + 1) == L.DASO_ENOSPACE
    assert rc(fit * 2048 + 1, nb=2) == L.DASO_ENOSPACE
    assert rc(fit * 2048) == L.DASO_EHIP
    assert rc(fit * 2048 + 1, stats=False) == L.DASO_EHIP
    assert lib.daso_fused_sync_step(ctypes.byref(L.daso_sync_args()), None) == L.DASO_EINVAL


def test_global_merge_f32_rejects(lib):
    _no_gpu()
    f, n = lib.daso_global_merge_f32, 1000
    st = ptrs(A + MB, A + 2 * MB)
    ok_b = L.bucket_table([(0, 1000, 1)])
    assert f(A, ptrs(A + 2048, A + 2 * MB), 2, ok_b, 1, None, n, None) == L.DASO_EALIAS   # 4 B/elem overlap
    assert f(A, st, 2, ok_b, 1, A + MB + 3200, n, None) == L.DASO_EALIAS               # wire inside copy 0
    assert f(A, st, 2, L.bucket_table([(0, 999, 1)]), 1, None, n, None) == L.DASO_EINVAL
    assert f(A, st, 2, ok_b, 1, None, 0, None) == L.DASO_OK


def test_element_count_limit(lib):
    """n beyond DASO_MAX_N (2^56) is refused before any byte span is formed."""
    _no_gpu()
    big = (1 << 56) + 1
    assert lib.daso_pack_bf16(A, A + 8 * MB, big, None) == L.DASO_EINVAL
    assert lib.daso_local_avg(ptrs(A), 1, A + 8 * MB, big, None) == L.DASO_EINVAL
    assert lib.daso_global_merge(A, ptrs(A + MB), 1, L.bucket_table([(0, big, 1)]), 1, None, big,
                                 None) == L.DASO_EINVAL
    a, keep = _args()
    a.n = big
    assert lib.daso_fused_sync_step(ctypes.byref(a), None) == L.DASO_EINVAL


def _spans_overlap(p, nbytes, q, mbytes):
    return p < q + mbytes and q < p + nbytes


def _expected_fused(n, grads, stale, params, momentum, wire, grad_avg, stats, nb):
    """The aliasing rule of daso_fused_sync_step, written from its header comment:
    params, momentum, wire and stats overlap nothing else (inputs or outputs);
    grad_avg overlaps no output and no copy, and of the gradients at most the one
    buffer it equals exactly."""
    ins = [(g, 4 * n) for g in grads] + [(s, 2 * n) for s in stale]
    outs = [(params, 4 * n), (momentum, 4 * n)]
    if wire:
        outs.append((wire, 2 * n))
    if stats:
        outs.append((stats, 24 * nb))
    for i, o in enumerate(outs):
        if any(_spans_overlap(*o, *x) for x in outs[i + 1:] + ins):
            return L.DASO_EALIAS
    if grad_avg:
        ga = (grad_avg, 4 * n)
        if any(_spans_overlap(*ga, *o) for o in outs) or any(_spans_overlap(*ga, s, 2 * n) for s in stale):
            return L.DASO_EALIAS
        if any(g != grad_avg and _spans_overlap(*ga, g, 4 * n) for g in grads):
            return L.DASO_EALIAS
    return L.DASO_EHIP          # passes every check; with no GPU the launch then fails


def test_fused_aliasing_rule_on_random_layouts(lib):
    """Random buffer layouts in a small fake address range (so that overlaps are
    frequent), every pointer aligned and the buckets valid: the status must be
    exactly what the header's aliasing rule says."""
    _no_gpu()
    hypothesis = pytest.importorskip("hypothesis")
    st = hypothesis.strategies

    @hypothesis.settings(max_examples=400, deadline=None, derandomize=True)
    @hypothesis.given(st.data())
    def check(data):
        n = data.draw(st.integers(1, 64)) * 4
        g = data.draw(st.integers(1, 3))
        P = data.draw(st.integers(0, 3))
        slots = 48                                   # buffers start on a 16-byte grid of this many slots
        addr = st.integers(0, slots).map(lambda k: A + 16 * k * 8)
        grads = [data.draw(addr) for _ in range(g)]
        stale = [data.draw(addr) for _ in range(P)]
        params, momentum = data.draw(addr), data.draw(addr)
        wire = data.draw(st.one_of(st.none(), addr))
        grad_avg = data.draw(st.one_of(st.none(), addr, st.sampled_from(grads)))
        stats = data.draw(st.one_of(st.none(), addr))
        a = L.daso_sync_args()
        keep = [ptrs(*grads), ptrs(*stale), L.bucket_table([(0, n, 1)])]
        a.n, a.g, a.P = n, g, P
        a.grads, a.stale = keep[0], keep[1]
        a.params, a.momentum, a.wire, a.grad_avg, a.stats = params, momentum, wire, grad_avg, stats
        a.buckets, a.nbuckets = keep[2], 1
        a.lr, a.mu, a.weight_decay, a.flags = 0.1, 0.9, 0.0, 0
        want = _expected_fused(n, grads, stale, params, momentum, wire, grad_avg, stats, 1)
        assert lib.daso_fused_sync_step(ctypes.byref(a), None) == want

    check()


def test_merge_and_local_avg_aliasing_rules_on_random_layouts(lib):
    """As above for daso_global_merge (params and wire overlap neither each other
    nor a copy) and daso_local_avg (out may be exactly one gradient buffer and
    overlaps no other)."""
    _no_gpu()
    hypothesis = pytest.importorskip("hypothesis")
    st = hypothesis.strategies

    @hypothesis.settings(max_examples=300, deadline=None, derandomize=True)
    @hypothesis.given(st.data())
    def check(data):
        n = data.draw(st.integers(1, 64)) * 4
        addr = st.integers(0, 40).map(lambda k: A + 128 * k)
        # merge
        P = data.draw(st.integers(0, 4))
        stale = [data.draw(addr) for _ in range(P)]
        params = data.draw(addr)
        wire = data.draw(st.one_of(st.none(), addr))
        want = L.DASO_EHIP
        if any(_spans_overlap(params, 4 * n, s_, 2 * n) for s_ in stale):
            want = L.DASO_EALIAS
        if wire and (_spans_overlap(wire, 2 * n, params, 4 * n)
                     or any(_spans_overlap(wire, 2 * n, s_, 2 * n) for s_ in stale)):
            want = L.DASO_EALIAS
        got = lib.daso_global_merge(params, ptrs(*stale), P, L.bucket_table([(0, n, 2)]), 1, wire, n, None)
        assert got == want
        # local average
        g = data.draw(st.integers(1, 4))
        grads = [data.draw(addr) for _ in range(g)]
        out = data.draw(st.one_of(addr, st.sampled_from(grads)))
        want = L.DASO_EHIP
        if any(gr != out and _spans_overlap(out, 4 * n, gr, 4 * n) for gr in grads):
            want = L.DASO_EALIAS
        assert lib.daso_local_avg(ptrs(*grads), g, out, n, None) == want

    check()


# ----------------------------------------------------------- bucket plan
def test_plan_buckets_matches_the_workload_recipes(lib):
    """The library's layout planner reproduces the bucket tables of every
    workload (whose counts are pinned in test_workloads.py)."""
    from workloads import recipes as R
    for w in R.all_workloads():
        if w.name == "tiny":
            continue  # a single explicit bucket, not planned
        got = L.plan_buckets(list(w.numels), R.BUCKET_CAP_ELEMS, w.S_cycle)
        assert got == [(b.start, b.numel, b.S) for b in w.buckets], w.name


def test_plan_buckets_random_and_edges(lib):
    import numpy as np
    from workloads import recipes as R
    rng = np.random.default_rng(5)
    for _ in range(200):
        nt = int(rng.integers(0, 40))
        numels = rng.integers(0, 1000, nt).tolist()
        cap = int(rng.integers(1, 3000))
        cyc = rng.integers(0, 9, int(rng.integers(1, 5))).tolist()
        want = [(s, k, cyc[b % len(cyc)]) for b, (s, k) in enumerate(R.plan_buckets(numels, cap))]
        assert L.plan_buckets(numels, cap, cyc) == want
    assert L.plan_buckets([], 10) == []
    assert L.plan_buckets([5, 3, 4, 10, 1], 8, (2,)) == [(12, 11, 2), (0, 12, 2)]
    f = lib.daso_plan_buckets
    i64 = (ctypes.c_int64 * 2)(4, -1)
    one = (ctypes.c_int32 * 1)(1)
    assert f(i64, 2, 10, one, 1, None, 0) == L.DASO_EINVAL
    assert f((ctypes.c_int64 * 1)(4), 1, 0, one, 1, None, 0) == L.DASO_EINVAL
    assert f((ctypes.c_int64 * 1)(4), 1, 10, (ctypes.c_int32 * 1)(-2), 1, None, 0) == L.DASO_EINVAL
    assert f((ctypes.c_int64 * 1)(4), 1, 10, one, 1, None, 1) == L.DASO_EINVAL


# ----------------------------------------------------------- launch shape
def _tiles_of(start, end, tile):
    return 0 if end <= start else (end - 1) // tile - start // tile + 1


def _shape_args(n, g, P, buckets, wire=True, stats=True, f32=False):
    """Fake, disjoint 2 GiB-spaced buffers (never dereferenced) for a fused call."""
    GB2 = 2 << 30
    a = L.daso_sync_args()
    keep = [ptrs(*[A + r * GB2 for r in range(g)]), ptrs(*[A + (g + i) * GB2 for i in range(P)]),
            L.bucket_table(buckets)]
    a.n, a.g, a.P = n, g, P
    a.grads = keep[0]
    if f32:
        a.stale_f32, a.flags = keep[1], L.DASO_EXCHANGE_F32
    else:
        a.stale = keep[1]
    a.params, a.momentum = A + (g + P) * GB2, A + (g + P + 1) * GB2
    w = A + (g + P + 2) * GB2 if wire else None
    if f32:
        a.wire_f32 = w
    else:
        a.wire = w
    a.stats = A + (g + P + 3) * GB2 if stats else None
    a.buckets, a.nbuckets = keep[2], len(buckets)
    a.lr, a.mu = 0.1, 0.9
    return a, keep


def _config(lib, a):
    c = L.daso_launch_config()
    rc = lib.daso_fused_launch_config(ctypes.byref(a), ctypes.byref(c))
    return rc, {f: getattr(c, f) for f, _ in L.daso_launch_config._fields_}


def test_fused_launch_config_follows_the_stated_rule(lib):
    """daso_fused_launch_config against the rule in daso.h, written out here:
    tiles of 2048 elements when a vector's inputs fit in 48 registers (4g + 2P
    + 8 for bf16 copies, 4g + 4P + 8 for fp32), else 1024; from 9 streams, runs
    of ntiles / 512 tiles rounded down to a power of two; from 10 streams, LDS
    that lets 2 workgroups share a 160 KB CU."""
    from workloads import recipes as R
    cap_lds = 160 * 1024 // 2 - 1024
    cases = []
    for name in ("resnet50", "gpt_medium", "segnet", "resnet18"):
        w = R.workload(name)
        cases.append((w.n, w.g, w.P, [(b.start, b.numel, b.S) for b in w.buckets], True, False))
    cases += [(25_557_032, 4, 0, [(0, 25_557_032, 1)], True, False),     # 9 streams
              (1_000_000, 1, 0, [(0, 1_000_000, 1)], False, False),     # 5 streams
              (25_557_032, 4, 8, [(0, 25_557_032, 2)], True, True)]     # fp32 exchange
    for n, g, P, bks, wire, f32 in cases:
        a, keep = _shape_args(n, g, P, bks, wire=wire, f32=f32)
        rc, c = _config(lib, a)
        assert rc == L.DASO_OK
        regs = 4 * g + (4 if f32 else 2) * P + 8
        tile = 2048 if regs <= 48 else 1024
        ntiles = sum(_tiles_of(s, s + k, tile) for (s, k, _) in bks[:64])
        streams = g + P + 4 + (1 if wire else 0)
        run = 1
        if streams >= 9:
            while run * 2 <= ntiles // 512:
                run *= 2
        want = {"tile_elems": tile, "ntiles": ntiles, "xcd_run_tiles": run,
                "lds_bytes": cap_lds if streams >= 10 else 0}
        assert c == want, (n, g, P, c, want)
    w = R.workload("resnet50")
    a, keep = _shape_args(w.n, w.g, w.P, [(b.start, b.numel, b.S) for b in w.buckets])
    assert _config(lib, a)[1]["xcd_run_tiles"] == 16 and _config(lib, a)[1]["tile_elems"] == 2048
    a.momentum = a.params + 64                      # rejected as the step rejects it
    assert _config(lib, a)[0] == L.DASO_EALIAS
    assert lib.daso_fused_launch_config(ctypes.byref(a), None) == L.DASO_EINVAL


def test_fused_launch_config_overrides(tmp_path):
    """DASO_FUSED_RUN_ELEMS and DASO_FUSED_WG_PER_CU replace the run length and
    the occupancy cap (read once per process, so in a child process)."""
    import json
    import subprocess
    import sys
    code = (
        "import ctypes, json, sys; sys.path.insert(0, %r); from tests import test_abi_host as T; "
        "from paper_2104_05588_amd import _lib as L; lib = L.load(); "
        "a, k = T._shape_args(25_557_032, 4, 8, [(0, 25_557_032, 4)]); print(json.dumps(T._config(lib, a)[1]))"
        % ROOT)
    for env, want in (({"DASO_FUSED_RUN_ELEMS": "0", "DASO_FUSED_WG_PER_CU": "0"}, (1, 0)),
                      ({"DASO_FUSED_RUN_ELEMS": "131072", "DASO_FUSED_WG_PER_CU": "3"}, (64, 160 * 1024 // 3 - 1024)),
                      ({"DASO_FUSED_RUN_ELEMS": "junk"}, (16, 160 * 1024 // 2 - 1024))):
        out = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, check=True,
                             env=dict(os.environ, **env), cwd=ROOT).stdout
        c = json.loads(out.strip().splitlines()[-1])
        assert (c["xcd_run_tiles"], c["lds_bytes"]) == want, (env, c)
