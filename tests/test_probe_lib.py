"""The bench's access-pattern probe library (libdaso_ceiling.so, outside the C
ABI of include/daso.h): its host checks reject bad arguments before anything is
launched (no GPU needed), and on the GPU every probe writes exactly the
elements [0, n) of each output stream, with the values its loads imply, and
nothing past them, in every tile order and occupancy cap the bench uses."""
import ctypes
import os

import numpy as np
import pytest

from paper_2104_05588_amd import build as B

MB = 1 << 20
A = 0x10000000          # fake, 16-byte aligned "device" addresses, never dereferenced
VP, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64


@pytest.fixture(scope="module")
def plib():
    if not os.path.exists(B.PROBE_LIB):
        B.build_probes()
    lib = ctypes.CDLL(B.PROBE_LIB)
    lib.daso_probe_run.argtypes = [ctypes.POINTER(VP), I32, ctypes.POINTER(VP), I32, ctypes.POINTER(VP), I32,
                                   ctypes.POINTER(VP), I32, VP, I64, I32, I32, I32, VP]
    lib.daso_probe_run.restype = ctypes.c_int
    lib.daso_probe_phased.argtypes = [ctypes.POINTER(VP), I32, ctypes.POINTER(VP), I32, ctypes.POINTER(VP),
                                      ctypes.POINTER(VP), VP, VP, I64, I32, I32, I32, VP]
    lib.daso_probe_phased.restype = ctypes.c_int
    return lib


def _ptrs(k, base=A, step=16 * MB):
    arr = (VP * max(k, 1))()
    for i in range(k):
        arr[i] = base + i * step
    return arr


def _call(lib, r32=6, r16=8, w32=2, w16=1, n=4096, iters=2, run=1, lds=0, sink=A, rd32=None, rd16=None, wr32=None,
          wr16=None):
    rd32 = _ptrs(r32) if rd32 is None else rd32
    rd16 = _ptrs(r16, A + 1024 * MB) if rd16 is None else rd16
    wr32 = _ptrs(w32, A + 2048 * MB) if wr32 is None else wr32
    wr16 = _ptrs(w16, A + 3072 * MB) if wr16 is None else wr16
    return lib.daso_probe_run(rd32, r32, rd16, r16, wr32, w32, wr16, w16, sink, n, iters, run, lds, None)


def _no_gpu():
    import torch
    if torch.cuda.is_available():
        pytest.skip("argument-check tests use fake device addresses; run them without a GPU")


def test_probe_library_exports_its_entry(plib):
    assert hasattr(plib, "daso_probe_run")


@pytest.mark.parametrize("bad", [
    dict(n=0), dict(n=-8), dict(n=4098),                     # n not a positive multiple of 4
    dict(iters=3), dict(iters=-2),                           # no such form
    dict(iters=0, n=4100), dict(iters=-1, n=4100),           # 16-byte bf16 forms need n % 8 == 0
    dict(run=0), dict(lds=-1), dict(lds=160 * 1024 + 1),
    dict(sink=None),
    dict(r32=49), dict(w32=5), dict(r16=-1),
    dict(r32=5),                                             # a shape without an instance
    dict(iters=0, r16=4),                                    # the 16-byte forms exist for g=4, P=8 only
])
def test_probe_rejects_before_launch(plib, bad):
    _no_gpu()
    assert _call(plib, **bad) == -1


@pytest.mark.parametrize("which", ["rd32", "rd16", "wr32", "wr16"])
@pytest.mark.parametrize("how", ["null", "misaligned"])
def test_probe_rejects_bad_pointers(plib, which, how):
    _no_gpu()
    k = {"rd32": 6, "rd16": 8, "wr32": 2, "wr16": 1}[which]
    arr = _ptrs(k, A + 4096 * MB)
    arr[k - 1] = None if how == "null" else A + 4096 * MB + 8
    assert _call(plib, **{which: arr}) == -1


def _phased(lib, r32=6, r16=8, n=4096, iters=2, nwg=4, spin=1000, ctr=A + 8192 * MB, late=A + 8193 * MB,
            rd32=None, rd16=None, wr32=None, wr16=None):
    rd32 = _ptrs(r32) if rd32 is None else rd32
    rd16 = _ptrs(r16, A + 1024 * MB) if rd16 is None else rd16
    wr32 = _ptrs(2, A + 2048 * MB) if wr32 is None else wr32
    wr16 = _ptrs(1, A + 3072 * MB) if wr16 is None else wr16
    return lib.daso_probe_phased(rd32, r32, rd16, r16, wr32, wr16, ctr, late, n, iters, nwg, spin, None)


@pytest.mark.parametrize("bad", [
    dict(n=0), dict(n=4098), dict(nwg=0), dict(nwg=4097), dict(spin=0), dict(ctr=None), dict(late=None),
    dict(r32=5), dict(iters=1), dict(r32=10, r16=32, iters=2), dict(r16=16),
])
def test_phased_probe_rejects_before_launch(plib, bad):
    _no_gpu()
    assert _phased(plib, **bad) == -1


@pytest.mark.parametrize("which", ["rd32", "rd16", "wr32", "wr16"])
def test_phased_probe_rejects_misaligned_pointers(plib, which):
    _no_gpu()
    k = {"rd32": 6, "rd16": 8, "wr32": 2, "wr16": 1}[which]
    arr = _ptrs(k, A + 4096 * MB)
    arr[k - 1] = A + 4096 * MB + 8
    assert _phased(plib, **{which: arr}) == -1


# ------------------------------------------------------------------ GPU
GUARD = 4096
SENT32, SENT16 = np.uint32(0xA5C3E1F7), np.uint16(0xC3A5)


def _expect(form, r32, r16, w32, w16, X32, X16, n):
    """Expected u32 words of each fp32 output and u16 words of each bf16 output,
    from the probe's definition: a vector's value is a fixed pattern (its first
    element index, then small constants) XOR every fp32 stream's matching
    vector and (step layout) the bf16 vectors' words."""
    out32 = np.zeros(n, np.uint32)
    out16 = np.zeros(n // 2, np.uint32)          # bf16 output as u32 words
    X16w = [x.view(np.uint32) for x in X16]
    x32 = np.bitwise_xor.reduce(np.stack(X32), axis=0) if r32 else np.zeros(len(X32[0]) if X32 else n, np.uint32)
    x16 = np.bitwise_xor.reduce(np.stack(X16w), axis=0) if r16 else np.zeros(n // 2 + 4, np.uint32)
    if form in (1, 2):
        e0 = np.arange(0, n, 4, dtype=np.int64)
        v = np.stack([e0.astype(np.uint32), np.full_like(e0, 1, np.uint32), np.full_like(e0, 2, np.uint32),
                      np.full_like(e0, 3, np.uint32)], axis=1)
        v ^= x32[:n].reshape(-1, 4)
        v[:, 0] ^= x16[e0 // 2]
        v[:, 1] ^= x16[e0 // 2 + 1]
        out32[:] = v.ravel()
        out16[:] = v[:, :2].ravel()
        return out32, out16.view(np.uint16)
    tile = 2048
    ntiles = (n + tile - 1) // tile
    t = np.arange(ntiles, dtype=np.int64)[:, None]
    i = np.arange(256, dtype=np.int64)[None, :]
    e16 = (t * tile + 8 * i).ravel()
    if form == 0:
        ea, eb = e16, e16 + 4
    else:
        ea = (t * tile + 4 * i).ravel()
        eb = ea + 1024
    first = e16.astype(np.uint32)[:, None]
    v0 = np.concatenate([first, np.broadcast_to(np.array([1, 2, 3], np.uint32), (len(e16), 3))], axis=1)
    v1 = np.concatenate([first, np.broadcast_to(np.array([5, 6, 7], np.uint32), (len(e16), 3))], axis=1)
    xpad = np.concatenate([x32[:n], np.zeros(2048, np.uint32)])
    ina, inb, in16 = ea < n, eb < n, e16 < n
    v0[ina] ^= xpad[ea[ina, None] + np.arange(4)]
    v1[inb] ^= xpad[eb[inb, None] + np.arange(4)]
    v16 = v0 ^ v1
    v16[in16] ^= x16[e16[in16, None] // 2 + np.arange(4)]
    out32[ea[ina, None] + np.arange(4)] = (v0 ^ v16)[ina]
    out32[eb[inb, None] + np.arange(4)] = (v1 ^ v16)[inb]
    out16[e16[in16, None] // 2 + np.arange(4)] = v16[in16]
    return out32, out16.view(np.uint16)


CASES = [  # (r32, r16, w32, w16, form, n)
    (6, 8, 2, 1, 2, 4), (6, 8, 2, 1, 2, 2052), (6, 8, 2, 1, 2, 3 * 2048 + 4), (6, 8, 2, 1, 2, 65536 + 1028),
    (6, 16, 2, 1, 1, 1028), (6, 16, 2, 1, 1, 5 * 1024 + 12),
    (0, 0, 2, 1, 2, 3 * 2048 + 4), (1, 0, 1, 0, 2, 65536 + 12), (6, 8, 0, 0, 2, 2052),
    (6, 8, 2, 1, 0, 8), (6, 8, 2, 1, 0, 2056), (6, 8, 2, 1, 0, 65536 + 1032),
    (6, 8, 2, 1, -1, 8), (6, 8, 2, 1, -1, 1032), (6, 8, 2, 1, -1, 2056), (6, 8, 2, 1, -1, 65536 + 1032),
]


@pytest.mark.gpu
@pytest.mark.parametrize("run,lds", [(1, 0), (16, 80896)])
@pytest.mark.parametrize("case", CASES, ids=lambda c: "r%d_%d_w%d_%d_f%d_n%d" % c)
def test_probe_writes_exactly_its_elements(plib, case, run, lds):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r32, r16, w32, w16, form, n = case
    print(f"\n[case] probe {case} run={run} lds={lds}", flush=True)
    rng = np.random.default_rng(n * 7 + form + 3)
    X32 = [rng.integers(0, 2**32, n + GUARD, dtype=np.uint64).astype(np.uint32) for _ in range(r32)]
    X16 = [rng.integers(0, 2**16, n + GUARD, dtype=np.uint32).astype(np.uint16) for _ in range(r16)]
    d32 = [torch.from_numpy(x.view(np.int32)).cuda() for x in X32]
    d16 = [torch.from_numpy(x.view(np.int16)).cuda() for x in X16]
    o32 = [torch.full((n + GUARD,), int(SENT32.view(np.int32)), dtype=torch.int32, device="cuda") for _ in range(w32)]
    o16 = [torch.full((n + GUARD,), int(SENT16.view(np.int16)), dtype=torch.int16, device="cuda") for _ in range(w16)]
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")

    def arr(ts):
        a = (VP * max(len(ts), 1))()
        for k, t in enumerate(ts):
            a[k] = t.data_ptr()
        return a
    torch.cuda.synchronize()
    rc = plib.daso_probe_run(arr(d32), r32, arr(d16), r16, arr(o32), w32, arr(o16), w16, VP(sink.data_ptr()), n,
                             form, run, lds, VP(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert rc == 0
    want32, want16 = _expect(form, r32, r16, w32, w16, X32, X16, n)
    for o in o32:
        got = o.cpu().numpy().view(np.uint32)
        assert np.array_equal(got[:n], want32), f"fp32 output differs at {np.flatnonzero(got[:n] != want32)[:5]}"
        assert (got[n:] == SENT32).all(), "fp32 output written past n"
    for o in o16:
        got = o.cpu().numpy().view(np.uint16)
        assert np.array_equal(got[:n], want16), f"bf16 output differs at {np.flatnonzero(got[:n] != want16)[:5]}"
        assert (got[n:] == SENT16).all(), "bf16 output written past n"
    assert int(sink.abs().sum()) == 0           # the sink is written only on request, never here


PHASED_CASES = [  # (r32, r16, iters, n, workgroups): several rounds of staged tiles, ragged tails
    (6, 8, 2, 4, 1), (6, 8, 2, 2052, 3), (6, 8, 2, 30 * 2048 + 4, 3), (6, 8, 2, 61 * 2048 + 4, 2),
    (10, 32, 1, 4, 2), (10, 32, 1, 1028, 2), (10, 32, 1, 101 * 1024 + 4, 2),
]


@pytest.mark.gpu
@pytest.mark.parametrize("spin", [100_000, 1])
@pytest.mark.parametrize("case", PHASED_CASES, ids=lambda c: "r%d_%d_it%d_n%d_wg%d" % c)
def test_phased_probe_writes_exactly_its_elements(plib, case, spin):
    """The chip-wide phased probe writes the bare mix's values to exactly the
    elements [0, n) of the step's three output streams over several rounds;
    with a spin limit of one poll its waits give up early (each still ends)
    and the data is the same."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    r32, r16, iters, n, nwg = case
    print(f"\n[case] phased probe {case} spin={spin}", flush=True)
    rng = np.random.default_rng(n * 11 + iters)
    X32 = [rng.integers(0, 2**32, n + GUARD, dtype=np.uint64).astype(np.uint32) for _ in range(r32)]
    X16 = [rng.integers(0, 2**16, n + GUARD, dtype=np.uint32).astype(np.uint16) for _ in range(r16)]
    d32 = [torch.from_numpy(x.view(np.int32)).cuda() for x in X32]
    d16 = [torch.from_numpy(x.view(np.int16)).cuda() for x in X16]
    o32 = [torch.full((n + GUARD,), int(SENT32.view(np.int32)), dtype=torch.int32, device="cuda") for _ in range(2)]
    o16 = [torch.full((n + GUARD,), int(SENT16.view(np.int16)), dtype=torch.int16, device="cuda")]
    ctr = torch.zeros(4, dtype=torch.int32, device="cuda")
    late = torch.zeros(4, dtype=torch.int32, device="cuda")

    def arr(ts):
        a = (VP * max(len(ts), 1))()
        for k, t in enumerate(ts):
            a[k] = t.data_ptr()
        return a
    torch.cuda.synchronize()
    rc = plib.daso_probe_phased(arr(d32), r32, arr(d16), r16, arr(o32), arr(o16), VP(ctr.data_ptr()),
                                VP(late.data_ptr()), n, iters, nwg, spin, VP(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert rc == 0
    want32, want16 = _expect(iters, r32, r16, 2, 1, X32, X16, n)
    for o in o32:
        got = o.cpu().numpy().view(np.uint32)
        assert np.array_equal(got[:n], want32), f"fp32 output differs at {np.flatnonzero(got[:n] != want32)[:5]}"
        assert (got[n:] == SENT32).all(), "fp32 output written past n"
    got = o16[0].cpu().numpy().view(np.uint16)
    assert np.array_equal(got[:n], want16), f"bf16 output differs at {np.flatnonzero(got[:n] != want16)[:5]}"
    assert (got[n:] == SENT16).all(), "bf16 output written past n"
    tiles = (n + 1024 * iters - 1) // (1024 * iters)
    per_round = nwg * (72 * 1024 // (iters * 256 * 16))
    rounds = (tiles + per_round - 1) // per_round
    assert int(ctr[0]) == 2 * rounds * nwg        # every workgroup met twice per round
    if spin > 1:
        assert int(late[0]) == 0
