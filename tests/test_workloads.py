"""Workload recipes and seeded generators (host only, no GPU)."""
import numpy as np

from workloads import recipes as R
from workloads import generate as Gen


def test_published_parameter_counts():
    # torchvision's published totals for ResNet-18 and ResNet-50, GPT-2 medium's
    # embedding + 24-block shapes, and the segmentation recipe's stated size
    assert (len(R.resnet18_numels()), sum(R.resnet18_numels())) == (62, 11_689_512)
    assert (len(R.resnet50_numels()), sum(R.resnet50_numels())) == (161, 25_557_032)
    assert (len(R.segnet_numels()), sum(R.segnet_numels())) == (1800, 70_520_320)
    assert (len(R.gpt_medium_numels()), sum(R.gpt_medium_numels())) == (292, 354_823_168)


def test_every_tensor_is_a_multiple_of_8():
    for w in R.all_workloads():
        assert all(k % 8 == 0 for k in w.numels), w.name


def test_bucket_plans():
    ws = {w.name: w for w in R.all_workloads()}
    assert [len(ws[k].buckets) for k in ("tiny", "resnet18", "resnet50", "segnet", "gpt_medium")] == [1, 2, 4, 10, 37]
    assert [b.numel for b in ws["resnet18"].buckets] == [7_726_056, 3_963_456]
    per_S = {}
    for b in ws["gpt_medium"].buckets:
        per_S[b.S] = per_S.get(b.S, 0) + b.numel
    assert per_S == {1: 128_091_136, 2: 75_577_344, 4: 75_577_344, 8: 75_577_344}
    # the 51.5M-element token embedding is the first tensor and closes the last bucket
    assert ws["gpt_medium"].buckets[-1].start == 0
    assert ws["gpt_medium"].buckets[-1].numel >= 50257 * 1024


def test_buckets_tile_the_flat_buffer():
    for w in R.all_workloads():
        spans = sorted((b.start, b.numel) for b in w.buckets)
        pos = 0
        for s, k in spans:
            assert s == pos
            pos += k
        assert pos == w.n
        # bucket boundaries fall on tensor boundaries
        offs = set(R.tensor_offsets(w.numels)) | {w.n}
        assert all(b.start in offs for b in w.buckets)


def test_bucket_walk_closes_at_cap():
    numels = [5, 3, 4, 10, 1]
    # reverse walk: 1 + 10 = 11 >= 8 closes [12, 23); 4 + 3 = 7 < 8 stays open,
    # + 5 = 12 closes [0, 12)
    assert R.plan_buckets(numels, cap=8) == [(12, 11), (0, 12)]
    # a remainder below the cap forms the last bucket
    assert R.plan_buckets([2, 9, 1], cap=8) == [(2, 10), (0, 2)]


def test_algorithmic_bytes():
    assert R.algorithmic_bytes_per_param(4, 8) == 50
    assert R.algorithmic_bytes_per_param(8, 32) == 114


def test_host_generator_is_seeded_and_shaped():
    w = R.workload("tiny")
    a = Gen.host_inputs(w)
    b = Gen.host_inputs(w)
    assert np.array_equal(a["params"], b["params"])
    assert len(a["grads"]) == 4 and len(a["stale"]) == 2
    assert a["stale"][0].dtype == np.uint16
    assert abs(float(np.std(a["params"])) - 0.02) < 1e-3
    assert abs(float(np.std(a["grads"][1])) - 1e-3) < 5e-5
    assert not np.array_equal(a["grads"][0], a["grads"][1])
    # stale copies sit next to the parameters: within the bf16 step plus noise
    up = (a["stale"][1].astype(np.uint32) << 16).view(np.float32)
    assert np.max(np.abs(up - a["params"])) < 1e-3
    assert not np.any(a["momentum"])


def test_bucket_generation_matches_full_generation():
    w = R.workload("resnet18")
    full = Gen.host_inputs(w)
    bk = w.buckets[1]
    part = Gen.host_bucket_inputs(w, 1)
    sl = slice(bk.start, bk.start + bk.numel)
    assert np.array_equal(full["params"][sl], part["params"])
    assert np.array_equal(full["stale"][3][sl], part["stale"][3])
