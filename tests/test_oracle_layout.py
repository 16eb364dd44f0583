"""Pins of the oracle's layout planner to numbers the paper prints.

Each number comes from tests/golden/paper_layout_numbers.json, which cites
where the paper prints it.  Together they fix the reshape orientation
(n = first dimension), the inclusion of raw vectors in the factor buffers,
the bucket-closing rule and MB = MiB: changing any of them breaks at least one.
"""

import json
import os

import pytest

import synthgrad as sg
from oracle import layout as L

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_layout_numbers.json")))
MIB = 1 << 20


def _plan(params, r, cap=L.DEFAULT_CAP_BYTES):
    return L.plan([p.shape for p in params], r, cap)


def test_param_counts_table1():
    g = GOLD["params_millions"]
    assert round(sum(p.numel for p in sg.resnet50()) / 1e6, 1) == g["resnet50"]
    assert round(sum(p.numel for p in sg.resnet152()) / 1e6, 1) == g["resnet152"]
    assert round(sum(p.numel for p in sg.bert_base(full=True)) / 1e6, 1) == g["bert_base"]
    assert round(sum(p.numel for p in sg.bert_large(full=True)) / 1e6, 1) == g["bert_large"]
    # exact counts of the workload sets
    assert sum(p.numel for p in sg.resnet50()) == 25_557_032
    assert sum(p.numel for p in sg.resnet152()) == 60_192_808
    assert sum(p.numel for p in sg.bert_base()) == 108_890_112
    assert sum(p.numel for p in sg.bert_large()) == 334_090_240


def test_tensor_counts():
    for params, ntensors, nmat in [(sg.resnet50(), 161, 54), (sg.resnet152(), 467, 156),
                                   (sg.bert_base(), 196, 74), (sg.bert_large(), 388, 146)]:
        lay = _plan(params, 4)
        assert len(lay.tensors) == ntensors
        assert sum(t.compressed for t in lay.tensors) == nmat


def test_powersgd_ratio_table1():
    g = GOLD["powersgd_ratio"]
    got = {
        "resnet50_r4": L.powersgd_ratio(_plan(sg.resnet50(), 4)),
        "resnet152_r4": L.powersgd_ratio(_plan(sg.resnet152(), 4)),
        "bert_base_r32": L.powersgd_ratio(_plan(sg.bert_base(full=True), 32)),
        "bert_large_r32": L.powersgd_ratio(_plan(sg.bert_large(full=True), 32)),
    }
    for k, v in got.items():
        assert abs(v - g[k]) / g[k] <= 0.05, (k, v)


def test_resnet50_buckets():
    lay = _plan(sg.resnet50(), 4)
    assert round(lay.numel * 4 / MIB, 1) == GOLD["resnet50_gradient_mb"]["value"]
    assert len(lay.buckets) == GOLD["resnet50_buckets_25mb"]["value"]
    assert [round(b.grad_elems * 4 / MIB, 2) for b in lay.buckets] == [28.86, 25.04, 27.05, 16.55]
    # the alternative rule "never exceed the cap" would give 5 buckets
    sizes = [t.numel * 4 for t in lay.tensors]
    groups, cur, cb = [], [], 0
    for i in reversed(range(len(sizes))):
        if cur and cb + sizes[i] > L.DEFAULT_CAP_BYTES:
            groups.append(cur)
            cur, cb = [], 0
        cur.append(i)
        cb += sizes[i]
    groups.append(cur)
    assert len(groups) == 5


def test_resnet50_factor_sizes_and_rates():
    lay = _plan(sg.resnet50(), 4)
    p, q = L.factor_totals(lay)
    assert (p, q) == (164_360, 273_844)
    g = GOLD["resnet50_r4_factor_mb"]
    assert round(p * 4 / MIB, 2) == g["P"] and round(q * 4 / MIB, 2) == g["Q"]
    rp, rq = L.compression_rates(lay)
    g = GOLD["resnet50_r4_rate_percent"]
    assert round(rp * 100, 2) == g["P"] and round(rq * 100, 2) == g["Q"]
    g = GOLD["resnet50_r4_compressed_cap_mb"]
    assert round(25 * rp, 2) == g["P"] and round(25 * rq, 2) == g["Q"]
    gp, gq = L.compressed_fusion_groups(lay)
    g = GOLD["resnet50_r4_compressed_groups"]
    assert (len(gp), len(gq)) == (g["P"], g["Q"])


def test_reshape_orientation_and_vectors_matter():
    """Swapping n and m, or leaving the raw vectors out, contradicts the printed rates."""
    lay = _plan(sg.resnet50(), 4)
    n1 = sum(t.numel for t in lay.tensors if not t.compressed)
    sum_n = sum(t.n for t in lay.tensors if t.compressed)
    sum_m = sum(t.m for t in lay.tensors if t.compressed)
    N = lay.numel
    swapped = ((sum_m * 4 + n1) / N * 100, (sum_n * 4 + n1) / N * 100)
    no_vec = (sum_n * 4 / N * 100, sum_m * 4 / N * 100)
    g = GOLD["resnet50_r4_rate_percent"]
    assert (round(swapped[0], 2), round(swapped[1], 2)) != (g["P"], g["Q"])
    assert (round(no_vec[0], 2), round(no_vec[1], 2)) != (g["P"], g["Q"])


def test_bert_large_size_and_r256_ratio():
    lay = _plan(sg.bert_large(full=True), 256)
    assert round(lay.numel * 4 / MIB, 1) == GOLD["bert_large_mb"]["value"]
    assert round(L.acp_ratio(lay), 1) == GOLD["bert_large_r256_acp_ratio"]["value"]


def test_small_tensor_share_increase():
    lay = _plan(sg.resnet50(), 4)
    thr = GOLD["small_tensor_share_increase"]["threshold"]
    before = sum(t.numel < thr for t in lay.tensors) / len(lay.tensors)
    after_sizes = []
    for t in lay.tensors:
        if t.compressed:
            after_sizes += [t.n * 4, t.m * 4]
        else:
            after_sizes.append(t.numel)
    after = sum(s < thr for s in after_sizes) / len(after_sizes)
    assert abs((after - before) - GOLD["small_tensor_share_increase"]["value"]) < 0.05


@pytest.mark.parametrize("name,nb", [("conv256x576_r4", 1), ("resnet50_r4", 4), ("resnet152_r4", 9),
                                     ("bert_base_r4", 13), ("bert_large_r4", 37)])
def test_workload_bucket_counts(name, nb):
    wl = sg.WORKLOADS[name]
    lay = L.plan([p.shape for p in wl.params], wl.rank, wl.cap_bytes)
    assert len(lay.buckets) == nb
    # every tensor lands in exactly one bucket; offsets are packed
    seen = sorted(t for b in lay.buckets for t in b.tids)
    assert seen == list(range(len(wl.params)))
    for b in lay.buckets:
        off = 0
        for tid, go in zip(b.tids, b.grad_off):
            assert go == off
            off += lay.tensors[tid].numel
        assert off == b.grad_elems


def test_eligibility_rule():
    assert not L.plan_tensor(0, (64,), 4).compressed
    assert L.plan_tensor(0, (64, 3, 7, 7), 4).compressed
    t = L.plan_tensor(0, (64, 3, 7, 7), 4)
    assert (t.n, t.m) == (64, 147)
    assert not L.plan_tensor(0, (2, 768), 32).compressed    # r >= min(n, m)
    assert not L.plan_tensor(0, (4, 768), 4).compressed
    assert L.plan_tensor(0, (5, 768), 4).compressed
