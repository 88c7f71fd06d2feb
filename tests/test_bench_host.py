"""Host logic of bench.py (CPU only): the algorithmic bytes it prices each
workload at, the placement of its timed window, the layout report and the
refusal of more than one GPU."""

from __future__ import annotations

import math
import os
import subprocess
import sys
import types

import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("name,step,norm", [("adam_n2_k2_p1m", 36, 0), ("adam_n3_k4_p16m", 44, 0),
                                            ("adopt_n2_k8_p124m_bf16", 30, 0), ("adam_n3_k4_p1311m", 44, 0),
                                            ("sgdm_n2_k16_p354m_clip", 28, 4)])
def test_algorithmic_bytes(name, step, norm):
    """Read and write of x, every u^j and v, one read of g (bf16 x and g at
    2 bytes), and one more read of g for the clip norm."""
    w = synth.WORKLOADS[name]
    assert bench.step_bytes_per_element(w) == step
    assert bench.norm_bytes_per_element(w) == norm


def _periods(w):
    return [h for h in (w.period_x, *w.period_u, w.period_v if w.has_v else 0) if h > 0]


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
@pytest.mark.parametrize("steps", [1, 2, 20, 256, 1000])
@pytest.mark.parametrize("warmup", [0, 5, 8])
def test_window_holds_the_all_states_event(name, steps, warmup):
    """The timed window s = start + warmup + 1 .. start + warmup + steps
    holds the first step at which every state is due together whenever the
    run is long enough to reach it, and starts at s >= 1."""
    w = synth.WORKLOADS[name]
    start = bench.window_start(w, steps, warmup)
    assert start >= 0
    lo, hi = start + warmup + 1, start + warmup + steps
    lcm = math.lcm(*_periods(w))
    if start > 0 or lcm <= hi:
        assert lo <= lcm <= hi, (start, lo, hi, lcm)
    # centred: the event sits in the middle of the window when the window can be placed freely
    if start > 0:
        assert abs((lcm - lo) - (hi - lcm)) <= 1


def test_layout_report_names_buffers():
    opt = types.SimpleNamespace(N=3, has_v=True, grad=object(), layout_order=[1, 0, 2, 3, 4, 5],
                                layout_report={"candidates": 24, "packed_ms": 2.0, "best_ms": 1.0, "worst_ms": 3.0,
                                               "order": [1, 0, 2, 3, 4, 5]})
    out = bench.layout_json(opt, "tuned")
    assert out["order"] == ["g", "x", "u1", "u2", "u3", "v"]
    assert out["candidates"] == 24 and out["best_ms"] == 1.0
    sgdm = types.SimpleNamespace(N=2, has_v=False, grad=None, layout_order=[0, 1, 2], layout_report=None)
    assert bench.layout_json(sgdm, "packed") == {"mode": "packed", "order": ["x", "u1", "u2"]}


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout.strip() == ""


def test_arena_carving_orders():
    """The optimizer's allocation (on the CPU here): every [K][P] buffer and
    the tail buffers are disjoint, 256-byte aligned, of the requested shape
    and type, laid out in the requested order, and returned in their own
    order whatever the layout."""
    import itertools

    import torch

    from paper_2510_05361_amd.optimizer import MtdaoOptimizer

    K, P = 3, 1001
    rows = [((K, P), torch.bfloat16), ((K, P), torch.bfloat16), ((K, P), torch.float32), ((K, P), torch.float32)]
    tail = [((P,), torch.float32)] * 2
    for order in itertools.permutations(range(len(rows))):
        opt = object.__new__(MtdaoOptimizer)
        opt._arena = None
        views = opt._carve(rows, tail, list(order), torch.device("cpu"))
        base = opt._arena.data_ptr()
        assert len(views) == len(rows) + len(tail)
        for v, (shape, dt) in zip(views, rows + tail):
            assert tuple(v.shape) == shape and v.dtype == dt and (v.data_ptr() - base) % 256 == 0
        spans = sorted((v.data_ptr(), v.data_ptr() + v.numel() * v.element_size()) for v in views)
        assert all(a[1] <= b[0] for a, b in zip(spans, spans[1:]))
        starts = [views[i].data_ptr() for i in order]
        assert starts == sorted(starts)
        assert min(v.data_ptr() for v in views[len(rows):]) > max(starts)
