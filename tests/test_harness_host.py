"""The parity harness itself, on the CPU: the oracle run over disjoint
column parts on threads equals the plain sequential run bit for bit, and
the comparison catches an error just over each tolerance.  (The GPU tests
rely on both.)"""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_harness import BF16_MAX_ULPS, OracleResult, bf16_bounds, compare, run_oracle, run_oracle_parallel


def _small(name, **kw):
    w = synth.small_variant(synth.WORKLOADS[name], 6_000, tail=13)
    return w.replace(steps=min(w.steps, 20), period_x=3, period_u=(4,) * w.n_moments, period_v=5, **kw)


def _assert_parts_equal(seq: OracleResult, par: OracleResult, P: int):
    for c, st in par.column_parts():
        cols = np.arange(P)[c] if isinstance(c, slice) else np.searchsorted(seq.idx, c) if seq.idx is not None else c
        for a, b in zip(st.arrays(), seq.state.arrays()):
            assert np.array_equal(a, b[:, cols])
        if st.x_outer is not None:
            assert np.array_equal(st.x_outer, seq.state.x_outer[cols])
            assert np.array_equal(st.outer_mom, seq.state.outer_mom[cols])


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_parallel_oracle_equals_sequential(name):
    w = _small(name)
    steps = list(range(1, w.steps + 1))
    seq = run_oracle(w, steps)
    par = run_oracle_parallel(w, steps, threads=3)
    assert par.masks == seq.masks and any(par.masks)
    assert len(par.column_parts()) == 3
    _assert_parts_equal(seq, par, w.numel)


def test_parallel_oracle_on_a_sample_and_with_nesterov():
    w = _small("adam_n3_k4_p16m")
    steps = list(range(1, w.steps + 1))
    idx = synth.sample_indices(w, n_stride=1000, edge=8)
    seq = run_oracle(w, steps, idx, outer=(0.7, 0.9))
    par = run_oracle_parallel(w, steps, idx, outer=(0.7, 0.9), threads=4)
    assert par.masks == seq.masks
    _assert_parts_equal(seq, par, w.numel)


class _FakeOpt:
    """The compared interface of MtdaoOptimizer over host tensors."""

    def __init__(self, w, st: oracle.OracleState, mu: float = 0.0):
        def t(a):
            a = np.ascontiguousarray(a)
            if a.dtype == np.uint16:
                return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16)
            return torch.from_numpy(a.copy())

        self._s = [t(a) for a in st.arrays()]
        self.x_outer = None if st.x_outer is None else t(st.x_outer)
        self.x_outer_mom = None if st.outer_mom is None else t(st.outer_mom)
        self.cfg = type("C", (), {"outer_momentum": mu})()

    def states(self):
        return self._s


@pytest.mark.parametrize("name", ["adam_n3_k4_p16m", "adopt_n2_k8_p124m_bf16"])
def test_compare_catches_errors_over_the_tolerance(name):
    w = _small(name)
    steps = list(range(1, w.steps + 1))
    o = run_oracle_parallel(w, steps, threads=2)
    full = run_oracle(w, steps)
    report = compare(w, _FakeOpt(w, full.state), o, "self")
    for k, m in report.items():
        assert m.get("rel_err", 0.0) == 0.0 and m.get("max_ulps", 0.0) == 0.0, (k, m)
    # one element of u^1 off by 2e-5 of the floor
    bad = full.state.copy()
    i = int(np.argmax(np.abs(bad.u[0][1])))
    bad.u[0][1, i] = np.float32(bad.u[0][1, i] * (1 + 2e-5))
    with pytest.raises(AssertionError):
        compare(w, _FakeOpt(w, bad), o, "planted-u")
    if w.param_dtype == "bf16":
        # elements whose largest magnitude lies in their final binade, above
        # the rms floor: an offset of k ulps there is k units
        xf = np.abs(synth.bf16_bits_to_f32(full.state.x)).astype(np.float64).reshape(-1)
        top = full.x_absmax[0].astype(np.float64).reshape(-1)
        rms = float(np.sqrt(np.mean(xf * xf)))
        ok = np.flatnonzero((np.floor(np.log2(np.maximum(xf, 1e-30))) == np.floor(np.log2(np.maximum(top, 1e-30))))
                            & (xf > 2 * rms) & ((full.state.x.reshape(-1) & 0x7F) < 0x70))
        bad = full.state.copy()
        bad.x.reshape(-1)[ok[0]] += np.uint16(BF16_MAX_ULPS + 1)
        with pytest.raises(AssertionError):
            compare(w, _FakeOpt(w, bad), o, "planted-x")
        # one-ulp offsets on more elements than the flip rate allows
        bad = full.state.copy()
        n_bad = int(bf16_bounds(bad.x.size, len(o.masks))[0]) + 1
        assert ok.size >= n_bad
        bad.x.reshape(-1)[ok[:n_bad]] += np.uint16(1)
        with pytest.raises(AssertionError):
            compare(w, _FakeOpt(w, bad), o, "planted-flips")


def test_sample_covers_index_boundaries():
    w = synth.WORKLOADS["adam_n3_k4_p1311m"]
    idx = synth.sample_indices(w)
    mask = synth.strided_mask(w, idx)
    assert mask.sum() == 1 << 20 and idx.size >= (1 << 20)
    P = w.numel
    for flat in (1 << 31, 1 << 32):
        m, c = divmod(flat, P)
        assert c in set(idx.tolist()) and c - 1 in set(idx.tolist()), flat
    offs = w.tensor_offsets()
    assert set(offs[:-1].tolist()) <= set(idx.tolist()) and set((offs[1:] - 1).tolist()) <= set(idx.tolist())
