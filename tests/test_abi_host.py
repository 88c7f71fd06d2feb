"""Host-side checks of the C ABI and the input generators (no GPU).

The library is loaded and every symbol the header declares must be
exported; validation, the sync schedule, the step counter and the error
paths are exercised through calls that never launch a kernel (a handle
over never-dereferenced addresses with init_states = 1, or numel = 0).
"""

import re

import numpy as np
import pytest
import torch

import oracle
import synth
from paper_2510_05361_amd import mtdao as abi
from synth.device import DeviceInputs

HEADER = __import__("os").path.join(__import__("os").path.dirname(__file__), "..", "include", "mtdao.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(mtdao_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) >= 9, names
    L = abi.lib()
    for n in names:
        assert hasattr(L, n), n


def test_header_enums_match_binding():
    text = open(HEADER).read()
    for name in ["MTDAO_OUTER_AVERAGE", "MTDAO_OUTER_NESTEROV", "MTDAO_SYNC_AFTER_STEP", "MTDAO_SYNC_MOMENTA_IN_STEP",
                 "MTDAO_ADAM", "MTDAO_ADOPT", "MTDAO_SGDM", "MTDAO_F32", "MTDAO_BF16", "MTDAO_OK",
                 "MTDAO_ERR_INVALID_ARG", "MTDAO_ERR_ALIGN", "MTDAO_ERR_HIP", "MTDAO_ERR_RANGE",
                 "MTDAO_ERR_WORKSPACE", "MTDAO_ADOPT_PREV", "MTDAO_ADOPT_CUR"]:
        m = re.search(rf"\b{name}\s*=\s*(-?\d+)", text)
        assert m and int(m.group(1)) == getattr(abi, name), name
    assert "0xFFFFFFFFu" in text and abi.MTDAO_SYNC_AUTO == 0xFFFFFFFF


def good_cfg(**kw):
    raw = {k[4:]: kw.pop(k) for k in list(kw) if k.startswith("raw_")}
    base = dict(form="adam", replicas=4, beta1=(0.9, 0.99), omega=(0.5, 0.3), numel=1024,
                period_x=4, period_u=(8, 8), period_v=16)
    base.update(kw)
    cfg = abi.make_config(**base)
    for k, v in raw.items():
        setattr(cfg, k, v)
    return cfg


BAD = [
    dict(form=3), dict(replicas=0), dict(replicas=abi.MTDAO_MAX_REPLICAS + 1),
    dict(beta1=(), omega=()), dict(beta1=(0.9,) * 5, omega=(0.1,) * 5),
    dict(beta1=(1.0, 0.99)), dict(beta1=(-0.1, 0.99)), dict(beta1=(float("nan"), 0.9)),
    dict(omega=(0.7, 0.4)), dict(omega=(-0.1, 0.3)), dict(omega=(1.5, 0.0)),
    dict(beta2=1.0), dict(beta2=-0.5), dict(eps=-1.0), dict(eps=float("inf")),
    dict(param_dtype=2), dict(grad_dtype=7), dict(adopt_order=2), dict(raw_bias_correction=3), dict(raw_n_tensors=-1),
    dict(period_x=-1), dict(period_u=(4, -2)), dict(period_v=-3), dict(start_step=-1),
    dict(numel=-5), dict(form="adopt", clip_rho=1.0), dict(clip_rho=float("nan")),
    dict(tensor_numel=[1000, 23]), dict(tensor_numel=[1024, -1, 1]),
    dict(numel=1 << 39, replicas=8), dict(sync_order=2), dict(sync_order=1), dict(form="adopt", sync_order=1),
    dict(outer_opt=2), dict(outer_opt=1, outer_lr=0.0), dict(outer_opt=1, outer_lr=float("inf")),
    dict(outer_opt=1, outer_momentum=1.0), dict(outer_opt=1, outer_momentum=-0.1),
    dict(form="sgdm", outer_opt=1, sync_order=1),
]


@pytest.mark.parametrize("kw", BAD, ids=[str(k) for k in BAD])
def test_invalid_config_rejected(kw):
    cfg = good_cfg(**kw)
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_workspace_bytes(cfg)
    assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
    assert abi.mtdao_last_error(None) != ""


def test_valid_edge_configs_accepted():
    for kw in [dict(omega=(0.5, 0.5)), dict(omega=(0.0, 0.0)), dict(beta1=(0.0, 0.0)),
               dict(replicas=1), dict(numel=0), dict(period_x=0, period_u=(0, 0), period_v=0),
               dict(form="sgdm", beta2=5.0, eps=-1.0, clip_rho=1.0), dict(tensor_numel=[1000, 0, 24]),
               dict(beta1=(0.9,) * 4, omega=(0.25,) * 4, period_u=(1, 2, 3, 4)),
               dict(omega=(0.5, 0.5000005))]:
        abi.mtdao_workspace_bytes(good_cfg(**kw))


def test_workspace_bytes():
    assert abi.mtdao_workspace_bytes(good_cfg()) == 0
    ws = abi.mtdao_workspace_bytes(good_cfg(form="sgdm", replicas=16, clip_rho=1.0))
    assert 16 * 4 <= ws <= 1 << 20
    assert abi.mtdao_workspace_bytes(good_cfg(form="adam", clip_rho=0.5)) > 0


def test_schedule_matches_oracle():
    """The library's schedule equals the oracle's for random configurations
    (host logic parity, bit for bit)."""
    rng = np.random.default_rng(3)
    for trial in range(200):
        form = ["adam", "adopt", "sgdm"][trial % 3]
        n = int(rng.integers(1, 5))
        hx, hv = int(rng.integers(0, 10)), int(rng.integers(0, 10))
        hu = [int(a) for a in rng.integers(0, 10, n)]
        cfg = abi.make_config(form, 3, (0.9,) * n, (0.1,) * n, 10, period_x=hx, period_u=hu,
                              period_v=hv)
        ocfg = oracle.OracleConfig(form=form, beta1=(0.9,) * n, omega=(0.1,) * n, period_x=hx,
                                   period_u=tuple(hu), period_v=hv)
        for s in range(1, 60):
            assert abi.mtdao_schedule(cfg, s) == oracle.schedule(ocfg, s), (trial, s)
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_schedule(good_cfg(), 0)
    assert e.value.code == abi.MTDAO_ERR_RANGE


def _fake_handle(cfg, base=1 << 40, stride=1 << 36):
    """Handle over addresses that are never dereferenced (init_states = 1
    makes mtdao_init enqueue nothing)."""
    n = cfg.n_moments
    u = [base + (1 + j) * stride for j in range(n)]
    v = base + (1 + n) * stride if cfg.form != abi.MTDAO_SGDM else None
    bufs = abi.make_buffers(base, u, v, True)
    ws = abi.mtdao_workspace_bytes(cfg)
    return abi.mtdao_init(cfg, bufs, (base + 8 * stride) if ws else None, ws, None)


def test_init_argument_errors():
    cfg = good_cfg()
    bufs = abi.make_buffers(1 << 40, [1 << 41], 1 << 42, True)  # u[1] missing
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(cfg, bufs, None, 0, None)
    assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
    bufs = abi.make_buffers((1 << 40) + 4, [1 << 41, 1 << 42], 1 << 43, True)
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(cfg, bufs, None, 0, None)
    assert e.value.code == abi.MTDAO_ERR_ALIGN
    bufs = abi.make_buffers(1 << 40, [(1 << 40) + 4096, 1 << 42], 1 << 43, True)  # overlaps x
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(cfg, bufs, None, 0, None)
    assert e.value.code == abi.MTDAO_ERR_INVALID_ARG and "overlap" in abi.mtdao_last_error(None)
    clip = good_cfg(form="sgdm", clip_rho=1.0)
    bufs = abi.make_buffers(1 << 40, [1 << 41, 1 << 42], None, True)
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(clip, bufs, None, 0, None)
    assert e.value.code == abi.MTDAO_ERR_WORKSPACE
    ws = abi.mtdao_workspace_bytes(clip)
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(clip, bufs, 1 << 44, ws - 8, None)
    assert e.value.code == abi.MTDAO_ERR_WORKSPACE


def test_handle_host_paths():
    cfg = good_cfg()
    h = _fake_handle(cfg)
    try:
        assert abi.mtdao_step_count(h) == 0
        # sync before any step: nothing due
        assert abi.mtdao_sync(h, abi.MTDAO_SYNC_AUTO, None) == 0
        assert abi.mtdao_sync(h, 0, None) == 0
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync(h, 1 << 4, None)  # Adam N=2 has states 0..3
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_local_step(h, None, 1e-3, 0.0, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_local_step(h, (1 << 45) + 2, 1e-3, 0.0, None)
        assert e.value.code == abi.MTDAO_ERR_ALIGN
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_local_step(h, (1 << 40) + 64, 1e-3, 0.0, None)  # overlaps x
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_local_step(h, 1 << 45, float("nan"), 0.0, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_step_sync(h, 1 << 45, 1e-3, 0.0, 1 << 4, None)  # bad mask
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_step_sync(h, (1 << 45) + 8, 1e-3, 0.0, 0, None)
        assert e.value.code == abi.MTDAO_ERR_ALIGN
        assert abi.mtdao_step_count(h) == 0, "a rejected call must not advance the step"
        dst = np.zeros(8, dtype=np.float32)
        for args, code in [((4, 0, 0, 8), abi.MTDAO_ERR_INVALID_ARG), ((-1, 0, 0, 8), abi.MTDAO_ERR_INVALID_ARG),
                           ((0, 4, 0, 8), abi.MTDAO_ERR_RANGE), ((1, 0, 1020, 8), abi.MTDAO_ERR_RANGE),
                           ((1, 0, -1, 2), abi.MTDAO_ERR_RANGE)]:
            with pytest.raises(abi.MtdaoError) as e:
                abi.mtdao_read_state(h, *args, dst, None)
            assert e.value.code == code, args
        abi.mtdao_read_state(h, 1, 0, 5, 0, dst, None)  # empty read is fine
    finally:
        abi.mtdao_destroy(h)
    abi.mtdao_destroy(None)
    assert abi.mtdao_step_count(None) == -1


def test_outer_nesterov_host_rules():
    cfg = good_cfg(outer_opt=abi.MTDAO_OUTER_NESTEROV, outer_lr=0.7, outer_momentum=0.9)
    abi.mtdao_workspace_bytes(cfg)
    bufs = abi.make_buffers(1 << 40, [1 << 41, 1 << 42], 1 << 43, True)  # outer buffers missing
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(cfg, bufs, None, 0, None)
    assert e.value.code == abi.MTDAO_ERR_INVALID_ARG and "x_outer" in abi.mtdao_last_error(None)
    bufs = abi.make_buffers(1 << 40, [1 << 41, 1 << 42], 1 << 43, True, 1 << 44, (1 << 44) + 64)
    with pytest.raises(abi.MtdaoError) as e:  # outer buffers overlap each other
        abi.mtdao_init(cfg, bufs, None, 0, None)
    assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
    bufs = abi.make_buffers(1 << 40, [1 << 41, 1 << 42], 1 << 43, True, 1 << 44, (1 << 44) + 8)
    with pytest.raises(abi.MtdaoError) as e:
        abi.mtdao_init(cfg, bufs, None, 0, None)
    bufs = abi.make_buffers(1 << 40, [1 << 41, 1 << 42], 1 << 43, True, 1 << 44, 1 << 45)
    h = abi.mtdao_init(cfg, bufs, None, 0, None)
    try:
        dst = np.zeros(4, dtype=np.float32)
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_read_state(h, abi.MTDAO_STATE_X_OUTER, 1, 0, 4, dst, None)
        assert e.value.code == abi.MTDAO_ERR_RANGE
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_local_step(h, (1 << 44) + 128, 1e-3, 0.0, None)  # overlaps x_outer
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
    finally:
        abi.mtdao_destroy(h)
    h = _fake_handle(good_cfg())
    try:
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_read_state(h, abi.MTDAO_STATE_X_OUTER, 0, 0, 4, np.zeros(4, np.float32), None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
    finally:
        abi.mtdao_destroy(h)


def test_averaged_momenta_order_host_rules():
    """Algorithm 4's order: moment averaging only inside mtdao_step_sync."""
    cfg = good_cfg(form="sgdm", sync_order=abi.MTDAO_SYNC_MOMENTA_IN_STEP)
    h = _fake_handle(cfg)
    try:
        for mask in (0b010, 0b100, 0b111):
            with pytest.raises(abi.MtdaoError) as e:
                abi.mtdao_sync(h, mask, None)
            assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
            assert "inside mtdao_step_sync" in abi.mtdao_last_error(h)
    finally:
        abi.mtdao_destroy(h)
    # numel = 0: the x bit passes validation and launches nothing
    cfg0 = abi.make_config("sgdm", 3, (0.0, 0.9), (0.3, 0.7), 0, period_x=2, period_u=(4, 4),
                           sync_order=abi.MTDAO_SYNC_MOMENTA_IN_STEP)
    h = abi.mtdao_init(cfg0, abi.make_buffers(None, [None] * 2, None, False), None, 0, None)
    try:
        assert abi.mtdao_sync(h, 0b001, None) == 0b001
        assert abi.mtdao_step_sync(h, None, 1e-3, 0.0, 0b111, None) == 0b111
    finally:
        abi.mtdao_destroy(h)


def test_empty_problem_counts_steps_and_reports_masks():
    """numel = 0 launches nothing; the step counter and the applied masks
    still follow the schedule (and the oracle's)."""
    for form in ("adam", "adopt", "sgdm"):
        cfg = abi.make_config(form, 3, (0.9, 0.99, 0.5), (0.2, 0.2, 0.2), 0, period_x=3,
                              period_u=(2, 5, 0), period_v=4, start_step=7)
        ocfg = oracle.OracleConfig(form=form, beta1=(0.9, 0.99, 0.5), omega=(0.2,) * 3, period_x=3,
                                   period_u=(2, 5, 0), period_v=4)
        bufs = abi.make_buffers(None, [None] * 3, None, False)
        h = abi.mtdao_init(cfg, bufs, None, 0, None)
        try:
            for k in range(1, 30):
                abi.mtdao_local_step(h, None, 1e-3, 0.0, None)
                assert abi.mtdao_step_count(h) == 7 + k
                assert abi.mtdao_sync(h, abi.MTDAO_SYNC_AUTO, None) == oracle.schedule(ocfg, 7 + k)
            for k in range(30, 50):
                got = abi.mtdao_step_sync(h, None, 1e-3, 0.0, abi.MTDAO_SYNC_AUTO, None)
                assert abi.mtdao_step_count(h) == 7 + k
                assert got == oracle.schedule(ocfg, 7 + k)
            assert abi.mtdao_step_sync(h, None, 1e-3, 0.0, 0b101, None) == 0b101
        finally:
            abi.mtdao_destroy(h)


# ------------------------------------------------------------ input generators


def test_device_generator_matches_host_generator():
    """synth.device (torch) and synth.workloads (numpy) draw bit-identical
    gradients and x_0 (run here with torch on the CPU)."""
    for w in [synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 40_000, tail=37),
              synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 20_000, tail=3),
              synth.WORKLOADS["adam_n2_k2_p1m"]]:
        dev = DeviceInputs(w, torch.device("cpu"))
        tdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
        g = torch.empty((w.replicas, w.numel), dtype=tdt)
        for s in (1, 2, 17):
            dev.grads_into(s, g)
            host = synth.host_grad_rows(w, s)
            gd = g.view(torch.int16).numpy().view(np.uint16) if tdt == torch.bfloat16 else g.numpy()
            assert np.array_equal(gd, host), (w.name, s)
        x0 = dev.x0_row()
        hx = synth.host_x0_row(w)
        xd = x0.view(torch.int16).numpy().view(np.uint16) if w.param_dtype == "bf16" else x0.numpy()
        assert np.array_equal(xd, hx), w.name
        for stream, scale, absolute in [(11, 0.02, False), (15, 1e-6, True)]:
            t = torch.empty((w.replicas, w.numel), dtype=torch.float32)
            dev.pool_rows_into(stream, scale, t, absolute=absolute)
            assert np.array_equal(t.numpy(), synth.host_pool_rows(w, stream, scale, np.arange(w.numel),
                                                                  absolute=absolute))
        idx = synth.sample_indices(w, 500)
        assert np.array_equal(synth.host_grad_rows(w, 5, idx), synth.host_grad_rows(w, 5)[:, idx])


def test_workload_sizes():
    """Tensor lists of the five workloads have the element counts of the
    GPT shapes they stand for."""
    want = {"adam_n2_k2_p1m": 1_048_576, "adam_n3_k4_p16m": 16_785_920,
            "adopt_n2_k8_p124m_bf16": 123_605_760, "adam_n3_k4_p1311m": 1_311_180_800,
            "sgdm_n2_k16_p354m_clip": 353_600_512}
    for name, P in want.items():
        assert synth.WORKLOADS[name].numel == P
        assert P % 64 == 0


def test_bf16_input_conversion():
    a = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -2.5, 3.4e38, np.nan], dtype=np.float32)
    b = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(a))
    t = torch.from_numpy(a).to(torch.bfloat16).float().numpy()
    assert np.array_equal(b[:5], t[:5]) and np.isnan(b[5])


def test_binding_struct_layout_matches_header(tmp_path):
    """Every field of mtdao_config, mtdao_buffers and mtdao_device_step sits at the same offset
    with the same size in the ctypes binding as in the C header (a stale
    mirror would hand the library garbage pointers)."""
    import ctypes
    import os
    import subprocess

    structs = {"mtdao_config": abi.MtdaoConfig, "mtdao_buffers": abi.MtdaoBuffers,
               "mtdao_device_step": abi.MtdaoDeviceStep}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "mtdao.h"', "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'  printf("{cname} sizeof %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu %zu\\n", offsetof({cname}, {fname}), '
                         f'sizeof((({cname}*)0)->{fname}));')
    lines.append("  return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(HEADER))
    subprocess.run(["gcc", "-std=c11", "-I", inc, "-o", str(exe), str(src)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    seen = 0
    for line in out:
        if not line:
            continue
        parts = line.split()
        py = structs[parts[0]]
        if parts[1] == "sizeof":
            assert int(parts[2]) == ctypes.sizeof(py), line
        else:
            fld = getattr(py, parts[1])
            assert (fld.offset, fld.size) == (int(parts[2]), int(parts[3])), line
            seen += 1
    assert seen == sum(len(p._fields_) for p in structs.values())


def test_sync_stats_host_rules():
    cfg = good_cfg()
    n = abi.mtdao_stats_scratch_bytes(cfg)
    assert 0 < n < 64 << 20
    h = _fake_handle(cfg)
    try:
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync_stats(h, 1, None, 0, None)
        assert e.value.code == abi.MTDAO_ERR_WORKSPACE
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync_stats(h, 1, (1 << 44) + 64, n, None)
        assert e.value.code == abi.MTDAO_ERR_ALIGN
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync_stats(h, 1 << 4, 1 << 44, n, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        applied, st = abi.mtdao_sync_stats(h, 0, 1 << 44, n, None)  # nothing due: no launch
        assert applied == 0 and np.all(np.isnan(st))
    finally:
        abi.mtdao_destroy(h)
    # the static-scratch variant rejects what its fixed array cannot hold, before anything else
    huge = good_cfg(numel=1 << 30)
    assert abi.mtdao_stats_scratch_bytes(huge) > abi.MTDAO_STATIC_SCRATCH_BYTES
    h = _fake_handle(huge)
    try:
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync_stats_static(h, 1, None)
        assert e.value.code == abi.MTDAO_ERR_WORKSPACE and "static scratch" in abi.mtdao_last_error(h)
    finally:
        abi.mtdao_destroy(h)
    big = good_cfg(replicas=17)
    h = _fake_handle(big)
    try:
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync_stats(h, 1, 1 << 44, abi.mtdao_stats_scratch_bytes(big), None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG and "16" in abi.mtdao_last_error(h)
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_sync_stats_static(h, 1, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
    finally:
        abi.mtdao_destroy(h)


def test_device_step_host_rules():
    """mtdao_step_sync_device and mtdao_device_step_set reject bad arguments
    before anything is enqueued (the step count does not move), and ADOPT's
    first update (v only) must go through the host-scalar calls."""
    cfg = good_cfg()
    h = _fake_handle(cfg)
    g = (1 << 44) + (1 << 40)
    try:
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_device_step_set(h, None, 0, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_device_step_set(h, (1 << 44) + 8, 0, None)
        assert e.value.code == abi.MTDAO_ERR_ALIGN
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_device_step_set(h, 1 << 44, -1, None)
        assert e.value.code == abi.MTDAO_ERR_RANGE
        for d, lr, n, code in [(None, 1 << 45, 4, abi.MTDAO_ERR_INVALID_ARG), (1 << 44, None, 4, abi.MTDAO_ERR_INVALID_ARG),
                               ((1 << 44) + 4, 1 << 45, 4, abi.MTDAO_ERR_ALIGN), (1 << 44, 1 << 45, 0, abi.MTDAO_ERR_RANGE)]:
            with pytest.raises(abi.MtdaoError) as e:
                abi.mtdao_step_sync_device(h, g, d, lr, None, n, abi.MTDAO_SYNC_AUTO, None)
            assert e.value.code == code
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_step_sync_device(h, g, 1 << 44, 1 << 45, None, 4, 1 << 5, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG
        assert abi.mtdao_step_count(h) == 0
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_device_step_advance(h, (1 << 44) + 8, None)
        assert e.value.code == abi.MTDAO_ERR_ALIGN
        abi.mtdao_device_step_advance(h, 1 << 44, None)  # no calls since the last set: nothing enqueued
    finally:
        abi.mtdao_destroy(h)
    adopt = good_cfg(form="adopt", beta2=0.9999)
    h = _fake_handle(adopt)
    try:
        with pytest.raises(abi.MtdaoError) as e:
            abi.mtdao_step_sync_device(h, g, 1 << 44, 1 << 45, None, 4, abi.MTDAO_SYNC_AUTO, None)
        assert e.value.code == abi.MTDAO_ERR_INVALID_ARG and "first update" in abi.mtdao_last_error(h)
        assert abi.mtdao_step_count(h) == 0
    finally:
        abi.mtdao_destroy(h)
