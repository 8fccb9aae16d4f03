"""Host-side checks of the C-ABI library (no GPU): it loads, exports every symbol
include/wdc.h declares, and its host logic (weight layout, parameter defaults,
sizes) agrees with the inputs and readings the oracle uses."""
import ctypes as C
import os
import re
from dataclasses import asdict

import pytest

import synth
from oracle import params as oparams

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    src = open(os.path.join(ROOT, "include", "wdc.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(wdc_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def wdc():
    import paper_2608_01845_amd as pkg
    pkg.load()
    return pkg


def test_library_exports_every_declared_symbol(wdc):
    lib = wdc.load()
    declared = header_functions()
    assert len(declared) >= 20
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(wdc.exported_symbols()) == declared


def make_ctx(wdc, cfg, params=None):
    lib = wdc.load()
    d = wdc.desc_from_config(cfg)
    p = params or wdc.default_params()
    h = C.c_void_p()
    assert lib.wdc_create(C.byref(d), C.byref(p), None, C.byref(h)) == 0, lib.wdc_last_error(None)
    return lib, h


@pytest.mark.parametrize("name", ["tiny", "mid", "5b", "13b", "stress"])
def test_weight_layout_matches_parameter_inventory(wdc, name):
    cfg = synth.get_config(name)
    lib, h = make_ctx(wdc, cfg)
    try:
        specs = synth.weight_specs(cfg)
        assert lib.wdc_weight_count(h) == len(specs)
        prev_end = 0
        esz = 2 if cfg.dtype == "bf16" else 4
        for i, (nm, shp) in enumerate(specs):
            name_p = C.c_char_p()
            shape = (C.c_int64 * 2)()
            nd = C.c_int32()
            off = C.c_size_t()
            assert lib.wdc_weight_info(h, i, C.byref(name_p), shape, C.byref(nd), C.byref(off)) == 0
            assert name_p.value.decode() == nm
            assert nd.value == len(shp)
            assert tuple(shape[: nd.value]) == tuple(shp)
            assert off.value % 256 == 0 and off.value >= prev_end
            n = 1
            for s in shp:
                n *= s
            prev_end = off.value + n * esz
        assert lib.wdc_weights_bytes(h) >= prev_end
    finally:
        lib.wdc_destroy(h)


def test_param_defaults_match_oracle_readings(wdc):
    p = wdc.default_params()
    o = asdict(oparams.DEFAULTS)
    mapping = {"bank_capacity": "bank_capacity", "age_max": "age_max", "n_min": "n_min", "k_init": "k_init",
               "k_ref": "k_ref", "theta_sim": "theta_sim", "theta_q": "theta_q", "tau_in": "tau_in",
               "tau_obs": "tau_obs", "gamma_q": "gamma_q", "alpha_min": "alpha_min", "alpha_max": "alpha_max",
               "eps": "eps", "eps_nu": "eps_nu", "w_z": "w_z", "w_age": "w_age", "w_phase": "w_phase",
               "w_cam": "w_cam", "w_depth": "w_depth", "eta0": "eta0", "beta_d": "beta_d", "eta_min": "eta_min",
               "eta_max": "eta_max", "a_cam": "a_cam", "a_depth": "a_depth", "a_phase": "a_phase", "lam": "lam",
               "r0": "r0", "tau_risk": "tau_risk"}
    for c_name, o_name in mapping.items():
        assert getattr(p, c_name) == o[o_name], c_name
    # ablation variants: the defaults are the full method
    assert p.period == o["period"]
    assert (p.surrogate, o["surrogate"]) == (wdc.SURROGATE_LIFTED, "lifted")
    assert (p.observation, o["observation"]) == (wdc.OBS_KERNEL, "kernel")
    for name in ("lift_condition", "impact_weight", "calibrate", "support_constraint"):
        assert p.__getattribute__(name) == int(o[name]) == 1, name


def test_params_struct_mirrors_oracle_fields(wdc):
    """Every oracle parameter has a field of the same name in wdc_params."""
    from dataclasses import fields
    names = {f[0] for f in wdc.Params._fields_}
    for f in fields(oparams.Params):
        assert f.name in names, f.name
    src = open(os.path.join(ROOT, "include", "wdc.h")).read()
    body = src[src.index("typedef struct {\n  int32_t bank_capacity;"):src.index("} wdc_params;")]
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    declared = re.findall(r"\b([a-z_0-9]+)\s*[,;]", body)
    assert declared == [f[0] for f in wdc.Params._fields_]


def test_create_rejects_bad_variant_params(wdc):
    cfg = synth.get_config("tiny")
    for bad in (dict(period=0), dict(surrogate=2), dict(observation=-1)):
        lib = wdc.load()
        d = wdc.desc_from_config(cfg)
        p = wdc.default_params(**bad)
        h = C.c_void_p()
        assert lib.wdc_create(C.byref(d), C.byref(p), None, C.byref(h)) == 1, bad


def test_create_rejects_bad_descriptors(wdc):
    lib = wdc.load()
    bad = [
        synth.get_config("tiny", head_dim=32, heads=8),            # unsupported head size
        synth.get_config("tiny", latent=(8, 4, 16, 16)),            # summary needs 16 channels
        synth.get_config("tiny", latent=(16, 4, 15, 16)),           # not divisible by the patch
        synth.get_config("tiny", rope=(16, 24, 22)),                # rotary dims do not sum to head_dim
        synth.get_config("tiny", n_dual=1),                         # dual-stream blocks without text
        # bf16, 4,200,000 tokens at head size 128: one head's q would pass 2^30 bytes
        synth.get_config("tiny", dtype="bf16", heads=2, head_dim=128, rope=(16, 56, 56), latent=(16, 100, 300, 560)),
    ]
    for cfg in bad:
        d = wdc.desc_from_config(cfg)
        p = wdc.default_params()
        h = C.c_void_p()
        st = lib.wdc_create(C.byref(d), C.byref(p), None, C.byref(h))
        assert st != 0
        assert lib.wdc_last_error(None)
    # under the limit (4,110,000 tokens), and float32 past it, are accepted
    for cfg in (synth.get_config("tiny", dtype="bf16", heads=2, head_dim=128, rope=(16, 56, 56),
                                 latent=(16, 100, 300, 548)),
                synth.get_config("tiny", heads=2, head_dim=128, rope=(16, 56, 56), latent=(16, 100, 300, 560))):
        d = wdc.desc_from_config(cfg)
        assert lib.wdc_create(C.byref(d), C.byref(wdc.default_params()), None, C.byref(h)) == 0, \
            lib.wdc_last_error(None)
        lib.wdc_destroy(h)
    p = wdc.default_params(bank_capacity=9)
    d = wdc.desc_from_config(synth.get_config("tiny"))
    h = C.c_void_p()
    assert lib.wdc_create(C.byref(d), C.byref(p), None, C.byref(h)) == 1


def test_unbound_context_errors(wdc):
    cfg = synth.get_config("tiny")
    lib, h = make_ctx(wdc, cfg)
    try:
        log = wdc.StepLog()
        # no workspace / weights: compute calls fail with a status, not a crash
        assert lib.wdc_dit_forward(h, C.c_void_p(16), 1.0, None, None, None, C.c_void_p(16)) == 5
        assert b"workspace" in lib.wdc_last_error(h)
        assert lib.wdc_dit_block_forward(h, 7, C.c_void_p(16), C.c_void_p(16)) == 1
        assert lib.wdc_surrogate_step(h, None, C.c_void_p(16), 0, 8, C.c_void_p(16), C.byref(log)) == 1
        assert lib.wdc_bind_workspace(h, C.c_void_p(8), 1 << 40) == 4     # misaligned
        assert lib.wdc_bind_workspace(h, C.c_void_p(16), 16) == 5         # too small
    finally:
        lib.wdc_destroy(h)


def test_state_and_workspace_sizes(wdc):
    cfg = synth.get_config("13b")
    lib, h = make_ctx(wdc, cfg)
    try:
        E = cfg.numel
        assert lib.wdc_state_bytes(h) >= (2 + 4) * E * 4
        n = cfg.n_tokens
        assert lib.wdc_workspace_bytes(h) >= n * cfg.hidden * 4 + n * (cfg.hidden + 4 * cfg.hidden) * 2
        assert lib.wdc_attn_pad(67576) % 256 == 0 and lib.wdc_attn_pad(67576) >= 67576
    finally:
        lib.wdc_destroy(h)


def test_timing_classes_match_header(wdc):
    src = open(os.path.join(ROOT, "include", "wdc.h")).read()
    consts = {m.group(1).lower(): int(m.group(2)) for m in re.finditer(r"WDC_T_([A-Z_]+)\s*=\s*(\d+)", src)}
    count = consts.pop("count")
    from paper_2608_01845_amd import _binding
    assert len(_binding.TIMING_CLASSES) == count
    for name, idx in consts.items():
        assert _binding.TIMING_CLASSES[idx] == name
