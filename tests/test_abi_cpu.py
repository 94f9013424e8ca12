"""The C ABI without a GPU: the library loads, exports every function the
header declares, its structs match the binding's layout, and argument
validation that happens before any device call reports errors."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2606_20543_amd as ssd
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssd.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ssd.LIB_PATH):
        from paper_2606_20543_amd import _build
        _build.build()
    return ssd.lib()


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ssd_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_exported(lib):
    names = _declared()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(ssd.EXPORTED) == names


def test_struct_layouts_match_header(tmp_path):
    src = tmp_path / "layout.c"
    src.write_text(f"""
#include <stdio.h>
#include <stddef.h>
#include "{HEADER}"
int main(void) {{
  printf("%zu %zu %zu %zu\\n", sizeof(ssd_model_config), sizeof(ssd_verify_params), sizeof(ssd_schedule), sizeof(ssd_stats));
  printf("%zu %zu %zu %zu\\n", offsetof(ssd_verify_params, temperature), offsetof(ssd_verify_params, seed),
         offsetof(ssd_verify_params, round), offsetof(ssd_schedule, temperature));
  printf("%zu %zu %zu %zu\\n", offsetof(ssd_schedule, seed), offsetof(ssd_model_config, rope_theta),
         offsetof(ssd_schedule, cfg), offsetof(ssd_schedule, cfg_weight));
  printf("%zu %zu %zu\\n", offsetof(ssd_schedule, eol), offsetof(ssd_schedule, eol_id),
         offsetof(ssd_schedule, separate_commit));
  printf("%zu %zu %zu %zu %zu\\n", offsetof(ssd_schedule, truncate), offsetof(ssd_schedule, trunc_block),
         offsetof(ssd_stats, accepted_round), offsetof(ssd_stats, proposed_round), offsetof(ssd_stats, wall_ns));
  return 0;
}}
""")
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", str(src), "-o", str(exe)])
    out = subprocess.check_output([str(exe)]).decode().split()
    got = [int(x) for x in out]
    want = [ctypes.sizeof(ssd.ssd_model_config), ctypes.sizeof(ssd.ssd_verify_params),
            ctypes.sizeof(ssd.ssd_schedule), ctypes.sizeof(ssd.ssd_stats),
            ssd.ssd_verify_params.temperature.offset, ssd.ssd_verify_params.seed.offset,
            ssd.ssd_verify_params.round.offset, ssd.ssd_schedule.temperature.offset,
            ssd.ssd_schedule.seed.offset, ssd.ssd_model_config.rope_theta.offset,
            ssd.ssd_schedule.cfg.offset, ssd.ssd_schedule.cfg_weight.offset,
            ssd.ssd_schedule.eol.offset, ssd.ssd_schedule.eol_id.offset,
            ssd.ssd_schedule.separate_commit.offset,
            ssd.ssd_schedule.truncate.offset, ssd.ssd_schedule.trunc_block.offset,
            ssd.ssd_stats.accepted_round.offset, ssd.ssd_stats.proposed_round.offset, ssd.ssd_stats.wall_ns.offset]
    assert got == want


def _cfg(shape):
    c = ssd.ssd_model_config()
    c.n_layers, c.d_model, c.n_heads, c.n_kv_heads = shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads
    c.head_dim, c.d_ff, c.vocab = shape.head_dim, shape.d_ff, shape.vocab
    c.img_lo, c.img_hi = shape.img_lo, shape.img_hi
    c.dtype = ssd.SSD_BF16 if shape.dtype == "bf16" else ssd.SSD_F32
    c.rms_eps, c.rope_theta = 1e-5, 10000.0
    return c


def test_weights_numel_matches_generator(lib):
    for wl in synth.WORKLOADS.values():
        assert ssd.ssd_weights_numel(_cfg(wl.model)) == synth.n_params(wl.model)


def test_invalid_configs_rejected(lib):
    c = _cfg(synth.M1B)
    c.n_kv_heads = 5
    assert ssd.ssd_weights_numel(c) == -1
    c = _cfg(synth.M1B)
    c.d_model = 2000  # bf16 GEMM K must be a multiple of 256
    assert ssd.ssd_weights_numel(c) == -1
    c = _cfg(synth.TINY)
    c.img_hi = c.vocab + 1
    assert ssd.ssd_weights_numel(c) == -1
    with pytest.raises(ssd.SSDError) as e:
        ssd.ssd_init_model(c, 1)
    assert e.value.status == ssd.SSD_E_INVAL and "image range" in ssd.ssd_last_error()


def test_null_arguments_rejected_before_device_work(lib):
    L = lib
    out = ctypes.c_void_p()
    assert L.ssd_init_model(None, None, None, ctypes.byref(out)) == ssd.SSD_E_INVAL
    assert L.ssd_prefill(None, 1, 1, None, 2, 1, None, ctypes.byref(out)) == ssd.SSD_E_INVAL
    prm = ssd.ssd_verify_params()
    assert L.ssd_verify_step(None, 1, None, None, ctypes.byref(prm), None, None, None, None, None) == ssd.SSD_E_INVAL
    sc = ssd.ssd_schedule()
    assert L.ssd_decode_image(None, ctypes.byref(sc), 1, 1, None, None, None, None, None, None) == ssd.SSD_E_INVAL
    assert L.ssd_get_carry(None, None) == ssd.SSD_E_INVAL
    assert L.ssd_session_set_cfg(None, 5.0) == ssd.SSD_E_INVAL
    assert L.ssd_profile(None, 1) == ssd.SSD_E_INVAL
    assert L.ssd_draft_head_init(None, 256, None, 1, ctypes.byref(out)) == ssd.SSD_E_INVAL
    assert L.ssd_draft_head_run(None, 1, None, None, None, None) == ssd.SSD_E_INVAL
    assert L.ssd_draft_head_numel(None, 256) == -1
    L.ssd_free_draft_head(None)  # a no-op
    st = ssd.ssd_stats()
    assert L.ssd_decode_image_heads(None, ctypes.byref(sc), 1, 1, None, None, 0, None, 0, None, ctypes.byref(st),
                                    None) == ssd.SSD_E_INVAL
    assert "NULL" in ssd.ssd_last_error()
    assert L.ssd_plant_image(None, ctypes.byref(sc), 1, 1, None, None, None, None, None, ctypes.byref(st),
                             None) == ssd.SSD_E_INVAL
    assert "NULL" in ssd.ssd_last_error()
