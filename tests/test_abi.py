"""Host-only checks of the C ABI: the library loads, exports every symbol the
headers declare, and rejects bad shapes before touching a GPU."""
import ctypes
import os
import re

import pytest

from paper_2609_12075_amd import synth, vla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    names = set()
    for h in ("vla.h", "vla_debug.h", "vla_sched.h"):
        p = os.path.join(ROOT, "include", h)
        if not os.path.exists(p):
            continue
        src = open(p).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        for m in re.finditer(r"\b(vla_\w+)\s*\(", src):
            names.add(m.group(1))
    return names


def test_library_exports_every_declared_symbol():
    L = vla.lib()
    declared = declared_functions()
    assert "vla_prefill" in declared and "vla_step" in declared
    for name in sorted(declared):
        assert hasattr(L, name), f"{name} declared in include/ but not exported"
    for name in vla.EXPORTS:
        assert name in declared


def test_weight_count_matches_schema():
    for cfg in list(synth.CONFIGS.values()) + [synth.reduced(c) for c in synth.CONFIGS.values()]:
        assert vla.weight_count(cfg) == synth.weight_count(cfg), cfg.name


@pytest.mark.parametrize("field,value,msg", [
    ("n_q", 7, "multiple of n_kv"),
    ("head_dim", 60, "head_dim"),
    ("img_hw", 65, "multiple of patch"),
    ("act_layers", 3, "act_layers"),
    ("max_batch", 0, "max_batch"),
])
def test_invalid_shapes_rejected(field, value, msg):
    cfg = synth.CONFIGS["smolvla"].with_(**{field: value})
    with pytest.raises(vla.VlaError) as e:
        vla.weight_count(cfg)
    assert msg in str(e.value)


def test_create_rejects_wrong_buffer_size_without_gpu():
    cfg = synth.CONFIGS["tiny"]
    s = vla.config_struct(cfg)
    h = ctypes.c_void_p()
    buf = (ctypes.c_float * 16)()
    st = vla.lib().vla_create_model(ctypes.byref(s), buf, 16, 0, ctypes.byref(h))
    assert st == vla.VLA_EINVAL
    assert "shape needs" in vla.lib().vla_last_error().decode()
    assert not h.value


def test_null_arguments_rejected():
    L = vla.lib()
    assert L.vla_prefill(None, 1, None, None, None, None) == vla.VLA_EINVAL
    assert L.vla_denoise(None, 1, None, None, 4, None, None) == vla.VLA_EINVAL
    assert L.vla_kv_bytes(None, 1) == 0
    assert L.vla_step(None, None) == vla.VLA_EINVAL
    assert "null" in L.vla_last_error().decode()


def test_bf16_gemm_hook_rejects_bad_shapes_without_gpu():
    L = vla.lib()
    buf = (ctypes.c_char * 64)()
    p = ctypes.cast(buf, ctypes.c_void_p)
    # GeGLU with odd N (gate/up rows come in pairs), an activation on top of
    # the GeGLU, and an output row shorter than N / 2
    assert L.vla_debug_gemm_bf16(4, 7, 8, p, 8, p, 8, None, 1, 0, 0, 0.0, p, 8, None) == vla.VLA_EINVAL
    assert "even" in L.vla_last_error().decode()
    assert L.vla_debug_gemm_bf16(4, 8, 8, p, 8, p, 8, None, 1, 2, 0, 0.0, p, 8, None) == vla.VLA_EINVAL
    assert "act" in L.vla_last_error().decode()
    assert L.vla_debug_gemm_bf16(4, 32, 8, p, 8, p, 8, None, 1, 0, 0, 0.0, p, 8, None) == vla.VLA_EINVAL
    assert "leading dimensions" in L.vla_last_error().decode()
    assert L.vla_debug_gemm_bf16(4, 32, 8, p, 8, p, 8, None, 0, 0, 0, 0.0, p, 16, None) == vla.VLA_EINVAL
    # folded norm without a positive eps
    assert L.vla_debug_gemm_bf16(4, 32, 8, p, 8, p, 8, None, 0, 0, 1, 0.0, p, 32, None) == vla.VLA_EINVAL
    assert "rms" in L.vla_last_error().decode()


@pytest.mark.parametrize("args,msg", [
    ((3, 64, 10, 0, 100), "kind must be"),
    ((2, 300, 10, 0, 100), "grid must be"),
    ((2, 64, 0, 0, 100), "iters or words"),
    ((1, 64, 10, 20000, 100), "iters or words"),
    ((2, 64, 10, 0, 0), "spin_limit"),
])
def test_sync_probe_rejects_bad_arguments_without_gpu(args, msg):
    import ctypes
    from paper_2609_12075_amd import vla
    L = vla.lib()
    assert L.vla_debug_sync_probe(*args, None, None, None, ctypes.c_void_p(16), None) == 1
    assert msg in L.vla_last_error().decode()
    # a barrier run without its counter is refused before anything launches
    assert L.vla_debug_sync_probe(2, 64, 10, 0, 100, None, None, None, ctypes.c_void_p(16), None) == 1
    assert "missing buffer" in L.vla_last_error().decode()
