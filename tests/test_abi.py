"""CPU-side checks of the C-ABI library: it loads, exports every symbol the
header declares, and rejects bad configurations before touching a GPU."""
import ctypes
import os
import re

import pytest

from paper_2412_07210_amd import outer

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "edit_outer.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(edit_outer_\w+)\s*\(", text)))


def test_header_declarations_match_binding():
    assert _declared() == sorted(outer.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = outer.load_library()
    for name in _declared():
        assert hasattr(lib, name), name


def test_library_is_built_for_gfx950_only():
    data = open(outer.LIBRARY, "rb").read()
    assert b"gfx950" in data
    for other in (b"gfx942", b"gfx90a", b"gfx1100"):
        assert b"amdgcn-amd-amdhsa--" + other not in data


def test_struct_layouts():
    # int32, int32, ptr, int32, uint32, 6 doubles, int64
    assert ctypes.sizeof(outer._Config) == 4 + 4 + 8 + 4 + 4 + 6 * 8 + 8
    assert outer._Config.layer_numel.offset == 8
    assert outer._LayerState.ema_mean.offset == 24
    assert outer._LayerState.anomalous.offset == 24 + 4 * 16 * 8
    assert outer._LayerState.synced_norm.offset == 24 + 4 * 16 * 8 + 16


def test_strerror():
    lib = outer.load_library()
    assert lib.edit_outer_strerror(0) == b"ok"
    assert lib.edit_outer_strerror(-1) == b"invalid argument"
    assert lib.edit_outer_strerror(-5) == b"no gfx950 device"


def _init(**over):
    lib = outer.load_library()
    numel = over.pop("numel", [1024])
    arr = (ctypes.c_int64 * len(numel))(*numel)
    fields = dict(num_workers=4, num_layers=len(numel), layer_numel=arr, replica_dtype=1,
                  flags=7, outer_lr=0.8, momentum=0.85, clip_threshold=10.0, clip_eps=1e-6,
                  ema_alpha=0.02, z_threshold=3.0, ema_warmup_rounds=10)
    fields.update(over)
    cfg = outer._Config(**fields)
    h = ctypes.c_void_p()
    rc = lib.edit_outer_init(ctypes.byref(cfg), ctypes.byref(h))
    return rc, lib.edit_outer_last_error().decode()


@pytest.mark.parametrize("over,needle", [
    (dict(num_workers=0), "num_workers"),
    (dict(num_workers=17), "num_workers"),
    (dict(num_layers=0), "num_layers"),
    (dict(replica_dtype=7), "replica_dtype"),
    (dict(flags=16), "flag"),
    (dict(flags=8 | 1), "EDIT_ONE_PASS"),
    (dict(flags=8 | 4), "EDIT_ONE_PASS"),
    (dict(ema_alpha=0.0), "ema_alpha"),
    (dict(ema_alpha=1.5), "ema_alpha"),
    (dict(clip_eps=0.0), "clip_eps"),
    (dict(clip_threshold=-1.0), "clip_threshold"),
    (dict(outer_lr=float("nan")), "finite"),
    (dict(ema_warmup_rounds=-1), "warmup"),
    (dict(numel=[10, -1]), "negative"),
])
def test_init_rejects_bad_config(over, needle):
    rc, msg = _init(**over)
    assert rc == outer.EDIT_EINVAL
    assert needle in msg


def test_null_arguments_are_rejected():
    lib = outer.load_library()
    h = ctypes.c_void_p()
    assert lib.edit_outer_init(None, ctypes.byref(h)) == outer.EDIT_EINVAL
    assert lib.edit_outer_step_layer(None, 0, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_outer_step_round(None, 1, None, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_outer_step_round_host(None, 1, None, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_outer_gram_layer(None, 0, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_outer_apply_layer(None, 0, None, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_outer_state_get(None, 0, None) == outer.EDIT_EINVAL
    assert lib.edit_outer_copy_probe(None, None, 15, None) == outer.EDIT_EINVAL
    lib.edit_outer_destroy(None)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(outer, "_lib", None)
    monkeypatch.setattr(outer, "LIBRARY", str(tmp_path / "missing.so"))
    with pytest.raises(outer.EditOuterError):
        outer.load_library()
