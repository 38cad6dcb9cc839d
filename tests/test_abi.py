"""CPU-side checks of the C-ABI library: it loads, exports every symbol the
header declares, and rejects bad configurations before touching a GPU."""
import ctypes
import math
import os
import re

import pytest

from paper_2412_07210_amd import outer

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "edit_outer.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(edit_(?:outer|group)_\w+)\s*\(", text)))


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
    assert outer.MAX_K == 32
    assert outer._LayerState.anomalous.offset == 24 + 4 * 32 * 8
    assert outer._LayerState.synced_norm.offset == 24 + 4 * 32 * 8 + 32


def test_strerror():
    lib = outer.load_library()
    assert lib.edit_outer_strerror(0) == b"ok"
    assert lib.edit_outer_strerror(-1) == b"invalid argument"
    assert lib.edit_outer_strerror(-5) == b"no gfx950 device"


def _init(**over):
    lib = outer.load_library()
    rank = over.pop("rank", None)
    numel = over.pop("numel", [1024])
    arr = (ctypes.c_int64 * len(numel))(*numel)
    fields = dict(num_workers=4, num_layers=len(numel), layer_numel=arr, replica_dtype=1,
                  flags=7, outer_lr=0.8, momentum=0.85, clip_threshold=10.0, clip_eps=1e-6,
                  ema_alpha=0.02, z_threshold=3.0, ema_warmup_rounds=10)
    fields.update(over)
    cfg = outer._Config(**fields)
    h = ctypes.c_void_p()
    if rank is None:
        rc = lib.edit_outer_init(ctypes.byref(cfg), ctypes.byref(h))
    else:
        rc = lib.edit_group_init(ctypes.byref(cfg), rank, ctypes.byref(h))
    return rc, lib.edit_outer_last_error().decode()


@pytest.mark.parametrize("over,needle", [
    (dict(num_workers=0), "num_workers"),
    (dict(num_workers=33), "num_workers"),
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
    (dict(ema_warmup_rounds=5), "ema_warmup_rounds must be >= 6"),
    (dict(ema_warmup_rounds=0), "ema_warmup_rounds must be >= 6"),
    (dict(ema_alpha=0.005, ema_warmup_rounds=10), "ema_warmup_rounds must be >= 22"),
    (dict(z_threshold=0.0), "z_threshold must be > 0"),
    (dict(z_threshold=-1.0), "z_threshold must be > 0"),
    (dict(numel=[10, -1]), "negative"),
])
def test_init_rejects_bad_config(over, needle):
    rc, msg = _init(**over)
    assert rc == outer.EDIT_EINVAL
    assert needle in msg


@pytest.mark.parametrize("over,needle", [
    (dict(rank=-1), "rank"),
    (dict(rank=4), "rank"),
    (dict(rank=0, flags=8), "EDIT_ONE_PASS"),
    (dict(rank=0, num_workers=33), "num_workers"),
    (dict(rank=0, ema_warmup_rounds=2), "ema_warmup_rounds must be >= 6"),
    (dict(rank=0, ema_alpha=0.0), "ema_alpha"),
    (dict(rank=1, numel=[5, -2]), "negative"),
])
def test_group_init_rejects_bad_config(over, needle):
    """The sync-group worker validates like edit_outer_init, plus its rank."""
    rc, msg = _init(**over)
    assert rc == outer.EDIT_EINVAL
    assert needle in msg


@pytest.mark.parametrize("over", [
    dict(ema_warmup_rounds=6),                   # the paper's alpha and delta: 6 rounds suffice
    dict(flags=0, ema_warmup_rounds=0),          # no anomaly elimination: no warm-up needed
    dict(flags=6, ema_warmup_rounds=0, z_threshold=0.0),
    dict(num_workers=32),
])
def test_init_accepts_config(over):
    """Accepted configurations get past validation (here, without a GPU, the
    device check then fails instead)."""
    rc, msg = _init(**over)
    assert rc != outer.EDIT_EINVAL, msg


def _closed_form_z(alpha, k):
    """z-score of a worker whose norm G never changes, against the EMA of
    Eq. 1 after k updates from zero: mu_k = G(1 - (1-alpha)^k) and
    sigma_k = G (1-alpha)^((k+1)/2) sqrt(1 - (1-alpha)^k) (closed form of the
    recurrence, independent of the library's iteration)."""
    a = 1.0 - alpha
    return a ** ((k - 1) / 2) / math.sqrt(1.0 - a ** k)


@pytest.mark.parametrize("alpha,delta", [(0.02, 3.0), (0.02, 2.0), (0.02, 5.0), (0.1, 3.0), (0.005, 3.0),
                                         (0.3, 1.5)])
def test_min_warmup_matches_closed_form(alpha, delta):
    """edit_outer_min_warmup is the first k whose closed-form z-score is at
    most delta (the z-test flags G - mu > delta sigma)."""
    k = 1
    while _closed_form_z(alpha, k) > delta:
        k += 1
    assert outer.min_warmup(alpha, delta) == k
    # the paper's alpha = 0.02 and delta = 3 (Sec. 3.2)
    assert outer.min_warmup() == 6
    assert _closed_form_z(0.02, 5) > 3.0 > _closed_form_z(0.02, 6)


def test_min_warmup_rejects_impossible():
    assert outer.min_warmup(0.02, 0.0) == -1
    assert outer.min_warmup(0.02, -2.0) == -1
    assert outer.min_warmup(0.0, 3.0) == -1
    assert outer.min_warmup(1.5, 3.0) == -1
    assert outer.min_warmup(0.02, float("nan")) == -1


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
    assert lib.edit_group_init(None, 0, ctypes.byref(h)) == outer.EDIT_EINVAL
    assert lib.edit_group_norm(None, 0, None, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_group_weights(None, 0, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_group_apply(None, 0, None, None, None, None, None) == outer.EDIT_EINVAL
    assert lib.edit_group_state_get(None, 0, None) == outer.EDIT_EINVAL
    assert lib.edit_group_state_set(None, 0, None) == outer.EDIT_EINVAL
    lib.edit_group_destroy(None)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(outer, "_lib", None)
    monkeypatch.setattr(outer, "LIBRARY", str(tmp_path / "missing.so"))
    with pytest.raises(outer.EditOuterError):
        outer.load_library()


def test_header_layout_matches_binding(tmp_path):
    """Compile a C program against include/edit_outer.h and compare every
    struct size, field offset and constant with the ctypes mirrors."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    cfg_fields = [f for f, _ in outer._Config._fields_]
    st_fields = [f for f, _ in outer._LayerState._fields_]
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "edit_outer.h"', 'int main(void) {',
             '  printf("cfg_size %zu\\n", sizeof(edit_outer_config_t));',
             '  printf("state_size %zu\\n", sizeof(edit_layer_state_t));']
    lines += [f'  printf("cfg.{f} %zu\\n", offsetof(edit_outer_config_t, {f}));' for f in cfg_fields]
    lines += [f'  printf("state.{f} %zu\\n", offsetof(edit_layer_state_t, {f}));' for f in st_fields]
    consts = ["EDIT_MAX_K", "EDIT_AE", "EDIT_WA", "EDIT_GC", "EDIT_ONE_PASS", "EDIT_OK", "EDIT_EINVAL",
              "EDIT_ENOMEM", "EDIT_EHIP", "EDIT_ESTATE", "EDIT_ENODEV", "EDIT_F32", "EDIT_BF16"]
    lines += [f'  printf("{c} %ld\\n", (long)({c}));' for c in consts]
    lines += ['  return 0;', '}']
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    got = dict(line.split() for line in subprocess.run([str(exe)], check=True, capture_output=True,
                                                       text=True).stdout.splitlines())
    assert int(got["cfg_size"]) == ctypes.sizeof(outer._Config)
    assert int(got["state_size"]) == ctypes.sizeof(outer._LayerState)
    for f in cfg_fields:
        assert int(got[f"cfg.{f}"]) == getattr(outer._Config, f).offset, f
    for f in st_fields:
        assert int(got[f"state.{f}"]) == getattr(outer._LayerState, f).offset, f
    py = {"EDIT_MAX_K": outer.MAX_K, "EDIT_AE": outer.AE, "EDIT_WA": outer.WA, "EDIT_GC": outer.GC,
          "EDIT_ONE_PASS": outer.ONE_PASS, "EDIT_OK": outer.EDIT_OK, "EDIT_EINVAL": outer.EDIT_EINVAL,
          "EDIT_ENOMEM": outer.EDIT_ENOMEM, "EDIT_EHIP": outer.EDIT_EHIP, "EDIT_ESTATE": outer.EDIT_ESTATE,
          "EDIT_ENODEV": outer.EDIT_ENODEV, "EDIT_F32": outer.F32, "EDIT_BF16": outer.BF16}
    for c, v in py.items():
        assert int(got[c]) == v, c
