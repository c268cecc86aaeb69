"""The C-ABI library loads and exports every entry point declared in
include/freqcache.h, and argument errors come back as status codes without any
device work (these run without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "freqcache.h")


def declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(fc_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def fc():
    import paper_2604_24391_amd as fc
    fc.lib()
    return fc


def test_header_declares_the_three_calls():
    names = declared()
    for n in ("fc_select", "fc_layer_forward", "fc_cache_update", "fc_create", "fc_destroy",
              "fc_last_error"):
        assert n in names


def test_every_declared_symbol_is_exported(fc):
    lib = fc.lib()
    missing = [n for n in declared() if not hasattr(lib, n)]
    assert not missing, missing
    assert sorted(fc.EXPORTS) == declared()


def test_version_and_error_text(fc):
    assert "gfx950" in fc.fc_version()
    assert isinstance(fc.fc_last_error(), str)


def test_null_arguments_are_rejected_without_a_device(fc):
    lib = fc.lib()
    assert lib.fc_create(None, 0, None) == 1
    assert lib.fc_select(None, None, None, None, 1, 224, 224, None, None) == 1
    assert "null" in fc.fc_last_error()
    assert lib.fc_layer_forward(None, None, None, None, None, None, None, 1, None) == 1
    assert lib.fc_cache_update(None, None, None, None, None, None, None, 16, 1, None) == 1
    assert lib.fc_cache_update_layers(None, None, 2, None, None, None, None, None, 16, 1,
                                      None) == 1
    assert lib.fc_profile_enable(None, 1) == 1
    assert lib.fc_destroy(None) == 1


def test_create_without_gpu_reports_no_device(fc):
    """On a machine without a GPU, fc_create fails with FC_ERR_NO_DEVICE (on a GPU
    box it succeeds)."""
    caps = fc.Caps(max_batch=1, max_height=224, max_width=224, max_tokens=256, max_seq=288,
                   max_d_model=256, max_ffn=1024, max_qkv=768)
    try:
        ctx = fc.Context(caps)
    except fc.FcError as e:
        assert e.status == 5
    else:
        ctx.close()


def test_bad_caps_rejected(fc):
    caps = fc.Caps(max_batch=0)
    with pytest.raises(fc.FcError) as e:
        fc.Context(caps)
    assert e.value.status == 1
    with pytest.raises(fc.FcError) as e:
        fc.Context(fc.Caps(max_tokens=4096))
    assert e.value.status == 6


def test_struct_layouts_match_the_header(fc, tmp_path):
    """ctypes mirrors of the C structs have the size and field offsets that the C
    compiler gives the header's structs (a small C program prints them)."""
    import shutil
    import subprocess
    structs = [fc.freqcache.fc_caps, fc.freqcache.fc_select_params, fc.freqcache.fc_select_out,
               fc.freqcache.fc_kv_cache, fc.freqcache.fc_layer_desc, fc.freqcache.fc_vit_desc,
               fc.freqcache.fc_vit_cache, fc.freqcache.fc_merger_desc]
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "freqcache.h"', 'int main(void) {']
    for st in structs:
        lines.append(f'  printf("%zu\\n", sizeof({st.__name__}));')
        for name, _ in st._fields_:
            lines.append(f'  printf("%zu\\n", offsetof({st.__name__}, {name}));')
    lines += ['  return 0;', '}']
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run([cc, "-I", inc, str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], check=True, capture_output=True,
                                          text=True).stdout.split()]
    want = []
    for st in structs:
        want.append(ctypes.sizeof(st))
        want += [getattr(st, name).offset for name, _ in st._fields_]
    assert got == want


def test_cache_update_layers_binding_checks_lengths(fc):
    """The binding refuses per-layer lists of different lengths before any call."""
    with pytest.raises(ValueError, match="one entry per layer"):
        fc.fc_cache_update_layers(None, None, [], [], [], None, None, 16)
    with pytest.raises(ValueError, match="one entry per layer"):
        fc.fc_cache_update_layers(None, None, [object()], [object(), object()], [object()], None,
                                  None, 16)


def test_select_noalloc_rejects_before_device_work(fc):
    """fc_select_noalloc checks its arguments and its scratch limit synchronously: null
    arguments are FC_ERR_INVALID_ARG and a batch whose workspace exceeds the static
    16 MiB scratch is FC_ERR_CAPACITY, both without a GPU (no pointer is touched)."""
    lib = fc.lib()
    assert lib.fc_select_noalloc(None, None, None, 1, 224, 224, None, None) == 1
    fake = fc.freqcache.fc_select_out(*([1] * 9))
    prm = fc.SelectParams().c()
    st = lib.fc_select_noalloc(ctypes.byref(prm), None, ctypes.c_void_p(1), 64, 448, 448,
                               ctypes.byref(fake), None)
    assert st == 3 and "scratch" in fc.fc_last_error()
    st = lib.fc_select_noalloc(ctypes.byref(prm), None, ctypes.c_void_p(1), 1, 100, 224,
                               ctypes.byref(fake), None)
    assert st == 2


def test_select_state_bytes_and_carry_errors(fc):
    """The carried selection state of one 448x448 frame: 1024 patches x 100 amplitude bins
    (float32, 16-patch chunks) and 1024 patch means (float64), each part 256-B aligned;
    sizes without a patch give 0.  fc_select_carry rejects null or aliased arguments
    before any device work."""
    assert fc.select_state_bytes(1, 448, 448) == 409600 + 8192
    assert fc.select_state_bytes(2, 224, 448) == 2 * 16 * 32 * 100 * 4 + 2 * 512 * 8
    assert fc.select_state_bytes(0, 448, 448) == 0 and fc.select_state_bytes(1, 10, 448) == 0
    lib = fc.lib()
    assert lib.fc_select_carry(None, None, None, None, None, 1, 224, 224, None, None) == 1


def test_debug_mode_switch(fc):
    """fc_debug sets and reports the process-wide debug mode; a negative argument only
    reads it."""
    start = fc.fc_debug()
    try:
        assert fc.fc_debug(True) == start
        assert fc.fc_debug() is True
        assert fc.lib().fc_debug(-5) == 1
        assert fc.fc_debug(False) is True
        assert fc.fc_debug() is False
    finally:
        fc.fc_debug(start)


@pytest.mark.parametrize("value,expect", [("1", 1), ("yes", 1), ("0", 0), ("", 0), (None, 0)])
def test_debug_mode_from_environment(fc, value, expect):
    """The mode starts from FC_DEBUG as the library loads (a fresh process loads it)."""
    import subprocess
    import sys
    env = dict(os.environ)
    env.pop("FC_DEBUG", None)
    if value is not None:
        env["FC_DEBUG"] = value
    code = ("import ctypes; L = ctypes.CDLL(%r); L.fc_debug.restype = ctypes.c_int32; "
            "print(L.fc_debug(-1))" % fc.freqcache.LIB)
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                         timeout=60)
    assert out.returncode == 0, out.stderr
    assert int(out.stdout.strip()) == expect
