"""C ABI checks that need no GPU: the built library loads, exports every
function include/ts3.h declares with the binding's signature table, and
rejects bad descriptors before touching the device."""
import ctypes as ct
import os
import re

import pytest

from paper_2602_04940_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ts3.h")


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return set(re.findall(r"^\s*(?:const\s+char\s*\*|ts3_status)\s*(ts3_\w+)\s*\(", src, flags=re.M))


def test_header_declares_the_binding_table():
    assert header_functions() == set(L.SIGNATURES)


def test_library_exports_every_declared_symbol():
    lib = L.lib()
    for name in header_functions():
        assert hasattr(lib, name), name


def test_struct_layouts_match_header():
    assert ct.sizeof(L.Desc) == 48
    assert L.Desc.group_span.offset == 32 and L.Desc.max_points.offset == 40
    assert ct.sizeof(L.Weights) == 9 * ct.sizeof(ct.c_void_p)
    assert ct.sizeof(L.Grads) == 9 * ct.sizeof(ct.c_void_p)


def _desc(**kw):
    d = dict(C=128, H=8, M=64, dh=16, temperature=0.5, eps=0.0, io_dtype=L.TS3_BF16, accum=L.TS3_ACCUM_FP32,
             group_span=1024, max_points=4096)
    d.update(kw)
    return L.Desc(**d)


@pytest.mark.parametrize("kw,status", [
    (dict(C=0), L.TS3_ERR_INVALID_ARG),
    (dict(H=4), L.TS3_ERR_UNSUPPORTED),           # H*dh != C
    (dict(C=72, H=8, dh=9), L.TS3_ERR_UNSUPPORTED),         # C not a multiple of 16
    (dict(M=24), L.TS3_ERR_UNSUPPORTED),                    # M not a multiple of 16
    (dict(C=640, H=8, dh=80, M=16), L.TS3_ERR_UNSUPPORTED),  # C beyond the runtime-shape kernels' 512
    (dict(M=272, H=16, dh=8), L.TS3_ERR_UNSUPPORTED),       # M beyond the runtime-shape kernels' 256
    (dict(C=128, H=2, dh=64, M=128), L.TS3_ERR_UNSUPPORTED),  # token attention over 160 KiB of LDS
    (dict(io_dtype=7), L.TS3_ERR_INVALID_ARG),
    (dict(accum=2), L.TS3_ERR_INVALID_ARG),
    (dict(accum=-1), L.TS3_ERR_INVALID_ARG),
    (dict(temperature=0.0), L.TS3_ERR_INVALID_ARG),
    (dict(temperature=float("nan")), L.TS3_ERR_INVALID_ARG),
    (dict(eps=-1.0), L.TS3_ERR_INVALID_ARG),
    (dict(group_span=0), L.TS3_ERR_INVALID_ARG),
    (dict(max_points=-1), L.TS3_ERR_INVALID_ARG),
])
def test_bad_descriptor_is_rejected_before_any_device_call(kw, status):
    lib = L.lib()
    h = ct.c_void_p(1)
    d = _desc(**kw)
    assert lib.ts3_state_create(ct.byref(d), ct.byref(h)) == status
    assert h.value is None
    assert lib.ts3_last_error()


def test_null_arguments():
    lib = L.lib()
    assert lib.ts3_state_create(None, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_state_free(None) == L.TS3_OK
    assert lib.ts3_slice_accumulate(None, None, None, 0, 0, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_deslice(None, None, None, 0, None, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_status_string(L.TS3_ERR_BAD_STATE) == b"call out of order"
    assert lib.ts3_state_get_spans(None, 0, 1, None, 0, None) == L.TS3_ERR_INVALID_ARG


def test_block_weight_layout_matches_header():
    assert ct.sizeof(L.BlockWeights) == 17 * ct.sizeof(ct.c_void_p)
    assert L.BlockWeights.ln1_g.offset == ct.sizeof(L.Weights)


@pytest.mark.parametrize("kw,blocks,hidden,status", [
    (dict(), 0, 512, L.TS3_ERR_INVALID_ARG),                                 # no blocks
    (dict(), 2, 384, L.TS3_ERR_UNSUPPORTED),                                 # hidden != 4C
    (dict(io_dtype=L.TS3_FP32), 2, 512, L.TS3_ERR_UNSUPPORTED),              # activations are bf16
    (dict(C=256, H=8, dh=32, M=24), 2, 1024, L.TS3_ERR_UNSUPPORTED),         # M not a multiple of 16
    (dict(temperature=-1.0), 2, 512, L.TS3_ERR_INVALID_ARG),
])
def test_bad_stack_is_rejected_before_any_device_call(kw, blocks, hidden, status):
    h = ct.c_void_p(1)
    d = _desc(**kw)
    assert L.lib().ts3_stack_create(ct.byref(d), blocks, hidden, ct.byref(h)) == status
    assert h.value is None


def test_stack_calls_reject_null_arguments():
    lib = L.lib()
    assert lib.ts3_stack_create(None, 1, 512, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_stack_free(None) == L.TS3_OK
    assert lib.ts3_stack_forward(None, None, None, 1, 1, 1, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_stack_decode(None, None, None, 1, 1, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_stack_feedforward(None, None, 0, None, None, 1, None, None) == L.TS3_ERR_INVALID_ARG
    assert lib.ts3_stack_layer(None, 0, None) == L.TS3_ERR_INVALID_ARG


def test_package_import_loads_nothing_and_product_has_no_oracle_dependency():
    import importlib
    import sys
    pkg = importlib.import_module("paper_2602_04940_amd")
    assert pkg.__name__
    pkg_dir = os.path.join(ROOT, "paper_2602_04940_amd")
    for dirpath, _, files in os.walk(pkg_dir):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in text and "from oracle" not in text, f
                assert "ts3_synth" not in text, f
    # Importing the package (and its binding) in a fresh interpreter pulls in
    # neither the oracle nor the input generators.
    import subprocess
    code = ("import sys, paper_2602_04940_amd; from paper_2602_04940_amd import _lib, layer, stack; "
            "print(sorted(m for m in sys.modules if m.split('.')[0] in ('oracle', 'ts3_synth')))")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "[]", r.stdout


def test_noalloc_rejects_a_call_beyond_its_fixed_scratch_before_any_device_call():
    """ts3_layer_forward_noalloc checks its scratch need on the host: 1e9 points
    in spans of 1,024 need ~1 GB of run sums, far past the 64 MiB array."""
    lib = L.lib()
    d = _desc(group_span=1024, max_points=0)
    w = L.Weights(*([0x1000] * 9))
    fake = ct.c_void_p(0x10000)  # aligned, never dereferenced: the call fails before touching it
    st = lib.ts3_layer_forward_noalloc(ct.byref(d), ct.byref(w), fake, 10 ** 9, 1 << 20, 1 << 20, fake, None)
    assert st == L.TS3_ERR_INVALID_ARG
    assert b"scratch" in lib.ts3_last_error()
    d2 = _desc(group_span=1000)
    assert lib.ts3_layer_forward_noalloc(ct.byref(d2), ct.byref(w), fake, 4096, 1024, 1024, fake,
                                         None) == L.TS3_ERR_INVALID_ARG  # tile not a multiple of the span
