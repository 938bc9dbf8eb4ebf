"""The C-ABI library loads and exports every symbol include/wf.h declares; host-side
argument validation (no GPU needed: none of these calls reaches the device)."""
import ctypes
import os
import re
import subprocess

import pytest

from wf_fixtures import MICRO, TINY, LARGE_V3, full_manifest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wf.h")


def _lib():
    from paper_2609_32869_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libwf.so not built")
    return binding, binding.load_library()


def declared_symbols():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(wf_\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_step_entry_points():
    syms = declared_symbols()
    for name in ("wf_init_weights", "wf_encode_memory_set", "wf_draft", "wf_verify_accept", "wf_step"):
        assert name in syms


def test_library_exports_every_declared_symbol():
    binding, lib = _lib()
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (wf_\w+)", out))
    missing = [s for s in declared_symbols() if s not in exported]
    assert not missing, missing
    assert sorted(binding.EXPORTS) == declared_symbols()
    for s in declared_symbols():
        assert hasattr(lib, s)


@pytest.mark.parametrize("cfg", [MICRO, TINY, LARGE_V3, LARGE_V3.with_(draft_audio=False),
                                 LARGE_V3.with_(draft_history=False), LARGE_V3.with_(draft_pos="abs"),
                                 LARGE_V3.with_(n_draft_layer=5),
                                 MICRO.with_(draft_audio=False, draft_history=False, draft_pos="abs")],
                         ids=["micro", "tiny", "large-v3", "no-audio", "no-history", "abs-pos", "five-layers", "micro-all"])
def test_weight_manifest_matches_fixture_order(cfg):
    binding, lib = _lib()
    c = binding.make_config(cfg, 1)
    n = ctypes.c_int()
    assert lib.wf_weight_count(ctypes.byref(c), ctypes.byref(n)) == 0
    man = full_manifest(cfg)
    assert n.value == len(man)
    for i, (name, shape) in enumerate(man):
        k = ctypes.c_int64()
        assert lib.wf_weight_numel(ctypes.byref(c), i, ctypes.byref(k)) == 0
        numel = 1
        for s in shape:
            numel *= s
        assert k.value == numel, name


def test_workspace_grows_with_batch_and_rejects_bad_configs():
    binding, lib = _lib()
    sizes = []
    for b in (1, 2, 16):
        c = binding.make_config(LARGE_V3, b)
        n = ctypes.c_size_t()
        assert lib.wf_workspace_bytes(ctypes.byref(c), ctypes.byref(n)) == 0
        sizes.append(n.value)
    assert sizes[0] < sizes[1] < sizes[2]
    bad = [dict(n_head=7), dict(block_k=4), dict(n_ctx=500), dict(n_ctx=440), dict(dtype=5), dict(max_batch=0),
           dict(eos_id=10 ** 6), dict(n_tap=0)]
    for kw in bad:
        c = binding.make_config(LARGE_V3, 1)
        for k, v in kw.items():
            setattr(c, k, v)
        n = ctypes.c_size_t()
        assert lib.wf_workspace_bytes(ctypes.byref(c), ctypes.byref(n)) == -1, kw
        assert lib.wf_last_error(None)
    c = binding.make_config(LARGE_V3, 1)
    c.taps[1] = c.taps[0]
    assert lib.wf_workspace_bytes(ctypes.byref(c), ctypes.byref(ctypes.c_size_t())) == -1


def test_init_rejects_bad_arguments_before_touching_the_device():
    binding, lib = _lib()
    c = binding.make_config(MICRO, 1)
    h = ctypes.c_void_p()
    n = ctypes.c_size_t()
    lib.wf_workspace_bytes(ctypes.byref(c), ctypes.byref(n))
    cnt = ctypes.c_int()
    lib.wf_weight_count(ctypes.byref(c), ctypes.byref(cnt))
    arr = (ctypes.c_void_p * cnt.value)(*([4096] * cnt.value))
    # misaligned workspace
    assert lib.wf_init_weights(ctypes.byref(h), ctypes.byref(c), arr, cnt.value, ctypes.c_void_p(4100), n.value, None) == -1
    # too small
    assert lib.wf_init_weights(ctypes.byref(h), ctypes.byref(c), arr, cnt.value, ctypes.c_void_p(4096), 100, None) == -3
    # wrong count
    assert lib.wf_init_weights(ctypes.byref(h), ctypes.byref(c), arr, cnt.value - 1, ctypes.c_void_p(4096), n.value, None) == -1
    # null weight pointer
    arr2 = (ctypes.c_void_p * cnt.value)(*([4096] * (cnt.value - 1) + [None]))
    assert lib.wf_init_weights(ctypes.byref(h), ctypes.byref(c), arr2, cnt.value, ctypes.c_void_p(4096), n.value, None) == -1
    assert lib.wf_strerror(-3) == b"workspace too small"
    # calls on a null handle
    assert lib.wf_draft(None, 0, 1, None, None) == -1
    assert lib.wf_release(None) == -1


def test_bench_refuses_several_gpus_without_touching_a_device():
    """bench.py measures one GPU; asking for more exits with status 2 and a message
    before any device or library is touched (so it also runs here, with no GPU)."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""
