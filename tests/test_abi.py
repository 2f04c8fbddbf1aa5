"""The C-ABI library loads, exports every symbol include/dllm.h declares, and
rejects invalid arguments on the host before touching the GPU (CPU only)."""
import ctypes
import math
import os
import re

import pytest

from paper_2608_22646_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dllm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dllm_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for must in ("dllm_step", "dllm_generate", "dllm_commit", "dllm_forward", "dllm_model_create",
                 "dllm_workspace_size", "dllm_last_error"):
        assert must in names


def test_library_exports_every_declared_symbol():
    lib = B.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
        assert name in B._SIGS, f"binding has no signature for {name}"


def test_struct_sizes_match_the_c_layout():
    # natural alignment of the C structs (x86-64 SysV)
    assert ctypes.sizeof(B.ModelCfg) == 56
    assert ctypes.sizeof(B.State) == 7 * 8
    assert ctypes.sizeof(B.WsLayout) == 10 * 8
    assert B.CaiParams.flags.offset + 4 == ctypes.sizeof(B.CaiParams) - 4 or \
        B.CaiParams.flags.offset + 4 == ctypes.sizeof(B.CaiParams)


def _cfg(**kw):
    base = dict(n_layers=1, d_model=256, n_heads=2, n_kv_heads=2, head_dim=128, d_ff=256, vocab=64, mask_id=63,
                rms_eps=1e-5, rope_base=1e4, dtype=B.DLLM_BF16)
    base.update(kw)
    return B.ModelCfg(**base)


@pytest.mark.parametrize("kw,code", [
    (dict(n_heads=3, n_kv_heads=2), -1),          # heads not a multiple of kv heads
    (dict(mask_id=64), -1),                       # mask id out of range
    (dict(head_dim=64), -5),                      # bf16 path needs head_dim 128
    (dict(dtype=7), -1),
    (dict(rms_eps=float("nan")), -1),
    (dict(d_model=0), -1),
])
def test_model_create_rejects_bad_shapes(kw, code):
    lib = B.lib()
    cfg = _cfg(**kw)
    n = 3 + 9 * cfg.n_layers
    ptrs = (ctypes.c_void_p * n)(*([0x1000] * n))
    h = ctypes.c_void_p()
    rc = lib.dllm_model_create(ctypes.byref(cfg), ptrs, n, None, 0, None, ctypes.byref(h))
    assert rc == code, lib.dllm_last_error()
    assert lib.dllm_last_error().decode() != ""


def test_model_create_rejects_wrong_weight_count_and_nulls():
    lib = B.lib()
    cfg = _cfg()
    ptrs = (ctypes.c_void_p * 5)(*([0x1000] * 5))
    h = ctypes.c_void_p()
    assert lib.dllm_model_create(ctypes.byref(cfg), ptrs, 5, None, 0, None, ctypes.byref(h)) == -1
    ptrs = (ctypes.c_void_p * 12)(*([0x1000] * 11 + [None]))
    assert lib.dllm_model_create(ctypes.byref(cfg), ptrs, 12, None, 0, None, ctypes.byref(h)) == -1
    assert lib.dllm_model_create(None, ptrs, 12, None, 0, None, ctypes.byref(h)) == -1


def test_model_buffer_size():
    """The model buffer holds the bf16 LM head's tiled copy: vocabulary rows padded
    to 256, d bf16 values each; an fp32 model needs none."""
    lib = B.lib()
    n = ctypes.c_size_t()
    for V, d in ((64, 256), (126464, 4096), (152064, 3584), (257, 512)):
        cfg = _cfg(vocab=V, mask_id=V - 1, d_model=d)
        assert lib.dllm_model_buffer_size(ctypes.byref(cfg), ctypes.byref(n)) == 0, lib.dllm_last_error()
        assert n.value == -(-V // 256) * 256 * d * 2
    cfg = _cfg(dtype=B.DLLM_F32, head_dim=64)
    assert lib.dllm_model_buffer_size(ctypes.byref(cfg), ctypes.byref(n)) == 0 and n.value == 0
    assert lib.dllm_model_buffer_size(ctypes.byref(_cfg(mask_id=64)), ctypes.byref(n)) == -1
    assert lib.dllm_model_buffer_size(None, ctypes.byref(n)) == -1


def test_model_create_checks_the_caller_buffer():
    """A bf16 model keeps its LM-head copy in the caller's buffer: a missing,
    misaligned or short buffer is rejected before any device work."""
    lib = B.lib()
    cfg = _cfg()
    n = 3 + 9 * cfg.n_layers
    ptrs = (ctypes.c_void_p * n)(*([0x1000] * n))
    need = ctypes.c_size_t()
    assert lib.dllm_model_buffer_size(ctypes.byref(cfg), ctypes.byref(need)) == 0
    h = ctypes.c_void_p()
    assert lib.dllm_model_create(ctypes.byref(cfg), ptrs, n, None, need.value, None, ctypes.byref(h)) == -1
    assert lib.dllm_model_create(ctypes.byref(cfg), ptrs, n, ctypes.c_void_p(0x1080), need.value, None,
                                 ctypes.byref(h)) == -1
    assert lib.dllm_model_create(ctypes.byref(cfg), ptrs, n, ctypes.c_void_p(0x1000), need.value - 256, None,
                                 ctypes.byref(h)) == -4
    assert "model_buf" in lib.dllm_last_error().decode()


def test_library_allocates_no_device_memory():
    """Every device buffer is the caller's: no allocation, free or device-wide
    synchronisation anywhere in the library's sources."""
    csrc = os.path.join(ROOT, "paper_2608_22646_amd", "csrc")
    banned = re.compile(r"\b(hipMalloc\w*|hipFree\w*|hipExtMalloc\w*|hipMallocManaged|hipDeviceSynchronize|"
                        r"hipMemset\w*)\s*\(")
    for f in sorted(os.listdir(csrc)):
        text = re.sub(r"//[^\n]*|/\*.*?\*/", "", open(os.path.join(csrc, f)).read(), flags=re.S)
        assert not banned.findall(text), (f, banned.findall(text))


def _commit_rc(ctl=None, **kw):
    lib = B.lib()
    p = (ctl or B.Controller()).to_c()
    for k, v in kw.items():
        setattr(p, k, v)
    st = B.State(*([0x1000] * 7))
    args = dict(B_=1, P=4, G=64, block=0, t=0)
    return lib.dllm_commit(ctypes.byref(p), ctypes.byref(st), ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000),
                           args["B_"], args["P"], args["G"], args["block"], args["t"], 99, None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(theta_s=float("nan")), -1),
    (dict(warmup=1.0), -1),
    (dict(warmup=-0.1), -1),
    (dict(block_len=65), -5),
    (dict(block_len=0), -5),
    (dict(patience=0), -1),
    (dict(theta_fb=float("inf")), -1),
    (dict(clip_lo=0.99, clip_hi=0.2), -1),
])
def test_commit_rejects_bad_controller_constants(kw, code):
    assert _commit_rc(**kw) == code


def test_commit_rejects_bad_indices():
    lib = B.lib()
    p = B.Controller().to_c()
    st = B.State(*([0x1000] * 7))
    c = ctypes.c_void_p(0x1000)
    # block index past G / block_len, step past T, G not a multiple of block_len, batch > 16
    assert lib.dllm_commit(ctypes.byref(p), ctypes.byref(st), c, c, 1, 4, 64, 2, 0, 99, None, None) == -2
    assert lib.dllm_commit(ctypes.byref(p), ctypes.byref(st), c, c, 1, 4, 64, 0, 32, 99, None, None) == -2
    assert lib.dllm_commit(ctypes.byref(p), ctypes.byref(st), c, c, 1, 4, 65, 0, 0, 99, None, None) == -2
    assert lib.dllm_commit(ctypes.byref(p), ctypes.byref(st), c, c, 17, 4, 64, 0, 0, 99, None, None) == -5
    st0 = B.State(*([0x1000] * 6 + [None]))
    assert lib.dllm_commit(ctypes.byref(p), ctypes.byref(st0), c, c, 1, 4, 64, 0, 0, 99, None, None) == -1
    assert lib.dllm_commit(None, ctypes.byref(st), c, c, 1, 4, 64, 0, 0, 99, None, None) == -1


def test_null_model_is_rejected():
    lib = B.lib()
    n = ctypes.c_size_t()
    assert lib.dllm_workspace_size(None, 1, 8, 8, ctypes.byref(n)) == -1
    assert lib.dllm_model_destroy(None) == 0


def test_library_has_no_undefined_internal_symbols():
    """Every kernel the launchers reference is defined (a kernel whose host stub
    the compiler dropped shows up as an undefined dllm:: symbol)."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-C", "--undefined-only", B.LIB_PATH], capture_output=True, text=True, check=True)
    bad = [l for l in out.stdout.splitlines() if "dllm::" in l]
    assert not bad, bad
