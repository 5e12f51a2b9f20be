"""The C-ABI library loads and exports every symbol include/mtp.h
declares; host-side argument checks that need no GPU."""
import ctypes
import os
import re

from paper_2609_03181_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "mtp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return set(re.findall(r"^\s*(?:mtp_status|void|size_t)\s+(\w+)\s*\(", src, flags=re.M))


def test_library_exports_every_declared_symbol():
    lib = _lib.load()
    names = _declared()
    assert names == set(_lib.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def test_struct_layouts_match_header():
    # 15 int32 then 2 doubles
    assert ctypes.sizeof(_lib.MtpConfig) == 15 * 4 + 4 + 16
    assert ctypes.sizeof(_lib.MtpWeights) == len(_lib.WEIGHT_FIELDS) * 8
    src = open(os.path.join(ROOT, "include", "mtp.h")).read()
    body = src[src.index("typedef struct {\n  const void *embed"):src.index("} mtp_weights;")]
    fields = re.findall(r"\*?(\w+)[,;]", body.replace("const void", "").replace("const float", ""))
    assert tuple(fields) == _lib.WEIGHT_FIELDS


def test_host_validation_without_gpu():
    lib = _lib.load()
    cfg = _lib.MtpConfig(2, 256, 4, 64, 8, 2, 1, 128, 384, 4096, 1, 0, 1, 64, 3, 1e4, 1e-6)
    w = _lib.MtpWeights()
    out = ctypes.c_void_p()
    assert lib.mtp_create(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(out)) == _lib.MTP_EINVAL
    bad = _lib.MtpConfig(2, 256, 4, 96, 8, 2, 1, 128, 384, 4096, 1, 0, 1, 64, 3, 1e4, 1e-6)
    assert lib.mtp_create(ctypes.byref(bad), ctypes.byref(w), ctypes.byref(out)) == \
        _lib.MTP_EUNSUPPORTED
    assert lib.mtp_create(None, None, None) == _lib.MTP_EINVAL
    assert lib.greedy_accept(0, 3, None, None, None, None, None) == _lib.MTP_EINVAL
    assert lib.moe_verify_step(None, 1, 3, *([None] * 12), 0, None) == _lib.MTP_EINVAL
    assert lib.mtp_draft_k(None, 1, 3, *([None] * 10), 0, None) == _lib.MTP_EINVAL
    assert lib.mtp_workspace_bytes(None, 1, 4) == 0
    assert lib.mtp_context_bytes(None) == 0
    st = ctypes.c_int32(0)
    assert lib.mtp_status_read(None, None, ctypes.byref(st)) == _lib.MTP_EINVAL
    assert lib.kv_commit_rollback(None, 1, 3, *([None] * 9), 0, None, None) == _lib.MTP_EINVAL


def _param_types(name):
    src = open(os.path.join(ROOT, "include", "mtp.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    m = re.search(r"\b" + name + r"\s*\(([^)]*)\)\s*;", src)
    params = [p.strip() for p in m.group(1).split(",")]
    out = []
    for p in params:
        if "*" in p:
            out.append("ptr")
        elif p.startswith("size_t"):
            out.append("size")
        elif p.startswith("int32_t"):
            out.append("i32")
        else:
            raise AssertionError(p)
    return out


def test_ctypes_signatures_match_header():
    lib = _lib.load()
    kind = {ctypes.c_void_p: "ptr", ctypes.c_int32: "i32", ctypes.c_size_t: "size"}
    for name in _lib.EXPORTS:
        want = _param_types(name)
        got = [kind[t] for t in getattr(lib, name).argtypes]
        assert got == want, name
