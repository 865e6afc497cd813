"""Host-side tests of the C ABI: the library loads without a GPU, exports every
symbol the header declares, and rejects bad arguments before any device work."""
import ctypes
import math
import os
import re

import pytest

import paper_2201_12854_amd as mca
from paper_2201_12854_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mca.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mca_[a-z_]+)\s*\(", text)))


def test_header_symbols_exported():
    lib = mca.load_library()
    names = _declared_functions()
    assert len(names) >= 10
    for name in names:
        assert hasattr(lib, name), name


def test_header_enums_match_binding():
    text = open(HEADER).read()
    for name, val in [("MCA_OK", 0), ("MCA_ERR_INVALID_ARGUMENT", 1), ("MCA_ERR_UNSUPPORTED", 2),
                      ("MCA_ERR_WORKSPACE_TOO_SMALL", 3), ("MCA_ERR_HIP", 4), ("MCA_F32", 0), ("MCA_BF16", 1),
                      ("MCA_NUM_STAGES", 5), ("MCA_SAMPLING_TOKEN", 0), ("MCA_SAMPLING_WEIGHT", 1)]:
        assert re.search(rf"\b{name}\s*=\s*{val}\b", text), name
    # struct layout: the binding's ctypes mirror has the header's field order
    body = re.search(r"typedef struct mca_forward_desc \{(.*?)\} mca_forward_desc;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = re.findall(r"(\w+);", body)
    assert fields == [f for f, _ in binding.ForwardDesc._fields_]


def test_status_strings_and_stages():
    lib = mca.load_library()
    for code, name in [(0, "MCA_OK"), (1, "MCA_ERR_INVALID_ARGUMENT"), (2, "MCA_ERR_UNSUPPORTED"),
                       (3, "MCA_ERR_WORKSPACE_TOO_SMALL"), (4, "MCA_ERR_HIP")]:
        assert mca.status_string(code) == name
    assert lib.mca_num_stages() == 5
    assert [lib.mca_stage_name(i).decode() for i in range(5)] == list(binding.STAGES)
    assert lib.mca_stage_name(99).decode() == "unknown"


def _desc(**kw):
    args = dict(batch=2, seq=128, heads=12, d_in=768, dtype_code=1, alpha=0.4, seed=0)
    args.update(kw)
    return mca.make_desc(args["batch"], args["seq"], args["heads"], args["d_in"], args["dtype_code"],
                         args["alpha"], args["seed"])


def test_workspace_size_formula():
    B, n, H, d = 2, 128, 12, 768
    got = mca.workspace_size(_desc())
    tokens = B * n
    parts = H * ((n + 63) // 64)

    def a(v):
        return (v + 255) // 256 * 256

    # colmax partials, row normalisers, H~ (bf16), sample lists (8 bytes per row slot,
    # slack after the last list), list layouts
    expect = (a(4 * tokens * parts) + a(4 * tokens * H) + a(2 * tokens * H * 64) + a(8 * (tokens * ((d + 2) // 2 * 2) + 2 * ((d + 2) // 2 * 2) + 64))
              + a(4 * tokens))
    assert got == expect
    assert mca.workspace_size(_desc(dtype_code=0)) > got  # float32 H~
    # median rule: every probability per key, 4 B n H n more
    d = _desc()
    d.importance = binding.MCA_IMPORTANCE_MEDIAN
    assert mca.workspace_size(d) == expect + a(4 * tokens * H * n)
    d.importance = binding.MCA_IMPORTANCE_MEAN
    assert mca.workspace_size(d) == expect
    d.window = 64  # a window only with the max rule
    with pytest.raises(binding.MCAError):
        mca.workspace_size(d)



def test_workspace_partials_per_query_tile():
    # one column-max partial per (head, query tile): tiles of 64 queries up to 8 key tiles
    # (n <= 512), of 128 queries beyond (the streaming score pass)
    def a(v):
        return (v + 255) // 256 * 256

    def parts_bytes(n):
        base = mca.workspace_size(_desc(batch=1, seq=n, heads=4, d_in=256))
        return base
    for n, qt in ((512, 64), (513, 128), (600, 128), (4096, 128)):
        H, tokens, d = 4, n, 256
        parts = H * ((n + qt - 1) // qt)
        expect = (a(4 * tokens * parts) + a(4 * tokens * H) + a(2 * tokens * H * 64)
                  + a(8 * (tokens * ((d + 2) // 2 * 2) + 2 * ((d + 2) // 2 * 2) + 64)) + a(4 * tokens))
        assert parts_bytes(n) == expect, n

def test_prepared_size_formula():
    for dt, esz in ((0, 4), (1, 2)):
        for d_in, d_out in ((768, 768), (45, 256), (1, 64)):
            # rownorm, W_v^T in fragment order, the Eq. 6 prefix-sum table (uint64 [d_in])
            off = (4 * d_in + 255) // 256 * 256
            end_wt = off + ((d_out + 15) // 16 * 16) * ((d_in + 127) // 128 * 128) * esz
            assert mca.prepared_size(dt, d_in, d_out) == (end_wt + 255) // 256 * 256 + 8 * d_in


@pytest.mark.parametrize("field,value,status", [
    ("alpha", 0.0, binding.MCA_ERR_INVALID_ARGUMENT),
    ("alpha", -0.5, binding.MCA_ERR_INVALID_ARGUMENT),
    ("alpha", math.nan, binding.MCA_ERR_INVALID_ARGUMENT),
    ("alpha", math.inf, binding.MCA_ERR_INVALID_ARGUMENT),
    ("batch", 0, binding.MCA_ERR_INVALID_ARGUMENT),
    ("seq", 0, binding.MCA_ERR_INVALID_ARGUMENT),
    ("d_in", 0, binding.MCA_ERR_INVALID_ARGUMENT),
    ("d_in", 2049, binding.MCA_ERR_UNSUPPORTED),
    ("heads", 3, binding.MCA_ERR_UNSUPPORTED),    # d_out = 192 is not a multiple of 256
    ("heads", 36, binding.MCA_ERR_UNSUPPORTED),   # d_out = 2304 > 2048
    ("d_head", 128, binding.MCA_ERR_UNSUPPORTED),
    ("dtype", 7, binding.MCA_ERR_INVALID_ARGUMENT),
    ("sampling", 2, binding.MCA_ERR_INVALID_ARGUMENT),
    ("sampling", -1, binding.MCA_ERR_INVALID_ARGUMENT),
    ("window", -2, binding.MCA_ERR_INVALID_ARGUMENT),
    ("window", 3, binding.MCA_ERR_INVALID_ARGUMENT),
    ("window", 1 << 26, binding.MCA_ERR_INVALID_ARGUMENT),
    ("importance", 3, binding.MCA_ERR_INVALID_ARGUMENT),
    ("importance", -1, binding.MCA_ERR_INVALID_ARGUMENT),
    ("exact_from", -1, binding.MCA_ERR_INVALID_ARGUMENT),
])
def test_desc_validation(field, value, status):
    d = _desc()
    setattr(d, field, value)
    with pytest.raises(binding.MCAError) as e:
        mca.workspace_size(d)
    assert e.value.status == status
    assert mca.load_library().mca_last_error().decode() != ""


def test_forward_rejects_null_and_small_workspace_without_device_work():
    lib = mca.load_library()
    d = _desc(batch=1, seq=16, heads=4, d_in=64)
    ws = mca.workspace_size(d)
    fake = ctypes.c_void_p(0x10000)  # aligned, never dereferenced: the checks fail first
    st = lib.mca_attention_forward(ctypes.byref(d), None, fake, fake, fake, fake, fake, fake, fake, ws, None)
    assert st == binding.MCA_ERR_INVALID_ARGUMENT
    st = lib.mca_attention_forward(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, ws - 1, None)
    assert st == binding.MCA_ERR_WORKSPACE_TOO_SMALL
    mis = ctypes.c_void_p(0x10004)
    st = lib.mca_attention_forward(ctypes.byref(d), mis, fake, fake, fake, fake, fake, fake, fake, ws, None)
    assert st == binding.MCA_ERR_INVALID_ARGUMENT
    st = lib.mca_attention_forward(None, fake, fake, fake, fake, fake, fake, fake, fake, ws, None)
    assert st == binding.MCA_ERR_INVALID_ARGUMENT
    d.seq_lens = 0x10008  # misaligned optional pointer
    st = lib.mca_attention_forward(ctypes.byref(d), fake, fake, fake, fake, fake, fake, fake, fake, ws, None)
    assert st == binding.MCA_ERR_INVALID_ARGUMENT


def test_prepare_weights_rejects_bad_arguments():
    lib = mca.load_library()
    fake = ctypes.c_void_p(0x10000)
    big = 1 << 30
    assert lib.mca_prepare_weights(None, 0, 8, 8, fake, big, None) == binding.MCA_ERR_INVALID_ARGUMENT
    assert lib.mca_prepare_weights(fake, 3, 8, 8, fake, big, None) == binding.MCA_ERR_INVALID_ARGUMENT
    assert lib.mca_prepare_weights(fake, 0, 0, 8, fake, big, None) == binding.MCA_ERR_INVALID_ARGUMENT
    assert lib.mca_prepare_weights(fake, 0, 4097, 8, fake, big, None) == binding.MCA_ERR_INVALID_ARGUMENT
    assert lib.mca_prepare_weights(fake, 0, 8, 8, ctypes.c_void_p(0x10002), big, None) == \
        binding.MCA_ERR_INVALID_ARGUMENT
    need = mca.prepared_size(0, 8, 8)
    assert lib.mca_prepare_weights(fake, 0, 8, 8, fake, need - 1, None) == binding.MCA_ERR_INVALID_ARGUMENT
    with pytest.raises(binding.MCAError):
        mca.prepared_size(5, 8, 8)


def test_profiler_lifecycle_without_device_work():
    p = mca.Profiler()
    stats = p.collect()  # nothing recorded: all zero
    assert all(v == (0.0, 0) for v in stats.values())
    p.close()


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError):
        binding._lib_saved = binding._lib
        try:
            binding._lib = None
            binding.load_library(str(tmp_path / "missing.so"))
        finally:
            binding._lib = binding._lib_saved


def test_binding_rejects_unknown_rule_names():
    with pytest.raises(ValueError):
        binding._importance_code("mode")
    with pytest.raises(ValueError):
        binding._sampling_code("rows")
    assert [binding._importance_code(r) for r in ("max", "mean", "median")] == [0, 1, 2]


def test_build_flags():
    # every HIP source is compiled for gfx950 without packed-fp32 code generation and with
    # MFMA results in ordinary VGPRs
    from paper_2201_12854_amd import build_lib

    flags = build_lib.CXXFLAGS
    assert "--offload-arch=gfx950" in flags
    i = flags.index("-packed-fp32-ops")
    assert flags[i - 3:i] == ["-Xclang", "-target-feature", "-Xclang"]
    assert "-amdgpu-mfma-vgpr-form" in flags


def test_issue_probe_library_rejects_bad_arguments():
    # the probe library (measurement support, include/mca_probe.h) loads without a GPU,
    # exports its entry point, and rejects invalid arguments before any device work
    path = os.path.join(ROOT, "paper_2201_12854_amd", "libmca_probe.so")
    if not os.path.exists(path):
        pytest.skip("libmca_probe.so not built")
    lib = ctypes.CDLL(path)
    f = lib.mca_issue_probe
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(ctypes.c_longlong), ctypes.c_int,
                  ctypes.POINTER(ctypes.c_int)]
    buf = (ctypes.c_longlong * 16)()
    nw = ctypes.c_int(-5)
    for kind, w, rounds in [(9, 1, 10), (-1, 1, 10), (0, 3, 10), (0, 8, 10), (4, 1, 10), (6, 4, 10), (0, 1, 0),
                            (2, 2, 1 << 21)]:
        assert f(kind, w, rounds, buf, 4, ctypes.byref(nw)) == -1, (kind, w, rounds)
    assert f(0, 1, 10, None, 4, ctypes.byref(nw)) == -1
    assert f(0, 1, 10, buf, 4, None) == -1
    assert nw.value == -5  # nothing written on rejection
