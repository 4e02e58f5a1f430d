"""The C ABI library loads without a GPU, exports every symbol the header
declares, and rejects malformed manifests before touching the device
(extent past its window, extent length disagreeing with the object size,
duplicate objects, bad shapes): the rejection conditions of the paper's
bounded source service and manifest ("A Shared Cross-Adapter Plan Core",
"Bounded Source Service")."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "msi.h")).read()
    return sorted(set(re.findall(r"^\s*(?:msi_status|const char \*|uint32_t)\s*(msi_\w+)\s*\(", src, re.M)))


def test_header_matches_binding_exports():
    import paper_2608_23805_amd as msi
    assert sorted(msi.EXPORTS) == _header_functions()


def test_library_exports_every_symbol():
    import paper_2608_23805_amd as msi
    lib = ctypes.CDLL(msi.LIB_PATH)
    for name in _header_functions():
        assert hasattr(lib, name), name
    assert msi.lib.msi_abi_version() == msi.MSI_ABI_VERSION


def _desc(msi, **over):
    """A small valid-looking manifest whose pool pointer is never dereferenced
    (creation fails during validation)."""
    d, I, E = 256, 128, 4
    ob = msi.object_nbytes(d, I, "bf16")
    win = (ctypes.c_uint8 * (4 * ob))()
    wins = (ctypes.c_void_p * 1)(ctypes.addressof(win))
    objs = over.pop("objects", [(0, e, 0, e * ob, ob) for e in range(E)])
    arr = (msi.msi_object_desc * len(objs))(*[msi.msi_object_desc(l, e, w, 0, o, n) for l, e, w, o, n in objs])
    kw = dict(abi_version=msi.MSI_ABI_VERSION, n_layers=1, n_experts=E, d_model=d, d_ff=I, top_k=2,
              wdtype=msi.MSI_W_BF16, slots_per_layer=2, transient_slots=0, policy=0,
              slot_pool=1 << 20, slot_pool_bytes=2 * ob + 4096, slot_stride=(ob + 255) // 256 * 256,
              windows=ctypes.cast(wins, ctypes.POINTER(ctypes.c_void_p)), n_windows=1, n_objects=len(objs),
              window_bytes=4 * ob, objects=ctypes.cast(arr, ctypes.POINTER(msi.msi_object_desc)))
    kw.update(over)
    return msi.msi_plan_desc(**kw), (win, wins, arr), ob


def _create(msi, **over):
    desc, keep, ob = _desc(msi, **over)
    h = ctypes.c_void_p()
    st = msi.lib.msi_plan_create(ctypes.byref(desc), ctypes.byref(h))
    return st, msi.last_error()


@pytest.mark.parametrize("case,status,fragment", [
    ("extent_past_window", -2, "past its window"),
    ("short_extent", -2, "extent length"),
    ("duplicate", -1, "duplicate"),
    ("bad_topk", -1, "top_k"),
    ("bad_d", -1, "d_model"),
    ("bad_stride", -1, "slot_stride"),
    ("bad_version", -1, "abi_version"),
    ("window_index", -1, "out of range"),
    ("bad_wdtype", -1, "unknown wdtype"),
    ("kq_d_ff", -1, "multiple of 256"),
])
def test_manifest_rejections(case, status, fragment):
    import paper_2608_23805_amd as msi
    ob = msi.object_nbytes(256, 128, "bf16")
    over = {
        "extent_past_window": dict(objects=[(0, 0, 0, 3 * ob + 16, ob)]),
        "short_extent": dict(objects=[(0, 0, 0, 0, ob - 2)]),
        "duplicate": dict(objects=[(0, 1, 0, 0, ob), (0, 1, 0, ob, ob)]),
        "bad_topk": dict(top_k=5),
        "bad_d": dict(d_model=200),
        "bad_stride": dict(slot_stride=1000),
        "bad_version": dict(abi_version=99),
        "window_index": dict(objects=[(0, 0, 3, 0, ob)]),
        "bad_wdtype": dict(wdtype=4),
        "kq_d_ff": dict(wdtype=msi.MSI_W_KQ),        # d_ff = 128: not whole 256-element super-blocks
    }[case]
    st, err = _create(msi, **over)
    assert st == status and fragment in err, (st, err)


def test_object_sizes_agree():
    """The binding's object sizes are the generators' for every format
    (the quantized mix: two k4 matrices and one k6 matrix)."""
    import paper_2608_23805_amd as msi
    import synth
    for wd in ("f32", "bf16", "q4b32", "kq"):
        for d, I in ((256, 256), (2048, 512), (512, 768)):
            assert msi.object_nbytes(d, I, wd) == synth.object_nbytes(d, I, wd), (wd, d, I)
    # 4.5 bits per weight for Wg / Wu, 6.5625 for Wd
    assert synth.k4_matrix_nbytes(512, 2048) * 8 == 4.5 * 512 * 2048
    assert synth.k6_matrix_nbytes(2048, 512) * 8 == 6.5625 * 512 * 2048


def test_null_arguments():
    import paper_2608_23805_amd as msi
    assert msi.lib.msi_plan_create(None, None) == msi.MSI_E_INVALID_ARG
    assert msi.lib.msi_route(None, None, None) == msi.MSI_E_INVALID_ARG
    assert msi.lib.msi_moe_forward(None, None, None, None) == msi.MSI_E_INVALID_ARG
    assert msi.lib.msi_plan_destroy(None) == msi.MSI_OK
    assert msi.stream_threshold() == 16



def _source_create(msi, tmp_path, ext_over=None, over=None, src_over=None, win_bytes=None, win_misalign=0,
                   write_file=True):
    """A plan over 4 source-backed objects (3 extents each) in one file;
    creation is expected to fail in validation, before any device call."""
    d, I, E = 256, 128, 4
    comps = [I * d * 2, I * d * 2, d * I * 2]
    ob = sum(comps)
    path = str(tmp_path / "canon.bin")
    if write_file:
        with open(path, "wb") as fh:
            fh.write(b"\x11" * (E * ob + 10000))
    extents, off = [], 100
    for e in range(E):
        for c, n in enumerate(comps):
            extents.append((0, e, c, 0, off, n))
            off += n
    if ext_over:
        extents = ext_over(extents)
    wb = win_bytes or (ob + 4 * 8192) // 4096 * 4096
    raw = (ctypes.c_uint8 * (wb + 8192))()
    base = (ctypes.addressof(raw) + 4095) // 4096 * 4096 + win_misalign
    wins = (ctypes.c_void_p * 1)(base)
    names = (ctypes.c_char_p * 1)(path.encode())
    arr = (msi.msi_extent_desc * len(extents))(*[msi.msi_extent_desc(*x) for x in extents])
    skw = dict(files=names, n_files=1, inflight=8, flags=1, align=4096,
               extents=ctypes.cast(arr, ctypes.POINTER(msi.msi_extent_desc)), n_extents=len(extents), reserved=0)
    skw.update(src_over or {})
    src = msi.msi_source_desc(**skw)
    objs = (msi.msi_object_desc * 1)(msi.msi_object_desc(0, 0, 0, 0, 0, ob))
    kw = dict(abi_version=msi.MSI_ABI_VERSION, n_layers=1, n_experts=E, d_model=d, d_ff=I, top_k=2,
              wdtype=msi.MSI_W_BF16, slots_per_layer=2, transient_slots=0, policy=0,
              slot_pool=1 << 20, slot_pool_bytes=2 * ob + 4096, slot_stride=(ob + 255) // 256 * 256,
              windows=ctypes.cast(wins, ctypes.POINTER(ctypes.c_void_p)), n_windows=1, n_objects=0,
              window_bytes=wb, objects=ctypes.cast(objs, ctypes.POINTER(msi.msi_object_desc)),
              source=ctypes.pointer(src))
    kw.update(over or {})
    desc = msi.msi_plan_desc(**kw)
    h = ctypes.c_void_p()
    st = msi.lib.msi_plan_create(ctypes.byref(desc), ctypes.byref(h))
    return st, msi.last_error()


@pytest.mark.parametrize("case,status,fragment", [
    ("extent_past_file", -2, "past the end of its file"),
    ("size_disagreement", -2, "add up to"),
    ("duplicate_component", -1, "duplicate component"),
    ("component_gap", -1, "gap"),
    ("objects_and_source", -1, "takes its objects"),
    ("misaligned_window", -1, "aligned"),
    ("inflight", -1, "in-flight"),
    ("window_too_small", -1, "covering reads"),
    ("missing_file", -1, "cannot open"),
])
def test_source_manifest_rejections(tmp_path, case, status, fragment):
    """Rejection conditions of the bounded source service at plan creation:
    extent overflow, object-size disagreement, malformed bundles, windows
    that are misaligned or too small, an in-flight limit outside 1..8, a file
    that cannot be opened."""
    import paper_2608_23805_amd as msi
    kw = {
        "extent_past_file": dict(ext_over=lambda x: x[:-1] + [(0, 3, 2, 0, 10 ** 7, x[-1][5])]),
        "size_disagreement": dict(ext_over=lambda x: x[:-1] + [x[-1][:5] + (x[-1][5] - 2,)]),
        "duplicate_component": dict(ext_over=lambda x: x + [x[0]]),
        "component_gap": dict(ext_over=lambda x: [e for e in x if not (e[1] == 1 and e[2] == 1)]),
        "objects_and_source": dict(over=dict(n_objects=1)),
        "misaligned_window": dict(win_misalign=512),
        "inflight": dict(src_over=dict(inflight=9)),
        "window_too_small": dict(win_bytes=4096 * 16),
        "missing_file": dict(write_file=False),
    }[case]
    st, err = _source_create(msi, tmp_path, **kw)
    assert st == status and fragment in err, (st, err)


def test_source_manifest_valid_until_device(tmp_path):
    """The same manifest without a fault passes validation and stops only at
    the device (no GPU here) -- so each rejection above is the validator's."""
    import paper_2608_23805_amd as msi
    st, err = _source_create(msi, tmp_path)
    assert st == msi.MSI_E_DEVICE, (st, err)
