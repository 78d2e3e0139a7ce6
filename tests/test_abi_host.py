"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every symbol bevpool.h declares, and rejects bad arguments before any device
work."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bevpool.h")


@pytest.fixture(scope="module")
def binding():
    from paper_2205_13542_amd import _binding, build
    if not os.path.exists(_binding.LIB_PATH):
        build.build()
    _binding.load()
    return _binding


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"BEVPOOL_API\s+[\w\s\*]+?\b(bevpool_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    assert {"bevpool_plan", "bevpool_forward", "bevpool_forward_timed"} <= set(names)
    assert len(names) == 14


def test_library_exports_every_declared_symbol(binding):
    lib = ctypes.CDLL(binding.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name
    assert set(_declared_functions()) == set(binding.EXPORTED)


def test_version(binding):
    assert binding.bevpool_version() >= 100


def _geom(**over):
    from paper_2205_13542_amd import bevpool_geometry
    import workloads as wl
    r = wl.tiny_rig()
    vals = dict(n_cams=r.n_cams, feat_h=r.feat_h, feat_w=r.feat_w, n_depth=r.n_depth,
                depth_min=r.depth_min, depth_step=r.depth_step, pixel_offset=r.pixel_offset,
                nx=r.nx, ny=r.ny, x_min=r.x_min, y_min=r.y_min, cell_x=r.cell_x,
                cell_y=r.cell_y, z_min=r.z_min, z_cell=r.z_cell)
    vals.update(over)
    return bevpool_geometry(**vals), r


def _plan_rc(binding, intr, extr, geom, null_out=False):
    lib = binding.load()
    dp = ctypes.POINTER(ctypes.c_double)
    out = ctypes.c_void_p(12345)
    rc = lib.bevpool_plan(None if intr is None else intr.ctypes.data_as(dp),
                          None if extr is None else extr.ctypes.data_as(dp),
                          None if geom is None else ctypes.byref(geom), None,
                          None if null_out else ctypes.byref(out))
    return rc, out.value


@pytest.mark.parametrize("over,code", [
    (dict(n_cams=0), -1), (dict(feat_h=-2), -1), (dict(nx=0), -1),
    (dict(depth_step=0.0), -1), (dict(cell_x=-0.3), -1), (dict(z_cell=float("nan")), -1),
    (dict(x_min=float("inf")), -1),
    (dict(n_cams=6, feat_h=1024, feat_w=1024, n_depth=400), -4),   # 2.5e9 points
    (dict(nx=70000, ny=70000), -4),
])
def test_plan_rejects_bad_geometry(binding, over, code):
    geom, r = _geom(**over)
    n = max(1, geom.n_cams)
    intr = np.tile(r.intrinsics, (n, 1)).astype(np.float64)
    extr = np.tile(r.extrinsics, (n, 1)).astype(np.float64)
    rc, out = _plan_rc(binding, intr, extr, geom)
    assert rc == code, binding.bevpool_last_error()
    assert out is None                      # *out_plan cleared on failure
    assert binding.bevpool_last_error()


def test_plan_rejects_null_and_bad_calibration(binding):
    geom, r = _geom()
    intr, extr = r.intrinsics.copy(), r.extrinsics.copy()
    assert _plan_rc(binding, None, extr, geom)[0] == -1
    assert _plan_rc(binding, intr, None, geom)[0] == -1
    assert _plan_rc(binding, intr, extr, None)[0] == -1
    assert _plan_rc(binding, intr, extr, geom, null_out=True)[0] == -1
    bad = intr.copy()
    bad[0, 0] = 0.0
    assert _plan_rc(binding, bad, extr, geom)[0] == -1
    bad = extr.copy()
    bad[0, 5] = float("nan")
    assert _plan_rc(binding, intr, bad, geom)[0] == -1


def test_forward_rejects_bad_handles_before_device_work(binding):
    lib = binding.load()
    fake = ctypes.create_string_buffer(256)   # host memory, wrong magic
    vp = ctypes.c_void_p
    assert lib.bevpool_forward(vp(1), vp(1), None, vp(1), 1, 8, 0, None) == -1
    assert lib.bevpool_forward(vp(1), vp(1), ctypes.cast(fake, vp), vp(1), 1, 8, 0, None) == -1
    info = binding.bevpool_plan_info()
    assert lib.bevpool_plan_info_get(ctypes.cast(fake, vp), ctypes.byref(info)) == -1
    assert lib.bevpool_plan_export(None, None, None, None) == -1
    lib.bevpool_plan_destroy(None)            # NULL-safe
    lib.bevpool_plan_destroy(ctypes.cast(fake, vp))   # bad magic: ignored
    # plan import: null arguments, and a cell map entry outside [-1, nx*ny)
    out = ctypes.c_void_p(123)
    g, _ = _geom()
    assert lib.bevpool_plan_import(None, ctypes.byref(g), None, ctypes.byref(out)) == -1
    assert out.value is None
    import numpy as np
    n_points = g.n_cams * g.n_depth * g.feat_h * g.feat_w
    cop = np.full(n_points, -1, dtype=np.int32)
    cop[5] = g.nx * g.ny
    assert lib.bevpool_plan_import(cop.ctypes.data_as(vp), ctypes.byref(g), None,
                                   ctypes.byref(out)) == -1
    assert b"cell_of_point[5]" in lib.bevpool_last_error()
    cop[5] = -2
    assert lib.bevpool_plan_import(cop.ctypes.data_as(vp), ctypes.byref(g), None,
                                   ctypes.byref(out)) == -1
    # forward_ex: bad handle
    assert lib.bevpool_forward_ex(vp(1), vp(1), None, vp(1), 8, 1, 8, 0, 0, None) == -1
    assert lib.bevpool_forward_ex(vp(1), vp(1), ctypes.cast(fake, vp), vp(1), 8, 1, 8, 0, 2,
                                  None) == -1
    # backward: bad handle, and no output at all
    assert lib.bevpool_backward(vp(1), vp(1), vp(1), None, vp(1), vp(1), 1, 8, 0, None) == -1
    assert lib.bevpool_backward(vp(1), vp(1), vp(1), ctypes.cast(fake, vp), vp(1), vp(1), 1, 8, 0,
                                None) == -1


def test_package_fails_loudly_without_library(tmp_path):
    from paper_2205_13542_amd import _binding
    saved = _binding._lib
    _binding._lib = None
    try:
        with pytest.raises(ImportError):
            _binding.load(str(tmp_path / "missing.so"))
    finally:
        _binding._lib = saved


def _declaration_comments():
    """(name, comment) for every declared function: the block comment right
    before its declaration."""
    text = open(HEADER).read()
    out = []
    for m in re.finditer(r"/\*((?:(?!\*/).)*)\*/\s*(?:typedef[^;]*;\s*)?BEVPOOL_API\s+[\w\s\*]+?\b(bevpool_\w+)\s*\(",
                         text, flags=re.S):
        out.append((m.group(2), m.group(1)))
    return out


def test_every_operation_cites_its_passage():
    """Each entry point that computes or stores part of the method names the
    passage of the paper that defines it; utilities (error text, version,
    destroy) are exempt."""
    utilities = {"bevpool_last_error", "bevpool_version", "bevpool_plan_destroy"}
    found = dict(_declaration_comments())
    missing = set(_declared_functions()) - set(found)
    assert not missing, missing
    # the entry point that allocates nothing names its callers instead
    assert "cannot allocate" in found["bevpool_associate_noalloc"]
    for name, comment in found.items():
        if name in utilities or name == "bevpool_associate_noalloc":
            continue
        assert re.search(r"Sec\. III|Precomputation|Interval Reduction", comment), name
