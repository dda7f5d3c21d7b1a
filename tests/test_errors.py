"""Error paths of the C ABI that the host rejects before any HIP call, so they
run without a GPU: argument validation of cgtp_plan (degree, dtype, cover,
forced grids below exactness or of unsupported size) and of the forward entry
points (NULL plan).  Each case checks the documented status code and that no
plan handle is returned."""
import ctypes

import pytest

import paper_2602_21466_amd as lib


def _plan_rc(L, grid=None):
    h = ctypes.c_void_p()
    rc = lib._load().cgtp_plan(int(L), ctypes.byref(grid) if grid is not None else None, ctypes.byref(h))
    return rc, h.value


@pytest.mark.parametrize("L", [-1, -7])
def test_plan_negative_degree(L):
    assert _plan_rc(L) == (lib.CGTP_EINVAL, None)


@pytest.mark.parametrize("L", [33, 40, 1 << 20])
def test_plan_degree_above_the_build_limit(L):
    assert _plan_rc(L) == (lib.CGTP_EUNSUP, None)


@pytest.mark.parametrize("dtype", [2, 7, -1])
def test_plan_unknown_dtype(dtype):
    assert _plan_rc(4, lib._grid(dtype=dtype)) == (lib.CGTP_EDTYPE, None)


def test_plan_unknown_cover():
    assert _plan_rc(4, lib._grid(cover=5)) == (lib.CGTP_EINVAL, None)


def test_plan_negative_grid_sizes():
    assert _plan_rc(4, lib._grid(n_theta=-2)) == (lib.CGTP_EINVAL, None)
    assert _plan_rc(4, lib._grid(n_phi=-1)) == (lib.CGTP_EINVAL, None)


@pytest.mark.parametrize("L", [1, 4, 16, 32])
def test_plan_latitude_grid_below_exactness(L):
    # 2L Gauss-Legendre nodes integrate degree 4L - 1 exactly, one short of the products' 4L
    assert _plan_rc(L, lib._grid(n_theta=2 * L)) == (lib.CGTP_EGRID, None)


@pytest.mark.parametrize("L", [1, 4, 16, 32])
def test_plan_longitude_grid_below_exactness(L):
    # 4L longitudes alias the band-2L products
    assert _plan_rc(L, lib._grid(n_phi=4 * L)) == (lib.CGTP_EGRID, None)


@pytest.mark.parametrize("L", [2, 5, 16])
def test_plan_odd_latitude_grid(L):
    # exact (>= 2L + 1) but odd: the north-south fold needs an even node count
    assert _plan_rc(L, lib._grid(n_theta=2 * L + 3)) == (lib.CGTP_EUNSUP, None)


@pytest.mark.parametrize("L,n_phi", [(3, 13), (4, 17), (5, 21), (16, 65), (32, 129), (32, 160)])
def test_plan_longitude_size_not_2a3b(L, n_phi):
    # 4L + 1 (or anything) that is not 2^a 3^b, or above the largest transform
    assert _plan_rc(L, lib._grid(n_phi=n_phi)) == (lib.CGTP_EUNSUP, None)


def test_plan_null_output_handle():
    assert lib._load().cgtp_plan(3, None, None) == lib.CGTP_EINVAL


def test_forward_null_plan():
    f = lib._load()
    buf = ctypes.create_string_buffer(4096)
    p = ctypes.addressof(buf)
    assert f.cgtp_forward(None, ctypes.c_void_p(p), ctypes.c_void_p(p), ctypes.c_void_p(p + 2048), 1, None) \
        == lib.CGTP_EINVAL
    assert f.cgtp_forward_weighted(None, ctypes.c_void_p(p), ctypes.c_void_p(p), None, ctypes.c_void_p(p + 2048),
                                   1, None, None) == lib.CGTP_EINVAL


def test_destroy_null_is_a_no_op():
    assert lib._load().cgtp_destroy(None) == lib.CGTP_OK


def test_query_and_strerror_edges():
    f = lib._load()
    assert f.cgtp_plan_query(None, None, None, None, None, None) == lib.CGTP_EINVAL
    for code in (lib.CGTP_OK, lib.CGTP_EINVAL, lib.CGTP_EGRID, lib.CGTP_EDTYPE, lib.CGTP_ENOMEM, lib.CGTP_EHIP,
                 lib.CGTP_EUNSUP):
        assert lib.cgtp_strerror(code)
    assert lib.cgtp_strerror(12345)
    assert lib.cgtp_num_outputs(-1) < 0
    assert lib.cgtp_path_offset(3, 1, 1, 3) == -1 and lib.cgtp_path_offset(3, 4, 0, 4) == -1


def test_backward_null_plan_and_workspace_query():
    f = lib._load()
    buf = ctypes.create_string_buffer(8192)
    p = ctypes.addressof(buf)
    v = lambda o: ctypes.c_void_p(p + o)
    assert f.cgtp_backward(None, v(0), v(0), v(256), v(4096), v(4352), 1, v(6144), 1024, None) == lib.CGTP_EINVAL
    assert lib.cgtp_backward_workspace_bytes(None, 10) == -1
