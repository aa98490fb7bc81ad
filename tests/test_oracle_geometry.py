"""Pins of the oracle's stereographic tile coordinates (Sec. 3.3, Eq. 1) -- CPU only.

Each check rests on a fact fixed independently of the oracle's code: closed
forms of the stereographic projection, its conformality, cube-face adjacency and
the grid scales the paper prints (tests/golden/paper_scales.json)."""
import json
import os

import numpy as np
import pytest

from oracle import geometry as G

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_scales.json")
R_EARTH_KM = 6371.0


def test_centre_maps_to_origin():
    # G1: the tile centre itself projects to (0, 0) exactly.
    lat0, lon0 = 0.3, -1.1
    x, y = G.stereographic(np.array(lat0), np.array(lon0), lat0, lon0, 1.0)
    assert x == 0.0 and y == 0.0
    # odd tile: its middle token is the centre -> (0, 0) up to rounding
    c = G.tile_coords([2], [100], [37], 5, 5)
    assert abs(c[0, 2, 2, 0]) < 1e-9 and abs(c[0, 2, 2, 1]) < 1e-9


def test_meridian_closed_form():
    # G2: on the centre's meridian x = 0 and y = 2 tan(dlat/2) / l.
    lat0, lon0, ls = 0.4, 2.0, 7e-4
    dl = np.linspace(-0.2, 0.2, 41)
    x, y = G.stereographic(lat0 + dl, np.full_like(dl, lon0), lat0, lon0, ls)
    assert np.max(np.abs(x)) < 1e-12
    np.testing.assert_allclose(y * ls, 2 * np.tan(dl / 2), rtol=1e-12, atol=1e-15)


def test_equator_closed_form():
    # G3: centre on the equator, points on the equator: x = 2 tan(dlon/2)/l, y = 0.
    dl = np.linspace(-0.3, 0.3, 31)
    x, y = G.stereographic(np.zeros_like(dl), 0.7 + dl, 0.0, 0.7, 1.0)
    np.testing.assert_allclose(x, 2 * np.tan(dl / 2), rtol=1e-12, atol=1e-15)
    assert np.max(np.abs(y)) < 1e-15


def test_radial_distance_is_2tan_half_angle():
    # G4: |(x, y)| l = 2 tan(c/2), with c the great-circle distance (haversine form).
    r = np.random.default_rng(0)
    lat0, lon0 = 0.5, -0.3
    lat = lat0 + r.uniform(-0.3, 0.3, 200)
    lon = lon0 + r.uniform(-0.3, 0.3, 200)
    x, y = G.stereographic(lat, lon, lat0, lon0, 1.0)
    h = np.sin((lat - lat0) / 2) ** 2 + np.cos(lat) * np.cos(lat0) * np.sin((lon - lon0) / 2) ** 2
    c = 2 * np.arcsin(np.sqrt(h))
    np.testing.assert_allclose(np.hypot(x, y), 2 * np.tan(c / 2), rtol=1e-10)


def test_projection_is_conformal():
    # G5: the map (lat, lon) -> (x, y) preserves angles: with metric factors,
    # the Jacobian columns d/dlat and d/(cos(lat) dlon) are orthogonal and equally long.
    r = np.random.default_rng(1)
    lat0, lon0 = -0.6, 1.2
    eps = 1e-6
    for _ in range(20):
        lat = lat0 + r.uniform(-0.2, 0.2)
        lon = lon0 + r.uniform(-0.2, 0.2)
        def f(a, b):
            return np.array(G.stereographic(np.array(a), np.array(b), lat0, lon0, 1.0))
        j_lat = (f(lat + eps, lon) - f(lat - eps, lon)) / (2 * eps)
        j_lon = (f(lat, lon + eps) - f(lat, lon - eps)) / (2 * eps) / np.cos(lat)
        n1, n2 = np.linalg.norm(j_lat), np.linalg.norm(j_lon)
        assert abs(np.dot(j_lat, j_lon)) / (n1 * n2) < 1e-7
        assert abs(n1 / n2 - 1.0) < 1e-7


def test_cube_faces_tile_the_sphere():
    # Face centres point along the six axes, and neighbouring faces share their edges.
    axes = []
    for f in range(6):
        X, Y, Zc = G.cube_point(np.array([f]), np.array([0.0]), np.array([0.0]))
        axes.append(np.array([X[0], Y[0], Zc[0]]))
    A = np.abs(np.stack(axes))
    assert np.all(np.sort(A.sum(0)) == 2.0) and np.all(A.max(1) == 1.0)
    t = np.linspace(-np.pi / 4, np.pi / 4, 17)
    edges = []
    for f in range(6):
        for a, b in ((np.full_like(t, np.pi / 4), t), (np.full_like(t, -np.pi / 4), t),
                     (t, np.full_like(t, np.pi / 4)), (t, np.full_like(t, -np.pi / 4))):
            X, Y, Zc = G.cube_point(np.full(t.shape, f), a, b)
            P = np.stack([X, Y, Zc], 1)
            edges.append((f, np.round(P, 12)))
    # every edge polyline of a face appears (as a point set) on exactly one other face
    for i, (f, P) in enumerate(edges):
        key = set(map(tuple, P))
        partners = [g for j, (g, Q) in enumerate(edges) if j != i and set(map(tuple, Q)) == key]
        assert len(partners) == 1 and partners[0] != f


def test_paper_grid_scales():
    # The paper's printed scales: a 6 x 2048^2 cubed sphere of ~4.9-km cells,
    # 128 x 128-cell tiles ~576 km across, 36 x 36-cell windows ~160 km.
    g = json.load(open(GOLDEN))
    ls = G.l_scale(g["face_cells"])
    assert 6 * g["face_cells"] ** 2 == pytest.approx(g["grid_points"], rel=0.02)
    cell_km = ls * R_EARTH_KM
    assert cell_km == pytest.approx(g["grid_km"], rel=0.1)
    r = np.random.default_rng(2)
    for _ in range(8):
        f = int(r.integers(0, 6))
        T = g["train_tile_cells"] // 4
        oy, ox = (int(v) for v in r.integers(0, 512 - T + 1, 2))
        c = G.tile_coords([f], [oy], [ox], T, T)[0]
        span = np.mean(np.hypot(*(c[:, -1, :] - c[:, 0, :]).T))
        width_km = span * ls * R_EARTH_KM * T / (T - 1)
        assert width_km == pytest.approx(g["train_tile_km"], rel=0.25)
        Wn = g["window_cells"] // 4
        cw = G.tile_coords([f], [oy], [ox], Wn, Wn)[0]
        wspan = np.mean(np.hypot(*(cw[:, -1, :] - cw[:, 0, :]).T))
        wkm = wspan * ls * R_EARTH_KM * Wn / (Wn - 1)
        assert wkm == pytest.approx(g["window_km"], rel=0.3)


def test_tile_frame_axes():
    # x grows eastward and y northward in the tile frame: on face 0 (+X, lon 0 at
    # centre) columns run east and rows run north.
    c = G.tile_coords([0], [200], [200], 16, 16)[0]
    assert np.all(np.diff(c[:, :, 0], axis=1) > 0)
    assert np.all(np.diff(c[:, :, 1], axis=0) > 0)


# ----------------------------------------------------------------------------- wind frame (Eq. 2)

def test_wind_frame_is_identity_at_the_centre():
    r = np.random.default_rng(80)
    lat0, lon0 = 0.3, -1.1
    U, V = r.standard_normal(5), r.standard_normal(5)
    u, v = G.wind_to_tile_frame(U, V, lat0, lon0, lat0, lon0)
    np.testing.assert_allclose(u, U, atol=1e-15)
    np.testing.assert_allclose(v, V, atol=1e-15)


def test_wind_frame_on_the_equator_closed_form():
    # centre and points on the equator: n = n0 = z, e . e0 = cos(dlon)
    r = np.random.default_rng(81)
    lon = r.uniform(-1.2, 1.2, 7)
    U, V = r.standard_normal(7), r.standard_normal(7)
    u, v = G.wind_to_tile_frame(U, V, 0.0, lon, 0.0, 0.4)
    np.testing.assert_allclose(u, U * np.cos(lon - 0.4), atol=1e-14)
    np.testing.assert_allclose(v, V, atol=1e-14)


def test_wind_frame_on_the_centre_meridian_closed_form():
    # same longitude: e = e0, n . n0 = cos(dlat)
    r = np.random.default_rng(82)
    lat = r.uniform(-1.0, 1.0, 7)
    U, V = r.standard_normal(7), r.standard_normal(7)
    u, v = G.wind_to_tile_frame(U, V, lat, 0.7, 0.2, 0.7)
    np.testing.assert_allclose(u, U, atol=1e-14)
    np.testing.assert_allclose(v, V * np.cos(lat - 0.2), atol=1e-14)


def test_wind_frame_keeps_the_tangential_length():
    # U_loc^2 + V_loc^2 = |v|^2 - (v . r0)^2 with |v|^2 = U^2 + V^2
    r = np.random.default_rng(83)
    lat, lon = r.uniform(-1.3, 1.3, 50), r.uniform(-3, 3, 50)
    lat0, lon0 = 0.5, 2.0
    U, V = r.standard_normal(50), r.standard_normal(50)
    u, v = G.wind_to_tile_frame(U, V, lat, lon, lat0, lon0)
    e, n, _ = G.east_north_radial(lat, lon)
    _, _, r0 = G.east_north_radial(lat0, lon0)
    vr = np.sum((U[:, None] * e + V[:, None] * n) * r0, -1)
    np.testing.assert_allclose(u * u + v * v, U * U + V * V - vr * vr, atol=1e-12)


def test_wind_tiles_cut_the_face_and_use_each_tile_centre():
    n = 64
    r = np.random.default_rng(84)
    field = r.standard_normal((2, n, n, 2))
    t = G.wind_tiles(field, 4, n, 2, 3, 16, 12, 40, 20)
    assert t.shape == (6, 2, 16, 12, 2)
    # tile (1, 2): cells (40.., 40..); centre at the mean angles of its first and last cells
    rows, cols = 40 + np.arange(16), 40 + np.arange(12)
    beta, alpha = G.cell_angle(rows, n), G.cell_angle(cols, n)
    lat0, lon0 = G.latlon(4, (alpha[0] + alpha[-1]) / 2, (beta[0] + beta[-1]) / 2)
    lat, lon = G.latlon(4, alpha[5], beta[3])
    u, v = G.wind_to_tile_frame(field[1, 43, 45, 0], field[1, 43, 45, 1], lat, lon, lat0, lon0)
    np.testing.assert_allclose(t[5, 1, 3, 5], [u, v], atol=1e-15)


# ----------------------------------------------------------------------------- Duo-grid padding (App. F)

def test_duo_extended_mesh_continues_the_face():
    # on the face's own plane the extended mesh keeps the angular spacing: a halo
    # cell's point is the cube point at the extended equiangular angles
    p = G.cell_point(0, -1, 5, 16)
    X, Y, Zc = G.cube_point(0, G.cell_angle(5, 16), G.cell_angle(-1, 16))
    np.testing.assert_allclose(p, np.array([X, Y, Zc]) / np.sqrt(X * X + Y * Y + Zc * Zc), atol=1e-15)


@pytest.mark.parametrize("face", range(6))
def test_duo_halo_points_land_on_the_neighbouring_faces(face):
    # a point half a cell beyond an edge lies on the face across that edge, next to it
    n = 16
    for i, j in ((-1, 7), (n, 7), (7, -1), (7, n)):
        fp, rows, cols, w = G.duo_halo_neighbours(face, i, j, n)
        assert fp != face
        assert np.isclose(w.sum(), 1.0) and np.all(w >= 0)
        on_edge = (rows.min() == 0) or (rows.max() == n - 1) or (cols.min() == 0) or (cols.max() == n - 1)
        assert on_edge


@pytest.mark.parametrize("face", range(6))
def test_duo_points_on_an_edge_belong_to_the_lower_face_at_equal_distances(face):
    # halo cells on the diagonal beyond a face corner project onto the edge
    # shared by the two faces across that corner: both faces contain the point,
    # their 4 nearest cells are mirror images at the same distances, and the
    # lower-numbered face is taken
    n = 20
    normals = np.array([G.FACE_AXES[g][0] for g in range(6)], dtype=np.float64)
    for k in range(3):
        for i, j in ((-1 - k, -1 - k), (-1 - k, n + k), (n + k, -1 - k), (n + k, n + k)):
            p = G.cell_point(face, i, j, n)
            s = normals @ p
            both = np.flatnonzero(s > s.max() - 1e-12)
            assert len(both) == 2 and face not in both
            fp, _, _, _ = G.duo_halo_neighbours(face, i, j, n)
            assert fp == both.min()
            dists = []
            for g in both:
                I, J = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
                c = G.cell_point(np.full(I.shape, g), I, J, n).reshape(-1, 3)
                dists.append(np.sort(np.arccos(np.clip(c @ p, -1, 1)))[:4])
            np.testing.assert_allclose(dists[0], dists[1], atol=1e-7)


def test_duo_nearest_cells_lie_in_the_lattice_block_around_the_point():
    # the four nearest cells of the containing face always lie within the 6 x 6
    # block of its cell lattice around the point's (clamped) floor index: a
    # local search finds them
    for n, h in ((16, 4), (17, 3), (20, 3), (32, 8), (48, 6)):
        for f in range(6):
            for i in range(-h, n + h):
                for j in range(-h, n + h):
                    if 0 <= i < n and 0 <= j < n:
                        continue
                    fp, rows, cols, _ = G.duo_halo_neighbours(f, i, j, n)
                    nrm, right, up = (np.asarray(v, dtype=np.float64) for v in G.FACE_AXES[fp])
                    p = G.cell_point(f, i, j, n)
                    step = (np.pi / 2) / n
                    u = (np.arctan((p @ right) / (p @ nrm)) + np.pi / 4) / step - 0.5
                    v = (np.arctan((p @ up) / (p @ nrm)) + np.pi / 4) / step - 0.5
                    j0 = min(max(int(np.floor(u)), 0), n - 2)
                    i0 = min(max(int(np.floor(v)), 0), n - 2)
                    r0, c0 = min(max(i0 - 2, 0), n - 6), min(max(j0 - 2, 0), n - 6)
                    assert np.all((rows >= r0) & (rows < r0 + 6) & (cols >= c0) & (cols < c0 + 6)), (n, f, i, j)


def test_duo_pad_copies_the_interior_and_keeps_constants():
    n, h = 8, 2
    r = np.random.default_rng(86)
    field = r.standard_normal((6, 2, n, n, 3))
    out = G.duo_pad(field, h)
    np.testing.assert_array_equal(out[:, :, h:h + n, h:h + n], field)
    const = G.duo_pad(np.full((6, 1, n, n, 1), 2.5), h)
    np.testing.assert_allclose(const, 2.5, atol=1e-14)


def test_duo_pad_continues_a_smooth_field():
    # f(p) = p . g sampled at the cell centres of all faces: the halo holds f at the
    # halo point to within the inverse-distance interpolation error (<= the
    # largest neighbour distance times |g|), an O(1) error for a wrong face or
    # orientation
    n, h = 24, 3
    g = np.array([0.3, -1.1, 0.7])
    field = np.empty((6, 1, n, n, 1))
    I, J = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    for f in range(6):
        field[f, 0, :, :, 0] = G.cell_point(np.full(I.shape, f), I, J, n) @ g
    out = G.duo_pad(field, h)
    step = (np.pi / 2) / n
    m = n + 2 * h
    for f in range(6):
        Ip, Jp = np.meshgrid(np.arange(m) - h, np.arange(m) - h, indexing="ij")
        exact = G.cell_point(np.full(Ip.shape, f), Ip, Jp, n) @ g
        assert np.max(np.abs(out[f, 0, :, :, 0] - exact)) <= 2.0 * step * np.linalg.norm(g)


def test_duo_pad_vjp_is_the_adjoint_of_the_padding():
    # <P x, y> = <x, P^T y> for arbitrary x, y: a dropped term, a wrong weight
    # or a misplaced source cell breaks the identity
    rng = np.random.default_rng(5)
    n, h, P, C = 16, 4, 2, 3
    m = n + 2 * h
    x = rng.standard_normal((6, P, n, n, C))
    y = rng.standard_normal((6, P, m, m, C))
    lhs = float(np.sum(G.duo_pad(x, h) * y))
    rhs = float(np.sum(x * G.duo_pad_vjp(y, h)))
    assert abs(lhs - rhs) <= 1e-12 * (abs(lhs) + np.sum(np.abs(x)) * 1.0)


def test_duo_pad_vjp_conserves_the_total_and_copies_the_interior():
    n, h, P, C = 20, 3, 1, 2
    m = n + 2 * h
    # every halo cell's weights sum to 1: the total of P^T 1 counts every padded cell once
    ones = G.duo_pad_vjp(np.ones((6, P, m, m, C)), h)
    assert np.isclose(ones.sum(), 6 * P * C * m * m, rtol=1e-13)
    # no halo gradient: the interior is returned unchanged
    rng = np.random.default_rng(6)
    g = np.zeros((6, P, m, m, C))
    g[:, :, h:h + n, h:h + n] = rng.standard_normal((6, P, n, n, C))
    assert np.array_equal(G.duo_pad_vjp(g, h), g[:, :, h:h + n, h:h + n])
    # cells far from every edge receive no halo gradient
    inner = ones[:, :, h + 3:n - h - 3, h + 3:n - h - 3]
    assert np.array_equal(inner, np.ones_like(inner))
