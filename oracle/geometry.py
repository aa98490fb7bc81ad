"""Oracle: stereographic tile coordinates (test infrastructure, CPU only, float64).

This is the plain reference the HIP path is checked against; only tests, the
smoke check and the bench's CPU-baseline leg may use it.

Follows the paper's section on grid-invariant position encoding (Eq. 1): each
token's (lat, lon) is projected onto the tangent plane of a stereographic
projection centred on its tile, and the result divided by
l_scale = sqrt(4 pi / N_total).

Readings where the paper is silent (stated once here, listed in the design notes):
* equiangular cube: cell (i, j) of an n x n face has angles
  alpha = -pi/4 + (j + 1/2) (pi/2)/n (columns, x direction) and beta likewise from
  the row i (y direction); a token of a p x p patch (I, J) sits at the patch centre,
  alpha = -pi/4 + (p J + p/2)(pi/2)/n;
* face orientation, with a = tan(alpha), b = tan(beta):
  0: (1, a, b)   1: (-a, 1, b)   2: (-1, -a, b)   3: (a, -1, b)
  4: (-b, a, 1)  (north)          5: (b, a, -1)    (south);
* the tile centre is the point at the mean of the angles of the tile's first and
  last token on each axis;
* N_total counts native horizontal cells: 6 n^2.
"""
from __future__ import annotations

import numpy as np


def l_scale(n_cells: int = 2048) -> float:
    """Eq. 1 normaliser sqrt(4 pi / N_total) with N_total = 6 n^2 native cells."""
    return float(np.sqrt(4.0 * np.pi / (6.0 * n_cells * n_cells)))


def cube_point(face, alpha, beta):
    """Unnormalised point on the cube surface for equiangular angles (alpha, beta)."""
    face = np.asarray(face)
    a = np.tan(np.asarray(alpha, dtype=np.float64))
    b = np.tan(np.asarray(beta, dtype=np.float64))
    one = np.ones(np.broadcast(face, a, b).shape)
    a = a * one
    b = b * one
    face = face * np.ones(one.shape, dtype=np.int64)
    X = np.empty(one.shape)
    Y = np.empty(one.shape)
    Zc = np.empty(one.shape)
    table = {
        0: (one, a, b),
        1: (-a, one, b),
        2: (-one, -a, b),
        3: (a, -one, b),
        4: (-b, a, one),
        5: (b, a, -one),
    }
    for f, (x, y, z) in table.items():
        m = face == f
        X[m], Y[m], Zc[m] = x[m], y[m], z[m]
    return X, Y, Zc


def latlon(face, alpha, beta):
    """(lat, lon) in radians of the cube point for (face, alpha, beta)."""
    X, Y, Zc = cube_point(face, alpha, beta)
    lat = np.arctan2(Zc, np.hypot(X, Y))
    lon = np.arctan2(Y, X)
    return lat, lon


def token_angle(index, n_cells: int = 2048, patch: int = 4):
    """Equiangular angle of the centre of patch ``index`` along one face axis."""
    return -np.pi / 4 + (patch * np.asarray(index, dtype=np.float64) + patch / 2.0) * (np.pi / 2) / n_cells


def stereographic(lat, lon, lat0, lon0, lscale):
    """Eq. 1: tile-centred stereographic (x, y), divided by l_scale."""
    dl = lon - lon0
    cos_c = np.sin(lat0) * np.sin(lat) + np.cos(lat0) * np.cos(lat) * np.cos(dl)
    k = 2.0 / (1.0 + cos_c)
    x = (k / lscale) * np.cos(lat) * np.sin(dl)
    y = (k / lscale) * (np.cos(lat0) * np.sin(lat) - np.sin(lat0) * np.cos(lat) * np.cos(dl))
    return x, y


def tile_coords(face, oy, ox, H: int, W: int, n_cells: int = 2048, patch: int = 4,
                lscale: float | None = None) -> np.ndarray:
    """Stereographic coordinates coords[B, H, W, 2] (x, y) in float64 for tiles of H x W tokens.

    face/oy/ox: per-tile cube face and token origin (row, column)."""
    if lscale is None:
        lscale = l_scale(n_cells)
    face = np.asarray(face, dtype=np.int64)
    oy = np.asarray(oy, dtype=np.int64)
    ox = np.asarray(ox, dtype=np.int64)
    B = face.shape[0]
    out = np.empty((B, H, W, 2), dtype=np.float64)
    I = np.arange(H)
    J = np.arange(W)
    for t in range(B):
        beta = token_angle(oy[t] + I, n_cells, patch)       # rows
        alpha = token_angle(ox[t] + J, n_cells, patch)      # columns
        beta0 = 0.5 * (beta[0] + beta[-1])
        alpha0 = 0.5 * (alpha[0] + alpha[-1])
        lat0, lon0 = latlon(face[t], alpha0, beta0)
        A, Bt = np.meshgrid(alpha, beta, indexing="xy")      # [H, W]
        lat, lon = latlon(np.full(A.shape, face[t]), A, Bt)
        x, y = stereographic(lat, lon, lat0, lon0, lscale)
        out[t, :, :, 0] = x
        out[t, :, :, 1] = y
    return out


# ----------------------------------------------------------------------------- wind frame (Eq. 2)

def east_north_radial(lat, lon):
    """Unit vectors (e_hat, n_hat, r_hat) of the local East-North frame at (lat, lon), [..., 3]."""
    lat, lon = np.broadcast_arrays(np.asarray(lat, dtype=np.float64), np.asarray(lon, dtype=np.float64))
    e = np.stack([-np.sin(lon), np.cos(lon), np.zeros_like(lon)], -1)
    n = np.stack([-np.sin(lat) * np.cos(lon), -np.sin(lat) * np.sin(lon), np.cos(lat)], -1)
    r = np.stack([np.cos(lat) * np.cos(lon), np.cos(lat) * np.sin(lon), np.sin(lat)], -1)
    return e, n, r


def wind_to_tile_frame(U, V, lat, lon, lat0, lon0):
    """Eq. 2: v = U e + V n at (lat, lon); v_perp = v - (v . r0) r0 on the tangent
    plane of the tile centre (lat0, lon0); U_loc = v_perp . e0, V_loc = v_perp . n0.
    Reading: at a pole the frame is the formula's at the computed longitude."""
    e, n, _ = east_north_radial(lat, lon)
    e0, n0, r0 = east_north_radial(lat0, lon0)
    v = np.asarray(U, dtype=np.float64)[..., None] * e + np.asarray(V, dtype=np.float64)[..., None] * n
    vr = np.sum(v * r0, -1)
    vp = v - vr[..., None] * r0
    return np.sum(vp * e0, -1), np.sum(vp * n0, -1)


def cell_angle(index, n_cells: int = 2048):
    """Equiangular angle of the centre of cell ``index`` along one face axis."""
    return -np.pi / 4 + (np.asarray(index, dtype=np.float64) + 0.5) * (np.pi / 2) / n_cells


def wind_tiles(field, face: int, n_cells: int, nty: int, ntx: int, Ht: int, Wt: int, stride_y: int,
               stride_x: int) -> np.ndarray:
    """Tiles of a face's wind field in each tile's centre frame.

    field: [P, n_cells, n_cells, 2] float64 (U, V per cell of face ``face``);
    tile t = a * ntx + b covers cells (a stride_y + i, b stride_x + j), i < Ht,
    j < Wt; its centre is the point at the mean angles of its first and last
    cell on each axis.  Returns [nty * ntx, P, Ht, Wt, 2] float64."""
    field = np.asarray(field, dtype=np.float64)
    P = field.shape[0]
    out = np.empty((nty * ntx, P, Ht, Wt, 2))
    for a in range(nty):
        for b in range(ntx):
            rows = a * stride_y + np.arange(Ht)
            cols = b * stride_x + np.arange(Wt)
            beta, alpha = cell_angle(rows, n_cells), cell_angle(cols, n_cells)
            lat0, lon0 = latlon(face, 0.5 * (alpha[0] + alpha[-1]), 0.5 * (beta[0] + beta[-1]))
            A, Bt = np.meshgrid(alpha, beta, indexing="xy")
            lat, lon = latlon(np.full(A.shape, face), A, Bt)
            sub = field[:, rows[0]:rows[-1] + 1, cols[0]:cols[-1] + 1, :]
            u, v = wind_to_tile_frame(sub[..., 0], sub[..., 1], lat, lon, lat0, lon0)
            out[a * ntx + b, ..., 0] = u
            out[a * ntx + b, ..., 1] = v
    return out


# ----------------------------------------------------------------------------- KBD blend window (App. F)

def kbd_taper(overlap: int, beta: float) -> np.ndarray:
    """Rising half of the Kaiser-Bessel-derived window of length 2 * overlap:
    k[j] = I0(beta sqrt(1 - (2 j / overlap - 1)^2)), j = 0..overlap (the Kaiser
    window of length overlap + 1), w[n] = sqrt(sum_{j<=n} k[j] / sum_j k[j]),
    n = 0..overlap-1."""
    j = np.arange(overlap + 1, dtype=np.float64)
    k = np.i0(beta * np.sqrt(np.clip(1.0 - (2.0 * j / overlap - 1.0) ** 2, 0.0, None)))
    c = np.cumsum(k)
    return np.sqrt(c[:-1] / c[-1])


def kbd_window_2d(Ht: int, Wt: int, overlap: int, beta: float) -> np.ndarray:
    """Blend window [Ht * Wt]: per axis 1 in the interior and the KBD taper over
    ``overlap`` cells at each end (mirrored at the far end); the 2D window is the
    product of the two axes.  Reading: the taper spans the overlap, as the
    linear ramp does."""
    def axis(L):
        w = np.ones(L)
        t = kbd_taper(overlap, beta)
        w[:overlap] = np.minimum(w[:overlap], t)
        w[L - overlap:] = np.minimum(w[L - overlap:], t[::-1])
        return w
    return np.outer(axis(Ht), axis(Wt)).reshape(-1)


# ----------------------------------------------------------------------------- Duo-grid halo padding (App. F)

# Face axes: a point of face f is normal + a * right + b * up with a = tan(alpha)
# (columns) and b = tan(beta) (rows), the orientation table above.
FACE_AXES = {
    0: ((1, 0, 0), (0, 1, 0), (0, 0, 1)),
    1: ((0, 1, 0), (-1, 0, 0), (0, 0, 1)),
    2: ((-1, 0, 0), (0, -1, 0), (0, 0, 1)),
    3: ((0, -1, 0), (1, 0, 0), (0, 0, 1)),
    4: ((0, 0, 1), (0, 1, 0), (-1, 0, 0)),
    5: ((0, 0, -1), (0, 1, 0), (1, 0, 0)),
}


def _unit(v):
    v = np.asarray(v, dtype=np.float64)
    return v / np.linalg.norm(v, axis=-1, keepdims=True)


def cell_point(face, i, j, n_cells):
    """Unit sphere point of cell (row i, column j) of a face; indices may lie
    beyond [0, n) (the face's equiangular mesh extended on its own plane)."""
    X, Y, Zc = cube_point(face, cell_angle(j, n_cells), cell_angle(i, n_cells))
    return _unit(np.stack([X, Y, Zc], -1))


DUO_TIE = 1e-12  # face scores and distances are compared on this grid; equal ones by index


def duo_halo_neighbours(face, i, j, n_cells):
    """For the (extended) cell (i, j) of ``face``: the face f' containing its
    sphere point p (the axis of p's largest component; a point on an edge or
    corner, where components are equal on the 1e-12 grid, belongs to the
    lowest-numbered of its faces), the 4 cells of f' nearest to p (great-circle distance; distances equal on a 1e-12-radian grid
    ordered by row, then column), and their inverse-distance weights
    normalised to sum 1 (a cell at distance 0 takes weight 1).
    Returns (f', rows[4], cols[4], weights[4]), nearest first."""
    p = cell_point(face, i, j, n_cells)
    normals = np.array([FACE_AXES[f][0] for f in range(6)], dtype=np.float64)
    fp = int(np.argmax(np.round((normals @ p) / DUO_TIE).astype(np.int64)))
    I, J = np.meshgrid(np.arange(n_cells), np.arange(n_cells), indexing="ij")
    c = cell_point(np.full(I.shape, fp), I, J, n_cells).reshape(-1, 3)
    d = np.arctan2(np.linalg.norm(np.cross(c, p), axis=-1), c @ p)
    key = np.round(d / DUO_TIE).astype(np.int64)
    order = np.lexsort((J.reshape(-1), I.reshape(-1), key))[:4]
    rows, cols, dist = I.reshape(-1)[order], J.reshape(-1)[order], d[order]
    if dist[0] == 0.0:
        w = np.array([1.0, 0.0, 0.0, 0.0])
    else:
        w = 1.0 / dist
        w = w / w.sum()
    return fp, rows, cols, w


def duo_pad(field, halo: int) -> np.ndarray:
    """Duo-grid padding of all six faces: field [6, P, n, n, C] -> [6, P, n + 2h,
    n + 2h, C].  Interior cells are copied; every halo cell of face f extends
    f's equiangular mesh on its own plane, is projected to the sphere and takes
    the inverse-distance-weighted values of the 4 nearest cells of the face that
    contains it (summed nearest first)."""
    field = np.asarray(field, dtype=np.float64)
    _, P, n, _, C = field.shape
    m = n + 2 * halo
    out = np.empty((6, P, m, m, C))
    for f in range(6):
        out[f, :, halo:halo + n, halo:halo + n] = field[f]
        for ip in range(m):
            for jp in range(m):
                i, j = ip - halo, jp - halo
                if 0 <= i < n and 0 <= j < n:
                    continue
                fp, rows, cols, w = duo_halo_neighbours(f, i, j, n)
                acc = np.zeros((P, C))
                for k in range(4):
                    acc = acc + w[k] * field[fp, :, rows[k], cols[k]]
                out[f, :, ip, jp] = acc
    return out


def duo_pad_vjp(grad_padded, halo: int) -> np.ndarray:
    """Adjoint of the padding (the vector-Jacobian product of ``duo_pad``; App. F:
    P is a fixed sparse matrix, so gradients reach the faces through its
    transpose).  grad_padded [6, P, n + 2h, n + 2h, C] -> [6, P, n, n, C]: each
    face's interior gradient, plus, for every halo cell, its gradient times each
    of its 4 weights added to the source cell that weight belongs to."""
    g = np.asarray(grad_padded, dtype=np.float64)
    _, P, m, _, C = g.shape
    n = m - 2 * halo
    out = g[:, :, halo:halo + n, halo:halo + n].copy()
    for f in range(6):
        for ip in range(m):
            for jp in range(m):
                i, j = ip - halo, jp - halo
                if 0 <= i < n and 0 <= j < n:
                    continue
                fp, rows, cols, w = duo_halo_neighbours(f, i, j, n)
                for k in range(4):
                    out[fp, :, rows[k], cols[k]] += w[k] * g[f, :, ip, jp]
    return out
