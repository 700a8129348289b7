"""Reading a locality layout back from device memory, in the order the
library lays it out, and checking its sliced copy against P (shared by the
2-D and 3-D layout tests)."""
import numpy as np
import scipy.sparse as sp

TILE_ROWS, TILE_SEG, ITEM_MAX_TILES = 1024, 16384, 128
# tiles a row block may span (fp32 2-D: 16 always, up to 128 when the tiles are
# dense) and partial slots per row (so at most 32 tiles per row block on average)
TILE_MAX_SEG, TILE_NARROW_SEG, TILE_SLOTS, TILE_WIDE_ENTRIES = 128, 16, 32, 4096
SLICE, SLICES, CHUNK = 64, 16, 256  # rows per unit, units per tile, entries per chunk


def layout_arrays(lay, tiles=False, max_seg=None, narrow=None):
    """perm, rank, row_ptr, col, val of a layout (and the tile tables), read back
    from device memory in the order the library lays them out."""
    n, nnz = lay.n, lay.nnz
    mem = lay.mem.cpu().numpy()
    off = 0

    def take(nbytes, dtype, count):
        nonlocal off
        a = mem[off:off + nbytes].view(dtype)[:count]
        off = (off + nbytes + 255) // 256 * 256
        return a

    cap = nnz + 3 * n + 4  # rows padded to 4-entry vectors, plus a sentinel vector
    perm = take(4 * n, np.uint32, n)
    rank = take(4 * n, np.uint32, n)
    rp = take(8 * (n + 1), np.int64, n + 1)
    col = take(4 * cap, np.int32, cap)
    val = take(4 * cap, np.float32, cap)
    if not tiles:
        return perm, rank, rp, col, val
    max_seg = TILE_MAX_SEG if max_seg is None else max_seg
    narrow = TILE_NARROW_SEG if narrow is None else narrow
    blocks = (n + TILE_ROWS - 1) // TILE_ROWS
    max_tiles = blocks * TILE_SLOTS
    max_units = max_tiles * SLICES
    max_entries = nnz + nnz // 4 + CHUNK * SLICES * blocks * narrow + CHUNK
    t = dict(seg_lo=take(4 * blocks, np.int32, blocks), nseg=take(4 * blocks, np.int32, blocks))
    t["blk_tiles"] = take(4 * blocks * max_seg, np.int32, blocks * max_seg).reshape(blocks, max_seg)
    for k in ("tile_blk", "tile_seg", "tile_k"):
        t[k] = take(4 * max_tiles, np.int32, max_tiles)
    t["item_tiles"] = take(8 * max_tiles, np.int32, 2 * max_tiles).reshape(max_tiles, 2)
    t["run_len"] = take(4 * max_tiles * TILE_ROWS, np.int32, max_tiles * TILE_ROWS)
    t["tperm"] = take(2 * max_tiles * TILE_ROWS, np.uint16, max_tiles * TILE_ROWS)
    t["tpos"] = take(2 * max_tiles * TILE_ROWS, np.uint16, max_tiles * TILE_ROWS)
    for k in ("unit_of", "unit_chunks", "unit_tj", "unit_chunk0"):
        t[k] = take(4 * max_units, np.int32, max_units)
    t["item_units"] = take(16 * max_tiles, np.int32, 4 * max_tiles).reshape(max_tiles, 4)
    t["wave_units"] = take(16 * max_tiles * 16, np.int32, 4 * 16 * max_tiles).reshape(max_tiles, 16, 4)
    t["tcol"] = take(2 * max_entries, np.uint16, max_entries)
    t["tval"] = take(4 * max_entries, np.float32, max_entries)
    return (perm, rank, rp, col, val), t


def check_sliced_copy(lay, row_ptr, col_in, val_in, seg=TILE_SEG, max_seg=TILE_MAX_SEG, narrow=TILE_NARROW_SEG):
    """The tile tables of a tiled layout are consistent and its sliced copy
    (columns as offsets in windows of `seg` points) holds exactly P, relabelled.
    max_seg: tiles a row block may span; narrow: the span whose tiles bound the
    padding."""
    n = lay.n
    (perm, rank, rp, col, val), tt = layout_arrays(lay, tiles=True, max_seg=max_seg, narrow=narrow)
    T, I = lay.tiles, lay.items
    seg_lo, nseg, tile_blk, tile_seg = (tt[k] for k in ("seg_lo", "nseg", "tile_blk", "tile_seg"))
    blocks = (n + TILE_ROWS - 1) // TILE_ROWS
    # tiles: every (block, segment) pair once, segment-major, indexed both ways
    assert T == int(nseg[:blocks].sum()) and 0 < I <= T
    pairs = list(zip(tile_seg[:T].tolist(), tile_blk[:T].tolist()))
    assert pairs == sorted(pairs) and len(set(pairs)) == T
    for t in range(T):
        b = tile_blk[t]
        k = tile_seg[t] - seg_lo[b]
        assert 0 <= k < nseg[b] and tt["tile_k"][t] == k and tt["blk_tiles"][b, k] == t
    # rows of a tile sorted by decreasing run length, tperm and tpos inverse
    tperm = tt["tperm"][:T * TILE_ROWS].reshape(T, TILE_ROWS).astype(np.int64)
    tpos = tt["tpos"][:T * TILE_ROWS].reshape(T, TILE_ROWS).astype(np.int64)
    rlen = tt["run_len"][:T * TILE_ROWS].reshape(T, TILE_ROWS)
    for t in range(T):
        assert np.array_equal(np.sort(tperm[t]), np.arange(TILE_ROWS))
        assert np.array_equal(tpos[t][tperm[t]], np.arange(TILE_ROWS))
        assert np.all(np.diff(rlen[t][tperm[t]]) <= 0)
    # items: runs of tiles of one segment covering every tile once (stored
    # largest first); their units are every slice once, the ones with chunks
    # split among 16 waves whose chunks are contiguous
    itr = tt["item_tiles"][:I]
    assert np.all(itr[:, 1] > itr[:, 0]) and np.all(itr[:, 1] - itr[:, 0] <= ITEM_MAX_TILES)
    srt = itr[np.argsort(itr[:, 0])]
    assert srt[0, 0] == 0 and srt[-1, 1] == T and np.array_equal(srt[1:, 0], srt[:-1, 1])
    iu, wu = tt["item_units"][:I], tt["wave_units"][:I]
    uk, uj, uc = tt["unit_chunks"], tt["unit_tj"], tt["unit_chunk0"]
    assert iu[0, 0] == 0 and iu[-1, 2] == T * SLICES
    seen = np.zeros(T * SLICES, bool)
    chunk = 0
    for i in range(I):
        assert len(set(tile_seg[itr[i, 0]:itr[i, 1]].tolist())) == 1
        assert iu[i, 0] == (iu[i - 1, 2] if i else 0) and iu[i, 0] <= iu[i, 1] <= iu[i, 2]
        assert iu[i, 2] - iu[i, 0] == SLICES * (itr[i, 1] - itr[i, 0])
        for w in range(16):
            x, y, z, g = wu[i, w]
            assert x == (wu[i, w - 1, 1] if w else iu[i, 0]) and y >= x
            if y > x:
                assert z == chunk and g == int(uk[x:y].sum()) and np.all(uk[x:y] > 0)
                assert np.array_equal(uc[x:y], z + np.concatenate([[0], np.cumsum(uk[x:y])[:-1]]))
                chunk += g
        assert wu[i, 15, 1] == iu[i, 1] and np.all(uk[iu[i, 1]:iu[i, 2]] == 0)
        for d in range(iu[i, 0], iu[i, 2]):
            tj = uj[d]
            assert itr[i, 0] <= tj // SLICES < itr[i, 1] and not seen[tj] and tt["unit_of"][tj] == d
            seen[tj] = True
            t, j = divmod(int(tj), SLICES)
            assert uk[d] == (int(rlen[t][tperm[t][j * SLICE]]) + 3) // 4
    assert seen.all()
    assert lay.entries == chunk * CHUNK
    cost = [int(uk[iu[i, 0]:iu[i, 2]].sum()) for i in range(I)]
    assert cost == sorted(cost, reverse=True)  # largest item first
    # the sliced copy holds exactly P (padding carries zero values)
    rows_l, cols_l, vals_l = [], [], []
    tcol, tval = tt["tcol"], tt["tval"]
    lanes = np.arange(SLICE)
    for d in range(T * SLICES):
        if uk[d] == 0:
            continue
        t, j = divmod(int(uj[d]), SLICES)
        rows = tile_blk[t] * TILE_ROWS + tperm[t][j * SLICE + lanes]
        idx = (uc[d] + np.arange(uk[d]))[:, None, None] * CHUNK + lanes[None, :, None] * 4 + np.arange(4)[None, None, :]
        rows_l.append(np.broadcast_to(rows[None, :, None], idx.shape).ravel())
        cols_l.append(tcol[idx].astype(np.int64).ravel() + tile_seg[t] * seg)
        vals_l.append(tval[idx].ravel())
    rows_a, cols_a, vals_a = map(np.concatenate, (rows_l, cols_l, vals_l))
    keep = vals_a != 0
    assert np.all(rows_a[keep] < n)
    Pt = sp.csr_matrix((vals_a[keep], (rows_a[keep], cols_a[keep])), shape=(n, n))
    Po = sp.csr_matrix((val_in, col_in, row_ptr), shape=(n, n))
    ref = Po[perm.astype(np.int64)][:, perm.astype(np.int64)]
    assert abs(Pt - ref).max() == 0.0 and Pt.nnz == len(col_in)


def bfs_perm(rp, col, n):
    """The order (component, breadth-first level from the component's smallest
    point along P's rows, index), from scipy's graph routines."""
    import scipy.sparse.csgraph as cg
    A = sp.csr_matrix((np.ones(col.size), col, rp), shape=(n, n))
    nc, lab = cg.connected_components(A, directed=False)
    root = np.full(nc, n, np.int64)
    np.minimum.at(root, lab, np.arange(n))
    level = np.full(n, -1, np.int64)
    for r in root:
        order, pred = cg.breadth_first_order(A, int(r), directed=True, return_predecessors=True)
        level[r] = 0
        for v in order[1:]:  # breadth-first: a predecessor's level is set before its children's
            level[v] = level[pred[v]] + 1
    assert np.all(level >= 0)
    return np.lexsort((np.arange(n), level, root[lab])).astype(np.uint32)
