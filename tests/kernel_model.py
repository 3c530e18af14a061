"""Bounds-checked CPU model of the atomic backward's addressing (test infrastructure).

The atomic grad_value variant of the backward kernel (grad_value accumulated with fp32 buffer
atomics, Sec. 4.2's scatter-add done directly) is replayed here on the CPU exactly as the host
code launches it and as each lane forms its addresses:

  * the host's batch split (largest batch count per launch that keeps element offsets below
    2^29) and the launch geometry (channels per lane, lanes per query, queries per wave, grid
    padded to a multiple of 8);
  * the workgroup -> (batch, head, query chunk) arrangement over the eight XCDs: query eighths
    (XCD x takes the x-th eighth of every slab's query chunks) when there are at least half as many
    queries as value pixels, else slab ranges (XCD x takes a contiguous eighth of the slab-major
    work items); with as many queries as value pixels the eighths are bands of rows (XCD x takes
    the chunks whose first query lies in the x-th eighth of the rows of its level);
  * the sample split of small grids: a query chunk's K samples divided over up to 8 consecutive
    work items (at least 4 samples each, at most 4096 waves in all);
  * the per-sample description: fp32 image coordinates, the open range test, floor, the int32
    element offset of each corner row, and the out-of-range sentinel (2^29 elements) for corners
    off the map, samples off the map and queries past Lq;
  * every value-row load, grad_out read and grad_value atomic of every lane, with the buffer
    resource's range rule (an access whose byte range ends past the resource's size returns 0 /
    is dropped).

Each access is checked: in-range accesses address a whole row of the right (batch, pixel, head)
inside the launch's buffers, and every dropped access is one the definition says contributes
nothing. The atomics that land are then summed in fp64 and compared with the oracle. The model
imports neither the GPU library nor the oracle; the tests do the comparison.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

MAX_LAUNCH_ELEMS = 1 << 29  # per-launch element limit; also the off-map sentinel offset
MAX_INDEX = (1 << 31) - 1
WAVES_PER_BLOCK = 4
SMALL_GRID = 1024        # below this many four-wave workgroups, workgroups of one wave are launched
ATOMIC_ROW_FLOATS = 512  # grad_out floats of one wave staged for the row-coalesced atomics
K_SPLIT_MAX = 8          # most parts the backward splits a query chunk's samples into ...
K_SPLIT_MIN_SAMPLES = 4  # ... keeping at least this many samples per part ...
K_SPLIT_WAVES = 4096     # ... while the grid stays within this many waves
U32 = 1 << 32


def pick_vec(D: int, es: int) -> int:
    """Channels per lane: the widest row piece (<= 16 bytes) that divides D."""
    v = 16 // es
    while v > 1:
        if D % v == 0:
            return v
        v >>= 1
    return 1


def pick_lpp(D: int, vec: int) -> int:
    """Lanes per query: enough VEC-wide pieces to cover D, rounded up to a power of two (<= 64)."""
    need = (D + vec - 1) // vec
    lpp = 1
    while lpp < need and lpp < 64:
        lpp <<= 1
    return lpp


def batch_per_launch(S, M, D, Lq, L, P) -> int:
    nb = (MAX_LAUNCH_ELEMS - 1) // (S * M * D)
    per_q = Lq * M * max(L * P * 2, D)
    if per_q > 0 and MAX_INDEX // per_q < nb:
        nb = MAX_INDEX // per_q
    return max(nb, 1)


def fmaf32(x: np.ndarray, s: int, c: float) -> np.ndarray:
    """fp32 fma(x, s, c) with one rounding: x (fp32) * s (an integer below 2^24) is exact in the
    64-bit significand of long double, and so is the sum with c = -0.5 for every |x*s| >= 2^-30;
    below that both sides round to -0.5f."""
    r = x.astype(np.longdouble) * np.longdouble(s) + np.longdouble(c)
    return r.astype(np.float32)


@dataclass
class Launch:
    n0: int
    cnt: int
    vec: int
    lpp: int
    ppw: int
    waves: int
    q_per_block: int
    chunks: int
    num_blocks: int
    grid: int
    split: bool
    k_split: int
    bands: bool = False
    band_c: tuple = ()      # band_c[l][x]: first chunk of level l in band x (x = 0..8)
    band_count: tuple = ()  # chunks of one slab in band x
    band_cap: int = 0


class AddressError(AssertionError):
    pass


def band_table(shapes, qpb):
    """Chunk ranges of the bands of rows: row h of level l is in band floor(8 (h + 1/2) / H_l), and a
    query chunk goes with the band of its first query (query q is pixel q in level-major order)."""
    first_chunk = lambda q: (q + qpb - 1) // qpb
    start, bc = 0, []
    for H, W in shapes:
        row = []
        for x in range(8):
            r0 = max(0, -(-(x * H - 4) // 8))  # first row with 8 h + 4 >= x H
            row.append(first_chunk(start + r0 * W))
        start += H * W
        row.append(first_chunk(start))
        bc.append(tuple(row))
    count = tuple(sum(r[x + 1] - r[x] for r in bc) for x in range(8))
    return tuple(bc), count, max(count)


def launches(N, S, M, D, Lq, L, P, es, shapes=None):
    """The launches of the backward kernel; `shapes` ((H, W) per level) is needed where Lq == S."""
    nb = batch_per_launch(S, M, D, Lq, L, P)
    vec = pick_vec(D, es)
    lpp = pick_lpp(D, vec)
    ppw = 64 // lpp
    out = []
    for n0 in range(0, N, nb):
        cnt = min(nb, N - n0)
        chunks4 = (Lq + WAVES_PER_BLOCK * ppw - 1) // (WAVES_PER_BLOCK * ppw)
        waves = 1 if cnt * M * chunks4 < SMALL_GRID else WAVES_PER_BLOCK
        qpb = waves * ppw
        qchunks = (Lq + qpb - 1) // qpb
        ks = 1
        while (2 * ks <= K_SPLIT_MAX and 2 * ks * K_SPLIT_MIN_SAMPLES <= L * P and
               cnt * M * qchunks * waves * 2 * ks <= K_SPLIT_WAVES):
            ks *= 2
        chunks = qchunks * ks
        num_blocks = cnt * M * chunks
        split_grid = 8 * cnt * M * ((chunks + 7) // 8)
        split = 2 * Lq >= S and split_grid <= MAX_INDEX
        grid = split_grid if split else (num_blocks + 7) // 8 * 8
        ln = Launch(n0, cnt, vec, lpp, ppw, waves, qpb, chunks, num_blocks, grid, split, ks)
        if split and ks == 1 and Lq == S:
            if shapes is None:
                raise ValueError("the band arrangement needs the level shapes")
            bc, count, cap = band_table(shapes, qpb)
            band_grid = 8 * cnt * M * cap
            if band_grid <= MAX_INDEX:
                ln.bands, ln.band_c, ln.band_count, ln.band_cap, ln.grid = True, bc, count, cap, band_grid
        out.append(ln)
    return out


def _check(cond, msg):
    if not bool(np.all(cond)):
        raise AddressError(msg)


def wave_queries(ln: Launch, M: int):
    """(n, m, q, part) of every query slot of every wave of the launch, in the kernel's mapping:
    with x = b % 8 and i = b / 8, workgroup b runs the (i % cap)-th chunk of band x of slab i / cap
    (bands of rows: the chunks of band x, level after level), chunk x*chunks/8 + i % per of slab
    i / per (query eighths, per = ceil(chunks / 8)) or work item w = x * (G / 8) + i in slab-major
    order (slab ranges). Every (slab, chunk) must be run exactly once; a work item is query chunk
    chunk / k_split, sample part chunk % k_split."""
    b = np.arange(ln.grid, dtype=np.int64)
    x, i = b & 7, b >> 3
    if ln.bands:
        slab, k = i // ln.band_cap, i % ln.band_cap
        keep = (slab < ln.cnt * M) & (k < np.asarray(ln.band_count)[x])
        slab, k, xs = slab[keep], k[keep], x[keep]
        chunk = np.full(slab.shape, -1, dtype=np.int64)
        for l, row in enumerate(ln.band_c):
            row = np.asarray(row)
            c0, n = row[xs], row[xs + 1] - row[xs]
            take = (chunk < 0) & (k < n)
            chunk[take] = (c0 + k)[take]
            k = np.where(chunk < 0, k - n, k)
        _check(chunk >= 0, "band slot past its chunks")
    elif ln.split:
        per = (ln.chunks + 7) // 8
        slab = i // per
        chunk = ((x * ln.chunks) >> 3) + i % per
        keep = (slab < ln.cnt * M) & (chunk < (((x + 1) * ln.chunks) >> 3))
        slab, chunk = slab[keep], chunk[keep]
    else:
        w = x * (ln.grid >> 3) + i
        _check(np.unique(w).size == ln.grid, "workgroup renumbering is not a permutation")
        w = w[w < ln.num_blocks]
        slab, chunk = w // ln.chunks, w % ln.chunks
    item = slab * ln.chunks + chunk
    _check((chunk >= 0) & (chunk < ln.chunks), "work item chunk out of range")
    _check((np.unique(item).size == item.size) & (item.size == ln.num_blocks),
           "work items not covered exactly once")
    n, m = slab // M, slab % M
    part, qchunk = chunk % ln.k_split, chunk // ln.k_split
    wave = np.arange(ln.waves, dtype=np.int64)
    ps = np.arange(ln.ppw, dtype=np.int64)
    q = (qchunk[:, None, None] * ln.q_per_block + wave[None, :, None] * ln.ppw + ps[None, None, :])
    shp = q.shape
    bc = lambda a: np.broadcast_to(a[:, None, None], shp).ravel()
    return bc(n), bc(m), q.ravel(), bc(part)


def coalesced_atomics(D: int, vec: int, lpp: int) -> bool:
    """Whether the atomics take the row-coalesced mapping (one row piece per lane, PPW*D staged)."""
    return D == lpp * vec and (64 // lpp) * D <= ATOMIC_ROW_FLOATS


def coalesced_map(D: int, vec: int, lpp: int):
    """The row-coalesced atomics: instruction j, lane L add flat index f = 64 j + L of
    (query slot, corner, channel) = (f / 4D, (f / D) % 4, f % D); checked to cover every
    (query slot, corner, channel) of a wave exactly once, 32 consecutive lanes on one row."""
    ppw = 64 // lpp
    total = ppw * 4 * D
    _check(total % 64 == 0, "coalesced atomics need whole instructions")
    seen = np.zeros((ppw, 4, D), dtype=np.int64)
    for j in range(total // 64):
        f = 64 * j + np.arange(64)
        qq, r = f // (4 * D), f % (4 * D)
        c, ch = r // D, r % D
        np.add.at(seen, (qq, c, ch), 1)
    _check(np.all(seen == 1), f"coalesced atomics do not cover (query, corner, channel) once at D={D}")
    return total // 64


def lane_channel_maps(D: int, vec: int, lpp: int):
    """Channels read by value-row loads (lane sub, pass c0: [c0 + sub*vec, +vec)) and channels
    added by the atomics (lane sub, pass c0, element i: c0 + sub + lpp*i; or the row-coalesced
    mapping), each checked to cover [0, D) exactly once."""
    if coalesced_atomics(D, vec, lpp):
        coalesced_map(D, vec, lpp)
    loads, atom = [], []
    for c0 in range(0, D, lpp * vec):
        for sub in range(lpp):
            chan = c0 + sub * vec
            if chan < D:
                loads.append((chan, vec))
            for i in range(vec):
                ct = c0 + sub + lpp * i
                if ct < D:
                    atom.append(ct)
    cov = np.zeros(D, dtype=np.int64)
    for chan, v in loads:
        cov[chan:chan + v] += 1
    _check(np.all(cov == 1), f"value-row loads do not cover the {D} channels once")
    _check(sorted(atom) == list(range(D)), f"atomic lanes do not cover the {D} channels once")
    return loads, atom


def model_atomic_backward(value, shapes, starts, loc, attn, grad_out, plant_col_step=0):
    """Replay the atomic backward's addressing on the CPU; returns grad_value (fp64) summed from
    the atomics that land, and a dict of access counts. Raises AddressError on the first access
    that breaks an invariant. plant_col_step adds a planted error to the column step of the
    corner offsets (for the test that the model notices one)."""
    import scipy.sparse as sp

    N, S, M, D = value.shape
    _, Lq, _, L, P, _ = loc.shape
    K = L * P
    es = value.dtype.itemsize
    H = [int(h) for h, _ in shapes]
    W = [int(w) for _, w in shapes]
    st = [int(s) for s in starts]
    gv = np.zeros((N * S * M, D), dtype=np.float64)
    g = np.asarray(grad_out, dtype=np.float64).reshape(N * Lq * M, D)
    stats = {"launches": 0, "sample_slots": 0, "tail_slots": 0, "corner_atomics_landed": 0,
             "corner_atomics_dropped": 0}
    lns = launches(N, S, M, D, Lq, L, P, es, shapes=list(zip(H, W)))
    for ln in lns:
        stats["launches"] += 1
        loads, atom = lane_channel_maps(D, ln.vec, ln.lpp)
        elems = ln.cnt * S * M * D
        value_bytes, gv_bytes = elems * es, elems * 4
        _check(elems < MAX_LAUNCH_ELEMS, "launch exceeds the element limit")
        _check(ln.cnt * Lq * M * K * 2 <= MAX_INDEX and ln.cnt * Lq * M * D <= MAX_INDEX,
               "per-launch sample index range exceeds int32")
        n, m, q, part = wave_queries(ln, M)
        # every real (n, m, q, part) of the launch is served exactly once; the rest are tail slots
        real = q < Lq
        key = ((n[real] * M + m[real]) * Lq + q[real]) * ln.k_split + part[real]
        _check(np.unique(key).size == key.size == ln.cnt * M * Lq * ln.k_split, "queries not covered exactly once")
        # the part's samples [kb, ke), as the kernel forms them
        kper = (K + ln.k_split - 1) // ln.k_split
        kb = part * kper
        ke = np.minimum(kb + kper, K)
        # grad_out row read by each query slot (tail slots read query 0's row)
        gout_row = ((n * Lq + np.where(real, q, 0)) * M + m) * D
        _check((gout_row >= 0) & (gout_row + D <= ln.cnt * Lq * M * D), "grad_out row out of range")
        covered = np.zeros(K, dtype=np.int64)
        for k in range(K):
            l = k // P
            mine = (k >= kb) & (k < ke)  # the slots whose part holds sample k
            covered[k] = int(np.count_nonzero(mine & real))
            stats["sample_slots"] += int(np.count_nonzero(mine & real))
            stats["tail_slots"] += int(np.count_nonzero(mine & ~real))
            kn, km, kq, kreal, kgrow = n[mine], m[mine], q[mine], real[mine], gout_row[mine]
            qq = np.where(kreal, kq, 0)
            smp = ((kn * Lq + qq) * M + km) * K + k
            _check(smp[kreal] < ln.cnt * Lq * M * K, "sample index out of range")
            xy = loc[ln.n0:ln.n0 + ln.cnt].reshape(-1, 2)[smp]
            a = attn[ln.n0:ln.n0 + ln.cnt].reshape(-1)[smp].astype(np.float32)
            x = np.where(kreal, xy[:, 0], np.float32(-2.0)).astype(np.float32)
            y = np.where(kreal, xy[:, 1], np.float32(-2.0)).astype(np.float32)
            a = np.where(kreal, a, np.float32(0.0))
            w_im = fmaf32(x, W[l], -0.5)
            h_im = fmaf32(y, H[l], -0.5)
            ok = (h_im > -1) & (w_im > -1) & (h_im < H[l]) & (w_im < W[l])
            h0f, w0f = np.floor(h_im), np.floor(w_im)
            h0 = np.where(ok, h0f, 0).astype(np.int64)
            w0 = np.where(ok, w0f, 0).astype(np.int64)
            lh = np.where(ok, h_im - h0f, 0).astype(np.float32)
            lw = np.where(ok, w_im - w0f, 0).astype(np.float32)
            hh, hw = np.float32(1) - lh, np.float32(1) - lw
            a = np.where(ok, a, np.float32(0))
            base = ((kn * S + st[l] + h0 * W[l] + w0) * M + km) * D
            _check(np.abs(base[ok]) <= MAX_INDEX, "corner base offset overflows int32")
            top, bot, lef, rig = h0 >= 0, h0 + 1 < H[l], w0 >= 0, w0 + 1 < W[l]
            corners = [(top & lef, base, a * (hh * hw)),
                       (top & rig, base + M * D + plant_col_step, a * (hh * lw)),
                       (bot & lef, base + W[l] * M * D, a * (lh * hw)),
                       (bot & rig, base + (W[l] + 1) * M * D + plant_col_step, a * (lh * lw))]
            for dh_dw, (cv, off_if, wgt) in zip(((0, 0), (0, 1), (1, 0), (1, 1)), corners):
                valid = ok & cv
                off = np.where(valid, off_if, MAX_LAUNCH_ELEMS).astype(np.int64)
                # value-row loads: [(off << shift) + chan*es, + vec*es) against value_bytes
                for chan, v in loads:
                    lo_b = (off * es + chan * es) % U32
                    _check(off * es + chan * es < U32, "value load offset wraps 32 bits")
                    inr = lo_b + v * es <= value_bytes
                    _check(inr == valid, "a value-row load lands iff its corner is on the map")
                # the atomics: byte (off << 2) + ct*4 against gv_bytes
                for ct in (atom[0], atom[-1]):
                    byte = off * 4 + ct * 4
                    _check(byte < U32, "atomic offset wraps 32 bits")
                    _check((byte + 4 <= gv_bytes) == valid, "an atomic lands iff its corner is on the map")
                # a landed corner is the row of pixel (h0+dh, w0+dw) of this (batch, head)
                hc, wc = h0 + dh_dw[0], w0 + dh_dw[1]
                want = ((kn * S + st[l] + hc * W[l] + wc) * M + km) * D
                _check(off[valid] == want[valid], "landed corner is not the sampled pixel's row")
                _check(off[valid] % D == 0, "corner offset is not a row start")
                stats["corner_atomics_landed"] += int(valid.sum()) * D
                stats["corner_atomics_dropped"] += int((~valid).sum()) * D
                # accumulate: grad_value[row] += w * g[query row]
                rows = (off[valid] // D) + ln.n0 * S * M
                cols = kgrow[valid] // D + ln.n0 * Lq * M
                if rows.size:
                    A = sp.coo_matrix((wgt[valid].astype(np.float64), (rows, cols)), shape=(N * S * M, N * Lq * M))
                    gv += A.tocsr() @ g
        # each sample of each query is taken by exactly one part
        _check(np.all(covered == ln.cnt * M * Lq), "a sample of some query is in no part or in two")
    return gv.reshape(N, S, M, D), stats
