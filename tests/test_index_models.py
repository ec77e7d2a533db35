"""CPU models of kernel index arithmetic, checked before the kernels run.

Each model restates, in NumPy, how a kernel maps its workgroups, lanes and
copies onto the data, and checks on the CPU that every access stays inside
its buffer and that the mapped computation gives the intended product on
ragged shapes. They share no code with the library (they restate the
mapping), so a change to a kernel's indexing must be mirrored here.
"""

import math

import numpy as np
import pytest

# ---------------------------------------------------------------- helpers


def xcd_two_class_index(bid, nwg, n_first):
    """Workgroup bid -> logical job: every XCD (bid % 8) gets an even share of
    the first n_first jobs as one contiguous range, then of the rest."""
    xcd, idx = bid & 7, bid >> 3
    per, rem = nwg >> 3, nwg & 7
    fper, frem = n_first >> 3, n_first & 7
    f_cnt = fper + (1 if xcd < frem else 0)
    f_begin = xcd * fper + (xcd if xcd < frem else frem)
    if idx < f_cnt:
        return f_begin + idx
    begin = xcd * per + (xcd if xcd < rem else rem)
    return n_first + (begin - f_begin) + (idx - f_cnt)


@pytest.mark.parametrize("nwg,n_first", [(576, 512), (640, 512), (1, 0), (7, 3), (4096, 4096),
                                         (1000, 0), (9, 9), (513, 256)])
def test_xcd_two_class_index_is_a_permutation(nwg, n_first):
    jobs = [xcd_two_class_index(b, nwg, n_first) for b in range(nwg)]
    assert sorted(jobs) == list(range(nwg))


# ------------------------------------- k-major float32 kernel (tgemm_k32_kernel)

K32_ROWS = 32                               # k rows per slice
K32_STAGE = K32_ROWS * (64 + 256)           # floats of the largest slice (64 x 256 tile)
K32_MAX_COPIES = K32_STAGE // 256 // 4      # 1 KB copies per wave


def k32_tile(M):
    return (64, 256) if M <= 64 else (128, 128)


def k32_slice(G, A, M, N, tmi, tni, q, sumsq):
    """One slice q of tile (tmi, tni) through the kernel's copies and operand
    reads. Returns the tile's 32-row product (and checks every access)."""
    TM, TN = k32_tile(M)
    nm, ncopy = TM // 8, (TM + TN) // 8
    assert ncopy <= 4 * K32_MAX_COPIES
    lds = np.zeros(K32_STAGE, np.float64) if sumsq else np.full(K32_STAGE, np.nan)
    for wave in range(4):
        for p in range(K32_MAX_COPIES):
            c = wave + 4 * p
            if c >= ncopy:
                continue
            mside = c < nm
            W, R, X = (TM, M, G) if mside else (TN, N, A)
            lane = np.arange(64)
            f = 256 * (c if mside else c - nm) + 4 * lane
            k, pc = f // W, f & (W - 1)
            col = (tmi * TM if mside else tni * TN) + ((pc + W - 32 * (k & 1)) & (W - 1))
            voff = k * R * 4 + np.minimum(col, R - 4) * 4
            assert np.all(voff < 2 ** 32) and np.all(k < K32_ROWS)
            byte0 = q * K32_ROWS * R * 4 + voff
            assert np.all(byte0 + 16 <= X.size * 4) and np.all(byte0 % 16 == 0)
            dst = 1024 * c + 16 * lane
            assert np.all(dst + 16 <= K32_STAGE * 4)
            for ln in range(64):
                if sumsq and col[ln] >= R:
                    continue          # the norm variant leaves these words at zero
                b0 = byte0[ln] // 4
                lds[dst[ln] // 4: dst[ln] // 4 + 4] = X.reshape(-1)[b0:b0 + 4]
    wc = TN // 64
    out = np.zeros((TM, TN))
    for wave in range(4):
        wm, wn = wave // wc, wave % wc
        for a in range(2):
            for b in range(2):
                D = np.zeros((32, 32))
                lane = np.arange(64)
                h, c32 = lane >> 5, lane & 31
                oa = h * TM + ((wm * 64 + 32 * a + 32 * h) & (TM - 1)) + c32
                ob = K32_ROWS * TM + h * TN + ((wn * 64 + 32 * b + 32 * h) & (TN - 1)) + c32
                for kp in range(K32_ROWS // 2):
                    ia, ib = oa + 2 * kp * TM, ob + 2 * kp * TN
                    assert np.all(ia < K32_ROWS * TM)
                    assert np.all((K32_ROWS * TM <= ib) & (ib < K32_ROWS * (TM + TN)))
                    Aop = np.zeros((32, 2))
                    Bop = np.zeros((2, 32))
                    Aop[c32, h] = lds[ia]
                    Bop[h, c32] = lds[ib]
                    D += Aop @ Bop
                out[wm * 64 + 32 * a: wm * 64 + 32 * a + 32,
                    wn * 64 + 32 * b: wn * 64 + 32 * b + 32] = D
    return out


@pytest.mark.parametrize("M,N", [(64, 576), (64, 16), (128, 1152), (12, 100), (100, 36),
                                 (64, 144), (132, 260), (256, 2304)])
def test_k32_copies_and_reads_give_the_tile_product(M, N):
    """Ragged widths, both tile shapes: the clip variant's tile equals
    G_sliceᵀ A_slice on its valid part, and the norm variant's tile (copies
    past the edge skipped, words left at zero) has exactly the valid part's
    sum of squares."""
    T, B = 64, 2
    rng = np.random.default_rng(M * 1000 + N)
    G = rng.standard_normal((B * T, M)).astype(np.float32)
    A = rng.standard_normal((B * T, N)).astype(np.float32)
    TM, TN = k32_tile(M)
    tiles = [(tmi, tni) for tmi in range(-(-M // TM)) for tni in range(-(-N // TN))]
    if len(tiles) > 6:
        tiles = tiles[:3] + tiles[-3:]
    for tmi, tni in tiles:
        for q in (0, B * T // K32_ROWS - 1):
            rows = slice(q * K32_ROWS, (q + 1) * K32_ROWS)
            ref = G[rows].astype(np.float64).T @ A[rows].astype(np.float64)
            m0, n0 = tmi * TM, tni * TN
            mv, nv = min(TM, M - m0), min(TN, N - n0)
            out = k32_slice(G, A, M, N, tmi, tni, q, sumsq=False)
            assert not np.isnan(out[:mv, :nv]).any()
            np.testing.assert_allclose(out[:mv, :nv], ref[m0:m0 + mv, n0:n0 + nv], atol=1e-9)
            sq = k32_slice(G, A, M, N, tmi, tni, q, sumsq=True)
            assert math.isclose(float(np.sum(sq * sq)),
                                float(np.sum(ref[m0:m0 + mv, n0:n0 + nv] ** 2)), rel_tol=1e-12)


def test_k32_every_wave_has_copies():
    for TM, TN in ((64, 256), (128, 128)):
        nc = (TM + TN) // 8
        assert nc * 1024 <= K32_STAGE * 4
        for wave in range(4):
            assert sum(1 for p in range(K32_MAX_COPIES) if wave + 4 * p < nc) >= 4


# ------------------------------------------- float32 Gram form (gram64_kernel)

G64_COLS = 64


def g64_word(t, k):
    """Word of (row t, column k) in a slice: row t rotated by t 16-byte units."""
    return t * G64_COLS + 4 * (((k >> 2) + t) & 15) + (k & 3)


@pytest.mark.parametrize("T,d_in,d_out", [(64, 128, 64), (37, 64, 128), (2, 64, 64), (63, 192, 64)])
def test_gram64_copies_and_reads_give_the_norm(T, d_in, d_out):
    """Example ex of B: the slices' copies (rows past T never copied, slots
    zeroed) and the MFMA operand reads give Σ (A Aᵀ)∘(G Gᵀ) = ||Gᵀ A||²."""
    B, ex = 2, 1
    rng = np.random.default_rng(T + d_in)
    A = rng.standard_normal((B * T, d_in)).astype(np.float32)
    G = rng.standard_normal((B * T, d_out)).astype(np.float32)
    na, ns = d_in // G64_COLS, d_in // G64_COLS + d_out // G64_COLS
    accA, accG = np.zeros((64, 64)), np.zeros((64, 64))
    assert all(g64_word(t, k) < 64 * 64 for t in range(64) for k in range(64))
    assert len({g64_word(t, k) for t in range(64) for k in range(64)}) == 64 * 64
    for s in range(ns):
        lds = np.zeros(64 * 64)
        is_a = s < na
        X, d = (A, d_in) if is_a else (G, d_out)
        col0 = (s if is_a else s - na) * G64_COLS
        base = ex * T * d + col0
        for wave in range(4):
            for p in range(4):
                c = wave + 4 * p
                for lane in range(64):
                    t, u = 4 * c + (lane >> 4), lane & 15
                    col = 4 * ((u - t) & 15)
                    voff = t * d * 4 + col * 4
                    assert voff < 2 ** 32
                    if t >= T:
                        continue
                    f = base + voff // 4
                    assert f + 4 <= X.size and col0 + col + 4 <= d
                    dst = 1024 * c + 16 * lane
                    assert dst + 16 <= 64 * 64 * 4
                    lds[dst // 4: dst // 4 + 4] = X.reshape(-1)[f:f + 4]
        acc = accA if is_a else accG
        for wave in range(4):
            bm, bn = wave >> 1, wave & 1
            for kp in range(32):
                Aop, Bop = np.zeros((32, 2)), np.zeros((2, 32))
                for lane in range(64):
                    h, c32 = lane >> 5, lane & 31
                    k = 2 * kp + h
                    Aop[c32, h] = lds[g64_word(32 * bm + c32, k)]
                    Bop[h, c32] = lds[g64_word(32 * bn + c32, k)]
                acc[32 * bm:32 * bm + 32, 32 * bn:32 * bn + 32] += Aop @ Bop
    got = float((accA * accG).sum())
    Ai = A[ex * T:(ex + 1) * T].astype(np.float64)
    Gi = G[ex * T:(ex + 1) * T].astype(np.float64)
    ref = float(((Gi.T @ Ai) ** 2).sum())
    assert math.isclose(got, ref, rel_tol=1e-9)


# ------------------------------- stored per-example gradient, MFMA form (bf16)

def v_perm(src0, src1, sel):
    """v_perm_b32: byte i of the result is byte (sel >> 8 i) & 0xFF of the
    eight bytes {src1 (bytes 0-3), src0 (bytes 4-7)}."""
    pool = int(src1) | (int(src0) << 32)
    out = 0
    for i in range(4):
        b = (sel >> (8 * i)) & 0xFF
        out |= ((pool >> (8 * b)) & 0xFF) << (8 * i)
    return out


def bf16_values(words):
    """uint32 words -> their two bf16 halves as floats (low half first)."""
    out = []
    for wd in words:
        for h in (wd & 0xFFFF, wd >> 16):
            out.append(float(np.array([h << 16], np.uint32).view(np.float32)[0]))
    return out


def mfma_16x16x32(a_lane, b_lane, acc):
    """v_mfma_f32_16x16x32_bf16: lane l supplies A[l % 16][8 (l // 16) + e]
    and B[8 (l // 16) + e][l % 16] (e = 0..7); output v of lane l is
    D[4 (l // 16) + v][l % 16]."""
    A = np.zeros((16, 32))
    Bm = np.zeros((32, 16))
    for ln in range(64):
        A[ln % 16, 8 * (ln // 16): 8 * (ln // 16) + 8] = a_lane[ln]
        Bm[8 * (ln // 16): 8 * (ln // 16) + 8, ln % 16] = b_lane[ln]
    D = A @ Bm
    for ln in range(64):
        for v in range(4):
            acc[ln][v] += D[4 * (ln // 16) + v, ln % 16]


@pytest.mark.parametrize("T,d_w,r,narrow_is_a,chunk,t0,t1", [
    (37, 256, 16, True, 1, 0, 37), (64, 384, 5, False, 2, 8, 45), (29, 128, 4, True, 0, 3, 29),
    (16, 136, 16, False, 1, 0, 16)])
def test_skinny_mfma_lanes_form_the_gradient(T, d_w, r, narrow_is_a, chunk, t0, t1):
    """One wave of the MFMA stored-gradient kernel, bit by bit on bf16 data:
    its loads (wide columns past d_w, narrow columns past r and rows past the
    range read as zero), the in-register 8 x 8 transposes, the MFMAs and the
    stores give g = N^T W over rows [t0, t1) of the chunk's 128 columns, in
    the layout of G^T A."""
    rng = np.random.default_rng(T * d_w + r)
    to_bf16 = lambda x: (x.astype(np.float32).view(np.uint32) >> 16).astype(np.uint32)
    Nb = to_bf16(rng.standard_normal((T, r)))
    Wb = to_bf16(rng.standard_normal((T, d_w)))
    f = lambda b: (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    acc = np.zeros((8, 64, 4))
    for tg in range(t0, t1, 32):
        a_lane, b_lanes = [], [[] for _ in range(8)]
        for ln in range(64):
            g, cl = ln // 16, ln % 16
            col = chunk * 128 + 8 * cl
            rows = []      # the lane's eight 16-byte loads, as four uint32 words each
            nv = []
            for kk in range(8):
                t = tg + 8 * g + kk
                words = [0, 0, 0, 0]
                n = 0
                if t < t1:
                    if col < d_w:
                        assert col + 8 <= d_w
                        e = Wb[t, col:col + 8]
                        words = [int(e[2 * q]) | (int(e[2 * q + 1]) << 16) for q in range(4)]
                    if cl < r:
                        n = int(Nb[t, cl])
                rows.append(words)
                nv.append(n)
            a_lane.append(bf16_values([nv[2 * q] | (nv[2 * q + 1] << 16) for q in range(4)]))
            for j in range(8):
                sel = 0x05040100 if j % 2 == 0 else 0x07060302
                wq = [v_perm(rows[2 * q + 1][j // 2], rows[2 * q][j // 2], sel) for q in range(4)]
                b_lanes[j].append(bf16_values(wq))
        for j in range(8):
            mfma_16x16x32(a_lane, b_lanes[j], acc[j])
    got = np.zeros((r, d_w)) if not narrow_is_a else np.zeros((d_w, r))
    written = np.zeros_like(got, dtype=bool)
    for ln in range(64):
        m0, col = 4 * (ln // 16), chunk * 128 + 8 * (ln % 16)
        if col >= d_w or m0 >= r:
            continue
        for j in range(8):
            for v in range(4):
                if m0 + v < r:
                    idx = (col + j, m0 + v) if narrow_is_a else (m0 + v, col + j)
                    got[idx] = acc[j][ln][v]
                    written[idx] = True
    ref = f(Nb[t0:t1]).T @ f(Wb[t0:t1])           # [r][d_w]
    if narrow_is_a:
        ref = ref.T
    c0, c1 = chunk * 128, min(d_w, chunk * 128 + 128)
    sl = (slice(c0, c1), slice(None)) if narrow_is_a else (slice(None), slice(c0, c1))
    assert written[sl].all() and written.sum() == written[sl].size
    np.testing.assert_allclose(got[sl], ref[sl], rtol=1e-12, atol=1e-12)
    # The wave's norm partial (every output, zeros included) is the chunk's.
    assert math.isclose(float(np.sum(acc ** 2)), float(np.sum(ref[sl] ** 2)), rel_tol=1e-12)


# ------------------------- bf16 Gram form on 256-row tiles (ghost_tile256_kernel)
#
# WAVES waves own a 256 x 256 tile (p, q): a (WAVES / 2) x 2 grid of sub-tiles
# of MB x 4 blocks of 32 x 32 (MB = 16 / WAVES). Slices of BK columns of row
# blocks p and q are copied into LDS (1 KB per copy instruction) and read back
# as the 32x32x16 MFMA operands; GA is parked per lane in the workspace; a
# diagonal tile is computed whole.

G4_ROWS = 256


def g4_swz(bk, r):
    return ((r >> 1) & 7) if bk == 64 else ((r >> 2) & 3)


def xcd_logical_index(bid, nwg):
    per, rem, xcd, idx = nwg >> 3, nwg & 7, bid & 7, bid >> 3
    return xcd * (per + 1) + idx if xcd < rem else rem * (per + 1) + (xcd - rem) * per + idx


def g4_stage(bk, waves, T, d, p, q, s):
    """LDS stage of slice s of a d-wide operand: {16-byte slot: (row, chunk)}."""
    row_bytes, chunks = 2 * bk, bk // 8
    rpc = 1024 // row_bytes
    per = G4_ROWS // rpc // waves
    diag = p == q
    rows_p, rows_q = min(256, T - 256 * p), min(256, T - 256 * q)
    lds = {}
    for wave in range(waves):
        r0 = rpc * wave + np.arange(64) // chunks              # row of copy u = 0 per lane
        chunk = (np.arange(64) % chunks) ^ np.array([g4_swz(bk, r) for r in r0])
        for u in range(per if diag else 2 * per):
            second = u >= per
            j = wave + waves * (u % per)
            for lane in range(64):
                r = rpc * j + lane // chunks
                assert r == r0[lane] + rpc * waves * (u % per)
                assert g4_swz(bk, r) == g4_swz(bk, int(r0[lane])), "swizzle depends on u"
                rv = rows_q if second else rows_p
                row = 256 * (q if second else p) + min(r, rv - 1)
                off = row * d * 2 + 16 * int(chunk[lane]) + s * bk * 2
                assert 0 <= off and off + 16 <= T * d * 2 and off % 16 == 0
                dst = (G4_ROWS * row_bytes if second else 0) + 1024 * j + 16 * lane
                assert dst + 16 <= 2 * G4_ROWS * row_bytes
                assert dst not in lds, "an LDS slot written twice"
                lds[dst] = (row, s * chunks + int(chunk[lane]))
    expect = (1 if diag else 2) * G4_ROWS * row_bytes // 16
    assert len(lds) == expect, "an LDS slot left unwritten"
    return lds


def g4_gram(bk, waves, X, T, p, q):
    """GA (or GG) of tile (p, q) as the waves' accumulators: {(wave, a, b): 32x32}."""
    d = X.shape[1]
    row_bytes = 2 * bk
    mb, nb = 16 // waves, 4
    diag = p == q
    acc = {}
    for s in range(d // bk):
        lds = g4_stage(bk, waves, T, d, p, q, s)
        for wave in range(waves):
            wm, wn = wave >> 1, wave & 1
            row_a = 32 * mb * wm * row_bytes
            row_b = (0 if diag else G4_ROWS * row_bytes) + 32 * nb * wn * row_bytes
            for st in range(bk // 16):
                frag = {}
                for which, base, nblk in (("a", row_a, mb), ("b", row_b, nb)):
                    for blk in range(nblk):
                        rows, ks, addrs = [], [], []
                        for lane in range(64):
                            g = lane >> 5
                            rd = (lane & 31) * row_bytes + 16 * ((2 * st + g) ^ g4_swz(bk, lane & 31))
                            addr = base + 32 * blk * row_bytes + rd
                            addrs.append(addr)
                            row, chunk = lds[addr]
                            rows.append(row)
                            ks.append(chunk)
                        # 16-lane groups read 16 distinct 16-byte bank groups (256 B of banks).
                        for g16 in range(4):
                            grp = {(a // 16) % 16 for a in addrs[16 * g16:16 * g16 + 16]}
                            assert len(grp) == 16, "LDS bank conflict in an operand read"
                        # lane l: row (l % 32) of the 32-row block, k chunk 2 st + l / 32
                        assert all(rows[i] == rows[i + 32] and ks[i + 32] == ks[i] + 1 for i in range(32))
                        frag[(which, blk)] = (rows, ks)
                for a in range(mb):
                    for b in range(nb):
                        ra, ka = frag[("a", a)]
                        rb, kb = frag[("b", b)]
                        A32 = np.stack([X[ra[i], 8 * ka[i]:8 * ka[i] + 16] for i in range(32)])
                        B32 = np.stack([X[rb[i], 8 * kb[i]:8 * kb[i] + 16] for i in range(32)])
                        key = (wave, a, b)
                        acc[key] = acc.get(key, np.zeros((32, 32))) + A32 @ B32.T
    return acc


def g4_wave_sums(bk, waves, A, G, T, p, q):
    """Each wave's masked sum of GA * GG over its sub-tile of tile (p, q),
    through the park slots (every slot written once, read back by its lane)."""
    GA = g4_gram(bk, waves, A, T, p, q)
    GG = g4_gram(bk, waves, G, T, p, q)
    mb, nb = 16 // waves, 4
    per_wave = 256 * 256 // waves
    rows_p, rows_q = min(256, T - 256 * p), min(256, T - 256 * q)
    park = np.full(256 * 256, np.nan)
    lane = np.arange(64)
    v = np.arange(16)
    # Lane l, element v: block row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32.
    br = 8 * (v[None, :] >> 2) + 4 * (lane[:, None] >> 5) + (v[None, :] & 3)
    bc = np.broadcast_to(lane[:, None] & 31, br.shape)
    sums = {}
    for wave in range(waves):
        total = 0.0
        wm, wn = wave >> 1, wave & 1
        for a in range(mb):
            for b in range(nb):
                lane_ga = GA[(wave, a, b)][br, bc]
                # Park: float4 k = 4 (NB a + b) + c holds elements 4c..4c+3.
                offs = [per_wave * wave + 256 * (4 * (nb * a + b) + c) + 4 * lane[:, None]
                        + np.arange(4)[None, :] for c in range(4)]
                for c in range(4):
                    assert np.all(offs[c] < 256 * 256)
                    assert np.all(np.isnan(park[offs[c]])), "park slot written twice"
                    park[offs[c]] = lane_ga[:, 4 * c:4 * c + 4]
                back = np.concatenate([park[o] for o in offs], axis=1)
                row = 32 * (mb * wm + a) + br
                col = 32 * (nb * wn + b) + bc
                mask = (row < rows_p) & (col < rows_q)
                total += float(np.sum(np.where(mask, back * GG[(wave, a, b)][br, bc], 0.0)))
        sums[wave] = total
    assert not np.any(np.isnan(park)), "park slot never written"
    return sums


def g4_tile_sum(bk, waves, A, G, T, p, q):
    return sum(g4_wave_sums(bk, waves, A, G, T, p, q).values())


@pytest.mark.parametrize("bk,waves", [(64, 8), (64, 4), (32, 8)])
@pytest.mark.parametrize("T,d_in,d_out", [(300, 64, 128), (257, 128, 64), (520, 64, 64),
                                          (512, 64, 64)])
def test_ghost256_tiles_give_the_norm(bk, waves, T, d_in, d_out):
    rng = np.random.default_rng(T + d_in + bk + waves)
    A = rng.integers(-3, 4, (T, d_in)).astype(np.float64)
    G = rng.integers(-3, 4, (T, d_out)).astype(np.float64)
    nt = -(-T // 256)
    total = 0.0
    seen = set()
    for pr0 in range(nt * (nt + 1) // 2):
        pr, p = pr0, 0
        while pr >= nt - p:
            pr -= nt - p
            p += 1
        q = p + pr
        assert p <= q < nt and (p, q) not in seen
        seen.add((p, q))
        t = g4_tile_sum(bk, waves, A, G, T, p, q)
        total += t if p == q else 2.0 * t
    assert len(seen) == nt * (nt + 1) // 2
    want = float(np.sum((G.T @ A) ** 2))
    assert total == pytest.approx(want, rel=1e-12)


# Jobs of one example without a column split (ghost_tile256_kernel): with
# halves, diagonal tile k for k < nt, then the two 128-row halves of every
# off-diagonal tile o (row-major over p < q); otherwise the upper-triangle
# tiles in row-major order. Eight waves; a diagonal tile skips waves 4 and 6
# (the sub-tiles below its 128-row diagonal) and weights waves 1 and 3 by 2;
# an off-diagonal tile weights every wave by 2, and half h keeps waves
# 4 h .. 4 h + 3. Partial columns: diagonal tile p, then nt + 2 o + h.
G4_DIAG_ACT, G4_DIAG_W2 = 0xAF, 0x0A


def g4_off_pq(nt, o):
    p = 0
    while o >= nt - 1 - p:
        o -= nt - 1 - p
        p += 1
    return p, p + 1 + o


def g4_off_index(nt, p, q):
    return p * (nt - 1) - p * (p - 1) // 2 + (q - p - 1)


def g4_jobs(nt, halves):
    """(p, q, act, w2, columns written) per job of one example."""
    out = []
    for k in range(nt * nt if halves else nt * (nt + 1) // 2):
        half = -1
        if halves and k < nt:
            p = q = k
        elif halves:
            p, q = g4_off_pq(nt, (k - nt) >> 1)
            half = (k - nt) & 1
        else:
            pr, p = k, 0
            while pr >= nt - p:
                pr -= nt - p
                p += 1
            q = p + pr
        if p == q:
            out.append((p, q, G4_DIAG_ACT, G4_DIAG_W2, [p]))
            continue
        c = nt + 2 * g4_off_index(nt, p, q)
        act = 0xFF if half < 0 else 0x0F << (4 * half)
        out.append((p, q, act, 0xFF, [c, c + 1] if half < 0 else [c + half]))
    return out


@pytest.mark.parametrize("nt", range(1, 9))
@pytest.mark.parametrize("halves", [False, True])
def test_ghost256_jobs_weight_every_entry_once(nt, halves):
    """The active sub-tiles' weights, added to their mirror images, count every
    entry of the symmetric T x T product once, and every partial column is
    written by exactly one job."""
    T = 256 * nt
    weight = np.zeros((T, T))
    cols = np.zeros(nt * nt, int)
    for p, q, act, w2, written in g4_jobs(nt, halves):
        for wave in range(8):
            if (act >> wave) & 1:
                wm, wn = wave >> 1, wave & 1
                r0, c0 = 256 * p + 64 * wm, 256 * q + 128 * wn
                weight[r0:r0 + 64, c0:c0 + 128] += 2.0 if (w2 >> wave) & 1 else 1.0
        for c in written:
            cols[c] += 1
    assert np.all(weight + weight.T == 2.0)
    assert np.all(cols == 1)
    for o in range(nt * (nt - 1) // 2):
        p, q = g4_off_pq(nt, o)
        assert p < q < nt and g4_off_index(nt, p, q) == o


@pytest.mark.parametrize("halves", [False, True])
@pytest.mark.parametrize("T,d_in,d_out", [(300, 64, 128), (520, 128, 64), (777, 64, 64)])
def test_ghost256_job_decode_gives_the_norm(halves, T, d_in, d_out):
    """Wave sums of the modelled kernel, kept by the job's masks and weights,
    add up to ||G^T A||^2 on ragged T (rows past T masked out)."""
    rng = np.random.default_rng(T + d_in + (7 if halves else 0))
    A = rng.integers(-3, 4, (T, d_in)).astype(np.float64)
    G = rng.integers(-3, 4, (T, d_out)).astype(np.float64)
    nt = -(-T // 256)
    cache, total = {}, 0.0
    for p, q, act, w2, _ in g4_jobs(nt, halves):
        if (p, q) not in cache:
            cache[(p, q)] = g4_wave_sums(64, 8, A, G, T, p, q)
        for wave, ws in cache[(p, q)].items():
            if (act >> wave) & 1:
                total += (2.0 if (w2 >> wave) & 1 else 1.0) * ws
    assert total == pytest.approx(float(np.sum((G.T @ A) ** 2)), rel=1e-12)


@pytest.mark.parametrize("jobs", [1, 7, 160, 192, 511, 512, 513, 1080, 4099])
def test_ghost256_grid_visits_every_job_once(jobs):
    grid = min(jobs, 512)
    visits = []
    for bid in range(grid):
        job = xcd_logical_index(bid, grid)
        while job < jobs:
            visits.append(job)
            job += grid
    assert sorted(visits) == list(range(jobs))


# ------------------------ 384x256-tile clip kernel, ragged last row tile (tgemm_wide_kernel)
#
# A row tile covers 384 columns of G (output rows). In the last row tile of a
# d_out that is a multiple of 32 but not of 384, a lane's G copy reads column
# block min(blk, nvb - 1) of its k-row (blk 0..11, 32 columns each), and the
# store skips the 32-row blocks at or past nvb.

def wide_tile_rule(T, d_in, d_out, cus=256):
    tiles_m = -(-d_out // 384)
    pad = tiles_m * 384 - d_out
    ragged = d_out % 32 == 0 and 50 * pad <= 3 * d_out and tiles_m * (d_in // 256) >= cus
    return d_in % 256 == 0 and T % 64 == 0 and (d_out % 384 == 0 or ragged)


@pytest.mark.parametrize("M", [384, 736, 4064, 11008, 4096])
def test_wide_ragged_row_tile_copies_stay_in_bounds(M):
    assert wide_tile_rule(64, 256 * 256, M)
    tiles_m = -(-M // 384)
    for tm in range(tiles_m):
        nvb = min(12, (M - 384 * tm) // 32)
        assert nvb >= 1
        cols_read, rows_stored = set(), set()
        for t in range(48):                      # the slot's G copies (16 waves x 3)
            for lane in range(64):
                l_unit, l_byte = lane >> 4, 16 * (lane & 3)
                blk = 4 * (t % 3) + l_unit
                byte = 384 * tm * 2 + 64 * min(blk, nvb - 1) + l_byte   # within one k-row of G
                assert 0 <= byte and byte + 16 <= M * 2
                cols_read.add(byte // 2 // 8)
        for wave in range(16):
            wm = wave // 4
            for i in range(3):
                if wm * 3 + i >= nvb:
                    continue
                for r in range(32):
                    rows_stored.add(384 * tm + 32 * (wm * 3 + i) + r)
        assert rows_stored == set(range(384 * tm, min(384 * (tm + 1), M)))
        # every valid 8-column group of the tile is read
        assert {c for c in cols_read} >= set(range(384 * tm // 8, min(384 * (tm + 1), M) // 8))


@pytest.mark.parametrize("d_in,d_out,ok", [(256, 384, True), (4096, 11008, True), (6144, 4064, True),
                                           (4096, 4096, False), (65536, 4096, True),
                                           (65536, 512, False), (65536, 416, False), (256, 736, False)])
def test_wide_tile_rule(d_in, d_out, ok):
    """Whole row tiles always; a ragged last row tile only with at most 6 %
    padding and at least one tile per CU (256)."""
    assert wide_tile_rule(64, d_in, d_out) == ok


@pytest.mark.parametrize("n,nA,S", [(236, 64, 3), (64, 16, 4), (49, 24, 3), (60, 12, 1), (17, 1, 1),
                                    (2, 1, 4), (3, 1, 4), (3, 2, 4)])
def test_ghost256_split_parts_cover_the_slices(n, nA, S):
    """Part p of a split tile takes slices [n p / S, n (p + 1) / S); the
    combine adds GA over the parts that hold A slices (lo < nA) and GG over
    those that hold G slices (hi > nA): every slice once, in part order."""
    # A small layer in a launch whose split suits a larger one (n < S) has
    # empty parts; an empty part that starts before A's end parks a zero GA,
    # one between A and G parks nothing, and neither changes the sums.
    seen = []
    a_parts, g_parts = [], []
    for p in range(S):
        lo, hi = n * p // S, n * (p + 1) // S
        assert lo <= hi and (lo < hi or n < S)
        seen.extend(range(lo, hi))
        if lo < nA:
            a_parts.append(p)
        if hi > nA:
            g_parts.append(p)
    assert seen == list(range(n))
    assert sorted({s for p in a_parts for s in range(n * p // S, n * (p + 1) // S) if s < nA}) \
        == list(range(nA))
    assert sorted({s for p in g_parts for s in range(n * p // S, n * (p + 1) // S) if s >= nA}) \
        == list(range(nA, n))
    # The combine's clamping: A parts are the prefix 0 .. pa - 1, G parts the
    # suffix pg .. S - 1; part p reads A slot min(p, pa - 1) and G slot
    # max(p, pg), always written, and keeps them only when it owns them.
    pa = max(p + 1 for p in range(S) if n * p // S < nA)
    pg = min(p for p in range(S) if n * (p + 1) // S > nA)
    assert a_parts == list(range(pa)) and g_parts == list(range(pg, S))
    for p in range(S):
        assert min(p, pa - 1) in a_parts and max(p, pg) in g_parts
        assert (p < pa) == (p in a_parts) and (p >= pg) == (p in g_parts)
