"""CPU model of the wave-tile kernels (csrc/whtmix_wave.hip), no GPU.

Re-states in numpy:
* the cross-lane primitives as the gfx9/gfx950 ISA defines them -- DPP
  (quad_perm, row_shl, row_shr with row and bank masks, bound_ctrl off) and
  v_permlane16_swap / v_permlane32_swap on a register pair;
* the kernel's wave butterflies built from them (lane_partner, lane_bfly,
  swap_k2, wave_bfly, wht9) on a 64-lane x 8-register file;
* the layouts V4 / V8, the workspace run map and the gain index of the three
  passes;
* the single-launch scheduler: workgroup w takes tiles w, w + P, ... of each
  pass; per-slice counters order the passes; bounded waits; the last
  workgroup out resets the counters (the three-launch form runs the same
  tiles, one per workgroup, with kernel boundaries between the passes).

and checks that the butterflies transform exactly the bits they claim, that
every load and store stays inside its buffer and touches each element once,
that the modelled pipeline reproduces the CPU oracle, and that the schedule
terminates (and resets its counters) for every shape, including after a wait
that gives up.  Test code only; nothing in the product path uses it.
"""
import numpy as np
import pytest

from oracle import oracle as oracle_mod

TB, NV, LANES = 9, 8, 64
COUNTER_WORDS = 4096


# ---------------------------------------------------------------- primitives
def update_dpp(old, src, ctrl, row_mask, bank_mask, bound_ctrl=False):
    """One lane-permuting DPP move on 64 lanes (gfx9 semantics)."""
    out = np.array(old, copy=True)
    for lam in range(LANES):
        row, bank = lam >> 4, (lam >> 2) & 3
        if not ((row_mask >> row) & 1 and (bank_mask >> bank) & 1):
            continue
        if ctrl <= 0xFF:                                  # quad_perm
            s = (lam & ~3) | ((ctrl >> (2 * (lam & 3))) & 3)
        elif 0x101 <= ctrl <= 0x10F:                      # row_shl: read lane + n
            n = ctrl - 0x100
            s = lam + n if (lam & 15) + n < 16 else None
        elif 0x111 <= ctrl <= 0x11F:                      # row_shr: read lane - n
            n = ctrl - 0x110
            s = lam - n if (lam & 15) >= n else None
        else:
            raise ValueError(hex(ctrl))
        if s is None:
            if bound_ctrl:
                out[lam] = 0
            continue
        out[lam] = src[s]
    return out


def permlane_swap(a, b, width):
    """v_permlane{16,32}_swap_b32 a, b: odd 16-lane rows (width 16) or the
    upper 32 lanes (width 32) of a trade places with the even rows / lower
    lanes of b."""
    a2, b2 = np.array(a, copy=True), np.array(b, copy=True)
    for lam in range(LANES):
        if lam & width:
            a2[lam], b2[lam - width] = b[lam - width], a[lam]
    return a2, b2


def lane_partner(x, J):
    if J == 0:
        return update_dpp(np.zeros_like(x), x, 0xB1, 0xF, 0xF)
    if J == 1:
        return update_dpp(np.zeros_like(x), x, 0x4E, 0xF, 0xF)
    if J == 2:
        hi = update_dpp(np.zeros_like(x), x, 0x114, 0xF, 0xA)
        return update_dpp(hi, x, 0x104, 0xF, 0x5)
    hi = update_dpp(np.zeros_like(x), x, 0x118, 0xF, 0xC)
    return update_dpp(hi, x, 0x108, 0xF, 0x3)


LANE = np.arange(LANES)


def reg_bfly(v, J):
    v = v.copy()
    for k in range(NV):
        if not k & (1 << J):
            a, b = v[k].copy(), v[k | (1 << J)].copy()
            v[k], v[k | (1 << J)] = a + b, a - b
    return v


def lane_bfly(v, J):
    s = np.where(LANE & (1 << J), -1.0, 1.0)
    return np.stack([s * v[k] + lane_partner(v[k], J) for k in range(NV)])


def swap_k2(v, width):
    v = v.copy()
    for k in range(4):
        v[k], v[k + 4] = permlane_swap(v[k], v[k + 4], width)
    return v


def wave_bfly(v, J0):
    v = reg_bfly(v, 2)
    for J in range(max(J0, 0), 4):
        v = lane_bfly(v, J)
    if J0 <= 4:
        v = reg_bfly(swap_k2(v, 16), 2)
        v = swap_k2(v, 16)
    v = reg_bfly(swap_k2(v, 32), 2)
    return swap_k2(v, 32)


def wht9(v):
    return wave_bfly(reg_bfly(reg_bfly(v, 0), 1), 0)


# ---------------------------------------------------------------- layouts
def t_index(layout):
    """[8, 64] tile index of (register k, lane) in layout "V4" or "V8"."""
    k = np.arange(NV)[:, None]
    lam = LANE[None, :]
    if layout == "V4":
        return (k & 3) | (lam << 2) | ((k >> 2) << 8)
    return k | (lam << 3)


def group_t(layout, g):
    return (LANE << 2) | (g << 8) if layout == "V4" else (LANE << 3) | (g << 2)


def run_off(t, R):
    return ((t >> R) << TB) | (t & ((1 << R) - 1))


def dense_wht(n):
    i = np.arange(n)
    return np.array([[(-1.0) ** bin(a & b).count("1") for b in i] for a in i])


def bitwise_wht(x, bits):
    """Unnormalised butterflies of a vector over the given index bits."""
    x = x.astype(np.float64).copy()
    for j in bits:
        h = 1 << j
        idx = np.arange(x.size)
        lo = idx[(idx & h) == 0]
        a, b = x[lo].copy(), x[lo | h].copy()
        x[lo], x[lo | h] = a + b, a - b
    return x


# ---------------------------------------------------------------- tests
def test_dpp_partners_are_lane_xor():
    x = np.arange(LANES, dtype=np.float64) + 100.0
    for J in range(4):
        assert np.array_equal(lane_partner(x, J), x[LANE ^ (1 << J)]), J


def test_permlane_swap_transposes_a_lane_bit_with_register_bit_2():
    """After swap_k2(W), register k holds what (k ^ 4 if its lane bit is set
    ...) held: register bit 2 and lane bit log2(W) trade roles."""
    v = np.arange(NV * LANES, dtype=np.float64).reshape(NV, LANES)   # value = k*64 + lane
    for W, lb in ((16, 4), (32, 5)):
        s = swap_k2(v, W)
        for k in range(NV):
            for lam in range(LANES):
                k2, l5 = (k >> 2) & 1, (lam >> lb) & 1
                src_k = (k & 3) | (l5 << 2)
                src_l = (lam & ~(1 << lb)) | (k2 << lb)
                assert s[k, lam] == v[src_k, src_l]
        assert np.array_equal(swap_k2(s, W), v)            # an involution


@pytest.mark.parametrize("layout", ["V4", "V8"])
def test_wht9_is_the_full_tile_transform(layout):
    rng = np.random.default_rng(7)
    tile = rng.standard_normal(512)
    T = t_index(layout)
    v = tile[T]
    out = np.empty(512)
    out[T] = wht9(v)
    np.testing.assert_allclose(out, dense_wht(512) @ tile, rtol=0, atol=1e-9)


@pytest.mark.parametrize("R", [2, 3, 4, 5, 6])
def test_wave_bfly_transforms_the_high_bits_only(R):
    rng = np.random.default_rng(R)
    tile = rng.standard_normal(512)
    T = t_index("V4")
    out = np.empty(512)
    out[T] = wave_bfly(tile[T], R - 2)
    np.testing.assert_allclose(out, bitwise_wht(tile, range(R, TB)), rtol=0, atol=1e-9)


def run_pipeline(x, g, K, B, nvalid, dtype_layout):
    """The three passes on flat slices (numpy float64), with every index the
    kernel computes; returns y and per-buffer touch counts."""
    HB = K - TB
    R = TB - HB
    tiles = 1 << HB
    ws = np.full(B << K, np.nan)
    y = np.full(B * nvalid, np.nan)
    ws_writes = np.zeros(B << K, int)
    x_reads = np.zeros(B * nvalid, int)
    g_reads = np.zeros(1 << K, int)
    y_writes = np.zeros(B * nvalid, int)
    T_io = t_index(dtype_layout)
    T4 = t_index("V4")
    io_group = 4 if dtype_layout == "V4" else 8
    for b in range(B):                                   # pass 1
        for hi in range(tiles):
            start = hi << TB
            valid = max(0, min(nvalid - start, 512))
            v = np.zeros((NV, LANES))
            ok = T_io < valid
            v[ok] = x[b * nvalid + start + T_io[ok]]
            np.add.at(x_reads, b * nvalid + start + T_io[ok], 1)
            v = wht9(v)
            off = (b << K) + (hi << R) + run_off(T_io, R)
            assert off.min() >= b << K and off.max() < (b + 1) << K
            ws[off] = v
            np.add.at(ws_writes, off, 1)
    assert np.all(ws_writes == 1)
    scale = 2.0 ** -K
    for b in range(B):                                   # pass 2
        for run in range(tiles):
            base = (b << K) + (run << TB)
            v = ws[base + T4]
            u = T4
            f = ((u >> R) << TB) | (run << R) | (u & ((1 << R) - 1))
            assert f.min() >= 0 and f.max() < 1 << K
            np.add.at(g_reads, f, 1)
            v = wave_bfly(v, R - 2)
            v = v * (g[f] * scale)
            v = wave_bfly(v, R - 2)
            ws[base + T4] = v
            np.add.at(ws_writes, base + T4, 1)
    assert np.all(ws_writes == 2)
    assert np.all(g_reads == B)
    for b in range(B):                                   # pass 3
        for hi in range(tiles):
            start = hi << TB
            valid = max(0, min(nvalid - start, 512))
            if valid == 0:
                continue
            off = (b << K) + (hi << R) + run_off(T_io, R)
            v = wht9(ws[off])
            ok = T_io < valid
            y[b * nvalid + start + T_io[ok]] = v[ok]
            np.add.at(y_writes, b * nvalid + start + T_io[ok], 1)
    assert np.all(x_reads == 1) and np.all(y_writes == 1)
    # 16-byte groups are all-valid or all-padding when nvalid % 8 == 0
    assert nvalid % io_group == 0 or nvalid % 8 != 0
    return y


def wave_tile(blk, nblk, R):
    """The wave-tile kernels' block renumbering (tile::outer_block)."""
    if R >= 5:
        return blk
    g = 1 << (5 - R)
    if nblk % (8 * g):
        return blk
    return (blk & ~(8 * g - 1)) | ((blk & 7) * g) | ((blk >> 3) & (g - 1))


@pytest.mark.parametrize("K", [12, 13, 14, 15, 16])
@pytest.mark.parametrize("B", [1, 2, 3, 16])
@pytest.mark.parametrize("layout", ["V4", "V8"])
def test_shared_lines_stay_on_one_xcd(K, B, layout):
    """Blocks are dealt round-robin over the 8 XCDs (block i on XCD i mod 8).
    After the renumbering every 128-byte line of the workspace that passes 1
    and 3 write or read, and every line of the gain that pass 2 reads, is
    touched by blocks of one XCD only; the renumbering is a permutation."""
    HB = K - TB
    R = TB - HB
    nblk = B << HB
    wave_tile_map = [wave_tile(i, nblk, R) for i in range(nblk)]
    assert sorted(wave_tile_map) == list(range(nblk))
    T_io = t_index(layout)
    T4 = t_index("V4")
    ws_line_xcd, g_line_xcd = {}, {}
    for blk, i in enumerate(wave_tile_map):
        b, t = i >> HB, i & ((1 << HB) - 1)
        xcd = blk % 8
        off = (b << K) + (t << R) + run_off(T_io, R)           # passes 1 and 3 (t = hi)
        for line in np.unique(off >> 5):
            assert ws_line_xcd.setdefault(int(line), xcd) == xcd
        f = ((T4 >> R) << TB) | (t << R) | (T4 & ((1 << R) - 1))   # pass 2 (t = run)
        for line in np.unique(f >> 5):
            assert g_line_xcd.setdefault((b, int(line)), xcd) == xcd
    assert len(ws_line_xcd) == (B << K) >> 5


@pytest.mark.parametrize("K,B,N,C,layout", [
    (12, 1, 64, 64, "V4"), (13, 2, 128, 64, "V8"), (14, 1, 256, 64, "V4"),
    (15, 3, 256, 128, "V8"), (16, 1, 1024, 64, "V4"), (16, 2, 1024, 64, "V8"),
    (16, 1, 1000, 64, "V4"), (15, 2, 200, 128, "V8"), (13, 1, 33, 128, "V4"),
])
def test_pipeline_matches_oracle(K, B, N, C, layout):
    P = 1 << max(0, (N - 1).bit_length())
    assert P * C == 1 << K
    rng = np.random.default_rng(K * 100 + N)
    x = rng.standard_normal((B, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    y = run_pipeline(x.reshape(-1), g.reshape(-1), K, B, N * C, layout)
    ref = oracle_mod.whtmix(x, g)
    np.testing.assert_allclose(y.reshape(B, N, C), ref, rtol=0, atol=1e-9 * np.abs(ref).max())


# ---------------------------------------------------------------- scheduler
def simulate(B, K, P, spin_limit=10 ** 9, stall=None):
    """Round-robin interleaving of P resident one-wave workgroups, each a
    sequence of steps: pass-1 tiles (signal c0), pass-2 tiles (wait c0, signal
    c1), pass-3 tiles (wait c1), exit.  `stall`: (wg, polls) makes workgroup
    wg sit idle for that many rounds before its first tile (a slow wave).
    Returns (rounds, counters after the run, error flags)."""
    HB = K - TB
    tiles = 1 << HB
    ntiles = B << HB
    ctr = np.zeros(COUNTER_WORDS, np.int64)
    c0, c1 = 0, B
    EXITED, CALL_ERR, STICKY = COUNTER_WORDS - 3, COUNTER_WORDS - 2, COUNTER_WORDS - 1
    progs = []
    for w in range(P):
        items = [(1, i) for i in range(w, ntiles, P)] + \
                [(2, i) for i in range(w, ntiles, P)] + [(3, i) for i in range(w, ntiles, P)]
        progs.append({"items": items, "pos": 0, "polls": 0, "ok": True, "done": False,
                      "idle": stall[1] if stall and stall[0] == w else 0})
    rounds = 0
    while not all(p["done"] for p in progs):
        rounds += 1
        assert rounds < 10 ** 6, "schedule did not finish"
        for w, p in enumerate(progs):
            if p["done"]:
                continue
            if p["idle"]:
                p["idle"] -= 1
                continue
            if p["pos"] == len(p["items"]) or not p["ok"]:
                prior = ctr[EXITED]
                ctr[EXITED] += 1
                if prior == P - 1:
                    if ctr[CALL_ERR]:
                        ctr[STICKY] |= ctr[CALL_ERR]
                    ctr[:2 * B] = 0
                    ctr[CALL_ERR] = 0
                    ctr[EXITED] = 0
                p["done"] = True
                continue
            pas, i = p["items"][p["pos"]]
            b = i >> HB
            if pas == 1:
                ctr[c0 + b] += 1
                p["pos"] += 1
                continue
            need = c0 + b if pas == 2 else c1 + b
            if ctr[need] < tiles:
                if ctr[CALL_ERR]:
                    p["ok"] = False
                    continue
                p["polls"] += 1
                if p["polls"] > spin_limit:
                    ctr[CALL_ERR] = 1
                    p["ok"] = False
                continue
            p["polls"] = 0
            if pas == 2:
                ctr[c1 + b] += 1
            p["pos"] += 1
    return rounds, ctr


@pytest.mark.parametrize("B,K,P", [(1, 16, 128), (2, 16, 256), (47, 16, 700), (3, 12, 5),
                                   (16, 14, 33), (5, 15, 1), (2046, 12, 4096)])
def test_schedule_completes_and_resets(B, K, P):
    P = min(P, B << (K - TB))
    _, ctr = simulate(B, K, P)
    assert not ctr.any()


def test_wait_that_gives_up_still_drains_and_flags():
    """A tiny poll limit with one slow workgroup: some wait gives up, every
    workgroup still exits, the counters return to zero and only the sticky
    word remains set (the host reads and clears it)."""
    _, ctr = simulate(2, 14, 16, spin_limit=0, stall=(0, 50))
    assert ctr[COUNTER_WORDS - 1] == 1
    ctr[COUNTER_WORDS - 1] = 0
    assert not ctr.any()


def test_batch_limit_matches_counter_block():
    assert 2 * 2046 + 3 <= COUNTER_WORDS < 2 * 2047 + 3


# ---------------------------------------------------------------- TWO_PASS
def fold_pass(x, g, K, B, nvalid, ws, counts):
    """The fold pass (fold_pass_kernel): workgroup (b, m) of 512 threads,
    8 waves of 64 lanes x 8 registers, with the kernel's M1 / M2 layouts,
    LDS addresses and workspace offsets.  Writes ws, counts every access."""
    HB = K - TB
    R, Q = TB - HB, 21 - K
    A, LJ = TB - Q, Q - 2
    W0 = 6 - LJ
    t = np.arange(512)
    j1, h1 = (t & ((1 << LJ) - 1)) << 2, t >> LJ
    j2, h2 = t & ((1 << Q) - 1), t >> Q

    def hi2(k):
        return (h2 & ((1 << W0) - 1)) | (k << W0) | ((h2 >> W0) << (HB - 1))

    def per_wave(v, fn):
        w = v.reshape(NV, 8, LANES)
        return np.stack([fn(w[:, i, :]) for i in range(8)], axis=1).reshape(NV, 512)

    def lane_stage(v):
        v = reg_bfly(reg_bfly(v, 0), 1)
        for J in range(LJ):
            v = lane_bfly(v, J)
        return v

    for b in range(B):
        for m in range(1 << A):
            gv = np.stack([g[(hi2(k) << TB) | (m << Q) | j2] for k in range(NV)]) * 2.0 ** -K
            np.add.at(counts["g"], np.stack([(hi2(k) << TB) | (m << Q) | j2
                                             for k in range(NV)]).ravel(), 1)
            v = np.zeros((NV, 512))
            for rr in range(2):
                row = (h1 | (rr << (HB - 1))) << TB
                for a in range(1 << A):
                    s = -1.0 if bin(m & a).count("1") & 1 else 1.0
                    i0 = row + (a << Q) + j1
                    ok = i0 < nvalid                       # whole 4-groups (nvalid % 8 == 0)
                    for e in range(4):
                        idx = b * nvalid + i0 + e
                        v[4 * rr + e, ok] += s * x[idx[ok]]
                        np.add.at(counts["x"], idx[ok], 1)
            v = per_wave(v, lane_stage)
            v = per_wave(v, lambda w: wave_bfly(w, LJ))
            lds = np.full(1 << (HB + Q), np.nan)
            lds_w = np.zeros(lds.size, int)
            for rr in range(2):
                a0 = ((h1 | (rr << (HB - 1))) << Q) | j1
                for wv in range(8):                        # a wave writes 1 KiB contiguous
                    seg = a0[wv * 64:(wv + 1) * 64]
                    assert np.array_equal(np.sort(seg), seg.min() + 4 * np.arange(64))
                for e in range(4):
                    lds[a0 + e] = v[4 * rr + e]
                    np.add.at(lds_w, a0 + e, 1)
            assert np.all(lds_w == 1)
            addr2 = np.stack([(hi2(k) << Q) | j2 for k in range(NV)])
            for k in range(NV):                            # 64 consecutive floats per wave
                for wv in range(8):
                    seg = addr2[k, wv * 64:(wv + 1) * 64]
                    assert np.array_equal(np.sort(seg), seg.min() + np.arange(64))
            assert np.array_equal(np.sort(addr2.ravel()), np.arange(lds.size))
            u = lds[addr2]
            u = reg_bfly(reg_bfly(reg_bfly(u, 0), 1), 2) * gv
            u = reg_bfly(reg_bfly(reg_bfly(u, 0), 1), 2)
            lds[addr2] = u
            for rr in range(2):
                a0 = ((h1 | (rr << (HB - 1))) << Q) | j1
                for e in range(4):
                    v[4 * rr + e] = lds[a0 + e]
            v = per_wave(v, lambda w: wave_bfly(w, LJ))
            t9 = (m << Q) | j1
            dst = (b << K) + ((t9 >> R) << TB) + (t9 & ((1 << R) - 1))
            for rr in range(2):
                for e in range(4):
                    off = dst + ((h1 | (rr << (HB - 1))) << R) + e
                    assert off.min() >= b << K and off.max() < (b + 1) << K
                    ws[off] = v[4 * rr + e]
                    np.add.at(counts["ws"], off, 1)


def run_two_pass(x, g, K, B, nvalid, layout):
    HB = K - TB
    R = TB - HB
    ws = np.full(B << K, np.nan)
    counts = {"x": np.zeros(B * nvalid, int), "g": np.zeros(1 << K, int),
              "ws": np.zeros(B << K, int)}
    fold_pass(x, g, K, B, nvalid, ws, counts)
    assert np.all(counts["ws"] == 1)
    assert np.all(counts["g"] == B)
    # each workgroup reads its whole slice once
    assert np.all(counts["x"] == 1 << (TB - (21 - K)))
    y = np.full(B * nvalid, np.nan)
    T_io = t_index(layout)
    for b in range(B):                                   # pass 3, as in run_pipeline
        for hi in range(1 << HB):
            start = hi << TB
            valid = max(0, min(nvalid - start, 512))
            if valid == 0:
                continue
            v = wht9(ws[(b << K) + (hi << R) + run_off(T_io, R)])
            ok = T_io < valid
            y[b * nvalid + start + T_io[ok]] = v[ok]
    return y


@pytest.mark.parametrize("K,B,N,C,layout", [
    (16, 1, 1024, 64, "V4"), (15, 2, 256, 128, "V8"), (16, 1, 1000, 64, "V4"),
    (15, 1, 200, 128, "V4"), (16, 2, 512, 128, "V8"),
])
def test_two_pass_matches_oracle(K, B, N, C, layout):
    """The fold pass then pass 3 reproduce the oracle (padded N included):
    the fold's signs, H over j, the hi butterflies split between M1 and M2
    and the run layout pass 3 gathers are all exercised."""
    P = 1 << max(0, (N - 1).bit_length())
    assert P * C == 1 << K
    rng = np.random.default_rng(K * 10 + B + N)
    x = rng.standard_normal((B, N, C))
    g = rng.uniform(0.5, 1.5, (P, C))
    y = run_two_pass(x.reshape(-1), g.reshape(-1), K, B, N * C, layout)
    ref = oracle_mod.whtmix(x, g)
    np.testing.assert_allclose(y.reshape(B, N, C), ref, rtol=0, atol=1e-9 * np.abs(ref).max())


@pytest.mark.parametrize("K", [15, 16])
def test_fold_workgroup_owns_whole_middle_tiles(K):
    """Workgroup m writes t9 in [m*2^Q, (m+1)*2^Q): 2^(Q-R) = 8 whole runs
    of pass 3's layout, i.e. 2^12 contiguous floats."""
    HB, Q = K - TB, 21 - K
    R = TB - HB
    assert Q - R == 3 and HB + Q == 12
    for m in range(1 << (TB - Q)):
        t9 = (m << Q) + np.arange(1 << Q)
        offs = np.concatenate([((t >> R) << TB) + (np.arange(1 << HB) << R) + (t & ((1 << R) - 1))
                               for t in t9])
        assert np.array_equal(np.sort(offs), (m << 12) + np.arange(1 << 12))


@pytest.mark.parametrize("K", [15, 16])
@pytest.mark.parametrize("B", [1, 3, 8, 13, 16, 47])
def test_fold_blocks_cover_each_slice_on_one_xcd(K, B):
    """fold_pass_kernel's block numbering: block i (on XCD i mod 8) takes
    slice ((i >> (A+3)) << 3) | (i & 7) and part (i >> 3) mod 2^A; the grid is
    B rounded up to 8 slices.  Every (slice, part) is taken once, the parts
    of a slice share one XCD, and only blocks past the last slice idle."""
    A = TB - (21 - K)
    grid = ((B + 7) // 8) << (A + 3)
    seen, xcd_of = {}, {}
    idle = 0
    for i in range(grid):
        b = ((i >> (A + 3)) << 3) | (i & 7)
        m = (i >> 3) & ((1 << A) - 1)
        if b >= B:
            idle += 1
            continue
        assert (b, m) not in seen
        seen[(b, m)] = i
        assert xcd_of.setdefault(b, i % 8) == i % 8
    assert len(seen) == B << A
    assert idle == grid - (B << A)
    assert grid * 512 < 1 << 32
