"""Host-side checks of the C ABI (no GPU needed).

* The packed metadata blob of dsv_segments_build equals, word for word, the
  blob of an independent Python packer written from the documented rules
  (plan.h / dsv.h): per-row adapter map, ascending training-row order, rows of
  each adapter for the rank-r shrink, the tile-group / gathered split decided
  per 128-row block, the GEMM tile lists, the backward chunks and items.
* Permuting the segment table leaves the blob unchanged.
* Every validation error returns its status and builds no plan.
* The library loads without a GPU and exports every function dsv.h declares.
"""
import os
import re
import struct
import subprocess

import numpy as np
import pytest

from paper_2607_28848_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dsv.h")

TILE_M, BLOCK_M, BLOCK_GROUPS, MAX_GROUPS, MIN_GROUP_ROWS = 256, 128, 4, 8, 4
ITEM_ROWS, RANK_ITEM_ROWS, CHUNK_ROWS = 16, 32, 256
TILE_WORDS = 4 + 3 * MAX_GROUPS


def _runs(ad, lo, hi):
    out, s = [], lo
    for t in range(lo + 1, hi + 1):
        if t == hi or ad[t] != ad[s]:
            out.append([s, t, ad[s]])
            s = t
    return out


def _chunked(items_src, limit):
    """[(adapter, begin, count, 0)] of consecutive same-adapter entries, <= limit each."""
    out, i = [], 0
    n = len(items_src)
    while i < n:
        a, j = items_src[i], i
        while j < n and items_src[j] == a and j - i < limit:
            j += 1
        out += [a, i, j - i, 0]
        i = j
    return out


def py_pack(segments, T, ranks, scales):
    """Independent packer of the plan blob (int32 words)."""
    n_ad = len(ranks)
    order = sorted([i for i, s in enumerate(segments) if s[1] > 0], key=lambda i: (segments[i][0], i))
    row_ad = [0] * T
    is_tr = [0] * T
    for i in order:
        st, ln, a, tr = segments[i]
        for t in range(st, st + ln):
            row_ad[t], is_tr[t] = a, tr
    train_rows = [t for t in range(T) if is_tr[t]]
    row_train = [-1] * T
    for i, t in enumerate(train_rows):
        row_train[t] = i
    tr_ad = [row_ad[t] for t in train_rows]
    Tt = len(train_rows)
    shrink_rows = sorted(range(T), key=lambda t: (row_ad[t], t))
    shrink_items = []
    i = 0
    while i < T:
        a, j = row_ad[shrink_rows[i]], i
        while j < T and row_ad[shrink_rows[j]] == a and j - i < RANK_ITEM_ROWS:
            j += 1
        shrink_items += [a, i, j - i, 0]
        i = j
    # per-128-row block: tile groups vs gathered rows
    gathered = [0] * T
    blocks = []
    for r0 in range(0, T, BLOCK_M):
        r1 = min(T, r0 + BLOCK_M)
        runs = _runs(row_ad, r0, r1)
        idx = sorted(range(len(runs)), key=lambda k: (-(runs[k][1] - runs[k][0]), k))
        groups = []
        for k in idx:
            if len(groups) < BLOCK_GROUPS and runs[k][1] - runs[k][0] >= MIN_GROUP_ROWS:
                groups.append(list(runs[k]))
        groups.sort(key=lambda g: g[0])
        glos = {g[0] for g in groups}
        hg = 0
        for r in runs:
            if r[0] not in glos:
                hg = 1
                for t in range(r[0], r[1]):
                    gathered[t] = 1
        blocks.append((groups, hg))

    def fwd_tiles(tm):
        out = []
        per = tm // BLOCK_M
        for b0 in range(0, len(blocks), per):
            r0, r1 = b0 * BLOCK_M, min(T, b0 * BLOCK_M + tm)
            groups, hg = [], 0
            for b in range(b0, min(b0 + per, len(blocks))):
                hg |= blocks[b][1]
                for g in blocks[b][0]:
                    if groups and groups[-1][1] == g[0] and groups[-1][2] == g[2]:
                        groups[-1][1] = g[1]
                    else:
                        groups.append(list(g))
            w = [r0, len(groups), hg, r1 - r0] + [0] * (3 * MAX_GROUPS)
            for k, (lo, hi, a) in enumerate(groups):
                w[4 + 3 * k: 7 + 3 * k] = [a, lo - r0, hi - r0]
            out += w
        return out

    gather_rows = [t for t in shrink_rows if gathered[t]]
    gslot = [-1] * T
    for s, t in enumerate(gather_rows):
        gslot[t] = s
    gather_items = _chunked([row_ad[t] for t in gather_rows], ITEM_ROWS)

    def bwd_tiles(tm):
        out, runs, k, r0 = [], _runs(tr_ad, 0, Tt), 0, 0
        while r0 < Tt:
            limit = min(Tt, r0 + tm)
            w = [r0, 0, 0, 0] + [0] * (3 * MAX_GROUPS)
            cur, ng = r0, 0
            while cur < limit and ng < MAX_GROUPS:
                hi = min(runs[k][1], limit)
                w[4 + 3 * ng: 7 + 3 * ng] = [runs[k][2], cur - r0, hi - r0]
                ng += 1
                cur = hi
                if cur == runs[k][1]:
                    k += 1
            w[1], w[3] = ng, cur - r0
            out += w
            r0 = cur
        return out

    train_ads = sorted(set(tr_ad))
    ad_slot = [-1] * n_ad
    for s, a in enumerate(train_ads):
        ad_slot[a] = s
    chunks, titems = [], []
    for lo, hi, a in (_runs(tr_ad, 0, Tt) if Tt else []):
        for b in range(lo, hi, CHUNK_ROWS):
            chunks += [a, b, min(CHUNK_ROWS, hi - b), ad_slot[a]]
        for b in range(lo, hi, ITEM_ROWS):
            titems += [a, b, min(ITEM_ROWS, hi - b), 0]
    n_chunks = len(chunks) // 4
    tad_ptr, tad_chunks = [0], []
    for s in range(len(train_ads)):
        tad_chunks += [c for c in range(n_chunks) if chunks[4 * c + 3] == s]
        tad_ptr.append(len(tad_chunks))
    scale_bits = list(np.asarray(scales, np.float32).view(np.int32))
    blob = []
    for arr in (row_ad, row_train, train_rows, tr_ad, shrink_rows, shrink_items, gslot, gather_rows,
                gather_items, fwd_tiles(TILE_M), fwd_tiles(BLOCK_M), bwd_tiles(TILE_M),
                bwd_tiles(BLOCK_M), chunks, titems, train_ads, ad_slot, tad_ptr, tad_chunks,
                list(ranks), scale_bits):
        blob += [0] * ((-len(blob)) % 64)
        blob += list(arr)
    blob += [0] * ((-len(blob)) % 64)
    return np.asarray(blob, np.int64).astype(np.int32)


def _dsv():
    from paper_2607_28848_amd import dsv
    return dsv


def _cases():
    rng = np.random.default_rng(2)
    pieces = [(int(l), int(a), 0) for l, a in zip(rng.integers(1, 40, 40), rng.integers(0, 6, 40))]
    pieces += [(300, 2, 1), (7, 4, 1), (1, 0, 1), (513, 2, 1)]
    order = rng.permutation(len(pieces))
    segs, s = [], 0
    for i in order:
        l, a, t = pieces[i]
        segs.append((s, l, a, t))
        s += l
    yield "mixed", segs, [8, 16, 64, 5, 32, 1], 64
    yield "tiny", wl.tiny().segments, [8, 8], 8
    w = wl.llama8b_mixed()
    yield "llama8b", w.segments, list(w.ranks), w.r_max
    w = wl.decode_heavy()
    yield "decode", w.segments, list(w.ranks), w.r_max
    w = wl.load_sweep(0.5)
    yield "sweep", w.segments, list(w.ranks), w.r_max
    yield "inference_only", [(0, 70, 1, 0), (70, 3, 0, 0)], [4, 4], 4
    yield "many_train_adapters", [(t, 1, t % 11, 1) for t in range(40)] + [(40, 9, 3, 0)], [3] * 11, 3


@pytest.mark.parametrize("name,segs,ranks,r_max", list(_cases()), ids=[c[0] for c in _cases()])
def test_blob_matches_independent_packer(name, segs, ranks, r_max):
    dsv = _dsv()
    T = sum(s[1] for s in segs)
    scales = np.linspace(0.5, 3.0, len(ranks)).astype(np.float32)
    plan = dsv.segments_build(segs, T, ranks, scales, r_max)
    got = plan.meta_words()
    ref = py_pack([tuple(s) for s in segs], T, ranks, scales)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    np.testing.assert_array_equal(got, ref)
    tr = [t for (st, l, a, x) in sorted(segs) if x for t in range(st, st + l)]
    np.testing.assert_array_equal(plan.train_rows(), sorted(tr))
    c = plan.counts()
    assert c["gathered_rows"] == len(plan.gathered_rows())
    # permuting the table changes nothing
    perm = [segs[i] for i in np.random.default_rng(0).permutation(len(segs))]
    np.testing.assert_array_equal(dsv.segments_build(perm, T, ranks, scales, r_max).meta_words(), got)


def _random_table(rng):
    """A random valid table: T in [0, 1200], pieces of 1..300 rows (mostly short),
    random adapters, ranks and training flags, in random table order, with a few
    zero-length entries mixed in."""
    n_ad = int(rng.integers(1, 12))
    r_max = int(rng.choice([1, 4, 8, 16, 33, 64]))
    ranks = [int(x) for x in rng.integers(1, r_max + 1, n_ad)]
    T_target = int(rng.integers(1, 1201)) if rng.random() > 0.08 else 0   # some empty batches
    segs, s = [], 0
    while s < T_target:
        ln = int(min(T_target - s, rng.choice([1, 2, 3, 5, 16, 40, 127, 300])))
        segs.append((s, ln, int(rng.integers(0, n_ad)), int(rng.random() < 0.4)))
        s += ln
    for _ in range(int(rng.integers(0, 3))):
        segs.append((int(rng.integers(0, s + 1)), 0, int(rng.integers(0, n_ad)), int(rng.integers(0, 2))))
    segs = [segs[i] for i in rng.permutation(len(segs))]
    return segs, s, ranks, r_max


def _corrupt(rng, segs, T, ranks, r_max):
    """Apply one defect; returns (segs, T, ranks, r_max, expected status name)."""
    nz = [i for i, x in enumerate(segs) if x[1] > 0]
    kind = int(rng.integers(0, 8))
    segs = list(segs)
    ranks = list(ranks)
    if kind == 0 and nz:                       # drop a non-empty entry: gap, or short of T
        del segs[nz[int(rng.integers(0, len(nz)))]]
        return segs, T, ranks, r_max, "ERR_LAYOUT"
    if kind == 1 and nz:                       # lengthen one entry: overlap, or past T
        i = nz[int(rng.integers(0, len(nz)))]
        st, ln, a, tr = segs[i]
        segs[i] = (st, ln + int(rng.integers(1, 4)), a, tr)
        return segs, T, ranks, r_max, "ERR_LAYOUT"
    if kind == 2 and segs:                     # adapter id out of range
        i = int(rng.integers(0, len(segs)))
        st, ln, a, tr = segs[i]
        segs[i] = (st, ln, int(rng.choice([-1, len(ranks), len(ranks) + 7])), tr)
        return segs, T, ranks, r_max, "ERR_RANGE"
    if kind == 3 and segs:                     # training flag not 0/1
        i = int(rng.integers(0, len(segs)))
        st, ln, a, tr = segs[i]
        segs[i] = (st, ln, a, int(rng.choice([-1, 2, 255])))
        return segs, T, ranks, r_max, "ERR_RANGE"
    if kind == 4:                              # one rank outside [1, r_max]
        ranks[int(rng.integers(0, len(ranks)))] = int(rng.choice([0, -3, r_max + 1]))
        return segs, T, ranks, r_max, "ERR_RANGE"
    if kind == 5:                              # r_max outside [1, 64]
        return segs, T, ranks, int(rng.choice([0, -1, 65, 1 << 30])), "ERR_RANGE"
    if kind == 6 and nz:                       # negative start or length
        i = nz[int(rng.integers(0, len(nz)))]
        st, ln, a, tr = segs[i]
        segs[i] = (-1 - st, ln, a, tr) if rng.random() < 0.5 else (st, -ln, a, tr)
        return segs, T, ranks, r_max, "ERR_LAYOUT"
    return segs, T, ranks, r_max, "OK"


@pytest.mark.parametrize("seed", range(40))
def test_random_tables_valid_and_defective(seed):
    """Random tables, half of them with one defect: a valid table packs to the
    independent packer's blob and answers every query consistently; a defective
    one returns its status and builds no plan.  (Also the workload of the
    host-sanitizer run of this file.)"""
    dsv = _dsv()
    rng = np.random.default_rng(1000 + seed)
    segs, T, ranks, r_max = _random_table(rng)
    scales = [float(x) for x in rng.uniform(-4, 4, len(ranks)).astype(np.float32)]
    if seed % 2:
        segs, T, ranks, r_max, status = _corrupt(rng, segs, T, ranks, r_max)
    else:
        status = "OK"
    if status != "OK":
        with pytest.raises(dsv.DsvError) as e:
            dsv.segments_build(segs, T, ranks, scales, r_max)
        assert e.value.status == getattr(dsv, status)
        return
    plan = dsv.segments_build(segs, T, ranks, scales, r_max)
    np.testing.assert_array_equal(plan.meta_words(), py_pack(segs, T, ranks, scales))
    tr = sorted(t for (st, l, a, x) in segs if x for t in range(st, st + l))
    np.testing.assert_array_equal(plan.train_rows(), tr)
    c = plan.counts()
    g = plan.gathered_rows()
    assert c["gathered_rows"] == len(g) and len(set(g.tolist())) == len(g)
    assert all(0 <= t < T for t in g.tolist())
    for dt in (dsv.BF16, dsv.F32):
        for K, N in ((8, 8), (4096, 14336), (14336, 4096)):
            assert dsv.fwd_workspace_bytes(plan, dt, K, N) >= 0
            assert dsv.bwd_workspace_bytes(plan, dt, K, N) >= 0


def test_zero_length_segments_are_ignored():
    dsv = _dsv()
    segs = [(0, 5, 0, 0), (5, 0, 1, 1), (5, 3, 1, 1), (8, 0, 0, 0)]
    a = dsv.segments_build(segs, 8, [2, 2], [1.0, 1.0], 2).meta_words()
    b = dsv.segments_build([segs[0], segs[2]], 8, [2, 2], [1.0, 1.0], 2).meta_words()
    np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("segs,T,ranks,r_max,status", [
    ([(0, 4, 0, 0), (5, 3, 0, 0)], 8, [2], 2, "ERR_LAYOUT"),      # gap
    ([(0, 5, 0, 0), (4, 4, 0, 0)], 8, [2], 2, "ERR_LAYOUT"),      # overlap
    ([(0, 7, 0, 0)], 8, [2], 2, "ERR_LAYOUT"),                    # does not reach T
    ([(0, 9, 0, 0)], 8, [2], 2, "ERR_LAYOUT"),                    # runs past T
    ([(-1, 9, 0, 0)], 8, [2], 2, "ERR_LAYOUT"),                   # negative start
    ([(0, 8, 0, 0), (3, -1, 0, 0)], 8, [2], 2, "ERR_LAYOUT"),     # negative length
    ([(0, 8, 1, 0)], 8, [2], 2, "ERR_RANGE"),                     # adapter id
    ([(0, 8, -1, 0)], 8, [2], 2, "ERR_RANGE"),
    ([(0, 8, 0, 2)], 8, [2], 2, "ERR_RANGE"),                     # is_train flag
    ([(0, 8, 0, 0)], 8, [3], 2, "ERR_RANGE"),                     # rank > r_max
    ([(0, 8, 0, 0)], 8, [0], 2, "ERR_RANGE"),                     # rank < 1
    ([(0, 8, 0, 0)], 8, [2], 65, "ERR_RANGE"),                    # r_max > 64
    ([(0, 8, 0, 0)], 8, [2], 0, "ERR_RANGE"),
])
def test_validation_errors(segs, T, ranks, r_max, status):
    dsv = _dsv()
    with pytest.raises(dsv.DsvError) as e:
        dsv.segments_build(segs, T, ranks, [1.0] * len(ranks), r_max)
    assert e.value.status == getattr(dsv, status)


def test_nonfinite_scale_rejected():
    dsv = _dsv()
    with pytest.raises(dsv.DsvError) as e:
        dsv.segments_build([(0, 4, 0, 0)], 4, [2], [float("nan")], 2)
    assert e.value.status == dsv.ERR_RANGE


def test_host_only_plan_rejected_by_fwd_bwd_and_shape_checks():
    import ctypes
    dsv = _dsv()
    lib = dsv.lib_handle()
    plan = dsv.segments_build([(0, 16, 0, 1)], 16, [4], [2.0], 4)
    fake = ctypes.c_void_p(4096)
    args = [fake] * 4
    rc = lib.dsv_cobatch_fwd(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, fake, 1 << 20, None)
    assert rc == dsv.ERR_ARG
    rc = lib.dsv_lora_bwd(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, fake, fake, fake, 0,
                          fake, 1 << 20, None)
    assert rc == dsv.ERR_ARG
    for K, N in ((60, 64), (64, 0), (-8, 64)):
        assert lib.dsv_cobatch_fwd(plan.handle, dsv.BF16, K, N, *args, fake, fake, fake, 0, None) == dsv.ERR_SIZE
    assert lib.dsv_cobatch_fwd(plan.handle, 7, 64, 64, *args, fake, fake, fake, 0, None) == dsv.ERR_RANGE
    assert lib.dsv_lora_bwd(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, fake, fake, fake, 2,
                            fake, 0, None) == dsv.ERR_RANGE
    assert lib.dsv_cobatch_fwd(None, dsv.BF16, 64, 64, *args, fake, fake, fake, 0, None) == dsv.ERR_ARG
    # workspace queries are pure host arithmetic
    assert dsv.fwd_workspace_bytes(plan, dsv.BF16, 64, 64) > 0
    assert dsv.bwd_workspace_bytes(plan, dsv.BF16, 64, 64) > 0


def test_status_strings():
    dsv = _dsv()
    lib = dsv.lib_handle()
    for s in (0, -1, -2, -3, -4, -5, 99):
        assert lib.dsv_status_string(s)


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dsv_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    dsv = _dsv()
    names = _declared_functions()
    assert len(names) >= 12
    out = subprocess.run(["nm", "-D", "--defined-only", dsv.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(l.split()[-1] for l in out.splitlines() if l.strip())
    missing = [n for n in names if n not in exported]
    assert not missing, missing
    lib = dsv.lib_handle()
    for n in names:
        assert getattr(lib, n) is not None


def test_dropout_argument_checks_on_host():
    """dsv_cobatch_fwd_dropout / dsv_lora_bwd_dropout reject a missing dropout
    (ERR_ARG) and p outside [0, 1) (ERR_RANGE) before looking at the plan's device
    state; the dropout workspace of the backward is at least the plain one."""
    import ctypes
    dsv = _dsv()
    lib = dsv.lib_handle()
    plan = dsv.segments_build([(0, 16, 0, 1)], 16, [4], [2.0], 4)
    fake = ctypes.c_void_p(4096)
    args = [fake] * 4
    for p in (-0.1, 1.0, 1.5, float("nan"), float("inf")):
        d = dsv.Dropout(p, 1, 0)
        assert lib.dsv_cobatch_fwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, ctypes.byref(d),
                                           fake, 1 << 20, None) == dsv.ERR_RANGE
        assert lib.dsv_lora_bwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, fake, fake, fake, 0,
                                        ctypes.byref(d), fake, 1 << 20, None) == dsv.ERR_RANGE
    assert lib.dsv_cobatch_fwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, None, fake, 1 << 20,
                                       None) == dsv.ERR_ARG
    assert lib.dsv_lora_bwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, fake, fake, fake, 0, None,
                                    fake, 1 << 20, None) == dsv.ERR_ARG
    # a mask buffer that is not 4-byte aligned
    d = dsv.Dropout(0.05, 1, 0, ctypes.c_void_p(4098))
    assert lib.dsv_cobatch_fwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, ctypes.byref(d), fake,
                                       1 << 20, None) == dsv.ERR_ARG
    assert lib.dsv_lora_bwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, fake, fake, fake, 0,
                                    ctypes.byref(d), fake, 1 << 20, None) == dsv.ERR_ARG
    d = dsv.Dropout(0.05, 1, 0)  # valid: the host-only plan is what is rejected
    assert lib.dsv_cobatch_fwd_dropout(plan.handle, dsv.BF16, 64, 64, *args, fake, fake, ctypes.byref(d), fake,
                                       1 << 20, None) == dsv.ERR_ARG
    for dt in (dsv.BF16, dsv.F32):
        plain = dsv.bwd_workspace_bytes(plan, dt, 520, 64)
        drop = dsv.bwd_workspace_bytes(plan, dt, 520, 64, dropout=True)
        assert drop >= plain


def test_grouped_argument_checks_on_host():
    """The grouped entry points reject a bad group size (ERR_RANGE), missing entries
    (ERR_ARG) and a bad shape in any entry (ERR_SIZE) before touching the device;
    a group of one has the single call's workspace; a group's workspace holds every
    projection's regions."""
    import ctypes
    dsv = _dsv()
    lib = dsv.lib_handle()
    plan = dsv.segments_build([(0, 16, 0, 1), (16, 300, 1, 0)], 316, [4, 4], [2.0, 2.0], 4)
    fake = ctypes.c_void_p(4096)
    arr = (dsv.FwdProj * 9)()
    for i in range(9):
        arr[i] = dsv.FwdProj(64, 64, fake, fake, fake, fake, fake, fake)
    for n in (0, -1, 9):
        assert lib.dsv_cobatch_fwd_grouped(plan.handle, dsv.BF16, n, arr, fake, 1 << 20, None) == dsv.ERR_RANGE
    assert lib.dsv_cobatch_fwd_grouped(plan.handle, dsv.BF16, 2, None, fake, 1 << 20, None) == dsv.ERR_ARG
    arr[1].K = 60
    assert lib.dsv_cobatch_fwd_grouped(plan.handle, dsv.BF16, 2, arr, fake, 1 << 20, None) == dsv.ERR_SIZE
    arr[1].K = 64
    assert lib.dsv_cobatch_fwd_grouped(plan.handle, dsv.BF16, 2, arr, fake, 1 << 20, None) == dsv.ERR_ARG
    barr = (dsv.BwdProj * 2)()
    for i in range(2):
        barr[i] = dsv.BwdProj(64, 64, fake, fake, fake, fake, fake, fake, fake, fake, fake)
    assert lib.dsv_lora_bwd_grouped(plan.handle, dsv.BF16, 2, barr, 2, fake, 1 << 20, None) == dsv.ERR_RANGE
    assert lib.dsv_lora_bwd_grouped(plan.handle, dsv.BF16, 2, barr, 0, fake, 1 << 20, None) == dsv.ERR_ARG
    for dt in (dsv.BF16, dsv.F32):
        assert dsv.fwd_grouped_workspace_bytes(plan, dt, [(520, 776)]) == dsv.fwd_workspace_bytes(plan, dt, 520, 776)
        assert dsv.bwd_grouped_workspace_bytes(plan, dt, [(520, 776)]) == dsv.bwd_workspace_bytes(plan, dt, 520, 776)
        shapes = [(520, 776), (4096, 1024), (136, 64)]
        # each projection's h / low-rank / partial regions, without split-tile partials
        assert dsv.fwd_grouped_workspace_bytes(plan, dt, shapes) >= sum(
            dsv.fwd_workspace_bytes(plan, dt, 64, 64) for _ in shapes)
        assert dsv.bwd_grouped_workspace_bytes(plan, dt, shapes) >= sum(
            dsv.bwd_workspace_bytes(plan, dt, K, 64) for K, _ in shapes) // 2


def test_row_strides_checked_on_host():
    """Row strides of the grouped calls: 0 (dense) and any multiple of 8 from the row
    length up to 2^20 pass the checks (the host-only plan then fails with ERR_ARG);
    a stride shorter than a row, not a multiple of 8, above 2^20 or negative fails
    with ERR_SIZE before anything else, in a group of one and of two, for every
    strided operand.  dsv_row_stride pads long bf16 rows whose byte length is a
    multiple of 4096; the binding passes a row-strided view's stride and refuses
    non-contiguous operands in the single-projection calls."""
    import ctypes
    import torch
    dsv = _dsv()
    lib = dsv.lib_handle()
    plan = dsv.segments_build([(0, 16, 0, 1), (16, 300, 1, 0)], 316, [4, 4], [2.0, 2.0], 4)
    fake = ctypes.c_void_p(4096)
    K, N = 72, 136
    lens = {"ldx": K, "ldw": K, "ldy": N, "lddy": N, "lddx": K, "ldwt": N}
    for n in (1, 2):
        arr = (dsv.FwdProj * n)()
        for i in range(n):
            arr[i] = dsv.FwdProj(K, N, fake, fake, fake, fake, fake, fake)
        assert lib.dsv_cobatch_fwd_grouped(plan.handle, dsv.BF16, n, arr, fake, 1 << 20, None) == dsv.ERR_ARG
        for f in ("ldx", "ldw", "ldy"):
            for v in (lens[f], lens[f] + 8, lens[f] + 64, 1 << 20):
                setattr(arr[n - 1], f, v)
                assert lib.dsv_cobatch_fwd_grouped(plan.handle, dsv.BF16, n, arr, fake, 1 << 20, None) == dsv.ERR_ARG
            for v in (lens[f] - 8, lens[f] + 4, (1 << 20) + 8, -8):
                setattr(arr[n - 1], f, v)
                for dt in (dsv.BF16, dsv.F32):
                    assert lib.dsv_cobatch_fwd_grouped(plan.handle, dt, n, arr, fake, 1 << 20, None) == dsv.ERR_SIZE, (f, v)
            setattr(arr[n - 1], f, 0)
        barr = (dsv.BwdProj * n)()
        for i in range(n):
            barr[i] = dsv.BwdProj(K, N, fake, fake, fake, fake, fake, fake, fake, fake, fake, fake)
        assert lib.dsv_lora_bwd_grouped(plan.handle, dsv.BF16, n, barr, 0, fake, 1 << 20, None) == dsv.ERR_ARG
        for f in ("ldx", "ldw", "lddy", "lddx", "ldwt"):
            setattr(barr[n - 1], f, lens[f] + 64)
            assert lib.dsv_lora_bwd_grouped(plan.handle, dsv.BF16, n, barr, 0, fake, 1 << 20, None) == dsv.ERR_ARG
            for v in (lens[f] - 8, lens[f] + 4, (1 << 20) + 8, -8):
                setattr(barr[n - 1], f, v)
                for dt in (dsv.BF16, dsv.F32):
                    assert lib.dsv_lora_bwd_grouped(plan.handle, dt, n, barr, 0, fake, 1 << 20, None) == dsv.ERR_SIZE, (f, v)
            setattr(barr[n - 1], f, 0)
    # the recommended stride
    assert dsv.row_stride(14336, dsv.BF16) == 14400
    assert dsv.row_stride(28672, dsv.BF16) == 28736
    for n in (4096, 8192, 1024, 10000, 14344, 8):
        assert dsv.row_stride(n, dsv.BF16) == n
    assert dsv.row_stride(14336, dsv.F32) == 14336
    assert dsv.row_stride(0, dsv.BF16) == 0 and dsv.row_stride(14336, 7) == 0
    # binding: the stride of a row-strided view, dense = 0, column-strided refused
    buf = torch.zeros((10, 88), dtype=torch.bfloat16)
    assert dsv._ld(buf[:, :72], 72) == 88
    assert dsv._ld(buf, 88) == 0 and dsv._ld(None, 72) == 0
    with pytest.raises(ValueError):
        dsv._ld(buf.t(), 10)
    with pytest.raises(ValueError):
        dsv._ld(buf[:, :72:2], 36)
    X = buf[:, :72]
    with pytest.raises(ValueError):
        dsv.cobatch_fwd(plan, X, torch.zeros((8, 72), dtype=torch.bfloat16), None, None)
    with pytest.raises(ValueError):
        dsv.lora_bwd(plan, X, torch.zeros((8, 72), dtype=torch.bfloat16), None, None, None, None)


def test_adamw_grouped_argument_checks_on_host():
    """dsv_adamw_step_grouped rejects a bad group size (ERR_RANGE), a NULL array
    (ERR_ARG), a bad shape in any entry (ERR_SIZE), bad hyper-parameters
    (ERR_RANGE) and a host-only plan (ERR_ARG) before touching the device."""
    import ctypes
    dsv = _dsv()
    lib = dsv.lib_handle()
    plan = dsv.segments_build([(0, 16, 0, 1)], 16, [4], [2.0], 4)
    fake = ctypes.c_void_p(4096)
    arr = (dsv.AdamWProj * 9)()
    for i in range(9):
        arr[i] = dsv.AdamWProj(64, 64, *([fake] * 10))
    hp = dsv.AdamWHparams(1e-3, 0.9, 0.999, 1e-8, 0.01)
    for n in (0, -1, 9):
        assert lib.dsv_adamw_step_grouped(plan.handle, dsv.BF16, n, arr, 1, ctypes.byref(hp), None) == dsv.ERR_RANGE
    assert lib.dsv_adamw_step_grouped(plan.handle, dsv.BF16, 2, None, 1, ctypes.byref(hp), None) == dsv.ERR_ARG
    arr[1].N = 60
    assert lib.dsv_adamw_step_grouped(plan.handle, dsv.BF16, 2, arr, 1, ctypes.byref(hp), None) == dsv.ERR_SIZE
    arr[1].N = 64
    assert lib.dsv_adamw_step_grouped(plan.handle, dsv.BF16, 2, arr, 1, ctypes.byref(hp), None) == dsv.ERR_ARG
    assert lib.dsv_adamw_step_grouped(None, dsv.BF16, 2, arr, 1, ctypes.byref(hp), None) == dsv.ERR_ARG
    assert lib.dsv_adamw_step(plan.handle, dsv.BF16, 64, 64, 1, ctypes.byref(hp), *([fake] * 10), None) == dsv.ERR_ARG
