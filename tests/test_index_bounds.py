"""A CPU model of the kernels' index arithmetic (no GPU): for seeded random
and extreme descriptors, every global address the work-order, partition and
merge kernels form stays inside its buffer, and the work order is a
permutation of the step's work items.

The model restates, formula by formula, what pda_order.hip,
pda_partition.hip and pda_merge.hip compute from a work item's index (its
partition, sequence, KV head and chunk group, or its shared-prefix group),
with the partition size, partition count and workspace taken from the
library's own plan (pda_plan / pda_plan_shared_prefix).  Tile loads are
bounds-checked by their buffer descriptors on the GPU; what is modelled here
is everything else: block-table entries read, query rows read, output rows
and partial states written, the workspace carving, and the LDS indices of the
staged path.
"""
import numpy as np
import pytest

import paper_2405_11143_amd as pda

BS = 16
WAVES, WAVE = 4, 64
MAX_GROUP = 16
ORDER_BUCKETS = 256
ID_WINDOW = 256


def plan_of(B, Hq, Hkv, D, mbps, mcl, tp, n, groups=None):
    prob = pda.make_problem(B, Hq, Hkv, D, 10 ** 6, mbps, mcl, tp, num_query_tokens=n)
    if groups is None:
        info = pda.pda_plan(prob)
    else:
        info = pda.pda_plan_shared_prefix(prob, pda.make_prefix_groups(len(groups["prefix"]), groups["max_size"],
                                                                         groups["max_prefix"]))
    G = Hq // Hkv
    qc = min(n, MAX_GROUP // G)
    nqc = -(-n // qc)
    cpg = 4 * WAVES if nqc > 2 * WAVES else 2 * WAVES if nqc > WAVES else WAVES
    ncg = -(-nqc // cpg)
    P = info["num_partitions"]
    Tp = info["partition_tokens"]
    Pp = -(-groups["max_prefix"] // Tp) if groups else 0
    MR = 64 // (n * G) if groups else 0  # members per row group (prefix item)
    RG = -(-min(groups["max_size"], B) // MR) if groups and len(groups["prefix"]) else 0
    regular = P * B * Hkv * ncg
    if groups:
        assert ncg == 1  # with groups both kinds of work-order pairs hold Hkv items
    items = regular + (len(groups["prefix"]) * Pp * RG * Hkv if groups else 0)
    split = P > 1 or groups is not None
    S = Pp + P
    slots = B * n * Hq * S if split else 0
    ws = slots * (D + 2) * 4 + items * 4 + (B * 4 if groups else 0)
    assert info["workspace_bytes"] == ws, (info, ws)  # the carving below matches the library's size
    return dict(G=G, qc=qc, nqc=nqc, cpg=cpg, ncg=ncg, P=P, Tp=Tp, Pp=Pp, MR=MR, RG=RG, regular=regular, items=items,
                S=S, slots=slots, split=split, ws=ws)


def chunk_visible(L, n, qc, c):
    i0 = c * qc
    nv = min(qc, n - i0)
    return L - n + i0 + nv


def model_order(B, Hkv, lens_c, mcl, pl, seq_prefix=None, groups=None):
    """The work-order kernel's writes: returns the order array (every slot
    written once, every value an item index)."""
    P, Tp, Pp, RG, HC = pl["P"], pl["Tp"], pl["Pp"], pl["RG"], Hkv * pl["ncg"]
    regular_pairs = B * P
    ngroups = len(groups["prefix"]) if groups else 0
    pairs = regular_pairs + ngroups * Pp * RG
    order = np.full(pairs * HC, -1, dtype=np.int64)

    def bucket(idx):
        if idx < regular_pairs:
            b, p = idx % B, idx // B
            L = lens_c[b]
            t0 = min(seq_prefix[b] if seq_prefix is not None else 0, L)
            tok = max(0, min(L, t0 + (p + 1) * Tp) - (t0 + p * Tp))
        else:  # (grp * Pp + pp) * RG + rg
            x = idx - regular_pairs
            rg, pp, grp = x % RG, (x // RG) % Pp, x // (RG * Pp)
            assert 0 <= grp < ngroups
            first = min(max(groups["start"][grp], 0), B)
            members = min(min(groups["start"][grp + 1], B) - first, groups["max_size"])
            plen = min(max(groups["prefix"][grp], 0), groups["max_prefix"])
            tok = max(0, min(plen, (pp + 1) * Tp) - pp * Tp) if rg * pl["MR"] < members else 0
        return ORDER_BUCKETS - 1 - min(-(-tok // BS), ORDER_BUCKETS - 1)

    classes = [bucket(i) for i in range(pairs)]
    counts = np.bincount(classes, minlength=ORDER_BUCKETS)
    start = np.concatenate([[0], np.cumsum(counts)[:-1]])
    for idx in range(pairs):  # one valid arrival order of the atomics
        pos = start[classes[idx]]
        start[classes[idx]] += 1
        if Hkv % 8 == 0:
            for x in range(HC):
                slot = pos * HC + x
                assert 0 <= slot < len(order) and order[slot] == -1
                order[slot] = idx * HC + (x % Hkv) * pl["ncg"] + x // Hkv
        else:
            r = pos % 8
            c = min(8, pairs - (pos - r))
            base = (pos - r) * HC + r
            for x in range(HC):
                slot = base + x * c
                assert 0 <= slot < len(order) and order[slot] == -1
                order[slot] = idx * HC + x
    assert sorted(order.tolist()) == list(range(pairs * HC)), "the order is a permutation of the work items"
    return order


def check_regular_item(item, B, Hq, Hkv, D, n, mbps, mcl, lens_c, pl, seq_prefix, touched):
    G, qc, nqc, cpg, ncg, Tp = pl["G"], pl["qc"], pl["nqc"], pl["cpg"], pl["ncg"], pl["Tp"]
    HC = Hkv * ncg
    gc = item % HC
    b = (item // HC) % B
    p = item // (HC * B)
    g, cg = gc // ncg, gc % ncg
    assert 0 <= b < B and 0 <= g < Hkv and 0 <= p < pl["P"] and 0 <= cg < ncg
    nw = 2 * WAVES if cpg > 2 * WAVES else WAVES  # wavefronts of the launch's workgroups
    nchunk = min(cpg, nqc - cg * cpg)  # the register-only variant runs only when every item has one chunk
    assert 1 <= nchunk <= (2 * nw if cpg > WAVES else nw)
    two = cpg > WAVES and nchunk > nw
    ntile = nw if two else nchunk
    slices = nw // ntile
    # the LDS epilogue arrays have nw entries: row_weights reads entry t + x * ntile (t < ntile, x < slices)
    assert slices >= 1 and ntile * slices <= nw
    if two:
        assert nchunk <= 2 * nw  # wavefront w folds chunks w and w + nw
    L = min(max(lens_c[b], 0), mcl)
    t0_all = seq_prefix[b] if seq_prefix is not None else 0
    rows_q = B * n * Hq

    def parts_of(c):
        lv = chunk_visible(L, n, qc, c)
        t0 = min(t0_all, max(lv, 0))
        return -(-(lv - t0) // Tp) if lv > 0 else 0

    chunks = [cg * cpg + t for t in range(nchunk)]
    assert all(c < nqc for c in chunks)
    nparts_max = max(parts_of(c) for c in chunks)
    for c in chunks:
        i0 = c * qc
        nv = min(qc, n - i0)
        assert nv >= 1
        for r in range(nv * G):  # query rows read, output rows written (zeros or final)
            row = (b * n + i0 + r // G) * Hq + g * G + r % G
            assert 0 <= row < rows_q
            if p == 0 and chunk_visible(L, n, qc, c) <= 0:
                touched["out"].add(row)
    if p >= nparts_max:
        return
    lv_last = chunk_visible(L, n, qc, chunks[-1])  # the kernel's first block: the item's last chunk's
    j_begin = (min(t0_all, max(lv_last, 0)) + p * Tp) // BS

    def block_end(lv, parts):
        t0 = min(t0_all, max(lv, 0))
        return -(-min(lv, t0 + (p + 1) * Tp) // BS) if p < parts else 0

    J1 = j_begin
    for c in chunks:
        J1 = max(J1, block_end(chunk_visible(L, n, qc, c), parts_of(c)))
    # block-table entries read: [j_begin, J1) of row b, within the blocks the context uses
    assert 0 <= j_begin <= J1 <= -(-L // BS) <= mbps, (j_begin, J1, L, mbps)
    # the staged path's id window and step buffers
    for jw in range(j_begin, J1, ID_WINDOW):
        assert min(J1, jw + ID_WINDOW) - jw <= ID_WINDOW
    for c in chunks:
        parts = parts_of(c)
        if p >= parts:
            continue
        i0 = c * qc
        nv = min(qc, n - i0)
        single = parts == 1 and min(t0_all, chunk_visible(L, n, qc, c)) == 0
        for h in range(nv * G):
            row = (b * n + i0 + h // G) * Hq + g * G + h % G
            if single:
                touched["out"].add(row)
            else:
                slot = row * pl["S"] + pl["Pp"] + p
                assert pl["split"] and 0 <= slot < pl["slots"], (slot, pl["slots"])
                touched["slots"].add(slot)


def check_prefix_item(pitem, B, Hq, Hkv, D, n, mcl, mbps, lens_c, pl, groups, touched):
    Pp, Tp, G, RG, MR = pl["Pp"], pl["Tp"], pl["G"], pl["RG"], pl["MR"]
    g = pitem % Hkv
    rg = (pitem // Hkv) % RG
    pp = (pitem // (Hkv * RG)) % Pp
    grp = pitem // (Hkv * RG * Pp)
    starts = groups["start"]
    assert 0 <= grp < len(groups["prefix"])
    first_g = min(max(starts[grp], 0), B)
    members_g = min(min(starts[grp + 1], B) - first_g, groups["max_size"])
    first = first_g + rg * MR
    members = min(MR, members_g - rg * MR)
    plen = groups["prefix"][grp]
    plen = 0 if plen < 0 else min(plen, groups["max_prefix"]) // BS * BS
    if members <= 0 or pp * Tp >= plen:
        return
    rows = members * n * G  # member-major, then the new tokens, then the G heads
    assert rows <= WAVES * MAX_GROUP
    j_begin, j_end = pp * Tp // BS, min(plen, (pp + 1) * Tp) // BS
    assert 0 <= first_g < B and 0 <= j_begin < j_end <= mbps  # table row of the group's first member
    for m in range(members):
        assert 0 <= first + m < B  # the lengths read for the rows' limits
    for rr in range(rows):
        m, i, h = rr // (n * G), (rr // G) % n, rr % G
        q_row = (first + m) * n + i
        row = q_row * Hq + g * G + h
        assert 0 <= row < B * n * Hq  # the query row read and the state written
        slot = row * pl["S"] + pp
        assert 0 <= slot < pl["slots"]
        touched["slots"].add(slot)


def check_merge(B, Hq, n, mcl, lens_c, pl, seq_prefix, touched):
    """Rows the merge reads (their slots) and writes."""
    Tp, S = pl["Tp"], pl["S"]
    for row in range(B * n * Hq):
        i = (row // Hq) % n
        b = row // (Hq * n)
        L = min(max(lens_c[b], 0), mcl)
        vis = chunk_visible(L, n, pl["qc"], i // pl["qc"])
        if vis <= 0:
            continue
        t0 = min(seq_prefix[b] if seq_prefix is not None else 0, vis)
        n_pre = -(-t0 // Tp)
        n_own = -(-(vis - t0) // Tp)
        if n_pre == 0 and n_own <= 1:
            assert row in touched["out"], "a final row that pass 1 did not write"
            continue
        for k in range(n_pre + n_own):
            slot = row * S + k + (pl["Pp"] - n_pre if k >= n_pre else 0)
            assert 0 <= slot < pl["slots"]
            assert slot in touched["slots"], "the merge reads a partial state pass 1 did not write"
        touched["out"].add(row)
    assert len(touched["out"]) == B * n * Hq, "every output row is written"


def staged_lds_indices(D, nw=WAVES):
    """The staging buffer's piece indices and the transposed V reads stay in one block."""
    TC = 16 * D * 2 // 16
    RP = D // 8
    block_pieces = TC + BS * (RP + 2)
    loads = 2 * 2 * TC // (nw * WAVE)
    assert loads * nw * WAVE == 2 * 2 * TC  # every piece of a step is loaded once
    for tid in range(nw * WAVE):
        for k in range(loads):
            ci = k * nw * WAVE + tid
            pc = ci % TC
            blk = ci // (2 * TC)
            dst = blk * block_pieces + (TC + pc // RP * (RP + 2) + pc % RP if (ci // TC) & 1 else pc)
            assert blk < 2 and 0 <= dst < 2 * block_pieces
            assert blk * block_pieces <= dst < (blk + 1) * block_pieces
    staged_row = D + 16
    for lane in range(WAVE):
        nn, kg = lane & 15, lane >> 4
        tr_off = (4 * kg + nn // 4) * staged_row + 4 * (nn % 4)
        for t in range(D // 16):
            e = tr_off + 16 * t
            assert 0 <= e and e + 4 <= BS * staged_row  # 4 elements read from the V part of the block
            assert (e % staged_row) + 4 <= D  # never into a row's padding


def run_case(rng, B, Hq, Hkv, D, n, mcl, tp, lens, mbps, groups=None):
    pl = plan_of(B, Hq, Hkv, D, mbps, mcl, tp, n, groups)
    lens_c = [min(max(int(x), 0), mcl) for x in lens]
    seq_prefix = None
    if groups:
        seq_prefix = [0] * B
        for grp in range(len(groups["prefix"])):
            first = min(max(groups["start"][grp], 0), B)
            last = min(min(groups["start"][grp + 1], B), first + groups["max_size"])
            plen = groups["prefix"][grp]
            plen = 0 if plen < 0 else min(plen, groups["max_prefix"]) // BS * BS
            for b in range(first, last):
                seq_prefix[b] = plen
    order = model_order(B, Hkv, lens_c, mcl, pl, seq_prefix, groups)
    assert len(order) == pl["items"]
    assert pl["slots"] * (D + 2) * 4 + len(order) * 4 <= pl["ws"]  # states, then the order (then prefixes)
    touched = {"out": set(), "slots": set()}
    for item in range(pl["items"]):
        if item < pl["regular"]:
            check_regular_item(item, B, Hq, Hkv, D, n, mbps, mcl, lens_c, pl, seq_prefix, touched)
        else:
            check_prefix_item(item - pl["regular"], B, Hq, Hkv, D, n, mcl, mbps, lens_c, pl, groups, touched)
    check_merge(B, Hq, n, mcl, lens_c, pl, seq_prefix, touched)


@pytest.mark.parametrize("D", [64, 128])
def test_staged_lds_indices(D):
    staged_lds_indices(D)
    staged_lds_indices(D, nw=2 * WAVES)  # workgroups of 8 wavefronts (items of more than 8 chunks)


def test_random_descriptors():
    rng = np.random.default_rng(11143)
    for _ in range(120):
        G = int(rng.choice([1, 2, 3, 4, 5, 7, 8, 16]))
        Hkv = int(rng.choice([1, 2, 3, 8]))
        n = int(rng.choice([1, 1, 2, 4, 7, 16, 33, 64]))
        B = int(rng.integers(1, 12))
        lens = rng.integers(-3, 900, B)
        lens[rng.integers(0, B)] = int(rng.choice([0, 1, 16, 17, n]))
        mcl = int(max(lens.max(), 0) + rng.choice([0, 0, 5, 100]))
        mbps = -(-max(mcl, 1) // BS) + int(rng.integers(0, 3))
        tp = int(rng.choice([0, 0, 16, 48, 256]))
        run_case(rng, B, G * Hkv, Hkv, int(rng.choice([64, 128])), n, mcl, tp, lens, mbps)


def test_shared_prefix_descriptors():
    rng = np.random.default_rng(7)
    for _ in range(160):
        G = int(rng.choice([1, 3, 4, 6, 8, 9, 16]))
        Hkv = int(rng.choice([1, 2, 8]))
        n = int(rng.choice([1, 1, 2, 3, 4, 7, 8, 10, 21]))
        if n * G > 64:
            continue
        # up to a few row groups of 64 / (n G) members
        max_size = int(rng.integers(1, 3 * (64 // (n * G)) + 2))
        ngroups = int(rng.integers(1, 5))
        sizes = rng.integers(0, max_size + 1, ngroups)
        start = np.concatenate([[0], np.cumsum(sizes)]).astype(int)
        B = int(start[-1] + rng.integers(0, 3))
        if B == 0:
            continue
        max_prefix = int(rng.choice([16, 64, 256, 512]))
        prefix = [int(rng.choice([0, 16, max_prefix, max_prefix + 16, -16])) for _ in range(ngroups)]
        lens = rng.integers(max_prefix, max_prefix + 700, B)
        lens[rng.integers(0, B)] = max_prefix + int(rng.integers(0, n + 1))  # new tokens inside the prefix
        mcl = int(lens.max())
        groups = dict(start=start.tolist(), prefix=prefix, max_size=max_size, max_prefix=max_prefix)
        run_case(rng, B, G * Hkv, Hkv, 128, n, mcl, int(rng.choice([0, 64])), lens, -(-mcl // BS), groups)


@pytest.mark.parametrize("n,G,Hkv,tp", [(1, 4, 8, 0), (4, 4, 8, 0), (32, 4, 8, 0), (64, 4, 8, 3840),
                                         (512, 4, 8, 0), (512, 8, 1, 256), (16, 8, 1, 0), (13, 16, 1, 16),
                                         (40, 4, 8, 0), (68, 4, 8, 0), (36, 8, 1, 0)])
def test_named_shapes(n, G, Hkv, tp):
    """Small batches in the shapes of the benchmarked steps (4 to 512 new
    tokens, wide items of 8 and 16 chunks, a last group of one chunk, two or
    more chunk groups, split contexts)."""
    rng = np.random.default_rng(n + G)
    lens = [1, n, n + 17, 600, 1500, 4096]
    run_case(rng, len(lens), G * Hkv, Hkv, 128, n, 4096, tp, lens, 256)
