"""Pins for the CPU enumeration of the WG -> (b, hq, m) mappings (CPU only).

What ties the enumeration (oracle/mapping.py) to the paper:
  * every mapping is a permutation of the grid, on many shapes including
    ragged ones (N not a multiple of NX, Hq < NX);
  * swizzled head-first equals the chiplet renumbering of Fig. "wg-swizzle"
    (new id = (wid mod NX) * N/NX + wid div NX) whenever N is a multiple of NX;
  * with one batch and Hq a multiple of NX it equals what the listing of
    Fig. "head-first code" computes: head = (wid mod NX) * Hq/NX +
    wid div (NX*NB) and block = (wid mod (NX*NB)) div NX;
  * the caption example of Sections 3.2/3.3 (8 heads, 128 row blocks, 4 XCDs)
    from tests/golden/caption_example.json;
  * "one ACC at a time" (Section 3.3) for every shape whose ACC count is a
    multiple of NX, including the GQA grouping of Section 3.1;
  * the block-major order inside an XCD's piece (an order option for swizzled
    head-first) keeps every XCD's set of tiles, dispatches whole-head pieces
    block-major so each group of four consecutive WGs of an XCD shares a row
    block when the piece holds a multiple of four heads, and leaves other
    pieces in head-major order;
  * swizzled block-first (Section 3.2) keeps the block-major order, puts each
    GQA group on one XCD when the group count equals NX, serves Hq/NX heads
    per row block on each XCD for MHA, and is naive block-first when NX = 1;
  * paired row blocks (an order option): hand-worked tables, every tile
    computed once, every slot of equal causal cost but one middle block per
    head, one ACC at a time, and equal work per shader engine where
    heavy-first order alone leaves it unequal.
Planted mistakes in the enumeration (monkeypatched) must fail a pin.
"""

import json
import os

import numpy as np
import pytest

from oracle import mapping as mp

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "caption_example.json")

SHAPES = [(B, Hq, NB, NX) for B in (1, 2, 3) for Hq in (1, 2, 3, 4, 5, 8, 12, 16)
          for NB in (1, 2, 3, 7, 9) for NX in (1, 2, 4, 8)]


def _table(m, mapping, B, Hq, NB, NX):
    return np.array([m.map_wid(mapping, w, B, Hq, NB, NX) for w in range(B * Hq * NB)])


def pin_permutation(m):
    for (B, Hq, NB, NX) in SHAPES:
        N = B * Hq * NB
        for mapping in mp.MAPPINGS:
            t = _table(m, mapping, B, Hq, NB, NX)
            keys = (t[:, 0] * Hq + t[:, 1]) * NB + t[:, 2]
            assert t.min() >= 0 and np.all(t[:, 0] < B) and np.all(t[:, 1] < Hq) \
                and np.all(t[:, 2] < NB)
            assert np.array_equal(np.sort(keys), np.arange(N)), (mapping, B, Hq, NB, NX)


def pin_chiplet_swizzle(m):
    """Fig. "wg-swizzle": XCD-major renumbering when NX divides N."""
    for (B, Hq, NB, NX) in SHAPES:
        N = B * Hq * NB
        if N % NX:
            continue
        for wid in range(N):
            renum = (wid % NX) * (N // NX) + wid // NX
            assert m.map_wid(mp.SWIZZLED_HEAD_FIRST, wid, B, Hq, NB, NX) == \
                m.unravel(renum, (B, Hq, NB))


def pin_head_first_listing(m):
    """Fig. "head-first code" for one batch and NX | Hq."""
    for (B, Hq, NB, NX) in SHAPES:
        if B != 1 or Hq % NX:
            continue
        for wid in range(Hq * NB):
            head = (wid % NX) * (Hq // NX) + wid // (NX * NB)
            block = (wid % (NX * NB)) // NX
            assert m.map_wid(mp.SWIZZLED_HEAD_FIRST, wid, 1, Hq, NB, NX) == (0, head, block)


def pin_caption_example(m):
    g = json.load(open(GOLDEN))
    s = g["shape"]
    B, Hq, NB, NX = s["B"], s["Hq"], s["row_blocks"], s["NX"]
    N = B * Hq * NB
    c = g["claims"]
    # naive block-first
    t = _table(m, mp.NAIVE_BLOCK_FIRST, B, Hq, NB, NX)
    for wid, (xcd, head, block) in enumerate(c["naive_block_first"]["first_dispatch"]):
        assert m.xcd_of(wid, NX) == xcd and tuple(t[wid][1:]) == (head, block)
    assert np.all(np.diff(t[:, 2]) >= 0)  # block-major: blocks never go back
    # naive head-first: head-major order, every head on all XCDs
    t = _table(m, mp.NAIVE_HEAD_FIRST, B, Hq, NB, NX)
    assert np.all(np.diff(t[:, 1]) >= 0)
    for h in range(Hq):
        xcds = {m.xcd_of(w, NX) for w in range(N) if t[w][1] == h}
        assert len(xcds) == c["naive_head_first"]["xcds_per_head"]
    # swizzled head-first: one XCD per head, one ACC at a time, blocks in order
    t = _table(m, mp.SWIZZLED_HEAD_FIRST, B, Hq, NB, NX)
    for h in range(Hq):
        wids = [w for w in range(N) if t[w][1] == h]
        assert len({m.xcd_of(w, NX) for w in wids}) == c["swizzled_head_first"]["xcds_per_head"]
        assert [t[w][2] for w in wids] == list(range(NB))
    seqs = m.xcd_acc_sequences(t, Hq, s["Hkv"], NX)
    for seq in seqs:
        assert all(a <= b for a, b in zip(seq, seq[1:]))
    # the illustration puts heads {2x, 2x+1} on XCD x
    for x in range(NX):
        assert sorted(set(seqs[x])) == [2 * x, 2 * x + 1]
    # swizzled block-first: block-major, and (4 groups of 2 heads) XCD x serves
    # heads {2x, 2x+1} of every row block
    cs = c["swizzled_block_first"]
    t = _table(m, mp.SWIZZLED_BLOCK_FIRST, B, Hq, NB, NX)
    assert np.all(np.diff(t[:, 2]) >= 0)
    per = cs["heads_per_xcd_per_block"]
    for w in range(N):
        assert t[w][1] // per == m.xcd_of(w, NX)


def pin_one_acc_at_a_time(m):
    """Section 3.3: with NX | B*Hkv every ACC lives on one XCD, XCDs never revisit an ACC."""
    shapes = [(1, 32, 32, 8192, 128), (1, 64, 8, 8192, 128), (8, 64, 64, 4096, 128),
              (1, 16, 16, 131072, 128), (2, 16, 4, 1000, 128), (1, 8, 8, 300, 64)]
    for (B, Hq, Hkv, Sq, BM) in shapes:
        NX = 8
        NB = m.num_row_blocks(Sq, BM)
        t = np.array([m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, B, Hq, NB, NX)
                      for w in range(B * Hq * NB)])
        seqs = m.xcd_acc_sequences(t, Hq, Hkv, NX)
        owner = {}
        for x, seq in enumerate(seqs):
            assert all(a <= b for a, b in zip(seq, seq[1:]))
            for a in seq:
                assert owner.setdefault(a, x) == x, "ACC split across XCDs"


def pin_gqa_groups_on_one_xcd(m):
    """Llama-3-70B-like GQA (Hq=64, Hkv=8, 64 row blocks): group x runs on XCD x."""
    B, Hq, Hkv, NB, NX = 1, 64, 8, 64, 8
    for wid in range(B * Hq * NB):
        _, hq, _ = m.map_wid(mp.SWIZZLED_HEAD_FIRST, wid, B, Hq, NB, NX)
        assert hq // (Hq // Hkv) == m.xcd_of(wid, NX)


def pin_swizzled_block_first(m):
    """Section 3.2: block-first order; GQA groups co-located when Hkv == NX."""
    for (B, Hq, Hkv, NB, NX) in [(1, 64, 8, 64, 8), (1, 32, 8, 16, 8), (2, 128, 8, 5, 8),
                                 (1, 8, 4, 128, 4), (3, 16, 4, 7, 4)]:
        N = B * Hq * NB
        t = _table(m, mp.SWIZZLED_BLOCK_FIRST, B, Hq, NB, NX)
        # block-major: every head of row block m (of batch b) before block m+1
        assert np.array_equal(t[:, 0] * NB + t[:, 2], np.arange(N) // Hq)
        for w in range(N):
            assert t[w][1] // (Hq // Hkv) == m.xcd_of(w, NX), (B, Hq, Hkv, NB, NX, w)
    # MHA with NX | Hq: each XCD serves the same Hq/NX heads of every row block
    B, Hq, NB, NX = 2, 32, 6, 8
    t = _table(m, mp.SWIZZLED_BLOCK_FIRST, B, Hq, NB, NX)
    for x in range(NX):
        heads = {int(t[w][1]) for w in range(x, B * Hq * NB, NX)}
        assert heads == set(range(x * Hq // NX, (x + 1) * Hq // NX))
    # one XCD: nothing to co-locate, the order is naive block-first
    for (B, Hq, NB) in [(1, 5, 3), (2, 8, 4)]:
        assert np.array_equal(_table(m, mp.SWIZZLED_BLOCK_FIRST, B, Hq, NB, 1),
                              _table(m, mp.NAIVE_BLOCK_FIRST, B, Hq, NB, 1))


def pin_xcd_block_major(m):
    """Order option for swizzled head-first: same XCD tile sets, block-major inside."""
    for (B, Hq, NB, NX) in SHAPES[::3] + [(1, 32, 32, 8), (1, 64, 32, 8), (8, 64, 16, 8),
                                          (1, 16, 512, 8), (2, 12, 3, 8), (1, 128, 16, 8),
                                          (2, 128, 8, 8), (1, 48, 5, 8), (3, 40, 4, 8),
                                          (1, 16, 64, 8), (1, 16, 65, 8), (1, 32, 128, 8),
                                          (1, 128, 16, 8), (2, 72, 16, 8), (1, 64, 17, 8),
                                          (1, 64, 15, 8)]:
        N = B * Hq * NB
        for heavy, short in ((False, False), (True, False), (True, True)):
            plain = _table(m, mp.SWIZZLED_HEAD_FIRST, B, Hq, NB, NX) if not heavy else \
                np.array([m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, B, Hq, NB, NX, True)
                          for w in range(N)])
            bm = np.array([m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, B, Hq, NB, NX, heavy, True, short)
                           for w in range(N)])
            keys = (bm[:, 0] * Hq + bm[:, 1]) * NB + bm[:, 2]
            assert np.array_equal(np.sort(keys), np.arange(N))       # a permutation
            for x in range(NX):
                sel = np.arange(x, N, NX)
                assert {tuple(r) for r in plain[sel]} == {tuple(r) for r in bm[sel]}
                L0, n = m.xcd_piece(x, N, NX)
                seq = bm[sel]
                if n == 0:
                    continue
                if NB <= 64 and L0 % NB == 0 and n % NB == 0:
                    hx = n // NB
                    # the expected order, built by nested loops: groups of G
                    # local heads in turn (16 for heads of at most 16 row
                    # blocks when short-head groups are asked for, else 4),
                    # each group block-major
                    G = 16 if short and NB <= 16 else 4
                    want = []
                    for g0 in range(0, hx, G):
                        group = range(g0, min(g0 + G, hx))
                        for blk in range(NB):
                            for h in group:
                                want.append((h, blk))
                    blocks = seq[:, 2] if not heavy else NB - 1 - seq[:, 2]
                    heads = seq[:, 0] * Hq + seq[:, 1]
                    got = list(zip((heads - L0 // NB).tolist(), blocks.tolist()))
                    assert got == want, (B, Hq, NB, NX, x)
                    # G consecutive WGs of a full group share a row block
                    full = (hx // G) * G * NB
                    assert all(len(set(blocks[i:i + G])) == 1 for i in range(0, full, G))
                    # at most G heads among any G*NB consecutive WGs of a group
                    for i in range(0, n, G * NB):
                        assert len(set(heads[i:i + G * NB].tolist())) <= G
                else:
                    assert np.array_equal(seq, plain[sel])
    with pytest.raises(ValueError):
        m.map_wid(mp.NAIVE_BLOCK_FIRST, 0, 1, 8, 4, 8, False, True)


def pin_ceil_blocks(m):
    assert m.num_row_blocks(256, 128) == 2 and m.num_row_blocks(257, 128) == 3
    assert m.num_row_blocks(1, 128) == 1 and m.grid_size(2, 3, 129, 128) == 12


def pin_heavy_first_order(m):
    """The order option keeps each (b, hq) on its XCD and reverses each head's block order."""
    for (B, Hq, NB, NX) in SHAPES[::7]:
        for mapping in mp.MAPPINGS:
            N = B * Hq * NB
            base = [m.map_wid(mapping, w, B, Hq, NB, NX) for w in range(N)]
            rev = [m.map_wid(mapping, w, B, Hq, NB, NX, True) for w in range(N)]
            assert sorted(rev) == sorted(base)
            for w in range(N):
                assert rev[w][:2] == base[w][:2] and rev[w][2] == NB - 1 - base[w][2]
    # swizzled head-first: each XCD sees every head's blocks in decreasing order
    B, Hq, NB, NX = 1, 16, 12, 8
    seen = {}
    for w in range(B * Hq * NB):
        b, h, blk = m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, B, Hq, NB, NX, True)
        seen.setdefault((w % NX, h), []).append(blk)
    assert all(v == sorted(v, reverse=True) and len(v) == NB for v in seen.values())


def pin_paired(m):
    """Order option: one WG per slot p of a head computes row blocks NB-1-p, then p."""
    # worked by hand: B=1, Hq=2, NB=5 (three slots per head), NX=2, swizzled
    # head-first.  XCD 0 takes head 0's slots, XCD 1 head 1's; slot p first
    # computes block 4-p (blocks 4+0, 3+1, then the middle block 2 alone).
    t = [m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, 1, 2, 5, 2, paired=True) for w in range(6)]
    assert t == [(0, 0, 4), (0, 1, 4), (0, 0, 3), (0, 1, 3), (0, 0, 2), (0, 1, 2)]
    # the same with heavy-first order: the slots of each head in reverse
    t = [m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, 1, 2, 5, 2, True, paired=True) for w in range(6)]
    assert t == [(0, 0, 2), (0, 1, 2), (0, 0, 3), (0, 1, 3), (0, 0, 4), (0, 1, 4)]
    # naive block-first, B=1, Hq=3, NB=4: slot 0 of every head, then slot 1
    t = [m.map_wid(mp.NAIVE_BLOCK_FIRST, w, 1, 3, 4, 8, paired=True) for w in range(6)]
    assert t == [(0, 0, 3), (0, 1, 3), (0, 2, 3), (0, 0, 2), (0, 1, 2), (0, 2, 2)]
    assert [m.slot_blocks(mm, 5) for mm in (4, 3, 2)] == [[4, 0], [3, 1], [2]]
    for (B, Hq, NB, NX) in SHAPES[::5] + [(1, 32, 32, 8), (1, 16, 512, 8), (2, 12, 3, 8)]:
        for mapping in mp.MAPPINGS:
            for heavy, xbm in ((False, False), (True, False), (True, True)):
                if xbm and mapping != mp.SWIZZLED_HEAD_FIRST:
                    continue
                n = B * Hq * ((NB + 1) // 2)   # ceil(NB / 2) slots per head
                with pytest.raises(ValueError):
                    m.map_wid(mapping, n, B, Hq, NB, NX, heavy, xbm, paired=True)
                seen = []
                costs = []
                for w in range(n):
                    b, hq, first = m.map_wid(mapping, w, B, Hq, NB, NX, heavy, xbm, paired=True)
                    blocks = m.slot_blocks(first, NB)
                    assert blocks[0] == max(blocks), "the later block first"
                    seen += [(b, hq, blk) for blk in blocks]
                    costs.append(sum(blk + 1 for blk in blocks))   # causal: block m costs m+1
                # every tile of the grid exactly once
                assert sorted(seen) == [(b, h, k) for b in range(B) for h in range(Hq)
                                        for k in range(NB)], (mapping, B, Hq, NB, NX)
                # every slot costs NB+1, except one middle block per head when NB is odd
                odd = [c for c in costs if c != NB + 1]
                assert len(odd) == (B * Hq if NB % 2 else 0)
                assert all(c == (NB + 1) // 2 for c in odd)
    # one ACC at a time (Section 3.3) still holds for swizzled head-first
    for (B, Hq, Hkv, NB) in [(1, 32, 32, 32), (1, 64, 8, 32), (1, 16, 16, 512), (2, 16, 4, 9)]:
        n = B * Hq * ((NB + 1) // 2)
        t = np.array([m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, B, Hq, NB, 8, True, paired=True)
                      for w in range(n)])
        owner = {}
        for x, seq in enumerate(m.xcd_acc_sequences(t, Hq, Hkv, 8)):
            assert all(a <= c for a, c in zip(seq, seq[1:]))
            for a in seq:
                assert owner.setdefault(a, x) == x, "ACC split across XCDs"
    # shader-engine balance (the reason for the order): the k-th WG of an XCD
    # goes to engine k mod 4; on MHA B1 H32 with 32 row blocks each engine of
    # each XCD gets the same causal work, which heavy-first alone does not give
    B, Hq, NB, NX = 1, 32, 32, 8
    for paired, balanced in ((True, True), (False, False)):
        n = B * Hq * (((NB + 1) // 2) if paired else NB)
        work = np.zeros((NX, 4))
        for w in range(n):
            _, _, first = m.map_wid(mp.SWIZZLED_HEAD_FIRST, w, B, Hq, NB, NX, True, paired=paired)
            blocks = m.slot_blocks(first, NB) if paired else [first]
            work[w % NX, (w // NX) % 4] += sum(blk + 1 for blk in blocks)
        assert (work.max(axis=1) == work.min(axis=1)).all() == balanced


PINS = [pin_heavy_first_order, pin_permutation, pin_chiplet_swizzle, pin_head_first_listing, pin_caption_example,
        pin_one_acc_at_a_time, pin_gqa_groups_on_one_xcd, pin_swizzled_block_first,
        pin_xcd_block_major, pin_ceil_blocks, pin_paired]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(mp)


def test_enumerate_matches_map_wid():
    t = mp.enumerate_mapping(mp.SWIZZLED_HEAD_FIRST, 2, 12, 300, 128, 8)
    assert t.shape == (2 * 12 * 3, 3)
    assert tuple(t[5]) == mp.map_wid(2, 5, 2, 12, 3, 8)


def test_errors():
    with pytest.raises(ValueError):
        mp.map_wid(4, 0, 1, 1, 1, 8)
    with pytest.raises(ValueError):
        mp.map_wid(0, 4, 1, 2, 2, 8)


# ---------------------------------------------------------------- planted mistakes


class _Mutant:
    """The enumeration module with one function replaced."""

    def __init__(self, **overrides):
        self.__dict__.update({k: getattr(mp, k) for k in dir(mp) if not k.startswith("__")})
        self.__dict__.update(overrides)
        # map_wid must see the replaced helpers
        me = self

        def map_wid(mapping, wid, B, Hq, NB, NX, heavy_first=False, xcd_block_major=False,
                    short_head_groups=False, paired=False):
            if paired:
                b, hq, p = me.paired_slot(mapping, wid, B, Hq, NB, NX, heavy_first,
                                          xcd_block_major, short_head_groups)
                return b, hq, me.pair_first(p, NB)
            N = B * Hq * NB
            if not 0 <= wid < N:
                raise ValueError("wid out of range")
            if xcd_block_major and mapping != mp.SWIZZLED_HEAD_FIRST:
                raise ValueError("block-major order needs swizzled head-first")
            if mapping == mp.NAIVE_BLOCK_FIRST:
                b, mm, hq = me.unravel(wid, me.bf_radices(B, Hq, NB))
            elif mapping == mp.NAIVE_HEAD_FIRST:
                b, hq, mm = me.unravel(wid, (B, Hq, NB))
            elif mapping == mp.SWIZZLED_BLOCK_FIRST:
                b, mm, j = me.unravel(wid, me.bf_radices(B, Hq, NB))
                hq = me.sbf_head(j, Hq, NX)
            else:
                L = me.swizzled_rank(wid, N, NX)
                if xcd_block_major:
                    L = me.bm_rank(L, wid % NX, N, NX, NB, short_head_groups)
                b, hq, mm = me.unravel(L, (B, Hq, NB))
            if heavy_first:
                mm = me.reverse_block(mm, NB)
            return b, hq, mm
        self.map_wid = overrides.get("map_wid", map_wid)
        self.__dict__.setdefault("bf_radices", lambda B, Hq, NB: (B, NB, Hq))
        self.__dict__.setdefault("reverse_block", lambda mm, NB: NB - 1 - mm)
        self.__dict__.setdefault("sbf_head", lambda j, Hq, NX: me.swizzled_rank(j, Hq, NX))
        self.__dict__.setdefault("bm_rank", _bm_rank)
        self.__dict__.setdefault("pair_first", lambda p, NB: NB - 1 - p)
        self.__dict__.setdefault(
            "paired_slot", lambda mapping, wid, B, Hq, NB, NX, hf, xbm, sh: me.map_wid(
                mapping, wid, B, Hq, me.pair_slots(NB), NX, hf, xbm, sh))


def _bm_rank(L, x, N, NX, NB, short=False, G=4, max_blocks=64, G_short=16, short_blocks=16,
             ignore_flag=False):
    L0, n = mp.xcd_piece(x, N, NX)
    if NB > max_blocks or L0 % NB or n % NB:
        return L
    if (short or ignore_flag) and NB <= short_blocks:
        G = G_short
    hx = n // NB
    k = L - L0
    first = (k // (G * NB)) * G
    g = min(G, hx - first)
    j = k - first * NB
    return L0 + (first + j % g) * NB + j // g


def _bm_rank_whole_piece(L, x, N, NX, NB, short=False):
    """Block-major across all heads of the piece (no groups)."""
    L0, n = mp.xcd_piece(x, N, NX)
    if NB > 64 or L0 % NB or n % NB:
        return L
    hx = n // NB
    k = L - L0
    return L0 + (k % hx) * NB + k // hx


def _bm_rank_transposed(L, x, N, NX, NB, short=False):
    L0, n = mp.xcd_piece(x, N, NX)
    if NB > 64 or L0 % NB or n % NB:
        return L
    hx = n // NB
    k = L - L0
    first = (k // (4 * NB)) * 4
    g = min(4, hx - first)
    j = k - first * NB
    return L0 + first * NB + (j // NB) + (j % NB) * g if g == NB else L0 + first * NB + j


def _bm_rank_any_piece(L, x, N, NX, NB, short=False):
    L0, n = mp.xcd_piece(x, N, NX)
    if NB > 64:
        return L
    hx = max(1, -(-n // NB))
    k = L - L0
    first = (k // (4 * NB)) * 4
    g = max(1, min(4, hx - first))
    j = k - first * NB
    return L0 + (first + j % g) * NB + j // g


def _bm_rank_full_last_group(L, x, N, NX, NB, short=False):
    """Treats a short last group as four heads wide."""
    L0, n = mp.xcd_piece(x, N, NX)
    if NB > 64 or L0 % NB or n % NB:
        return L
    k = L - L0
    first = (k // (4 * NB)) * 4
    j = k - first * NB
    return min(L0 + n - 1, L0 + (first + j % 4) * NB + j // 4)


def _unravel_first_fastest(x, radices):
    digits = []
    for r in radices:
        digits.append(x % r)
        x //= r
    return tuple(digits)


def _rank_no_ragged_term(wid, N, NX):
    return (wid % NX) * (N // NX) + wid // NX


def _rank_floor_ceil_swap(wid, N, NX):
    q = -(-N // NX)
    return (wid % NX) * q + wid // NX if (wid % NX) * q + wid // NX < N else wid


MAP_MUTANTS = {
    "unravel_first_digit_fastest": dict(unravel=_unravel_first_fastest),
    "swizzle_without_ragged_term": dict(swizzled_rank=_rank_no_ragged_term),
    "swizzle_ceil_stride": dict(swizzled_rank=_rank_floor_ceil_swap),
    "swizzle_identity": dict(swizzled_rank=lambda wid, N, NX: wid),
    "block_first_head_outer": dict(bf_radices=lambda B, Hq, NB: (B, Hq, NB)),
    "floor_row_blocks": dict(num_row_blocks=lambda Sq, BM: Sq // BM),
    "heavy_first_off_by_one": dict(reverse_block=lambda mm, NB: (NB - mm) % NB),
    "block_first_swizzle_missing": dict(sbf_head=lambda j, Hq, NX: j),
    "block_major_transposed": dict(bm_rank=_bm_rank_transposed),
    "block_major_on_partial_pieces": dict(bm_rank=_bm_rank_any_piece),
    "block_major_whole_piece": dict(bm_rank=_bm_rank_whole_piece),
    "block_major_full_last_group": dict(bm_rank=_bm_rank_full_last_group),
    "block_major_at_any_length": dict(bm_rank=lambda L, x, N, NX, NB, sh=False: _bm_rank(
        L, x, N, NX, NB, sh, max_blocks=1 << 30)),
    "block_major_limit_off_by_one": dict(bm_rank=lambda L, x, N, NX, NB, sh=False: _bm_rank(
        L, x, N, NX, NB, sh, max_blocks=63)),
    "block_major_short_heads_in_fours": dict(bm_rank=lambda L, x, N, NX, NB, sh=False: _bm_rank(
        L, x, N, NX, NB, sh, G_short=4)),
    "block_major_short_limit_above": dict(bm_rank=lambda L, x, N, NX, NB, sh=False: _bm_rank(
        L, x, N, NX, NB, sh, short_blocks=17)),
    "block_major_short_limit_below": dict(bm_rank=lambda L, x, N, NX, NB, sh=False: _bm_rank(
        L, x, N, NX, NB, sh, short_blocks=15)),
    "block_major_short_groups_always": dict(bm_rank=lambda L, x, N, NX, NB, sh=False: _bm_rank(
        L, x, N, NX, NB, sh, ignore_flag=True)),
    "paired_slots_floor": dict(pair_slots=lambda NB: NB // 2),
    "paired_first_is_the_slot": dict(pair_first=lambda p, NB: p),
    "paired_mirror_off_by_one": dict(
        slot_blocks=lambda mm, NB: [mm] if NB - mm == mm else [mm, NB - mm]),
    "paired_order_flags_dropped": dict(paired_slot=lambda mapping, wid, B, Hq, NB, NX, hf, xbm, sh:
                                       mp.map_wid(mapping, wid, B, Hq, (NB + 1) // 2, NX)),
    "paired_slots_decoded_over_all_blocks": dict(
        paired_slot=lambda mapping, wid, B, Hq, NB, NX, hf, xbm, sh: mp.map_wid(
            mapping, wid, B, Hq, NB, NX, hf, xbm, sh)),
    "block_first_swizzle_transposed": dict(
        sbf_head=lambda j, Hq, NX: (j % (Hq // NX if Hq >= NX else 1)) * NX + j // max(Hq // NX, 1)
        if Hq % NX == 0 else j),
}


def test_mutant_harness_is_faithful():
    m = _Mutant()
    for pin in PINS:
        pin(m)


@pytest.mark.parametrize("name", sorted(MAP_MUTANTS))
def test_planted_mistake_is_caught(name):
    m = _Mutant(**MAP_MUTANTS[name])
    caught = []
    for pin in PINS:
        try:
            pin(m)
        except (AssertionError, ValueError, ZeroDivisionError, IndexError):
            caught.append(pin.__name__)
    assert caught, "planted mistake %s passed every pin" % name
