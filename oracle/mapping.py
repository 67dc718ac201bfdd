"""CPU enumeration of the workgroup -> (batch, head, row-block) mappings.

TEST INFRASTRUCTURE ONLY (the oracle): imported by the test suite, the smoke
check and the benchmark's CPU-baseline leg, never by the product path.  It is
written from the paper's definitions, shares no code with the HIP kernels, and
is deliberately plain Python so it can be read against the paper.

Setting (Sections 2.2, 3.1, 3.2, 3.3):
  * A FlashAttention-2 forward grid has one workgroup (WG) per
    (batch b, query head hq, query row block m); there are
    NB = ceil(Sq / BM) row blocks per head (the listing of Fig. "head-first
    code" computes blocks_per_head with a ceiling) and N = B * Hq * NB WGs in a
    1-D grid.
  * The hardware hands WG ``wid`` to die (XCD) ``wid mod NX``: chunked
    round-robin with chunk size one (Section 2.2).  Within one XCD the k-th WG
    it receives is ``wid = x + k * NX``.
  * An Attention Compute Cluster (ACC, Section 3.1) is the set of WGs reading
    the same K/V: one (batch, KV head) pair, the KV head of query head hq being
    hq // (Hq // Hkv).

The three mappings (integer ``mapping`` argument of the C ABI):
  0  naive block-first (Section 3.2): block 0 of every head, then block 1 of
     every head, ...; heads vary fastest, batch outermost.
  1  naive head-first (Section 3.2): every block of head 0, then of head 1,
     ...; blocks vary fastest, batch outermost.
  2  swizzled head-first (Section 3.3): the head-first order is cut into NX
     contiguous pieces and piece x is run by XCD x, in order.  WG ``wid`` is
     the k-th WG of XCD x = wid mod NX (k = wid div NX); its rank in the
     XCD-major listing is L = x*q + min(x, r) + k with q, r = divmod(N, NX),
     and L is decoded in head-first order.  When N is a multiple of NX this is
     exactly the chiplet swizzle of Fig. "wg-swizzle" (new id =
     xcd * (N / NX) + local id); the min(x, r) term extends it to grids that are
     not, where the first r XCDs take one WG more.  Batch is outermost
     throughout (the readings of the garbled per-batch line of the listing and
     of Hq < NX are recorded with the design notes).
  3  swizzled block-first (Section 3.2): block-first order, with the query
     heads of every (batch, row block) row renumbered so that the WGs one XCD
     receives from that row carry a contiguous range of heads -- so the heads
     of a GQA group land on one XCD when the group count equals NX.  The
     paper gives no formula; this is the chiplet swizzle applied within each
     row of Hq WGs: position j of the row (its WG goes to XCD
     (row start + j) mod NX) takes head (j mod NX)*qh + min(j mod NX, rh) +
     j div NX, with qh, rh = divmod(Hq, NX).  When NX divides Hq, XCD x gets
     heads x*Hq/NX .. (x+1)*Hq/NX - 1 of every row block.

Order options (not among the paper's mappings):
  * ``heavy_first`` replaces the row block m by NB-1-m after any mapping, so
    every (b, hq) keeps its XCD but each head's blocks are dispatched
    last-to-first.  Under a causal mask block m costs m+1 K/V tiles, so this
    starts the expensive blocks first.
  * ``xcd_block_major`` (swizzled head-first only): XCD x's piece of the
    head-major order, when it is made of whole heads (hx of them, starting at
    L0), is cut into groups of G consecutive heads (the last group may hold
    fewer) and each group is dispatched block-major: the
    group's row block 0 of each of its heads, then row block 1 of each, and so
    on.  Same tiles per XCD, different order inside the XCD.  The MI355X
    dispatcher hands an XCD its WGs one per shader engine in turn, four shader
    engines per XCD (measured), so under a causal mask four consecutive WGs
    then cost the same, while the WGs in flight still read the K/V of only
    G heads.  G = BLOCK_MAJOR_HEADS = 4, or, with ``short_head_groups`` (the
    library sets it for its 128-row blocks, head dimension 56 and 64, four
    workgroups per CU), BLOCK_MAJOR_HEADS_SHORT = 16 when a head has at most
    SHORT_HEAD_BLOCKS = 16 row blocks: short causal heads finish their blocks
    quickly and a longer heavy-first prefix over more heads balances the CUs
    better, while such heads' K/V streams are short.  It
    applies only when NB <= BLOCK_MAJOR_MAX_BLOCKS = 64: the engine imbalance
    of head-major order shrinks like 1/NB, and at long contexts the K/V
    streams in flight cost more than it saves (measured).
  * ``paired`` (head dimension 128, forward): the grid has P = ceil(NB/2)
    slots per head instead of NB row blocks.  The mapping and the options
    above place the B*Hq*P slots as they would place tiles with P row blocks
    per head, and the WG of slot p computes row block NB-1-p, then row block p
    (once when the two coincide, the middle block of an odd NB).  Under a
    causal mask with Sq == Skv block m costs m+1 block-widths of K/V, so every
    slot costs NB+1 except that middle one, whatever order the WGs start in.
    A table entry is the slot's first row block NB-1-p; ``slot_blocks`` lists
    both.
"""

from __future__ import annotations

import numpy as np

NAIVE_BLOCK_FIRST = 0
NAIVE_HEAD_FIRST = 1
SWIZZLED_HEAD_FIRST = 2
SWIZZLED_BLOCK_FIRST = 3
BLOCK_MAJOR_HEADS = 4
BLOCK_MAJOR_HEADS_SHORT = 16
SHORT_HEAD_BLOCKS = 16
BLOCK_MAJOR_MAX_BLOCKS = 64
MAPPINGS = (NAIVE_BLOCK_FIRST, NAIVE_HEAD_FIRST, SWIZZLED_HEAD_FIRST, SWIZZLED_BLOCK_FIRST)


def num_row_blocks(Sq: int, BM: int) -> int:
    """NB = ceil(Sq / BM): the last block may be partial."""
    return (Sq + BM - 1) // BM


def grid_size(B: int, Hq: int, Sq: int, BM: int) -> int:
    return B * Hq * num_row_blocks(Sq, BM)


def unravel(x: int, radices) -> tuple:
    """Mixed-radix digits of x, most significant first (last digit fastest)."""
    digits = []
    for r in reversed(radices):
        digits.append(x % r)
        x //= r
    assert x == 0, "index out of range for the given radices"
    return tuple(reversed(digits))


def xcd_of(wid: int, NX: int) -> int:
    """Hardware dispatch model: chunked round-robin with chunk size one."""
    return wid % NX


def swizzled_rank(wid: int, N: int, NX: int) -> int:
    """Rank L of ``wid`` when the grid is listed XCD by XCD (XCD-major)."""
    x = wid % NX
    k = wid // NX
    q, r = divmod(N, NX)
    return x * q + min(x, r) + k


def xcd_piece(x: int, N: int, NX: int) -> tuple:
    """(first rank L0, length) of XCD x's contiguous piece of the XCD-major listing."""
    q, r = divmod(N, NX)
    return x * q + min(x, r), q + (1 if x < r else 0)


def pair_slots(NB: int) -> int:
    """Slots per head of the paired order: ceil(NB / 2)."""
    return (NB + 1) // 2


def slot_blocks(m_first: int, NB: int) -> list:
    """Row blocks a paired slot computes, in order, from its first block."""
    second = NB - 1 - m_first
    return [m_first] if second == m_first else [m_first, second]


def map_wid(mapping: int, wid: int, B: int, Hq: int, NB: int, NX: int,
            heavy_first: bool = False, xcd_block_major: bool = False,
            short_head_groups: bool = False, paired: bool = False) -> tuple:
    """(b, hq, m) that WG ``wid`` computes under ``mapping`` (with ``paired``,
    m is the first row block of its slot)."""
    if paired:
        b, hq, p = map_wid(mapping, wid, B, Hq, pair_slots(NB), NX, heavy_first,
                           xcd_block_major, short_head_groups)
        return b, hq, NB - 1 - p
    N = B * Hq * NB
    if not 0 <= wid < N:
        raise ValueError("wid out of range")
    if xcd_block_major and mapping != SWIZZLED_HEAD_FIRST:
        raise ValueError("the block-major order is defined for swizzled head-first only")
    if mapping == NAIVE_BLOCK_FIRST:
        b, m, hq = unravel(wid, (B, NB, Hq))
    elif mapping == NAIVE_HEAD_FIRST:
        b, hq, m = unravel(wid, (B, Hq, NB))
    elif mapping == SWIZZLED_HEAD_FIRST:
        L = swizzled_rank(wid, N, NX)
        L0, n = xcd_piece(wid % NX, N, NX)
        if xcd_block_major and NB <= BLOCK_MAJOR_MAX_BLOCKS and L0 % NB == 0 and n % NB == 0:
            hx = n // NB                       # whole heads in the piece
            k = L - L0                         # position within the XCD's sequence
            G = BLOCK_MAJOR_HEADS_SHORT if short_head_groups and NB <= SHORT_HEAD_BLOCKS \
                else BLOCK_MAJOR_HEADS
            first = (k // (G * NB)) * G        # first head of k's group
            g = min(G, hx - first)             # heads in k's group
            j = k - first * NB                 # position within the group
            L = L0 + (first + j % g) * NB + j // g   # head j mod g, block j div g
        b, hq, m = unravel(L, (B, Hq, NB))
    elif mapping == SWIZZLED_BLOCK_FIRST:
        b, m, j = unravel(wid, (B, NB, Hq))
        hq = swizzled_rank(j, Hq, NX)
    else:
        raise ValueError("unknown mapping %r" % (mapping,))
    if heavy_first:
        m = NB - 1 - m
    return b, hq, m


def enumerate_mapping(mapping: int, B: int, Hq: int, Sq: int, BM: int, NX: int,
                      heavy_first: bool = False, xcd_block_major: bool = False,
                      short_head_groups: bool = False, paired: bool = False) -> np.ndarray:
    """Array [N, 3] of (b, hq, m) for wid = 0 .. N-1 (pure-Python loop); with
    ``paired``, N = B*Hq*ceil(NB/2) and m is each slot's first row block."""
    NB = num_row_blocks(Sq, BM)
    N = B * Hq * (pair_slots(NB) if paired else NB)
    out = np.empty((N, 3), dtype=np.int64)
    for wid in range(N):
        out[wid] = map_wid(mapping, wid, B, Hq, NB, NX, heavy_first, xcd_block_major,
                           short_head_groups, paired)
    return out


def split_flags(mapping_with_flags: int) -> tuple:
    """(base mapping, heavy_first, xcd_block_major, paired) of an ABI mapping value."""
    return (mapping_with_flags & 0xF, bool(mapping_with_flags & 0x10),
            bool(mapping_with_flags & 0x20), bool(mapping_with_flags & 0x40))


def acc_id(b: int, hq: int, Hq: int, Hkv: int) -> int:
    """Attention Compute Cluster of a WG: the (batch, KV head) it reads."""
    return b * Hkv + hq // (Hq // Hkv)


def xcd_acc_sequences(table: np.ndarray, Hq: int, Hkv: int, NX: int) -> list:
    """For each XCD, the ACC ids of the WGs it receives, in dispatch order."""
    seqs = [[] for _ in range(NX)]
    for wid in range(table.shape[0]):
        b, hq, _ = table[wid]
        seqs[xcd_of(wid, NX)].append(acc_id(int(b), int(hq), Hq, Hkv))
    return seqs
