"""The slot maps of the block kernels' LDS exchange, checked on the CPU.

A row spread over NW waves (C chunks of 8 values per lane) swaps its wave bits
with the low log2(NW) chunk bits through LDS: afterwards chunk k of wave w
holds tile chunk (k % NW)*C + (k // NW)*NW + w, where tile chunk W was chunk
W % C of wave W // C.  Each pass of the exchange stores every chunk (or half of
it) in one LDS slot, with one of two maps:

    direct:     wave w writes chunk k to slot w*C + k and reads its chunk k
                from slot (k % NW)*C + (k // NW)*NW + w;
    transposed: wave w writes chunk k to slot (k % NW)*C + (k // NW)*NW + w
                and reads its chunk k from slot w*C + k.

The kernels put a barrier only between the writes and the reads of a pass, and
take the two maps in turn from one pass to the next (two-pass rows take both,
the one-pass row loop alternates per row).  That is safe when, from each pass
to the next, the slots a wave writes are exactly the slots that wave read in
the previous pass: then no wave overwrites a slot another wave may still be
reading.  This file models the maps as the kernel source states them and checks
delivery, that each pass's writes are a bijection onto the slots, and that
hazard-freedom property, and that it would fail without the alternation.
"""
from __future__ import annotations

import pytest


def write_slot(w: int, k: int, C: int, NW: int, tr: bool) -> int:
    return (k % NW) * C + (k // NW) * NW + w if tr else w * C + k


def read_slot(w: int, k: int, C: int, NW: int, tr: bool) -> int:
    return w * C + k if tr else (k % NW) * C + (k // NW) * NW + w


def expected_tile_chunk(w: int, k: int, C: int, NW: int) -> int:
    return (k % NW) * C + (k // NW) * NW + w


SHAPES = [(C, NW) for NW in (2, 4, 8) for C in (2, 4, 8, 16) if NW <= C]


@pytest.mark.parametrize("C,NW", SHAPES)
@pytest.mark.parametrize("tr", [False, True], ids=["direct", "transposed"])
def test_each_map_delivers_every_chunk(C, NW, tr):
    slots = {}
    for w in range(NW):
        for k in range(C):
            s = write_slot(w, k, C, NW, tr)
            assert 0 <= s < NW * C
            assert s not in slots, "two chunks written to one slot"
            slots[s] = w * C + k  # the tile chunk wave w holds as its chunk k
    assert len(slots) == NW * C
    for w in range(NW):
        for k in range(C):
            assert slots[read_slot(w, k, C, NW, tr)] == expected_tile_chunk(w, k, C, NW)


def _written(w, C, NW, tr):
    return {write_slot(w, k, C, NW, tr) for k in range(C)}


def _read(w, C, NW, tr):
    return {read_slot(w, k, C, NW, tr) for k in range(C)}


def pass_maps(kernel: str, rows: int) -> list[bool]:
    """The map (True = transposed) of each exchange pass a workgroup runs."""
    if kernel == "block_one_pass":
        return [False]
    if kernel == "block_two_pass":
        return [False, True]
    if kernel == "loop_one_pass":  # rows alternate: peeled row direct, then T, F, T, ...
        return [r % 2 == 1 for r in range(rows)]
    if kernel == "loop_two_pass":  # every row: direct, then transposed
        return [p == 1 for r in range(rows) for p in range(2)]
    raise ValueError(kernel)


@pytest.mark.parametrize("C,NW", SHAPES)
@pytest.mark.parametrize("kernel", ["block_one_pass", "block_two_pass", "loop_one_pass",
                                    "loop_two_pass"])
def test_no_wave_overwrites_a_slot_another_wave_may_still_read(C, NW, kernel):
    maps = pass_maps(kernel, rows=7)
    for prev, nxt in zip(maps, maps[1:]):
        for w in range(NW):
            assert _written(w, C, NW, nxt) == _read(w, C, NW, prev)
            for u in range(NW):
                if u != w:
                    assert not (_written(w, C, NW, nxt) & _read(u, C, NW, prev))


@pytest.mark.parametrize("C,NW", SHAPES)
def test_the_same_map_twice_would_need_a_barrier(C, NW):
    """Without the alternation a fast wave's next writes land in slots that
    other waves read in the pass before: the model catches it."""
    for tr in (False, True):
        clash = any(_written(w, C, NW, tr) & _read(u, C, NW, tr)
                    for w in range(NW) for u in range(NW) if u != w)
        assert clash


@pytest.mark.parametrize("C,NW", SHAPES)
def test_adversarial_schedule_reads_the_right_values(C, NW):
    """Simulate a row loop on one LDS array where, in every pass, one slow wave
    reads only after every other wave has already written the next pass (the
    latest the barrier between writes and reads allows): every chunk read is
    still the one the reader expects."""
    rows = 6
    maps = pass_maps("loop_one_pass", rows)
    for slow in range(NW):
        lds = {}
        for r, tr in enumerate(maps):
            # all writes of pass r (the slow wave's too; it wrote before the barrier)
            for w in range(NW):
                for k in range(C):
                    lds[write_slot(w, k, C, NW, tr)] = (r, w * C + k)
            # every wave but the slow one reads pass r
            for w in range(NW):
                if w == slow:
                    continue
                for k in range(C):
                    assert lds[read_slot(w, k, C, NW, tr)] == (r, expected_tile_chunk(w, k, C, NW))
            # the others run ahead and write pass r + 1 before the slow wave reads pass r
            if r + 1 < len(maps):
                nxt = maps[r + 1]
                for w in range(NW):
                    if w != slow:
                        for k in range(C):
                            lds[write_slot(w, k, C, NW, nxt)] = (r + 1, w * C + k)
            for k in range(C):
                assert lds[read_slot(slow, k, C, NW, tr)] == (r, expected_tile_chunk(slow, k, C, NW))
            # the slow wave's own writes of pass r + 1 come after its reads of pass r
            if r + 1 < len(maps):
                for k in range(C):
                    lds[write_slot(slow, k, C, NW, maps[r + 1])] = (r + 1, slow * C + k)
