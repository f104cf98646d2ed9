"""The direct-to-LDS layouts of the ppd kernels, checked on the host.

A buffer_load_dwordx4 with the LDS flag writes lane i's 16 bytes at 16 i
past the instruction's LDS address, so the layout inside a 1 KB group of
rows is set by which 16-byte chunk of the (block, head) tile each lane
fetches.  This test places one 64-key step the way the kernels' staging
does (the same formulas as prefill_paged_attn.hip: dma_off, koff / k_addr,
voff / v_frag), then checks that every K operand read (ds_read_b128) and
every transposing V read (ds_read_b64_tr_b16, which hands lane j of a
16-lane group element j % 4 of the 8-byte rows 4 e + j / 4 its lanes
address) fetches the element the MFMA operand layout needs, and that the
reads are free of bank conflicts at 64 banks of 4 bytes: 16 lanes of a
b128 read, 32 lanes of a transposing b64 read, per pass.
"""

import pytest

KBN = 64


def layout(D):
    if D == 128:
        return 4, 4 * D + 8, lambda d: 4 * d
    return 8, 8 * D + 16, lambda d: 4 * ((d >> 1) & 1) + (d >> 2)


def place(D):
    """LDS element index -> (key, dim) after one step's staging."""
    rows, kgrp, swz = layout(D)
    cpr = D // 8
    lds = {}
    for grp in range(KBN // rows):
        for lane in range(64):
            d, cpos = lane // cpr, lane % cpr
            src = d * D + 8 * (cpos ^ swz(d))          # dma_off: element of the group's rows
            for e in range(8):
                lds[grp * kgrp + 8 * lane + e] = (grp * rows + (src + e) // D, (src + e) % D)
    return lds


def k_offset(D, lane, ks, mt):
    rows, kgrp, swz = layout(D)
    qi, half = lane & 31, lane >> 5
    if D == 128:
        koff = (qi >> 2) * kgrp + (qi & 3) * D + 8 * half + 32 * ((ks >> 1) ^ (qi & 3))
        return mt * 8 * kgrp + 16 * (ks & 1) + koff
    koff = (qi >> 3) * kgrp + (qi & 7) * D + 8 * ((2 * ks + half) ^ swz(qi & 7))
    return mt * 4 * kgrp + koff


def v_offset(D, lane, ks2, dt, hi):
    rows, kgrp, swz = layout(D)
    tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2)
    if D == 128:
        tr_d = tr_row & 3
        tr_base = (tr_row >> 2) * kgrp + tr_d * D + 8 * (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) + 4 * (lane & 1)
        voff = tr_base + 32 * (dt ^ tr_d)
    else:
        voff = tr_row * D + 8 * ((4 * dt + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ swz(tr_row)) + 4 * (lane & 1)
    slice_groups = 16 // rows
    return slice_groups * ks2 * kgrp + (slice_groups // 2) * kgrp * hi + voff


def conflicts(byte_addrs, width):
    """Extra bank cycles of one pass: accesses of `width` bytes each."""
    banks = [(a // 4 + w) % 64 for a in byte_addrs for w in range(width // 4)]
    return len(banks) - len(set(banks))


@pytest.mark.parametrize("D", [128, 64])
def test_k_operand_reads(D):
    lds = place(D)
    for ks in range(D // 16):
        for mt in range(2):
            offs = [k_offset(D, lane, ks, mt) for lane in range(64)]
            for lane, o in enumerate(offs):
                qi, half = lane & 31, lane >> 5
                got = [lds[o + e] for e in range(8)]
                assert got == [(mt * 32 + qi, ks * 16 + half * 8 + e) for e in range(8)]
            for q in range(4):
                assert conflicts([2 * o for o in offs[16 * q:16 * q + 16]], 16) == 0


@pytest.mark.parametrize("D", [128, 64])
def test_v_operand_transposing_reads(D):
    lds = place(D)
    for ks2 in range(4):
        for dt in range(D // 32):
            for hi in range(2):
                offs = [v_offset(D, lane, ks2, dt, hi) for lane in range(64)]
                for lane, o in enumerate(offs):
                    g, i = lane >> 4, lane & 15
                    key = 16 * ks2 + 8 * hi + 4 * (g >> 1) + (i >> 2)
                    dim = 32 * dt + 16 * (g & 1) + 4 * (i & 3)
                    assert [lds[o + e] for e in range(4)] == [(key, dim + e) for e in range(4)]
                # what the transpose hands lane j of a group: rows 4 e + j / 4,
                # element j % 4 -> keys 4 (l / 32) + e of dim l % 32 (the A operand)
                for lane in range(64):
                    g, j = lane >> 4, lane & 15
                    for e in range(4):
                        src = 16 * g + 4 * e + j // 4
                        key, dim = lds[offs[src] + j % 4]
                        assert (key, dim) == (16 * ks2 + 8 * hi + 4 * (lane >> 5) + e, 32 * dt + lane % 32)
                for q in range(2):
                    assert conflicts([2 * o for o in offs[32 * q:32 * q + 32]], 8) == 0


@pytest.mark.parametrize("D", [128, 64])
def test_staging_covers_every_element_once(D):
    lds = place(D)
    assert sorted(lds.values()) == [(k, d) for k in range(KBN) for d in range(D)]
    rows, kgrp, _ = layout(D)
    assert max(lds) < (KBN // rows) * kgrp
