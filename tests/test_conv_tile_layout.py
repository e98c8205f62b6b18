"""Host-side check of the LDS layout of the conv tile kernel's A operand when it is loaded straight
into LDS (paper_2407_11698_amd/csrc/conv_tile.hip, 64-channel chunks, 256-pixel tiles, W a
multiple of 16).

The test restates the kernel's address arithmetic: the lane-linear LDS-direct loads (LDS unit
4 q + (e ^ ((q >> 1) & 3)) holds channel group e of staged pixel q; staged rows of `apitch`
pixels, a multiple of 16) and the fragment reads (a per-fragment base, one of three per-lane
terms for column offsets -1, 0, +1 and a row offset). For every tile, wave, fragment, K-step
(tap) and lane it checks that the unit read holds the input pixel and channel group the
convolution needs (zero outside the image), that every access stays in the stage, that the four
lanes of each pixel load one contiguous 64-byte segment, and that each fragment read's lane
addresses, modulo 1 KiB, are those of a read pattern measured free of bank conflicts on gfx950
(rocprofv3 SQ_LDS_BANK_CONFLICT on a probe reading 64 (r + s) + 16 (g ^ (((r + s) >> 1) & 3)),
lane 16 g + r, s = 0 .. 3). Forward and input gradient (opposite tap offsets)."""
import pytest

NT, BM, TM = 512, 256, 4       # threads, output pixels per tile, 16-pixel fragments per wave
NPMAX = 576                    # staged pixels of a stage
NIA = (NPMAX * 4 + NT - 1) // NT


def geometry(n, h, w):
    rt = BM // w
    ns, rs = (1, rt) if rt <= h else (rt // h, h)
    apitch = (w + 2 + 15) // 16 * 16
    aseg = (rs + 2) * apitch
    return rt, ns, rs, apitch, aseg, ns * aseg


def staged_units(mt, n, h, w):
    """LDS unit -> (image, row, column, group) or 'zero' / 'pad', as the loads fill it."""
    rt, ns, rs, apitch, aseg, npx = geometry(n, h, w)
    img0, row0 = divmod(mt * rt, h)
    lds, srcs = {}, {}
    for tid in range(NT):
        wave, lane = divmod(tid, 64)
        for v in range(NIA):
            chunk = NT * v + 64 * wave
            if chunk >= 4 * npx:
                continue                       # a whole wave past the staged pixels loads nothing
            unit = tid + NT * v
            q = unit >> 2
            e = (unit & 3) ^ ((q >> 1) & 3)
            seg, r = divmod(q, aseg)
            lr, lc = divmod(r, apitch)
            img, hh, ww = img0 + seg, row0 + lr - 1, lc - 1
            if img < n and 0 <= hh < h and 0 <= ww < w:
                src = (img, hh, ww, e)
            else:
                src = "pad" if ww > w else "zero"
            dst = chunk + lane                 # lane-linear: LDS unit of this lane
            assert dst < NPMAX * 4 and dst not in lds
            lds[dst] = src
            srcs.setdefault(dst >> 2, set()).add(src if src in ("pad", "zero") else src[:3])
    # the four lanes of a pixel load groups of that one pixel (one 64-byte source segment)
    for q, ss in srcs.items():
        assert len(ss) == 1, (q, ss)
    return lds


def check(n, h, w, sgn):
    rt, ns, rs, apitch, aseg, npx = geometry(n, h, w)
    assert w % 16 == 0 and npx <= NPMAX
    for mt in range((n * h + rt - 1) // rt):
        img0, row0 = divmod(mt * rt, h)
        lds = staged_units(mt, n, h, w)
        for wave in range(8):
            wm = wave >> 1
            for i in range(TM):
                mloc0 = wm * 64 + 16 * i
                seg, rem = divmod(mloc0, rs * w)
                row, col0 = divmod(rem, w)
                for ks in range(9):
                    dr, dc = sgn * (ks // 3 - 1), sgn * (ks % 3 - 1)
                    pat = {}
                    for g4 in range(4):
                        for l in range(16):
                            base = (seg * aseg + (row + 1) * apitch + col0) * 64
                            t = l + 1 + dc
                            addr = base + 64 * t + 16 * (g4 ^ ((t >> 1) & 3)) + dr * apitch * 64
                            assert 0 <= addr and addr + 16 <= NPMAX * 64
                            got = lds.get(addr // 16)
                            m = mloc0 + l
                            sg, rm = divmod(m, rs * w)
                            rr, cc = divmod(rm, w)
                            img, hh, ww = img0 + sg, row0 + rr + dr, cc + dc
                            want = (img, hh, ww, g4) if (img < n and 0 <= hh < h and 0 <= ww < w) else "zero"
                            assert got == want, (mt, wave, i, ks, g4, l, got, want)
                            pat[16 * g4 + l] = addr % 1024
                    s = 1 + dc
                    assert pat == {16 * g + r: (64 * (r + s) + 16 * (g ^ (((r + s) >> 1) & 3))) % 1024
                                   for g in range(4) for r in range(16)}


@pytest.mark.parametrize("h,w", [(32, 32), (16, 16), (8, 64), (4, 64)])
@pytest.mark.parametrize("sgn", [1, -1], ids=["forward", "input_gradient"])
def test_direct_a_layout(h, w, sgn):
    check(2, h, w, sgn)
