"""LDS bank-conflict model of the kernels' LDS instructions.

The GPU analogue of the paper's cache-model study (Sec. 6.3: a model of one
memory level, evaluated per schedule against hardware counters), for the
level the kernels stage their operands in: LDS.  It predicts, per kernel
launch, the LDS cycles of every fragment read and staging write and how
many of them are bank-conflict cycles, the quantities rocprofv3 counts as
``SQ_LDS_IDX_ACTIVE`` and ``SQ_LDS_BANK_CONFLICT``.

Hardware model (gfx950, measured with an in-bounds per-lane-pair probe: for
each pair of lanes only those two were active, on the same banks at
different addresses, and ``SQ_LDS_BANK_CONFLICT`` showed whether the pair
shares a phase):

- banks of 4 bytes; within a phase, dword address ``a`` uses bank
  ``a % P``, where P (measured by scanning the address distance between two
  lanes of one phase) is 64 for ds_read_b128/b64/b64_tr_b16 and 32 for
  ds_read_b32 and every write form;
- an instruction is served in phases of lanes; a phase takes as many cycles
  as the largest number of distinct dwords any one bank must deliver (lanes
  reading the same dword share it);
- phases per instruction:
    ds_read_b128          4 phases of 16 lanes: {0-3, 12-15, 20-23, 24-27},
                          {4-11, 16-19, 28-31} and the same sets + 32;
    ds_read_b64, ds_read_b64_tr_b16, ds_read_b32
                          2 phases of 32 lanes (0-31, 32-63);
    ds_write_b128         8 phases of 8 consecutive lanes;
    ds_write_b64          4 phases of 16 consecutive lanes.
  Copies written into LDS by buffer loads (``... lds``) are not counted:
  they do not show in those counters (the bf16 GEMM's measured LDS-active
  cycles equal its predicted fragment-read cycles within 0.2%).

Each ``*_launch`` function below mirrors the addressing of one kernel family
in ``csrc/`` and returns a :class:`LdsCost` for one launch.
"""
from __future__ import annotations

import json
from dataclasses import dataclass

BANKS = 64

_B128 = [[0, 1, 2, 3, 12, 13, 14, 15, 20, 21, 22, 23, 24, 25, 26, 27],
         [4, 5, 6, 7, 8, 9, 10, 11, 16, 17, 18, 19, 28, 29, 30, 31]]
PHASES = {
    "ds_read_b128": _B128 + [[l + 32 for l in p] for p in _B128],
    "ds_read_b64": [list(range(32)), list(range(32, 64))],
    "ds_read_b64_tr_b16": [list(range(32)), list(range(32, 64))],
    "ds_read_b32": [list(range(32)), list(range(32, 64))],
    "ds_write_b128": [list(range(8 * i, 8 * i + 8)) for i in range(8)],
    "ds_write_b64": [list(range(16 * i, 16 * i + 16)) for i in range(4)],
    "ds_write_b32": [list(range(32)), list(range(32, 64))],
    "ds_write_b16": [list(range(32)), list(range(32, 64))],
}
WIDTH = {"ds_read_b128": 16, "ds_read_b64": 8, "ds_read_b64_tr_b16": 8, "ds_read_b32": 4,
         "ds_write_b128": 16, "ds_write_b64": 8, "ds_write_b32": 4, "ds_write_b16": 2}
# Banks a phase of the instruction sees: two lanes of one phase conflict when
# their dword addresses differ by a multiple of this (measured by scanning
# the address distance of two lanes of one phase).
PERIOD = {"ds_read_b128": 64, "ds_read_b64": 64, "ds_read_b64_tr_b16": 64, "ds_read_b32": 32,
          "ds_write_b128": 32, "ds_write_b64": 32, "ds_write_b32": 32, "ds_write_b16": 32}


def cycles(op: str, addrs) -> int:
    """LDS cycles of one wave instruction: ``addrs`` holds each lane's byte
    address (None for an inactive lane)."""
    words = max(1, WIDTH[op] // 4)       # a 2-byte access uses the bank of its dword
    nbanks = PERIOD.get(op, BANKS)
    total = 0
    for phase in PHASES[op]:
        banks = {}
        for lane in phase:
            a = addrs[lane]
            if a is None:
                continue
            w0 = a // 4
            for d in range(words):
                banks.setdefault((w0 + d) % nbanks, set()).add(w0 + d)
        total += max((len(s) for s in banks.values()), default=0)
    return total


def ideal(op: str) -> int:
    """Conflict-free cycles of one wave instruction (one per phase)."""
    return len(PHASES[op])


@dataclass
class LdsCost:
    """LDS cycles of one launch: ``active`` (every cycle an LDS instruction
    occupies, the counterpart of SQ_LDS_IDX_ACTIVE), ``conflict`` (the
    cycles beyond one per phase, SQ_LDS_BANK_CONFLICT), ``read_bytes`` and
    ``write_bytes`` (bytes the instructions move)."""
    active: int = 0
    conflict: int = 0
    read_bytes: int = 0
    write_bytes: int = 0

    def add(self, op: str, addrs, times: int = 1):
        c = cycles(op, addrs)
        self.active += c * times
        self.conflict += (c - ideal(op)) * times
        nb = WIDTH[op] * sum(a is not None for a in addrs) * times
        if op.startswith("ds_write"):
            self.write_bytes += nb
        else:
            self.read_bytes += nb

    def scaled(self, k: int) -> "LdsCost":
        return LdsCost(self.active * k, self.conflict * k, self.read_bytes * k, self.write_bytes * k)

    def __iadd__(self, o: "LdsCost"):
        self.active += o.active
        self.conflict += o.conflict
        self.read_bytes += o.read_bytes
        self.write_bytes += o.write_bytes
        return self

    @property
    def ratio(self) -> float:
        return self.conflict / self.active if self.active else 0.0


def _cdiv(a, b):
    return (a + b - 1) // b


# ---------------------------------------------------------------- bf16 GEMM

def swz_a_bf16(ca: int, row: int) -> int:
    """A-row chunk swizzle of the bf16 direct-to-LDS GEMM (csrc/gemm_bf16.hip)."""
    return (row >> 2) & 3 if ca == 4 else (row >> 1) & 7


def swz_b_bf16(k: int, mi: int = 32) -> int:
    return ((k & 1) * 6) ^ ((k & 2) * 5) ^ ((((k >> 3) & 1) * 2) if mi == 16 else 0)


def gemm_bf16_dma_stage(BM, BN, BK, WM, WN, MI, swz_a=swz_a_bf16) -> LdsCost:
    """LDS cost of one LDS stage of one workgroup (all its waves) of the
    bf16 direct-to-LDS GEMM: per MFMA k-step, TM ds_read_b128 A fragments and
    2*TN ds_read_b64_tr_b16 B fragment halves per wave."""
    NWN = BN // WN
    TM, TN = WM // MI, WN // MI
    KCH = 16 if MI == 32 else 32
    RA, CA, RB = BK * 2, BK // 8, BN * 2
    cost = LdsCost()
    for wave in range((BM // WM) * NWN):
        wm, wn = wave // NWN, wave % NWN
        for kk in range(0, BK, KCH):
            for i in range(TM):
                addrs = []
                for lane in range(64):
                    lrow, lgrp = lane % MI, lane // MI
                    row = wm * WM + i * MI + lrow
                    addrs.append(row * RA + (((kk >> 3) + lgrp) ^ swz_a(CA, row)) * 16)
                cost.add("ds_read_b128", addrs)
            for j in range(TN):
                for half in (0, 4):
                    addrs = []
                    for lane in range(64):
                        lrow, lgrp = lane % MI, lane // MI
                        rsub = (lane & 15) >> 2
                        chunk = (((wn * WN + j * MI + (lrow & ~15) + 4 * (lane & 3)) >> 3)
                                 ^ swz_b_bf16(8 * (lgrp & 1) + rsub, MI)) * 16 + 8 * (lane & 1)
                        addrs.append((kk + 8 * lgrp + rsub + half) * RB + chunk)
                    cost.add("ds_read_b64_tr_b16", addrs)
    return cost


def gemm_bf16_dma_launch(sched, M, N, K, swz_a=swz_a_bf16) -> LdsCost:
    """One launch of the bf16 direct-to-LDS GEMM: every stage of every tile
    (the stage's slot base is a multiple of 256 bytes, so every stage has the
    same bank pattern), plus the one fragment set read past the last stage."""
    s = sched
    stage = gemm_bf16_dma_stage(s["block_m"], s["block_n"], s["block_k"], s["wave_m"],
                                s["wave_n"], s["mfma_m"], swz_a)
    tiles = _cdiv(M, s["block_m"]) * _cdiv(N, s["block_n"])
    kt = _cdiv(K, s["block_k"])
    steps = s["block_k"] // (16 if s["mfma_m"] == 32 else 32)
    total = stage.scaled(kt * steps)
    # the per-stage cost is per step-set times steps; add one extra set
    per_set = LdsCost(stage.active // steps, stage.conflict // steps,
                      stage.read_bytes // steps, stage.write_bytes // steps)
    total += per_set
    return LdsCost(total.active * tiles // steps, total.conflict * tiles // steps,
                   total.read_bytes * tiles // steps, total.write_bytes * tiles // steps)


# ------------------------------------------------- fp32 balanced halo conv

def conv_f32_halo16_launch(N, C, H, W, OC, pad_h, pad_w, nh=2, plane_pad=16,
                           a_swizzle=False, tile_px=None) -> LdsCost:
    """One launch of the balanced halo-tiled fp32 conv (3x3, stride 1,
    csrc/conv2d_f32.hip): per instruction k-step (tap, 4-channel group) one
    ds_read_b32 A value and one ds_read_b32 B value per 16-pixel column
    block.  ``plane_pad``: floats between patch planes beyond the patch rows;
    ``a_swizzle``: output channel oc holds its channel c at slot
    c ^ (2 * ((oc >> 2) & 3)) (True, the kernel's layout), at c ^ f(oc % 16)
    for a callable f, or at c (False)."""
    BM, NB, CC, CO = 64, 13, 8, 4
    if callable(a_swizzle):
        a_xor = a_swizzle
    elif a_swizzle:
        a_xor = lambda lcol: ((lcol >> 2) & 3) << 1
    else:
        a_xor = lambda lcol: 0
    PR = 8 if nh == 1 else 10
    PLANE = PR * 64 + plane_pad
    OH, OW = H + 2 * pad_h - 2, W + 2 * pad_w - 2
    OHW = OH * OW
    BNmax = 16 * NB * nh
    if tile_px is None:
        t = _cdiv(OHW, BNmax)
        tile_px = _cdiv(OHW, t)
    chunks = _cdiv(OHW, tile_px)
    per_image = LdsCost()
    for ch in range(chunks):
        p0 = ch * tile_px
        pend = min(p0 + tile_px, OHW)
        oh0 = p0 // OW
        for wave in range(4 * nh):
            wq, half = wave & 3, wave >> 2
            nbw = NB - 1 if (nh == 2 and half == 1 and tile_px <= 16 * (2 * NB - 1)) else NB
            pw0 = p0 + 16 * NB * half
            offs = []
            for j in range(nbw):
                row = []
                for lane in range(64):
                    pix = pw0 + 16 * j + (lane & 15)
                    off = 0
                    if pix < pend:
                        oh, ow = divmod(pix, OW)
                        off = (oh - oh0) * 64 + ow - pad_w + CO
                    row.append(off)
                offs.append(row)
            for t in range(18):
                tap, s = t >> 1, t & 1
                kh, kw = divmod(tap, 3)
                a = []
                for lane in range(64):
                    lcol, lgrp = lane & 15, lane >> 4
                    c = lgrp + 4 * s
                    slot = c ^ a_xor(lcol)
                    a.append(4 * (tap * BM * CC + (wq * 16 + lcol) * CC + slot))
                per_image.add("ds_read_b32", a)
                for j in range(nbw):
                    b = [4 * ((lane >> 4) * PLANE + offs[j][lane] + 4 * s * PLANE + kh * 64 + kw)
                         for lane in range(64)]
                    per_image.add("ds_read_b32", b)
    # tiles per output-channel block; stages C / 8; images N
    return per_image.scaled(_cdiv(OC, BM) * (C // CC) * N)


# --------------------------------------------------- bf16 halo-tiled conv

def conv_bf16_halo_launch(N, C, H, W, OC, pad_h, pad_w, a_swizzle=False, rotate=False,
                          store_order=False, trailing_store=False) -> LdsCost:
    """One launch of the bf16 halo-tiled conv (3x3, stride 1,
    csrc/conv2d_bf16.hip): per stage and wave, the register-staged patch and
    weight stores (ds_write_b128) and, per tap, TM ds_read_b128 A fragments
    and TN ds_read_b128 B fragments (one 16-byte cell of 8 channels).
    ``a_swizzle``: output channels with bit 3 set hold their two 8-channel
    halves swapped; ``rotate``: patch row r is stored rotated by
    (r * OW) mod 16 cells in rows of 80 cells (else unrotated rows of 64);
    ``store_order``: a thread writes its two patch cells in the order bit 2
    of its column pair selects (else even cells first); ``trailing_store``:
    the last stage also stores a (never read) next stage, as the kernel did
    before its loads went two stages ahead."""
    BM, BN, WM, WN, MI = 64, 256, 64, 64, 32
    TM, TN, CC, PR, CO = WM // MI, WN // MI, 16, 8, 2
    PC = 80 if rotate else 64
    HALF = PR * PC * 16
    P_BYTES = 2 * HALF
    OH, OW = H + 2 * pad_h - 2, W + 2 * pad_w - 2
    OHW = OH * OW
    chunks = _cdiv(OHW, BN)

    def rot(r):
        return (r * OW) % 16 if rotate else 0

    stage_w = LdsCost()
    # patch stores: thread tid -> patch row tid >> 5, column pair tid & 31
    for wave in range(4):
        for h in range(2):
            for second in range(2):
                addrs = []
                for lane in range(64):
                    tid = wave * 64 + lane
                    pr, cp = tid >> 5, tid & 31
                    first = ((cp >> 2) & 1) if store_order else 0
                    addrs.append(h * HALF + (pr * PC + 2 * cp + (second ^ first) + rot(pr)) * 16)
                stage_w.add("ds_write_b128", addrs)
        if wave < 2:   # weight slabs: threads 0 .. 127
            for t in range(9):
                addrs = []
                for lane in range(64):
                    tid = wave * 64 + lane
                    woc, wh = tid >> 1, tid & 1
                    slot = wh ^ ((woc >> 3) & 1) if a_swizzle else wh
                    addrs.append(P_BYTES + ((t * BM + woc) * CC + 8 * slot) * 2)
                stage_w.add("ds_write_b128", addrs)
    per_image = LdsCost()
    for ch in range(chunks):
        p0 = ch * BN
        oh0 = p0 // OW
        for wave in range(4):
            cells = []
            for j in range(TN):
                row = []
                for lane in range(64):
                    pix = p0 + wave * WN + j * MI + lane % MI
                    if pix < OHW:
                        oh, ow = divmod(pix, OW)
                        row.append((oh - oh0, ow - pad_w + CO))
                    else:
                        row.append((0, 0))
                cells.append(row)
            for t in range(9):
                kh, kw = divmod(t, 3)
                for i in range(TM):
                    addrs = []
                    for lane in range(64):
                        lrow, lgrp = lane % MI, lane // MI
                        slot = lgrp ^ ((lrow >> 3) & 1) if a_swizzle else lgrp
                        addrs.append(P_BYTES + ((t * BM + i * MI + lrow) * CC + 8 * slot) * 2)
                    per_image.add("ds_read_b128", addrs)
                for j in range(TN):
                    addrs = []
                    for lane in range(64):
                        r, c = cells[j][lane]
                        addrs.append((lane // MI) * HALF + ((r + kh) * PC + c + kw + rot(r + kh)) * 16)
                    per_image.add("ds_read_b128", addrs)
        per_image += stage_w
    # the prologue's store of stage 0 and one store per stage but the last
    # (plus the last one's when ``trailing_store``)
    total = per_image.scaled(C // CC)
    if trailing_store:
        total += stage_w.scaled(chunks)
    return total.scaled(_cdiv(OC, BM) * N)


def rows_swz(c: int) -> int:
    """Cell-slot swizzle of the bf16 row-streaming conv (csrc/conv2d_bf16.hip)."""
    return ((c >> 1) ^ (c & ~3)) & 7


def conv_bf16_rows_launch(N, C, H, W, OC, pad_h, pad_w) -> LdsCost:
    """One launch of the bf16 row-streaming conv (3x3, stride 1, 64 input
    channels; csrc/conv2d_bf16.hip, k_order 3).  Per workgroup: the weight
    cells (ds_write_b128, two slabs of nine taps per thread) and band rows 0
    .. 3 once; per step of two output rows, the two new input rows (two
    ds_write_b128 per thread and row) and, per wave and (kw, 16-channel
    k-step) group, three weight and four pixel fragments (ds_read_b128);
    plus the first group of the step after the last; and per wave and output
    row of a step, the staging of the row for the stores (four ds_write_b128
    and four ds_read_b128)."""
    assert C == 64
    BM, NCG, RO, CO = 64, 8, 2, 2
    OH, OW = H + 2 * pad_h - 2, W + 2 * pad_w - 2
    per_img = _cdiv(OC, BM) * N
    nb = _cdiv(256, per_img)
    band = _cdiv(_cdiv(OH, nb), RO) * RO         # whole steps, as the launcher sizes bands
    nbands = _cdiv(OH, band)
    row_w = LdsCost()           # one input row into the ring (every thread)
    for wave in range(4):
        for second in range(2):
            addrs = []
            for lane in range(64):
                tid = wave * 64 + lane
                q, g = tid & 31, tid >> 5
                wodd = (q >> 2) & 1
                col = 2 * q + (wodd ^ second)
                addrs.append(col * NCG * 16 + ((g ^ rows_swz(col)) << 4))
            row_w.add("ds_write_b128", addrs)
    weights = LdsCost()
    for wave in range(4):
        for h in range(2):
            for t in range(9):
                addrs = []
                for lane in range(64):
                    s_ = wave * 64 + lane + 256 * h
                    oc, wg = s_ >> 3, s_ & 7
                    addrs.append(t * BM * NCG * 16 + oc * NCG * 16 + ((wg ^ rows_swz(oc)) << 4))
                weights.add("ds_write_b128", addrs)
    group = LdsCost()           # all (kw, k-step) groups of one step, all waves
    first_group = LdsCost()     # group (0, 0): also read ahead for the step after the last
    for wave in range(4):
        oc_l = [32 * (wave & 1) + lane % 32 for lane in range(64)]
        px_l = []
        for lane in range(64):
            px = 32 * (wave >> 1) + lane % 32
            if px >= OW:
                px = px - 32 if (px >= 32 and px - 32 < OW) else OW - 1
            px_l.append(px)
        for kw in range(3):
            for ks in range(C // 16):
                g = LdsCost()
                for kh in range(3):
                    g.add("ds_read_b128", [oc_l[l] * NCG * 16 + (((2 * ks + l // 32) ^ rows_swz(oc_l[l])) << 4)
                                           for l in range(64)])
                for i in range(RO + 2):
                    addrs = []
                    for l in range(64):
                        col = px_l[l] + kw - pad_w + CO
                        addrs.append(col * NCG * 16 + (((2 * ks + l // 32) ^ rows_swz(col)) << 4))
                    g.add("ds_read_b128", addrs)
                group += g
                if kw == 0 and ks == 0:
                    first_group += g
    staging = LdsCost()         # one output row of every wave, out and back
    for wave in range(4):
        for i in range(4):
            staging.add("ds_write_b128", [(l % 32) * 128 + (((2 * i + l // 32) ^ (l % 32 & 7)) << 4)
                                          for l in range(64)])
        for s4 in range(4):
            staging.add("ds_read_b128", [(8 * s4 + (l >> 3)) * 128 + (((l & 7) ^ (l >> 3)) << 4)
                                         for l in range(64)])
    total = LdsCost()
    for band_i in range(nbands):
        rows = min(band, OH - band_i * band)
        nsteps = _cdiv(rows, RO)
        total += weights
        total += row_w.scaled(2 * RO)                  # prologue: band rows 0 .. 3
        total += row_w.scaled(RO * nsteps)             # each step stores the next step's rows
        total += group.scaled(nsteps)
        total += first_group
        total += staging.scaled(RO * nsteps)
    return total.scaled(per_img)


# ---------------------------------------------------------------- fp32 GEMM

def swz_a_f32(ca: int, row: int) -> int:
    """A-row chunk swizzle of the fp32 direct-to-LDS GEMM (csrc/gemm_f32.hip)."""
    return (row >> 2) & 3 if ca == 4 else (row >> 1) & 7


def _waves(BM, BN, WM, WN):
    NWN = BN // WN
    return [(w // NWN, w % NWN) for w in range((BM // WM) * NWN)]


def gemm_f32_dma_stage(BM, BN, BK, WM, WN, MI, swz_a=swz_a_f32) -> LdsCost:
    """One LDS stage of one workgroup of the fp32 direct-to-LDS GEMM: per
    fragment set, TM ds_read_b128 A fragments and 4*TN ds_read_b32 B
    values per wave (B rows swizzled by lane group)."""
    KG = 2 if MI == 32 else 4
    KCH, SWB = 4 * KG, 16 // KG
    RA, CA, RB = BK * 4, BK // 4, BN * 4
    TM, TN = WM // MI, WN // MI
    cost = LdsCost()
    for wm, wn in _waves(BM, BN, WM, WN):
        for kk in range(0, BK, KCH):
            for i in range(TM):
                addrs = []
                for lane in range(64):
                    lrow, lgrp = lane % MI, lane // MI
                    row = wm * WM + i * MI + lrow
                    addrs.append(row * RA + (((kk >> 2) + lgrp) ^ swz_a(CA, row)) * 16)
                cost.add("ds_read_b128", addrs)
            for j in range(TN):
                for s in range(4):
                    addrs = []
                    for lane in range(64):
                        lrow, lgrp = lane % MI, lane // MI
                        boff = (4 * lgrp * BN + ((wn * WN + j * MI + lrow) ^ (4 * SWB * lgrp))) * 4
                        addrs.append((kk + s) * RB + boff)
                    cost.add("ds_read_b32", addrs)
    return cost


def gemm_f32_reg_stage(BM, BN, BK, WM, WN, MI, PAD):
    """(stores, reads) of one LDS stage of one workgroup of the fp32
    register-staged GEMM with 16-byte rows (padded A and B rows)."""
    NT = (BM // WM) * (BN // WN) * 64
    KG = 2 if MI == 32 else 4
    KCH = 4 * KG
    AS, BS = BK + PAD, BN + (8 if MI == 32 else 4)
    TM, TN = WM // MI, WN // MI
    st, rd = LdsCost(), LdsCost()
    for w in range(NT // 64):
        for i in range(BM * BK // (4 * NT)):
            addrs = []
            for lane in range(64):
                idx = w * 64 + lane + i * NT
                r, c = idx // (BK // 4), (idx % (BK // 4)) * 4
                addrs.append((r * AS + c) * 4)
            st.add("ds_write_b128", addrs)
        for i in range(BK * BN // (4 * NT)):
            addrs = []
            for lane in range(64):
                idx = w * 64 + lane + i * NT
                r, c = idx // (BN // 4), (idx % (BN // 4)) * 4
                addrs.append((r * BS + c) * 4)
            st.add("ds_write_b128", addrs)
    for wm, wn in _waves(BM, BN, WM, WN):
        for kk in range(0, BK, KCH):
            for i in range(TM):
                rd.add("ds_read_b128", [((wm * WM + lane % MI) * AS + 4 * (lane // MI) + i * MI * AS + kk) * 4
                                        for lane in range(64)])
            for j in range(TN):
                for s in range(4):
                    rd.add("ds_read_b32", [((4 * (lane // MI) + kk + s) * BS + wn * WN + lane % MI + j * MI) * 4
                                           for lane in range(64)])
    return st, rd


def gemm_f32_ksplit_tile(MI, TM, TN, KS) -> LdsCost:
    """The fixed-order reduction of one reduction-split tile: each of the KS
    waves writes its partial accumulators (ds_write_b32 of consecutive
    lanes), then the KS partials of every register are read back."""
    nacc = 16 if MI == 32 else 4
    nreg = TM * TN * nacc
    cost = LdsCost()
    contiguous = [4 * lane for lane in range(64)]
    cost.add("ds_write_b32", contiguous, times=KS * nreg)
    cost.add("ds_read_b32", contiguous, times=KS * nreg)
    return cost


# ---------------------------------------------------------------- bf16 GEMM (register-staged)

def gemm_bf16_reg_stage(BM, BN, BK, WM, WN, MI, PAD):
    """(stores, reads) of one LDS stage of the bf16 register-staged GEMM
    (16-byte chunks, padded A rows, B rows padded by 32 elements)."""
    NT = (BM // WM) * (BN // WN) * 64
    KG = 2 if MI == 32 else 4
    KCH = 8 * KG
    AS, BS = BK + PAD, BN + 32
    TM, TN = WM // MI, WN // MI
    st, rd = LdsCost(), LdsCost()
    for w in range(NT // 64):
        for i in range(BM * BK // (8 * NT)):
            addrs = []
            for lane in range(64):
                idx = w * 64 + lane + i * NT
                r, c = idx // (BK // 8), (idx % (BK // 8)) * 8
                addrs.append((r * AS + c) * 2)
            st.add("ds_write_b128", addrs)
        for i in range(BK * BN // (8 * NT)):
            addrs = []
            for lane in range(64):
                idx = w * 64 + lane + i * NT
                r, c = idx // (BN // 8), (idx % (BN // 8)) * 8
                addrs.append((r * BS + c) * 2)
            st.add("ds_write_b128", addrs)
    for wm, wn in _waves(BM, BN, WM, WN):
        for kk in range(0, BK, KCH):
            for i in range(TM):
                rd.add("ds_read_b128", [((wm * WM + lane % MI) * AS + 8 * (lane // MI) + i * MI * AS + kk) * 2
                                        for lane in range(64)])
            for j in range(TN):
                for half in (0, 4):
                    addrs = []
                    for lane in range(64):
                        lrow, lgrp = lane % MI, lane // MI
                        bs = ((8 * lgrp + ((lane & 15) >> 2)) * BS + wn * WN + (lrow & ~15)
                              + 4 * (lane & 3))
                        addrs.append((bs + (kk + half) * BS + j * MI) * 2)
                    rd.add("ds_read_b64_tr_b16", addrs)
    return st, rd


# ------------------------------------------------------- per-launch models

def matmul_launch(dtype: str, s: dict, M: int, N: int, K: int):
    """LDS cost of one launch of the matmul instance ``s`` (a schedule dict)
    on 16-byte-aligned row-major operands, or None if the instance's kernel
    is not modelled.  The instance's kernel is the one its launcher picks for
    such operands: the direct-to-LDS kernel for lds_pad -1, else the
    register-staged kernel, or for k_split > 1 the reduction-split kernel
    (lds_stages 0) or the direct-to-LDS kernel in k_split wave groups."""
    BM, BN, BK = s["block_m"], s["block_n"], s["block_k"]
    WM, WN, MI = s["wave_m"], s["wave_n"], s["mfma_m"]
    tiles = _cdiv(M, BM) * _cdiv(N, BN)
    kt = _cdiv(K, BK)
    if s.get("k_split", 1) > 1 and s.get("lds_stages", 0) > 0 and dtype == "f32" and s["lds_pad"] < 0:
        # k_split groups of waves, each the direct-to-LDS pipeline on every
        # k_split-th K-step (the same number of iterations in every group),
        # then the partial sums of groups 1.. through LDS, one lane-
        # contiguous dword per register, written once and read once
        ks = s["k_split"]
        stage = gemm_f32_dma_stage(BM, BN, BK, WM, WN, MI)
        steps = BK // (4 * (2 if MI == 32 else 4))
        ktg = _cdiv(kt, ks)
        one = stage.scaled(ktg * steps)
        one += stage
        tile = LdsCost(one.active * ks // steps, one.conflict * ks // steps,
                       one.read_bytes * ks // steps, one.write_bytes * ks // steps)
        nreg = (BM // WM) * (BN // WN) * (WM // MI) * (WN // MI) * (MI * MI // 64)
        lanes = [4 * l for l in range(64)]
        tile.add("ds_write_b32", lanes, times=(ks - 1) * nreg)
        tile.add("ds_read_b32", lanes, times=(ks - 1) * nreg)
        return tile.scaled(tiles)
    if s.get("k_split", 1) > 1:
        return gemm_f32_ksplit_tile(MI, BM // MI, BN // MI, s["k_split"]).scaled(tiles)
    if dtype == "bf16":
        if s["lds_pad"] < 0:
            return gemm_bf16_dma_launch(s, M, N, K)
        st, rd = gemm_bf16_reg_stage(BM, BN, BK, WM, WN, MI, s["lds_pad"])
        total = st.scaled(kt)
        total += rd.scaled(kt)
        return total.scaled(tiles)
    if s["lds_pad"] < 0:
        stage = gemm_f32_dma_stage(BM, BN, BK, WM, WN, MI)
        kch = 4 * (2 if MI == 32 else 4)
        steps = BK // kch
        total = stage.scaled(kt * steps)
        total += stage
        return LdsCost(total.active * tiles // steps, total.conflict * tiles // steps,
                       total.read_bytes * tiles // steps, total.write_bytes * tiles // steps)
    st, rd = gemm_f32_reg_stage(BM, BN, BK, WM, WN, MI, s["lds_pad"])
    total = st.scaled(kt)
    total += rd.scaled(kt)
    return total.scaled(tiles)


# ---------------------------------------------------- few-output-channel conv

def conv_f32_smallm_patch_launch(N, C, H, W, OC, R, S, sh, sw, ph, pw, vec=None):
    """One launch of the patch-staged few-output-channel fp32 conv
    (csrc/conv2d_f32.hip), or None when its patch does not fit (then the
    gather form runs, which uses LDS only for the k-offset table): per
    workgroup the staging stores (ds_write_b32 of consecutive lanes, spread
    over eight waves), per k-step and pixel block the table entry, the weight
    and the input value (ds_read_b32; the two halves of the waves take the
    two halves of the k-steps), and the second half's partial sums written
    and read back once (ds_write_b128 / ds_read_b128, lane-contiguous).
    ``vec``: 16-byte patch rows (the launcher's choice for widths that are
    a multiple of 4 and 16-byte aligned inputs, taken here for every such
    width): one ds_write_b128 per lane and row, the patch origin at a
    multiple of 4 columns."""
    BN, WAVES, SWAVES = 64, 4, 8
    if vec is None:
        vec = W % 4 == 0
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    OHW = OH * OW
    K = C * R * S
    KP = _cdiv(K, 32) * 32
    WS = KP + 2
    span = (BN - 1 + OW - 1) // OW + 1

    def geom(v):
        padl = _cdiv(pw, 4) * 4 if v else pw
        wp = (OW - 1) * sw + S - pw + padl
        if v:
            wp = _cdiv(wp, 4) * 4
        pr = (span - 1) * sh + R
        area = max(C * pr * wp, 32 * BN)        # the patch, later the partial sums
        fits = 4 * (area + 16 * (KP + 2)) + 4 * KP <= 48 * 1024 and wp <= 256 and KP <= 256
        return fits, pr, wp, padl, area
    fits, PR, WP, PADL, AREA = geom(vec)
    if vec and not fits:
        vec = False
        fits, PR, WP, PADL, AREA = geom(False)
    if not fits:
        return None
    PLANE = PR * WP

    def tab(k):
        if k >= K:
            return 0
        ic, rem = divmod(k, R * S)
        kh, kw = divmod(rem, S)
        return ic * PLANE + kh * WP + kw

    per_image = LdsCost()
    chunks = _cdiv(OHW, BN)
    contiguous = [4 * lane for lane in range(64)]
    for ch in range(chunks):
        p0 = ch * BN
        oh_a = p0 // OW
        # staging: patch rows (4 column groups each), weights, table
        rows = C * PR
        for w in range(SWAVES):
            nr = len(range(w, rows, SWAVES))
            if vec:
                # lanes past the row are masked; counted like the rest, as
                # for the 4-byte stores
                per_image.add("ds_write_b128", [16 * lane for lane in range(64)], times=nr)
            else:
                per_image.add("ds_write_b32", contiguous, times=nr * _cdiv(WP, 64))
            per_image.add("ds_write_b32", contiguous, times=2 * _cdiv(KP, 64))
        per_image.add("ds_write_b32", contiguous, times=_cdiv(KP, 64))
        red = [16 * lane for lane in range(64)]
        per_image.add("ds_write_b128", red, times=WAVES * 2)
        per_image.add("ds_read_b128", red, times=WAVES * 2)
        for w in range(WAVES):
            pb = []
            for lane in range(64):
                pix = p0 + w * 16 + (lane & 15)
                if pix < OHW:
                    oh, ow = divmod(pix, OW)
                    pb.append((oh - oh_a) * sh * WP + ow * sw + PADL - pw)
                else:
                    pb.append(0)
            for s in range(KP // 4):
                per_image.add("ds_read_b32", [4 * tab(4 * s + (lane >> 4)) for lane in range(64)])
                per_image.add("ds_read_b32", [4 * (AREA + (lane & 15) * WS + (lane >> 4) + 4 * s)
                                              for lane in range(64)])
                per_image.add("ds_read_b32", [4 * (pb[lane] + tab(4 * s + (lane >> 4))) for lane in range(64)])
    return per_image.scaled(_cdiv(OC, 16) * N)


# ------------------------------------------------ fp32 conv: gather kernels

def _ktab_build(K: int, NW: int, base: int) -> LdsCost:
    """Building the k-offset table at kernel start: thread t writes entries
    t, t + NT, ... (8 bytes each), one ds_write_b64 per wave and pass in
    which the wave has an entry."""
    NT = 64 * NW
    cost = LdsCost()
    n = sum(1 for i in range(_cdiv(K, NT)) for w in range(NW) if w * 64 + i * NT < K)
    cost.add("ds_write_b64", [base + 8 * lane for lane in range(64)], times=n)
    return cost


def conv_f32_gather_dma_launch(BM, BN, WM, WN, STAGES, N, C, H, W, OC, R, S, sh, sw, ph, pw,
                               tap: bool) -> LdsCost:
    """The fp32 direct-to-LDS gather conv kernels (block_k 32, 32x32x2
    instructions): the tap-major kernel (``tap``) and the k-table kernel.
    Both read fragments as the direct-to-LDS GEMM does (weight chunks
    swizzled by (m ^ m >> 3) & 7, pixel columns XOR 32 on odd groups of four
    k rows), K-stages x block_k / 8 fragment sets per workgroup.  The
    k-table kernel also builds its table and reads one entry (the same for
    every lane of a wave) per k row a wave gathers, in every stage it
    prepares: the STAGES of the prologue and one per K-stage."""
    BK, MI = 32, 32
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    K, NW = C * R * S, (BM // WM) * (BN // WN)
    KT = _cdiv(K, BK)
    tile = gemm_f32_dma_stage(BM, BN, BK, WM, WN, MI,
                              swz_a=lambda ca, row: (row ^ (row >> 3)) & 7).scaled(KT)
    if not tap:
        base = STAGES * (BM + BN) * BK * 4
        tile += _ktab_build(K, NW, base)
        tile.add("ds_read_b64", [base] * 64, times=(STAGES + KT) * BK)
    return tile.scaled(_cdiv(OC, BM) * _cdiv(N * OH * OW, BN))


def conv_f32_reg_launch(BM, BN, BK, WM, WN, MI, PAD, N, C, H, W, OC, R, S, sh, sw, ph, pw,
                        vec: bool) -> LdsCost:
    """The fp32 register-staged gather conv kernel: per K-stage the weight
    tile's 16-byte (``vec``) or 4-byte stores, one 4-byte store per gathered
    element (thread t owns pixel column t % BN), and the register-staged
    GEMM's fragment reads; at kernel start the k-offset table.  A wave reads
    the table entry of each k row it gathers (every lane the same entry, as
    two 4-byte reads) when one of its lanes has a pixel and k < K."""
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    K, Ng = C * R * S, N * OH * OW
    NW = (BM // WM) * (BN // WN)
    NT = 64 * NW
    KT = _cdiv(K, BK)
    AS, BS = BK + PAD, BN + (8 if MI == 32 else 4)
    WA = 4 if vec else 1
    _, stage = gemm_f32_reg_stage(BM, BN, BK, WM, WN, MI, PAD)
    for w in range(NW):
        for i in range(BM * BK // (WA * NT)):
            addrs = []
            for lane in range(64):
                idx = w * 64 + lane + i * NT
                r, c = idx // (BK // WA), (idx % (BK // WA)) * WA
                addrs.append((r * AS + c) * 4)
            stage.add("ds_write_b128" if vec else "ds_write_b32", addrs)
    brpp = NT // BN                       # gathered k rows per pass
    for w in range(NW):
        for i in range(BK // brpp):
            stage.add("ds_write_b32", [(((w * 64 + lane) // BN + i * brpp) * BS + (w * 64 + lane) % BN) * 4
                                       for lane in range(64)])
    tiles_m, tiles_n = _cdiv(OC, BM), _cdiv(Ng, BN)
    total = stage.scaled(KT * tiles_m * tiles_n)
    base = 2 * (BM * AS + BK * BS) * 4
    total += _ktab_build(K, NW, base).scaled(tiles_m * tiles_n)
    total.add("ds_read_b32", [base] * 64,
              times=_reg_table_reads(N, C, H, W, R, S, sh, sw, ph, pw, BN, NW, BK) * tiles_m)
    return total


def conv_bf16_gather_launch(BM, BN, BK, WM, WN, MI, PAD, N, C, H, W, OC, R, S, sh, sw, ph, pw) -> LdsCost:
    """The bf16 register-staged gather conv kernel: per K-stage the weight
    tile's 16-byte stores (2-byte ones when C*R*S is not a multiple of 8),
    one 2-byte store per gathered element, and the bf16 register-staged
    GEMM's fragment reads (transpose reads for the pixel operand); the
    k-offset table and its reads as in the fp32 kernel."""
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    K, Ng = C * R * S, N * OH * OW
    NW = (BM // WM) * (BN // WN)
    NT = 64 * NW
    KT = _cdiv(K, BK)
    AS, BS = BK + PAD, BN + 32
    vec = K % 8 == 0
    WA = 8 if vec else 1
    _, stage = gemm_bf16_reg_stage(BM, BN, BK, WM, WN, MI, PAD)
    for w in range(NW):
        for i in range(BM * BK // (WA * NT)):
            addrs = []
            for lane in range(64):
                idx = w * 64 + lane + i * NT
                r, c = idx // (BK // WA), (idx % (BK // WA)) * WA
                addrs.append((r * AS + c) * 2)
            stage.add("ds_write_b128" if vec else "ds_write_b16", addrs)
    brpp = NT // BN
    for w in range(NW):
        for i in range(BK // brpp):
            stage.add("ds_write_b16", [(((w * 64 + lane) // BN + i * brpp) * BS + (w * 64 + lane) % BN) * 2
                                       for lane in range(64)])
    tiles_m, tiles_n = _cdiv(OC, BM), _cdiv(Ng, BN)
    total = stage.scaled(KT * tiles_m * tiles_n)
    base = 2 * (BM * AS + BK * BS) * 2
    total += _ktab_build(K, NW, base).scaled(tiles_m * tiles_n)
    total.add("ds_read_b32", [base] * 64,
              times=_reg_table_reads(N, C, H, W, R, S, sh, sw, ph, pw, BN, NW, BK) * tiles_m)
    return total


def _reg_table_reads(N, C, H, W, R, S, sh, sw, ph, pw, BN, NW, BK) -> int:
    """Table reads of the register-staged gather conv kernels per output-
    channel tile row: a wave reads the entry of each k row it gathers (every
    lane the same entry) as two 4-byte reads, the first when one of its lanes
    has a pixel and k < K, the second (the input offset) only when the tap
    of k also falls inside the image for one of those lanes."""
    import numpy as np
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    K, Ng = C * R * S, N * OH * OW
    brpp = 64 * NW // BN
    ks = np.arange(K)
    kh, kw = (ks % (R * S)) // S, ks % S
    reads = 0
    for tn in range(_cdiv(Ng, BN)):
        for w in range(NW):
            cols = (w * 64 + np.arange(64)) % BN + tn * BN
            cols = cols[cols < Ng]
            if cols.size == 0:
                continue                  # no lane of the wave has a pixel
            pix = cols % (OH * OW)
            ih0, iw0 = (pix // OW) * sh - ph, (pix % OW) * sw - pw
            rin = ((ih0[None, :] + np.arange(R)[:, None] >= 0) &
                   (ih0[None, :] + np.arange(R)[:, None] < H))
            cin = ((iw0[None, :] + np.arange(S)[:, None] >= 0) &
                   (iw0[None, :] + np.arange(S)[:, None] < W))
            tap_in = (rin[:, None, :] & cin[None, :, :]).any(axis=2)      # [R][S]
            mine = ks[(ks % BK) % brpp == ((w * 64) // BN) % brpp]         # the k rows the wave gathers
            reads += mine.size + int(tap_in[kh[mine], kw[mine]].sum())
    return reads


def conv_f32_halo256_launch(N, C, H, W, OC, ph, pw) -> LdsCost:
    """The fp32 64x256 halo kernel (k_order 2 with 64x256 tiles): four 64x64
    waves of 32x32x2 instructions, one MFMA k-step per tap of an 8-channel
    stage.  Per tap a wave reads two weight fragments (ds_read_b128 of
    [tap][oc][8 channels] cells) and, per 32-pixel block, four ds_read_b32 of
    the patch at the lane's pixel plus the tap's offset (planes of 8 rows x
    64 columns + 8 floats).  Each workgroup reads C / 8 stages of nine taps
    plus the first tap of the stage after its last."""
    BM, BN, WN, MI, CC, PR, CO = 64, 256, 64, 32, 8, 8, 4
    PLANE = PR * 64 + 8
    A_BYTES = 9 * BM * CC * 4
    OH, OW = H + 2 * ph - 2, W + 2 * pw - 2
    OHW = OH * OW

    def tap_cost(p0, tap):
        oh0 = p0 // OW
        kh, kw = divmod(tap, 3)
        cost = LdsCost()
        for w in range(BN // WN):
            for i in range(BM // MI):
                cost.add("ds_read_b128", [((lane % 32) * CC + 4 * (lane // 32)) * 4 +
                                          (tap * BM * CC + i * MI * CC) * 4 for lane in range(64)])
            for j in range(WN // MI):
                base = []
                for lane in range(64):
                    pix = p0 + w * WN + j * MI + lane % 32
                    off = 0                       # past the image: patch position 0
                    if pix < OHW:
                        oh, ow = divmod(pix, OW)
                        off = (oh - oh0) * 64 + ow - pw + CO
                    base.append((4 * (lane // 32) * PLANE + off) * 4)
                for sub in range(4):
                    cost.add("ds_read_b32", [A_BYTES + b + (sub * PLANE + kh * 64 + kw) * 4 for b in base])
        return cost

    total = LdsCost()
    for chunk in range(_cdiv(OHW, BN)):
        stage = LdsCost()
        for tap in range(9):
            stage += tap_cost(chunk * BN, tap)
        total += stage.scaled(C // CC)
        total += tap_cost(chunk * BN, 0)
    return total.scaled(N * _cdiv(OC, BM))


# the tap-major instances' stages and their k-table fallback's stages
_TAP_FALLBACK = {(64, 256): 2, (64, 128): 3, (64, 64): 4, (128, 128): 3}


def _conv_f32_gather(s: dict, k_order: int, stages: int, dims) -> LdsCost:
    """The launchers' chain below the halo kernels: tap-major when C % 32 ==
    0, else the k-table direct-to-LDS kernel with the fallback stages, else
    (C*R*S not a multiple of 4) the register-staged kernel with 4-float
    padded rows."""
    N, C, H, W, OC, R, S, sh, sw, ph, pw = dims
    BM, BN, WM, WN = s["block_m"], s["block_n"], s["wave_m"], s["wave_n"]
    K = C * R * S
    if k_order == 1:
        if C % 32 == 0:
            return conv_f32_gather_dma_launch(BM, BN, WM, WN, stages, *dims, tap=True)
        stages = _TAP_FALLBACK[(BM, BN)]
    if K % 4 == 0:
        return conv_f32_gather_dma_launch(BM, BN, WM, WN, stages, *dims, tap=False)
    return conv_f32_reg_launch(BM, BN, 32, WM, WN, 32, 4, *dims, vec=False)


def conv_launch(dtype: str, s: dict, N, C, H, W, OC, R, S, stride, pad):
    """LDS cost of one conv launch of instance ``s``, or None when the kernel
    it runs for this shape is not modelled (the few-channel kernel's gather
    form, when the patch does not fit)."""
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    ph, pw = (pad, pad) if isinstance(pad, int) else pad
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    halo_class = R == 3 and S == 3 and sh == 1 and sw == 1
    dims = (N, C, H, W, OC, R, S, sh, sw, ph, pw)
    if dtype == "f32" and s["block_m"] == 16 and s["lds_stages"] == 0:
        return conv_f32_smallm_patch_launch(N, C, H, W, OC, R, S, sh, sw, ph, pw)
    if dtype == "f32" and s["k_order"] == 2 and s["block_n"] in (208, 416):
        nh = 1 if s["block_n"] == 208 else 2
        if halo_class and C % 8 == 0 and pw <= 4 and OW - pw + 5 <= 63:
            # the launcher's pixel tile: the fewest tiles per image of at most 208*nh
            ohw = OH * OW
            t = _cdiv(ohw, 208 * nh)
            pt = _cdiv(ohw, t)
            span = (pt - 1 + OW - 1) // OW + 1
            if span + 2 <= (8 if nh == 1 else 10):
                return conv_f32_halo16_launch(N, C, H, W, OC, ph, pw, nh=nh, a_swizzle=True, tile_px=pt)
        s = dict(s, block_n=256, wave_m=64, wave_n=64)   # falls back to the 64x256 halo kernel
    if dtype == "f32" and s["k_order"] == 2:
        span = (256 - 1 + OW - 1) // OW + 1
        if halo_class and C % 16 == 0 and pw <= 4 and OW - pw + 5 <= 63 and span + 2 <= 8:
            return conv_f32_halo256_launch(N, C, H, W, OC, ph, pw)
        return _conv_f32_gather(dict(s, block_m=64, block_n=256, wave_m=64, wave_n=64), 1, 2, dims)
    if dtype == "f32" and s["k_order"] == 1:
        return _conv_f32_gather(s, 1, s["lds_stages"], dims)
    if dtype == "f32" and s["k_order"] == 0 and s["lds_pad"] < 0:
        return _conv_f32_gather(s, 0, s["lds_stages"], dims)
    if dtype == "f32" and s["k_order"] == 0:
        return conv_f32_reg_launch(s["block_m"], s["block_n"], s["block_k"], s["wave_m"], s["wave_n"],
                                   s["mfma_m"], s["lds_pad"], *dims, vec=(C * R * S) % 4 == 0)
    if dtype == "bf16" and s["k_order"] == 3:
        if halo_class and C == 64 and W % 2 == 0 and pw <= 2 and OW % 4 == 0 and OW <= 64 and OW + 1 - pw + 2 <= 63:
            return conv_bf16_rows_launch(N, C, H, W, OC, ph, pw)
        s = dict(s, k_order=2, block_n=256)   # the launcher falls back to the halo kernel
    if dtype == "bf16" and s["k_order"] == 2:
        span = (256 - 1 + OW - 1) // OW + 1
        if halo_class and C % 16 == 0 and W % 2 == 0 and pw <= 2 and OW - pw + 3 <= 63 and span + 2 <= 8:
            return conv_bf16_halo_launch(N, C, H, W, OC, ph, pw, a_swizzle=True, rotate=True,
                                         store_order=True)
        # the halo launcher falls back to the gather kernel's 64x128 tiles
        s = dict(s, k_order=0, block_m=64, block_n=128, block_k=32, wave_m=32, wave_n=64, mfma_m=32,
                 lds_pad=8)
    if dtype == "bf16" and s["k_order"] == 0:
        return conv_bf16_gather_launch(s["block_m"], s["block_n"], s["block_k"], s["wave_m"], s["wave_n"],
                                       s["mfma_m"], s["lds_pad"], *dims)
    return None


# ----------------------------------------------------------- evaluation

def run(op: str, dtype: str, dims, order_path: str, reps: int = 2):
    """Launch every compiled instance of op/dtype ``reps`` times on the
    problem ``dims`` (matmul: M, N, K; conv: N, C, H, W, OC, R, S, stride,
    pad) and record the order, so that the profiler's per-dispatch counter
    rows can be matched to instances.  LDS traffic does not depend on the
    raster order, so raster 0 stands for all of them."""
    import torch

    import paper_2512_16512_amd as xtc
    from paper_2512_16512_amd import tune
    p = tune.Problem(op, dtype, tuple(dims))
    code = xtc.XTC_F32 if dtype == "f32" else xtc.XTC_BF16
    opc = xtc.XTC_OP_MATMUL if op == "matmul" else xtc.XTC_OP_CONV2D
    stream = torch.cuda.current_stream().cuda_stream
    entries = []
    for s in xtc.xtc_sched_list(opc, code):
        s.raster, s.xcd_remap = 0, 1
        for _ in range(reps):
            p.launch(s, stream)
        torch.cuda.synchronize()
        entries.append(s.as_dict())
    with open(order_path, "w") as f:
        json.dump({"op": op, "dtype": dtype, "dims": list(dims), "reps": reps, "schedules": entries}, f)
    print("launched %d instances x %d" % (len(entries), reps), flush=True)


def _counter_rows(csv_path: str, counter: str):
    import csv
    rows = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter or "xtc::" not in r["Kernel_Name"]:
            continue
        d = int(r["Dispatch_Id"])
        rows[d] = rows.get(d, 0.0) + float(r["Counter_Value"])
    return [rows[d] for d in sorted(rows)]


def predict(op: str, dtype: str, s: dict, dims):
    if op == "matmul":
        return matmul_launch(dtype, s, *dims)
    return conv_launch(dtype, s, *dims)


def correlate(order_path: str, csv_path: str):
    """Predicted vs measured LDS-active and bank-conflict cycles per
    instance; returns the table and (Pearson, Spearman) for both counters
    over the modelled instances."""
    from paper_2512_16512_amd.traffic_model import pearson, spearman
    o = json.load(open(order_path))
    act = _counter_rows(csv_path, "SQ_LDS_IDX_ACTIVE")
    con = _counter_rows(csv_path, "SQ_LDS_BANK_CONFLICT")
    reps = o["reps"]
    n = len(o["schedules"])
    if len(act) != reps * n or len(con) != reps * n:
        raise ValueError("%d/%d counter rows for %d instances x %d launches"
                         % (len(act), len(con), n, reps))
    table = []
    for i, s in enumerate(o["schedules"]):
        pred = predict(o["op"], o["dtype"], s, o["dims"])
        table.append({"sched": s,
                      "measured_active": sum(act[i * reps:(i + 1) * reps]) / reps,
                      "measured_conflict": sum(con[i * reps:(i + 1) * reps]) / reps,
                      "predicted_active": None if pred is None else pred.active,
                      "predicted_conflict": None if pred is None else pred.conflict})
    mod = [t for t in table if t["predicted_active"] is not None]
    stats = {}
    for key in ("active", "conflict"):
        x = [t["predicted_" + key] for t in mod]
        y = [t["measured_" + key] for t in mod]
        stats[key] = (pearson(x, y), spearman(x, y)) if len(mod) > 2 else (float("nan"),) * 2
    return table, stats


def main(argv=None):
    import argparse
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    r = sub.add_parser("run")
    r.add_argument("op", choices=["matmul", "conv2d"])
    r.add_argument("dtype", choices=["f32", "bf16"])
    r.add_argument("dims", type=int, nargs="+")
    r.add_argument("--order", required=True)
    r.add_argument("--reps", type=int, default=2)
    c = sub.add_parser("correlate")
    c.add_argument("order")
    c.add_argument("counters_csv")
    c.add_argument("--json", default=None)
    a = ap.parse_args(argv)
    if a.cmd == "run":
        run(a.op, a.dtype, a.dims, a.order, a.reps)
        return 0
    table, stats = correlate(a.order, a.counters_csv)
    for key, (r_, rho) in stats.items():
        print("%-8s Pearson r = %.4f  Spearman rho = %.4f" % (key, r_, rho))
    if a.json:
        with open(a.json, "w") as f:
            json.dump({"stats": stats, "rows": table}, f, indent=1)
    return 0


if __name__ == "__main__":
    import sys
    sys.exit(main())
