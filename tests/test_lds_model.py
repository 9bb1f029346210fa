"""Host-side model of the LDS traffic of the scan kernels, barrier interval by barrier
interval, per wave and per lane (no GPU).

Each kernel's LDS accesses are written out here from its source: for every thread, the
array, the byte range and the direction of every LDS read and write between two
workgroup barriers (the kernels' __syncthreads calls), for one 64-token chunk (sequence
kernels) or one block (block kernel), at every dstate the kernels are built for.  The
checks, per interval:

* no byte is written by one wave and read or written by another (with no barrier in
  between, such an access would race);
* no two lanes write the same byte with one instruction, and no two threads write the
  same byte in one interval at all (the stored value would depend on timing);
* every index stays inside its array (an index past the end would land in another
  array);
* every byte read was written earlier in the same chunk (LDS is not cleared between
  workgroups: a byte not rewritten would hold whatever the previous workgroup on that
  CU left there);
* the transposed B and x images of the sequence kernels: each (token, column) element
  is read from the slot it was written to, under the plain and the permuted layouts.

The permuted layouts are those of seg_state (used by it) and the same layouts applied
to seg_out (a variant that was measured and not kept: outputs changed in their last
bits from run to run).  The model finds no LDS hazard in either, so that variability did
not come from LDS ordering in the source.
"""
import collections

import pytest

P = 64          # head dim
KC = 64         # chunk length of the sequence kernels
THREADS = 256   # sequence kernels: 4 waves


# ----------------------------------------------------------------- index helpers
def img_idx(QN, f32, mt, q, grp, col):
    """Slot of the MFMA operand quad (token tile mt, dstate quad q, lane group grp,
    column col) in a B or C row image (bdlm_device.h, img_idx)."""
    chunk = (4 * q + grp) if f32 else (2 * q + (grp >> 1))
    return (mt * QN + q) * 64 + grp * 16 + (col ^ (chunk & 15))


def bt_slot(NS, tq, n):
    """Permuted slot of element (token quad tq, column n) of the transposed B image."""
    if NS == 16:
        t = (tq >> 1) & 7
    elif NS == 32:
        t = (tq & 7) | ((tq & 1) << 4)
    elif NS == 64:
        t = ((tq & 1) << 4) | (((n >> 4) & 1) << 2) | (((tq >> 1) & 1) << 1) | ((n >> 5) & 1)
    else:
        t = ((tq & 1) << 4) | ((n >> 4) & 1) | (((n >> 5) & 3) << 1)
    return tq * NS + (n ^ t)


def xt_slot(tq, p):
    """Permuted slot of element (token quad tq, column p) of the transposed x image."""
    t = ((tq & 1) << 4) | ((p >> 4) & 1) | (((tq >> 1) & 1) << 1) | (((p >> 5) & 1) << 2)
    return tq * P + (p ^ t)


# ------------------------------------------------------------------ the recorder
class Model:
    """Records LDS accesses: (interval, array, byte) -> [(thread, kind, instruction)]."""

    def __init__(self, arrays: dict):
        self.arrays = arrays                  # name -> size in bytes
        # a wave may rewrite bytes it wrote before in the same interval (with later
        # instructions: a wave's LDS instructions are served in order)
        self.same_wave_rewrites = False
        self.interval = 0
        self.acc = collections.defaultdict(list)
        self.oob = []
        self.elem = {}                        # (array, byte) -> logical element last written

    def barrier(self):
        self.interval += 1

    def access(self, tid, kind, instr, array, offset, nbytes, tag=None):
        size = self.arrays[array]
        if offset < 0 or offset + nbytes > size:
            self.oob.append((array, offset, nbytes, tid, instr))
            return
        for b in range(offset, offset + nbytes):
            self.acc[(self.interval, array, b)].append((tid, kind, instr))
            if tag is not None:
                if kind == "W":
                    self.elem[(array, b)] = tag
                else:
                    got = self.elem.get((array, b))
                    if got != tag:
                        self.mismatch.append((array, b, tag, got))

    mismatch: list

    def check(self):
        """Problems found: races, colliding writes, out-of-range indices, reads of bytes not
        written earlier in the chunk, and elements read from a slot another element was
        written to."""
        problems = [("out of range", o) for o in self.oob]
        written = set()                      # (array, byte) written in an earlier interval
        by_interval = collections.defaultdict(dict)
        for (iv, arr, b), lst in self.acc.items():
            by_interval[iv][(arr, b)] = lst
        for iv in sorted(by_interval):
            here = by_interval[iv]
            for key, lst in here.items():
                writers = {(t, i) for t, k, i in lst if k == "W"}
                wthreads = {t for t, _ in writers}
                readers = {t for t, k, _ in lst if k == "R"}
                if len(wthreads) > 1:
                    per_instr = collections.Counter(i for _, i in writers)
                    ok = (self.same_wave_rewrites and len({t // 64 for t in wthreads}) == 1 and
                          max(per_instr.values()) == 1)
                    if not ok:
                        problems.append(("two writers in one interval", iv, key, sorted(wthreads)[:4]))
                wwaves = {t // 64 for t in wthreads}
                rwaves = {t // 64 for t in readers}
                if wwaves and (rwaves - wwaves or len(wwaves) > 1):
                    problems.append(("cross-wave access to a written byte", iv, key,
                                     sorted(wwaves), sorted(rwaves)))
                if readers and not writers and key not in written:
                    problems.append(("read of a byte not written in this chunk", iv, key,
                                     sorted(readers)[:4]))
                if readers and writers:
                    # same wave: the read must come after the write in program order
                    first_w = min(i for _, i in writers)
                    if any(i < first_w for t, k, i in lst if k == "R"):
                        problems.append(("read before the write of the same wave", iv, key))
            written |= {k for k, lst in here.items() if any(x[1] == "W" for x in lst)}
        problems += [("element read from another element's slot", m) for m in self.mismatch[:8]]
        return problems


def new_model(arrays):
    m = Model(arrays)
    m.mismatch = []
    return m


# ------------------------------------------------------------- sequence kernels
def stage_chunk(m, NS, swz, with_rows, instr0=0, with_wr=False):
    """Stager::stage (bf16 storage): row images of B and C (with_rows), the transposed B
    image and the transposed x image, from the registers of one chunk; plus wave 0's
    decay sums."""
    QN = NS // 16
    BCPR = NS // 8
    BT = 16 * BCPR
    XCPR = P // 8
    XT = (KC // 2) * XCPR
    for tid in range(THREADS):
        for k in range(max(1, BT // THREADS)):
            task = tid + THREADS * k
            if task >= BT:
                continue
            g, pc = task // BCPR, task % BCPR
            if with_rows:
                for arr in ("sB", "sC"):
                    for r in range(4):
                        j = 4 * g + r
                        q0, q1 = 2 * pc, 2 * pc + 1
                        for qq in (q0, q1):
                            slot = img_idx(QN, False, j >> 4, qq >> 2, qq & 3, j & 15)
                            m.access(tid, "W", instr0 + 1, arr, slot * 8, 8,
                                     tag=(arr, j, 4 * qq))
            for d in range(4):
                for h in range(2):     # lo / hi halves: columns pc*8 + 2d + h
                    n = pc * 8 + 2 * d + h
                    slot = bt_slot(NS, g, n) if swz else g * NS + n
                    m.access(tid, "W", instr0 + 2, "sBt", slot * 8, 8, tag=("Bt", g, n))
        for k in range(max(1, XT // THREADS)):
            task = tid + THREADS * k
            if task >= XT:
                continue
            g, pc = task // XCPR, task % XCPR
            for d in range(4):
                for h in range(2):
                    p = pc * 8 + 2 * d + h
                    if swz:
                        word = xt_slot(g >> 1, p) * 2 + (g & 1)
                    else:
                        word = ((g >> 1) * P + p) * 2 + (g & 1)
                    m.access(tid, "W", instr0 + 3, "sXt", word * 4, 4, tag=("Xt", g, p))
    for lane in range(64):                    # wave 0: decay sums
        for arr in ("sDt", "sCs", "sEc", "sWs") + (("sWr",) if with_wr else ()):
            if arr in m.arrays:
                m.access(lane, "W", instr0 + 4, arr, lane * 4, 4, tag=(arr, lane))


def read_bt(m, tid, NS, swz, instr):
    """bt_read over every dstate tile: the transposed-B quads of tokens 16jt + 4grp ..,
    column 16q + col, and the elements they hold."""
    lane, grp, col = tid & 63, (tid & 63) >> 4, tid & 15
    for q in range(NS // 16):
        for jt in range(4):
            tq, n = 4 * jt + grp, 16 * q + col
            slot = bt_slot(NS, tq, n) if swz else tq * NS + n
            # the quad holds tokens 4tq .. 4tq+3 of column n: written as element (tq, n)
            m.access(tid, "R", instr, "sBt", slot * 8, 8, tag=("Bt", tq, n))


def read_xt(m, tid, swz, instr):
    """x operands: tokens 16jt + 4grp .. +3 of column p = 16 wave + col."""
    grp, col, wave = (tid & 63) >> 4, tid & 15, tid >> 6
    p = 16 * wave + col
    for jt in range(4):
        tq = 4 * jt + grp
        slot = xt_slot(tq, p) if swz else tq * P + p
        # two words: token pair 2tq (word 0) and 2tq + 1 (word 1)
        m.access(tid, "R", instr, "sXt", slot * 8, 4, tag=("Xt", 2 * tq, p))
        m.access(tid, "R", instr, "sXt", slot * 8 + 4, 4, tag=("Xt", 2 * tq + 1, p))


def seg_state_model(NS, both, swz=True):
    arrays = {"sBt": 16 * NS * 8, "sXt": 16 * P * 8}
    for a in ("sDt", "sCs", "sEc", "sWs", "sWr"):
        arrays[a] = KC * 4
    m = new_model(arrays)
    m.barrier()                                # kernel start / previous chunk's last barrier
    stage_chunk(m, NS, swz, with_rows=False, with_wr=both)
    m.barrier()
    for tid in range(THREADS):
        grp = (tid & 63) >> 4
        m.access(tid, "R", 10, "sCs", (KC - 1) * 4, 4, tag=("sCs", KC - 1))
        read_xt(m, tid, swz, 11)
        for jt in range(4):
            for r in range(4):
                t = 16 * jt + 4 * grp + r
                m.access(tid, "R", 12, "sWs", t * 4, 4, tag=("sWs", t))
                if both:
                    m.access(tid, "R", 12, "sWr", t * 4, 4, tag=("sWr", t))
        read_bt(m, tid, NS, swz, 13)
    m.barrier()                                # end of chunk
    return m


def seg_out_model(NS, sub, swz, want_y=True, carry=True):
    QN = NS // 16
    IMG = 4 * QN * 64
    arrays = {"sB": IMG * 8, "sC": IMG * 8, "sBt": 16 * NS * 8, "sXt": 16 * P * 8,
              "sM": 10 * 64 * 16}
    for a in ("sDt", "sCs", "sEc", "sWs"):
        arrays[a] = KC * 4
    m = new_model(arrays)
    m.barrier()
    stage_chunk(m, NS, swz, with_rows=True)
    m.barrier()
    # Gram tiles (wave w: tiles w, w + 4, w + 8) and the prefix term
    for tid in range(THREADS):
        wave, lane = tid >> 6, tid & 63
        grp, col = lane >> 4, lane & 15
        if want_y:
            for k in range(wave, 10, 4):
                mt = 0 if k < 1 else (1 if k < 3 else (2 if k < 6 else 3))
                jt = k - mt * (mt + 1) // 2
                for q in range(QN):
                    sb = img_idx(QN, False, jt, q, grp, col)
                    sc = img_idx(QN, False, mt, q, grp, col)
                    # quad (tile, q, grp, col) holds rows 16 tile + col, columns 16q + 4grp ..
                    m.access(tid, "R", 20, "sB", sb * 8, 8, tag=("sB", 16 * jt + col, 16 * q + 4 * grp))
                    m.access(tid, "R", 20, "sC", sc * 8, 8, tag=("sC", 16 * mt + col, 16 * q + 4 * grp))
                t = 16 * mt + col
                m.access(tid, "R", 21, "sCs", t * 4, 4, tag=("sCs", t))
                for r in range(4):
                    j = 16 * jt + 4 * grp + r
                    m.access(tid, "R", 21, "sCs", j * 4, 4, tag=("sCs", j))
                    m.access(tid, "R", 21, "sDt", j * 4, 4, tag=("sDt", j))
                m.access(tid, "W", 22, "sM", (k * 64 + lane) * 16, 16, tag=("sM", k, lane))
            for q in range(QN):
                for mt in range(4):
                    sc = img_idx(QN, False, mt, q, grp, col)
                    m.access(tid, "R", 23, "sC", sc * 8, 8, tag=("sC", 16 * mt + col, 16 * q + 4 * grp))
            for mt in range(4):
                for r in range(4):
                    t = 16 * mt + 4 * grp + r
                    m.access(tid, "R", 24, "sEc", t * 4, 4, tag=("sEc", t))
    m.barrier()                                # Gram tiles published
    for tid in range(THREADS):
        lane = tid & 63
        grp = lane >> 4
        read_xt(m, tid, swz, 30)
        if want_y:
            for mt in range(4):
                for jt in range(mt + 1):
                    k = mt * (mt + 1) // 2 + jt
                    m.access(tid, "R", 31, "sM", (k * 64 + lane) * 16, 16, tag=("sM", k, lane))
        if sub:
            for sb in range(KC // sub):
                m.access(tid, "R", 32, "sCs", ((sb + 1) * sub - 1) * 4, 4, tag=("sCs", (sb + 1) * sub - 1))
                for jt in range(sb * sub // 16, (sb + 1) * sub // 16):
                    for r in range(4):
                        t = 16 * jt + 4 * grp + r
                        m.access(tid, "R", 32, "sCs", t * 4, 4, tag=("sCs", t))
                        m.access(tid, "R", 32, "sDt", t * 4, 4, tag=("sDt", t))
                read_bt(m, tid, NS, swz, 33)
        elif carry:
            m.access(tid, "R", 34, "sCs", (KC - 1) * 4, 4, tag=("sCs", KC - 1))
            for jt in range(4):
                for r in range(4):
                    t = 16 * jt + 4 * grp + r
                    m.access(tid, "R", 34, "sWs", t * 4, 4, tag=("sWs", t))
            read_bt(m, tid, NS, swz, 35)
    m.barrier()                                # LDS is rewritten by the next chunk
    return m


# ----------------------------------------------------------------- block kernel
def block_model(LT, NS, commit, npart, want_y=True):
    """bdlm_block_kernel, bf16 storage, both branches from one input set (the step and the
    commit of the headline workload)."""
    QN, MT = NS // 16, LT // 16
    NT, NW = 256 * npart, 4 * npart
    QW = QN // npart
    IMG = MT * QN * 64
    XS = P + 4
    E = 8
    arrays = {"sC": IMG * 8, "sB": IMG * 8, "sX": LT * XS * 2, "sDt": 64 * 4, "sCs": 64 * 4,
              "sEx": 64 * 4, "sPar": 4 * 4, "sM": MT * MT * 64 * 16,
              "sRed": max(1, npart - 1) * 4 * MT * 64 * 16}
    m = new_model(arrays)
    CPR = NS // E
    BC_CH = LT * CPR
    X_CH = LT * (P // E)
    BC_PT = BC_CH // NT if BC_CH >= NT else 1
    X_PT = X_CH // NT if X_CH >= NT else 1
    # phase 1: images, x, parameters, decay sums
    for tid in range(NT):
        if tid < BC_CH:
            for k in range(BC_PT):
                i = tid + NT * k
                t, c = i // CPR, i % CPR
                at = img_idx(QN, False, t >> 4, c >> 1, 2 * (c & 1), t & 15)
                for arr in ("sC", "sB"):
                    # 8 bf16 of row t, columns 8c .. 8c + 7: two quads (groups 2(c&1), +1)
                    m.access(tid, "W", 1, arr, at * 8, 8, tag=(arr, t, 8 * c))
                    m.access(tid, "W", 1, arr, (at + 16) * 8, 8, tag=(arr, t, 8 * c + 4))
        if tid < X_CH:
            for k in range(X_PT):
                i = tid + NT * k
                j, c = i // (P // E), i % (P // E)
                for h in range(2):
                    for e in range(4):
                        m.access(tid, "W", 2, "sX", (j * XS + c * E + 4 * h + e) * 2, 2,
                                 tag=("sX", j, c * E + 4 * h + e))
        if tid < 3:
            m.access(tid, "W", 3, "sPar", tid * 4, 4, tag=("sPar", tid))
        if tid < 64:
            for a in ("sDt", "sCs", "sEx"):
                m.access(tid, "W", 4, a, tid * 4, 4, tag=(a, tid))
    m.barrier()
    # phase 2: decay-weighted Gram tiles
    for tid in range(NT):
        wave, lane = tid >> 6, tid & 63
        grp, col = lane >> 4, lane & 15
        for tile in range(wave, MT * MT, NW):
            mt, jt = tile // MT, tile % MT
            for q in range(0, QN, 2):
                for qq in sorted({q, q + 1 if q + 1 < QN else q}):
                    sb = img_idx(QN, False, jt, qq, grp, col)
                    sc = img_idx(QN, False, mt, qq, grp, col)
                    m.access(tid, "R", 10, "sB", sb * 8, 8, tag=("sB", 16 * jt + col, 16 * qq + 4 * grp))
                    m.access(tid, "R", 10, "sC", sc * 8, 8, tag=("sC", 16 * mt + col, 16 * qq + 4 * grp))
            t = 16 * mt + col
            m.access(tid, "R", 11, "sCs", t * 4, 4, tag=("sCs", t))
            m.access(tid, "R", 11, "sEx", t * 4, 4, tag=("sEx", t))
            for r in range(4):
                j = 16 * jt + 4 * grp + r
                for a in ("sCs", "sEx", "sDt"):
                    m.access(tid, "R", 11, a, j * 4, 4, tag=(a, j))
            m.access(tid, "W", 12, "sM", (tile * 64 + lane) * 16, 16, tag=("sM", tile, lane))
    m.barrier()
    # phase 3: x quads, intra product (first group), C quads, prefix partial products
    for tid in range(NT):
        wave, lane = tid >> 6, tid & 63
        pblk, part = wave & 3, wave >> 2
        grp, col = lane >> 4, lane & 15
        p = 16 * pblk + col
        q0 = part * QW
        for jt in range(MT):
            for r in range(4):
                j = 16 * jt + 4 * grp + r
                m.access(tid, "R", 20, "sX", (j * XS + p) * 2, 2, tag=("sX", j, p))
        if want_y:
            if part == 0:
                m.access(tid, "R", 21, "sPar", 4, 4, tag=("sPar", 1))
                m.access(tid, "R", 21, "sPar", 8, 4, tag=("sPar", 2))
                for mt in range(MT):
                    for jt in range(MT):
                        m.access(tid, "R", 22, "sM", ((mt * MT + jt) * 64 + lane) * 16, 16,
                                 tag=("sM", mt * MT + jt, lane))
                    for r in range(4):
                        t = 16 * mt + 4 * grp + r
                        m.access(tid, "R", 23, "sCs", t * 4, 4, tag=("sCs", t))
            for mt in range(MT):
                for k in range(QW):
                    sc = img_idx(QN, False, mt, q0 + k, grp, col)
                    m.access(tid, "R", 24, "sC", sc * 8, 8,
                             tag=("sC", 16 * mt + col, 16 * (q0 + k) + 4 * grp))
            if npart > 1 and part > 0:
                for mt in range(MT):
                    m.access(tid, "W", 25, "sRed", ((((part - 1) * 4 + pblk) * MT + mt) * 64 + lane) * 16,
                             16, tag=("sRed", part, pblk, mt, lane))
    if want_y and npart > 1:
        m.barrier()
        for tid in range(NT):
            wave, lane = tid >> 6, tid & 63
            pblk, part = wave & 3, wave >> 2
            if part == 0:
                for pt in range(1, npart):
                    for mt in range(MT):
                        m.access(tid, "R", 30, "sRed",
                                 ((((pt - 1) * 4 + pblk) * MT + mt) * 64 + lane) * 16, 16,
                                 tag=("sRed", pt, pblk, mt, lane))
    if commit:
        for tid in range(NT):
            wave, lane = tid >> 6, tid & 63
            part = wave >> 2
            grp, col = lane >> 4, lane & 15
            q0 = part * QW
            m.access(tid, "R", 40, "sCs", 63 * 4, 4, tag=("sCs", 63))
            for jt in range(MT):
                for r in range(4):
                    j = 16 * jt + 4 * grp + r
                    m.access(tid, "R", 40, "sCs", j * 4, 4, tag=("sCs", j))
                    m.access(tid, "R", 40, "sDt", j * 4, 4, tag=("sDt", j))
            for k in range(QW):
                q = q0 + k
                for jt in range(MT):
                    for r in range(4):
                        # B[16jt + 4grp + r, 16q + col]: quad (jt, q, group col >> 2, column
                        # 4grp + r), element col & 3
                        slot = img_idx(QN, False, jt, q, col >> 2, 4 * grp + r)
                        e = slot * 4 + (col & 3)
                        row, n0 = 16 * jt + 4 * grp + r, 16 * q + 4 * (col >> 2)
                        m.access(tid, "R", 41, "sB", e * 2, 2, tag=("sB", row, n0))
    m.barrier()
    return m


# ------------------------------------------------------------- long-block kernel
def long_model(NS, NCH, commit, want_y=True):
    """bdlm_long_block_kernel (bdlm_long.hip): wave c owns chunk c and its LDS region, which
    holds the chunk's C row image, then its B row image, then the local states it publishes;
    one barrier, after which every wave reads the other chunks' published states."""
    QN, RS = NS // 16, NS + 8
    REG = 64 * RS * 2
    PR, RPI = NS // 8, 64 // (NS // 8)
    names = ["Cs", "Ex", "Dt", "Ec", "Er", "Wf", "Wr", "La", "Lb", "Ua", "Ub"]
    arrays = {"reg": NCH * REG, "tot": 4 * NCH}
    arrays.update({n: NCH * 64 * 4 for n in names})
    m = new_model(arrays)
    m.same_wave_rewrites = True

    class Lockstep:
        """A wave's lanes issue each instruction together: accesses are collected per lane
        and replayed instruction by instruction."""
        def __init__(self):
            self.ops = []

        def access(self, tid, kind, instr, array, off, nbytes, tag=None):
            self.ops.append((instr, len(self.ops), tid, kind, array, off, nbytes, tag))

        def flush(self):
            for instr, _, tid, kind, array, off, nbytes, tag in sorted(self.ops, key=lambda o: o[:2]):
                outer.access(tid, kind, instr, array, off, nbytes, tag)
            self.ops = []
    outer = m
    for c in range(NCH):
        m = Lockstep()
        need_f, need_r = commit or c + 1 < NCH, want_y and c > 0
        base = c * REG
        for l in range(64):
            t, col, grp = 64 * c + l, l % 16, l // 16
            ins = 0

            def nxt():
                nonlocal ins
                ins += 1
                return ins
            for n in names:                       # per-token factors (lane = token)
                m.access(t, "W", nxt(), n, (c * 64 + l) * 4, 4, tag=(n, c, l))
            if l == 0:
                m.access(t, "W", nxt(), "tot", 4 * c, 4, tag=("tot", c))
            else:
                nxt()

            def stage(what):
                rl, pc = l // PR, l % PR
                for i in range(PR):
                    row = RPI * i + rl
                    off = base + (row * RS + pc * 8) * 2
                    i0 = nxt()
                    for e in range(8):
                        m.access(t, "W", i0, "reg", off + 2 * e, 2, tag=(what, row, pc * 8 + e))

            def quad(what, row, n0):
                i0 = nxt()
                for e in range(4):
                    m.access(t, "R", i0, "reg", base + (row * RS + n0 + e) * 2, 2, tag=(what, row, n0 + e))
            if want_y:
                stage("C")
                for mt in range(4):
                    for q in range(QN):
                        quad("C", 16 * mt + col, 16 * q + 4 * grp)
            stage("B")
            if want_y:
                for mt in range(4):
                    for n in ("Cs", "Ex", "La", "Ua"):
                        m.access(t, "R", nxt(), n, (c * 64 + 16 * mt + col) * 4, 4, tag=(n, c, 16 * mt + col))
                for jt in (0, 2):
                    for d in range(2):
                        for q in range(QN):
                            quad("B", 16 * (jt + d) + col, 16 * q + 4 * grp)
                    for d in range(2):
                        jj = jt + d
                        for n in ("Lb", "Ub", "Cs", "Ex", "Dt"):
                            i0 = nxt()
                            for r in range(4):
                                j = 16 * jj + 4 * grp + r
                                m.access(t, "R", i0, n, (c * 64 + j) * 4, 4, tag=(n, c, j))
            for jt in range(4):
                for n in ("Wf", "Wr"):
                    i0 = nxt()
                    for r in range(4):
                        j = 16 * jt + 4 * grp + r
                        m.access(t, "R", i0, n, (c * 64 + j) * 4, 4, tag=(n, c, j))
            for q in range(QN):                   # B read transposed
                for jt in range(4):
                    for r in range(4):
                        j = 16 * jt + 4 * grp + r
                        m.access(t, "R", nxt(), "reg", base + (j * RS + 16 * q + col) * 2, 2,
                                 tag=("B", j, 16 * q + col))
            for q in range(QN):                   # publish
                if need_f:
                    m.access(t, "W", nxt(), "reg", base + ((4 * q + grp) * 16 + col) * 16, 16,
                             tag=("F", c, q, grp, col))
                if need_r:
                    m.access(t, "W", nxt(), "reg", base + (QN * 64 + (4 * q + grp) * 16 + col) * 16, 16,
                             tag=("R", c, q, grp, col))
        m.flush()
    m = outer
    m.barrier()
    for c in range(NCH):
        for l in range(64):
            t, col, grp = 64 * c + l, l % 16, l // 16
            ins = 1000

            def rd(k, q, which):
                nonlocal ins
                ins += 1
                off = k * REG + ((QN * 64 if which == "R" else 0) + (4 * q + grp) * 16 + col) * 16
                m.access(t, "R", ins, "reg", off, 16, tag=(which, k, q, grp, col))
            for k in range(c):
                ins += 1
                m.access(t, "R", ins, "tot", 4 * k, 4, tag=("tot", k))
                for q in range(QN):
                    rd(k, q, "F")
            if commit and c == NCH - 1:
                for q in range(QN):
                    rd(c, q, "F")
            if want_y:
                for n, lo, hi in (("Ec", 0, 0), ("Er", 0, 0)):
                    for mt in range(4):
                        ins += 1
                        for r in range(4):
                            j = 16 * mt + 4 * grp + r
                            m.access(t, "R", ins, n, (c * 64 + j) * 4, 4, tag=(n, c, j))
                for k in range(NCH - 1, c, -1):
                    ins += 1
                    m.access(t, "R", ins, "tot", 4 * k, 4, tag=("tot", k))
                    for q in range(QN):
                        rd(k, q, "R")
    m.barrier()
    return m


# ---------------------------------------------------------------------- tests
@pytest.mark.parametrize("NS", [16, 32, 64, 128])
@pytest.mark.parametrize("both", [False, True])
@pytest.mark.parametrize("swz", [False, True])
def test_seg_state_lds(NS, both, swz):
    assert seg_state_model(NS, both, swz).check() == []


@pytest.mark.parametrize("NS", [16, 32, 64, 128])
@pytest.mark.parametrize("sub", [0, 16, 32])
@pytest.mark.parametrize("swz", [False, True])
def test_seg_out_lds(NS, sub, swz):
    assert seg_out_model(NS, sub, swz).check() == []


@pytest.mark.parametrize("NS", [16, 128])
def test_seg_out_lds_without_outputs(NS):
    assert seg_out_model(NS, 0, False, want_y=False).check() == []


@pytest.mark.parametrize("LT,NS", [(16, 16), (16, 128), (32, 64), (32, 128), (64, 32), (64, 128)])
@pytest.mark.parametrize("commit", [False, True])
def test_block_kernel_lds(LT, NS, commit):
    npart = 2 if (NS // 16) % 2 == 0 else 1
    assert block_model(LT, NS, commit, npart).check() == []
    if commit:
        assert block_model(LT, NS, True, npart, want_y=False).check() == []


@pytest.mark.parametrize("NS", [16, 32, 64, 128])
@pytest.mark.parametrize("NCH", [2, 3, 4])
@pytest.mark.parametrize("commit", [False, True])
def test_long_block_kernel_lds(NS, NCH, commit):
    assert long_model(NS, NCH, commit).check() == []
    if commit:
        assert long_model(NS, NCH, True, want_y=False).check() == []


def test_long_block_model_catches_a_cross_wave_rewrite():
    """Rewrites are allowed within a wave only: the same byte written by two waves in one
    interval, or by two lanes of one instruction, is still flagged."""
    w = new_model({"a": 256})
    w.same_wave_rewrites = True
    w.access(0, "W", 1, "a", 0, 4)
    w.access(1, "W", 2, "a", 0, 4)      # another lane of wave 0, a later instruction: fine
    assert w.check() == []
    w.access(64, "W", 3, "a", 0, 4)     # wave 1
    assert any(p[0] == "two writers in one interval" for p in w.check())
    v = new_model({"a": 256})
    v.same_wave_rewrites = True
    v.access(0, "W", 1, "a", 0, 4)
    v.access(1, "W", 1, "a", 0, 4)      # two lanes, one instruction
    assert any(p[0] == "two writers in one interval" for p in v.check())
    # the long-block kernel without its barrier: waves read states other waves publish
    m = long_model(32, 3, False)
    merged = new_model(m.arrays)
    merged.same_wave_rewrites = True
    for (iv, arr, b), lst in m.acc.items():
        merged.acc[(0, arr, b)].extend(lst)
    assert any(p[0] == "cross-wave access to a written byte" for p in merged.check())


def test_the_model_catches_planted_hazards():
    """The checks are live: a model with a missing barrier, a colliding write, an index
    past the end, a stale read or a mismatched slot is flagged."""
    m = seg_out_model(32, 0, False)
    assert m.check() == []
    # no barrier between the Gram tiles and their use: merge intervals 2 and 3
    merged = new_model(m.arrays)
    for (iv, arr, b), lst in m.acc.items():
        merged.acc[(2 if iv == 3 else iv, arr, b)].extend(lst)
    assert any(p[0] == "cross-wave access to a written byte" for p in merged.check())
    # two threads writing one byte
    w = new_model({"a": 8})
    w.barrier()
    w.access(0, "W", 1, "a", 0, 4)
    w.access(70, "W", 1, "a", 2, 4)
    assert any(p[0] == "two writers in one interval" for p in w.check())
    # index past the end
    o = new_model({"a": 8})
    o.access(0, "R", 1, "a", 6, 4)
    assert o.check()[0][0] == "out of range"
    # read of a byte never written
    r = new_model({"a": 8})
    r.barrier()
    r.access(3, "R", 1, "a", 0, 4)
    assert r.check()[0][0] == "read of a byte not written in this chunk"
    # an element read from a slot written with another element
    x = new_model({"a": 8})
    x.access(0, "W", 1, "a", 0, 4, tag="u")
    x.barrier()
    x.access(1, "R", 2, "a", 0, 4, tag="v")
    assert any(p[0] == "element read from another element's slot" for p in x.check())
