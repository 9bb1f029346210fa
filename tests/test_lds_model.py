"""Host-side model of the LDS traffic of the scan kernels, barrier interval by barrier
interval, per wave and per lane (no GPU).

Each kernel's LDS accesses are written out here from its source: for every thread, the
array, the byte range and the direction of every LDS read and write between two
workgroup barriers (the kernels' __syncthreads calls), for one 64-token chunk (sequence
kernels) or one block (block kernel, masked long-block kernel), at every dstate the
kernels are built for.  The
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
* the sequence kernels' row images of B and x, read back with the LDS transpose read:
  each (token, column quad) is read from the slot it was written to; separately, each
  lane's transpose-read address composed with the instruction's lane permutation (as
  measured on gfx950) gives exactly the MFMA operand element the kernels consume, and
  the staging writes, operand reads and transpose reads of the row images touch 16
  distinct 8-byte bank pairs per 16 lanes at dstate 64 and 128.
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


def row_slot(QN, t, Q):
    """Slot of quad (local token t, dstate quad Q) in a bf16 row image of B or C of the
    sequence kernels (bdlm_seq.hip, row_slot)."""
    q, a = Q >> 2, Q & 3
    return ((t >> 4) * QN + q) * 64 + a * 16 + ((t & 15) ^ (4 * a) ^ (q & 7))


def x_slot(t, PQ):
    """Slot of quad (local token t, column quad PQ) in the bf16 row image of x."""
    w, a = PQ >> 2, PQ & 3
    return ((t >> 4) * 4 + w) * 64 + a * 16 + ((t & 15) ^ (4 * a) ^ ((w & 1) | ((w & 2) << 1)))


def tr_tok(lane):
    """Token (within a 16-token tile) of the quad a lane reads for a transposed operand."""
    return 4 * (lane >> 4) + ((lane & 15) >> 2)


def tr_quad(lane):
    """Column quad (within a 16-column tile) of the quad a lane reads."""
    return lane & 3


def tr_source(lane, r):
    """LDS transpose read (ds_read_b64_tr_b16), as measured on gfx950: slot r of lane
    16g + 4a + b holds element b of the 8 bytes read by lane 16g + a + 4r.  Returns
    (source lane, element)."""
    g, a, b = lane >> 4, (lane & 15) >> 2, lane & 3
    return 16 * g + a + 4 * r, b


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
def stage_chunk(m, NS, with_c, instr0=0, with_wr=False):
    """Stager::stage (bf16 storage): row images of B (and C when loaded) and of x from
    the registers of one chunk; plus wave 0's decay sums."""
    BCPR = NS // 8
    BT = 16 * BCPR
    XCPR = P // 8
    XT = (KC // 2) * XCPR
    QN = NS // 16
    for tid in range(THREADS):
        for k in range(max(1, BT // THREADS)):
            task = tid + THREADS * k
            if task >= BT:
                continue
            g, pc = task // BCPR, task % BCPR
            for arr in ("sB", "sC") if with_c else ("sB",):
                for r in range(4):
                    j = 4 * g + r
                    for qq in (2 * pc, 2 * pc + 1):
                        m.access(tid, "W", instr0 + 1, arr, row_slot(QN, j, qq) * 8, 8,
                                 tag=(arr, j, 4 * qq))
        for k in range(max(1, XT // THREADS)):
            task = tid + THREADS * k
            if task >= XT:
                continue
            g, pc = task // XCPR, task % XCPR
            for r in range(2):
                t = 2 * g + r
                for pq in (2 * pc, 2 * pc + 1):
                    m.access(tid, "W", instr0 + 3, "sX", x_slot(t, pq) * 8, 8, tag=("sX", t, 4 * pq))
    for lane in range(64):                    # wave 0: decay sums
        for arr in ("sDt", "sCs", "sEc", "sWs") + (("sWr",) if with_wr else ()):
            if arr in m.arrays:
                m.access(lane, "W", instr0 + 4, arr, lane * 4, 4, tag=(arr, lane))


def read_bt(m, tid, NS, instr):
    """bt_read over every dstate tile: each lane's transpose-read quad of the B row
    image (token 16jt + tr_tok, dstate quad 4q + tr_quad)."""
    lane = tid & 63
    QN = NS // 16
    for q in range(QN):
        for jt in range(4):
            t, Q = 16 * jt + tr_tok(lane), 4 * q + tr_quad(lane)
            m.access(tid, "R", instr, "sB", row_slot(QN, t, Q) * 8, 8, tag=("sB", t, 4 * Q))


def read_xt(m, tid, instr):
    """x operands of wave w's columns: each lane's transpose-read quad of the x row
    image (token 16jt + tr_tok, column quad 4w + tr_quad)."""
    lane, wave = tid & 63, tid >> 6
    for jt in range(4):
        t, pq = 16 * jt + tr_tok(lane), 4 * wave + tr_quad(lane)
        m.access(tid, "R", instr, "sX", x_slot(t, pq) * 8, 8, tag=("sX", t, 4 * pq))


def seg_state_model(NS, both):
    QN = NS // 16
    arrays = {"sB": 4 * QN * 64 * 8, "sX": 16 * P * 8}
    for a in ("sDt", "sCs", "sEc", "sWs", "sWr"):
        arrays[a] = KC * 4
    m = new_model(arrays)
    m.barrier()                                # kernel start / previous chunk's last barrier
    stage_chunk(m, NS, with_c=False, with_wr=both)
    m.barrier()
    for tid in range(THREADS):
        grp = (tid & 63) >> 4
        m.access(tid, "R", 10, "sCs", (KC - 1) * 4, 4, tag=("sCs", KC - 1))
        read_xt(m, tid, 11)
        for jt in range(4):
            for r in range(4):
                t = 16 * jt + 4 * grp + r
                m.access(tid, "R", 12, "sWs", t * 4, 4, tag=("sWs", t))
                if both:
                    m.access(tid, "R", 12, "sWr", t * 4, 4, tag=("sWr", t))
        read_bt(m, tid, NS, 13)
    m.barrier()                                # end of chunk
    return m


def seg_out_model(NS, sub, want_y=True, carry=True):
    QN = NS // 16
    IMG = 4 * QN * 64
    arrays = {"sB": IMG * 8, "sC": IMG * 8, "sX": 16 * P * 8, "sM": 10 * 64 * 16}
    for a in ("sDt", "sCs", "sEc", "sWs"):
        arrays[a] = KC * 4
    m = new_model(arrays)
    m.barrier()
    stage_chunk(m, NS, with_c=True)
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
                    # lane (grp, col) reads quad 4q + grp of rows 16 tile + col
                    tb, tc, Q = 16 * jt + col, 16 * mt + col, 4 * q + grp
                    m.access(tid, "R", 20, "sB", row_slot(QN, tb, Q) * 8, 8, tag=("sB", tb, 4 * Q))
                    m.access(tid, "R", 20, "sC", row_slot(QN, tc, Q) * 8, 8, tag=("sC", tc, 4 * Q))
                t = 16 * mt + col
                m.access(tid, "R", 21, "sCs", t * 4, 4, tag=("sCs", t))
                for r in range(4):
                    j = 16 * jt + 4 * grp + r
                    m.access(tid, "R", 21, "sCs", j * 4, 4, tag=("sCs", j))
                    m.access(tid, "R", 21, "sDt", j * 4, 4, tag=("sDt", j))
                m.access(tid, "W", 22, "sM", (k * 64 + lane) * 16, 16, tag=("sM", k, lane))
            for q in range(QN):
                for mt in range(4):
                    tc, Q = 16 * mt + col, 4 * q + grp
                    m.access(tid, "R", 23, "sC", row_slot(QN, tc, Q) * 8, 8, tag=("sC", tc, 4 * Q))
            for mt in range(4):
                for r in range(4):
                    t = 16 * mt + 4 * grp + r
                    m.access(tid, "R", 24, "sEc", t * 4, 4, tag=("sEc", t))
    m.barrier()                                # Gram tiles published
    for tid in range(THREADS):
        lane = tid & 63
        grp = lane >> 4
        read_xt(m, tid, 30)
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
                read_bt(m, tid, NS, 33)
        elif carry:
            m.access(tid, "R", 34, "sCs", (KC - 1) * 4, 4, tag=("sCs", KC - 1))
            for jt in range(4):
                for r in range(4):
                    t = 16 * jt + 4 * grp + r
                    m.access(tid, "R", 34, "sWs", t * 4, 4, tag=("sWs", t))
            read_bt(m, tid, NS, 35)
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


# ------------------------------------------------------------- masked long-block kernel
def pair_idx(QP, mt, qp, grp, col):
    """16-byte entry of the quad pair (2qp, 2qp + 1) of lane (col, grp) of token tile mt in
    the masked long-block kernel's B and C images (bdlm_mask.hip, pair_idx)."""
    return (mt * QP + qp) * 64 + grp * 16 + (col ^ ((2 * qp + (grp >> 1)) & 15))


def mask_model(NS, MT, commit, want_y=True):
    """bdlm_mask_block_kernel (bdlm_mask.hip): eight waves, wave w owning the output rows of
    token tiles TPW w ..; the B image, the region that holds the C image and then the
    transposed x and the split state images, and the per-token decay arrays.  Elements are
    tagged, so every operand read is checked against the element the staging wrote there."""
    QN = NS // 16
    QP = (QN + 1) // 2
    NW, NT = 8, 512
    TPW = MT // NW
    NTOK = 16 * MT
    TPL = NTOK // 64
    LPT = 16 // TPL
    IMG, XTQ, SQP = MT * QP * 64, MT * 4 * 64, QP * 4 * 64
    REGION = max(IMG * 16, XTQ * 8 + SQP * 32)
    names = ["Dt", "Cs", "Ex", "Ec", "La", "Lb", "Ua", "Ub"] + (["Wc"] if commit else [])
    arrays = {"sB": IMG * 16, "sU": REGION, "sE": 4 * MT}
    arrays.update({n: NTOK * 4 for n in names})
    m = new_model(arrays)
    CPR = NS // 8
    BCN = NTOK * CPR
    BCK = BCN // NT if BCN >= NT else 1
    XN = 4 * MT * 8
    XK = XN // NT if XN >= NT else 1
    SN = 16 * NS
    SK = SN // NT if SN >= NT else 1
    S_OFF = XTQ * 8                     # state hi image in the region; lo follows
    # ---- interval 0: B and C images, the decay arrays (wave 0)
    for tid in range(NT):
        if tid >= BCN:
            continue
        for k in range(BCK):
            i = tid + NT * k
            t, c = i // CPR, i % CPR
            q, gr = c >> 1, 2 * (c & 1)
            at = 2 * pair_idx(QP, t >> 4, q >> 1, gr, t & 15) + (q & 1)
            at1 = 2 * pair_idx(QP, t >> 4, q >> 1, gr + 1, t & 15) + (q & 1)
            for arr, ok in (("sB", True), ("sU", want_y)):
                if not ok:
                    continue
                name = arr if arr == "sB" else "C"
                m.access(tid, "W", 1, arr, at * 8, 8, tag=(name, t, 16 * q + 4 * gr))
                m.access(tid, "W", 2, arr, at1 * 8, 8, tag=(name, t, 16 * q + 4 * gr + 4))
                if QN % 2 == 1 and q == QN - 1:
                    m.access(tid, "W", 3, arr, (at + 1) * 8, 8, tag=("Z",))
                    m.access(tid, "W", 4, arr, (at1 + 1) * 8, 8, tag=("Z",))
    for lane in range(64):
        for i in range(TPL):
            t = TPL * lane + i
            for n in names:
                m.access(lane, "W", 10, n, 4 * t, 4)
        if (lane & (LPT - 1)) == LPT - 1:
            m.access(lane, "W", 11, "sE", 4 * ((TPL * lane) >> 4), 4)
    m.barrier()
    # ---- interval 1: every wave's C quad pairs (then a barrier before the region is reused)
    if want_y:
        for tid in range(NT):
            w, lane = tid // 64, tid % 64
            col, grp = lane & 15, lane >> 4
            for mm in range(TPW):
                mt = TPW * w + mm
                for qp in range(QP):
                    e = pair_idx(QP, mt, qp, grp, col)
                    hi = ("Z",) if 2 * qp + 1 >= QN else ("C", 16 * mt + col, 32 * qp + 16 + 4 * grp)
                    m.access(tid, "R", 20, "sU", e * 16, 8, tag=("C", 16 * mt + col, 32 * qp + 4 * grp))
                    m.access(tid, "R", 20, "sU", e * 16 + 8, 8, tag=hi)
        m.barrier()
    # ---- interval 2: transposed x, the state's hi / lo images
    for tid in range(NT):
        if tid < XN:
            for k in range(XK):
                task = tid + NT * k
                tq, pc = task >> 3, task & 7
                for d in range(4):
                    for h in range(2):
                        pcol = pc * 8 + 2 * d + h
                        m.access(tid, "W", 30 + h, "sU", (tq * 64 + pcol) * 8, 8, tag=("X", tq, pcol))
        if want_y and tid < SN:
            for k in range(SK):
                i = tid + NT * k
                q, gp = i >> 8, i & 255
                at = 2 * ((q >> 1) * 256 + gp) + (q & 1)
                for img, off in (("SH", S_OFF), ("SL", S_OFF + SQP * 16)):
                    m.access(tid, "W", 32, "sU", off + at * 8, 8, tag=(img, q, gp))
                    if QN % 2 == 1 and q == QN - 1:
                        m.access(tid, "W", 33, "sU", off + (at + 1) * 8, 8, tag=("Z",))
    m.barrier()
    # ---- interval 3: the masked product, the diagonal tiles, the prefix term and stores,
    # the commit (reads only)
    for tid in range(NT):
        w, lane = tid // 64, tid % 64
        col, grp = lane & 15, lane >> 4
        mt0 = TPW * w

        def rd(instr, arr, off, n, tag=None):
            m.access(tid, "R", instr, arr, off, n, tag=tag)

        def xt(instr, tq, pcol):
            rd(instr, "sU", (tq * 64 + pcol) * 8, 8, tag=("X", tq, pcol))

        def b_pair(instr, jt, qp):
            e = pair_idx(QP, jt, qp, grp, col)
            rd(instr, "sB", e * 16, 8, tag=("sB", 16 * jt + col, 32 * qp + 4 * grp))
            hi = ("Z",) if 2 * qp + 1 >= QN else ("sB", 16 * jt + col, 32 * qp + 16 + 4 * grp)
            rd(instr, "sB", e * 16 + 8, 8, tag=hi)
        if want_y:
            for mm in range(TPW):
                t = 16 * (mt0 + mm) + col
                rd(40, "La", 4 * t, 4)
                rd(41, "Ua", 4 * t, 4)
            mm, jt = lane // MT, lane % MT
            mt = mt0 + (mm if mm < TPW else 0)
            for e in (mt - 1 if mt > 0 else 0, jt, jt - 1 if jt > 0 else 0, mt):
                rd(42, "sE", 4 * e, 4)
            for j0 in range(0, MT, 2):
                for d in range(2):
                    for qp in range(QP):
                        b_pair(43, j0 + d, qp)
                for mm in range(TPW):
                    mt = mt0 + mm
                    for d in range(2):
                        jt = j0 + d
                        rd(44, "Lb" if jt < mt else "Ub", 4 * (16 * jt + 4 * grp), 16)
                for pt in range(4):
                    xt(45, 4 * j0 + grp, 16 * pt + col)
                    xt(46, 4 * (j0 + 1) + grp, 16 * pt + col)
            for mm in range(TPW):
                mt = mt0 + mm
                for qp in range(QP):
                    b_pair(47, mt, qp)
                rd(48, "Cs", 4 * (16 * mt + col), 4)
                rd(48, "Ex", 4 * (16 * mt + col), 4)
                for n in ("Cs", "Ex", "Dt"):
                    rd(49, n, 4 * (16 * mt + 4 * grp), 16)
                for pt in range(4):
                    xt(50, 4 * mt + grp, 16 * pt + col)
                rd(51, "Ec", 4 * (16 * mt + 4 * grp), 16)
            for pt in range(4):
                for qp in range(QP):
                    e = (qp * 4 + grp) * 64 + 16 * pt + col
                    gp = grp * 64 + 16 * pt + col
                    for img, off in (("SH", S_OFF), ("SL", S_OFF + SQP * 16)):
                        hi = ("Z",) if 2 * qp + 1 >= QN else (img, 2 * qp + 1, gp)
                        rd(52, "sU", off + e * 16, 8, tag=(img, 2 * qp, gp))
                        rd(52, "sU", off + e * 16 + 8, 8, tag=hi)
                for mm in range(TPW):
                    xt(53, 4 * (mt0 + mm) + grp, 16 * pt + col)
        if commit:
            rd(60, "sE", 4 * (MT - 1), 4)
            pt = w & 3
            for jt in range(MT):
                rd(61, "Wc", 4 * (16 * jt + 4 * grp), 16)
                xt(62, 4 * jt + grp, 16 * pt + col)
            for i in range((4 * QN + NW - 1) // NW):
                kk = w + NW * i
                if kk >= 4 * QN:
                    break
                q = kk >> 2
                tt, ta = tr_tok(lane), tr_quad(lane)
                for jt in range(MT):
                    # one transpose read: the quad (token 16 jt + tt, dstate 16 q + 4 ta ..)
                    e = 2 * pair_idx(QP, jt, q >> 1, ta, tt) + (q & 1)
                    rd(63, "sB", e * 8, 8, tag=("sB", 16 * jt + tt, 16 * q + 4 * ta))
    m.barrier()
    return m

@pytest.mark.parametrize("NS", [16, 32, 64, 128])
@pytest.mark.parametrize("both", [False, True])
def test_seg_state_lds(NS, both):
    assert seg_state_model(NS, both).check() == []


@pytest.mark.parametrize("NS", [16, 32, 64, 128])
@pytest.mark.parametrize("sub", [0, 16, 32])
def test_seg_out_lds(NS, sub):
    assert seg_out_model(NS, sub).check() == []


@pytest.mark.parametrize("NS", [16, 128])
def test_seg_out_lds_without_outputs(NS):
    assert seg_out_model(NS, 0, want_y=False).check() == []


@pytest.mark.parametrize("NS", [16, 32, 64, 128])
def test_transpose_read_operands(NS):
    """Each lane's transpose-read address, composed with the instruction's lane
    permutation, yields the operands the MFMAs contract over tokens: lane (grp, col)
    slot r holds B[16jt + 4grp + r][16q + col] (state update) and x[16jt + 4grp + r]
    [16w + col] (intra term, skip term and state update of wave w)."""
    QN = NS // 16
    # what each row-image slot holds: (token, first column of its quad)
    b_at = {row_slot(QN, t, Q): (t, 4 * Q) for t in range(KC) for Q in range(NS // 4)}
    x_at = {x_slot(t, PQ): (t, 4 * PQ) for t in range(KC) for PQ in range(P // 4)}
    assert len(b_at) == KC * NS // 4 and len(x_at) == KC * P // 4
    for jt in range(4):
        for lane in range(64):
            grp, col = lane >> 4, lane & 15
            for r in range(4):
                src, e = tr_source(lane, r)
                for q in range(QN):
                    t, n0 = b_at[row_slot(QN, 16 * jt + tr_tok(src), 4 * q + tr_quad(src))]
                    assert (t, n0 + e) == (16 * jt + 4 * grp + r, 16 * q + col)
                for w in range(4):
                    t, p0 = x_at[x_slot(16 * jt + tr_tok(src), 4 * w + tr_quad(src))]
                    assert (t, p0 + e) == (16 * jt + 4 * grp + r, 16 * w + col)


def _bank_pairs_distinct(slots16):
    """8-byte accesses are served 16 lanes at a time over 32 four-byte banks: conflict
    free when the 16 slots fall on 16 distinct bank pairs."""
    return len({s % 16 for s in slots16}) == len(slots16)


@pytest.mark.parametrize("NS", [64, 128])
def test_row_images_are_bank_conflict_free(NS):
    QN, BCPR = NS // 16, NS // 8
    for r in range(4):                        # staging writes: one row r, one quad half
        for h in range(2):
            for base in range(0, THREADS, 16):
                sl = [row_slot(QN, 4 * (tid // BCPR) + r, 2 * (tid % BCPR) + h)
                      for tid in range(base, base + 16)]
                assert _bank_pairs_distinct(sl)
    for t0 in range(0, KC, 16):
        for q in range(QN):
            for grp in range(4):              # operand reads over dstate
                assert _bank_pairs_distinct([row_slot(QN, t0 + col, 4 * q + grp) for col in range(16)])
                # transpose reads: lanes 16grp .. 16grp + 15
                assert _bank_pairs_distinct([row_slot(QN, t0 + tr_tok(16 * grp + s), 4 * q + tr_quad(s))
                                             for s in range(16)])
    for r in range(2):                        # x staging writes and transpose reads
        for h in range(2):
            for base in range(0, THREADS, 16):
                assert _bank_pairs_distinct([x_slot(2 * (tid // 8) + r, 2 * (tid % 8) + h)
                                             for tid in range(base, base + 16)])
    for t0 in range(0, KC, 16):
        for w in range(4):
            for grp in range(4):
                assert _bank_pairs_distinct([x_slot(t0 + tr_tok(16 * grp + s), 4 * w + tr_quad(s))
                                             for s in range(16)])


@pytest.mark.parametrize("LT,NS", [(16, 16), (16, 128), (32, 64), (32, 128), (64, 32), (64, 128)])
@pytest.mark.parametrize("commit", [False, True])
def test_block_kernel_lds(LT, NS, commit):
    npart = 2 if (NS // 16) % 2 == 0 else 1
    assert block_model(LT, NS, commit, npart).check() == []
    if commit:
        assert block_model(LT, NS, True, npart, want_y=False).check() == []


@pytest.mark.parametrize("NS", [16, 32, 64, 128])
@pytest.mark.parametrize("MT", [8, 16])
@pytest.mark.parametrize("commit", [False, True])
def test_mask_block_kernel_lds(NS, MT, commit):
    assert mask_model(NS, MT, commit).check() == []
    if commit:
        assert mask_model(NS, MT, True, want_y=False).check() == []


@pytest.mark.parametrize("NS", [16, 32, 64, 128])
def test_mask_commit_transpose_read_operand(NS):
    """The masked long-block kernel's commit reads B transposed from its pair image: lane
    (grp, col) must receive B[16jt + 4grp + r][16q + col] in slot r.  Each lane's read
    (token 16jt + tr_tok, dstate quad piece tr_quad of quad q), composed with the
    instruction's lane permutation, gives exactly that element."""
    QN = NS // 16
    for q in range(QN):
        for jt in range(2):
            for lane in range(64):
                grp, col = lane >> 4, lane & 15
                for r in range(4):
                    src, e = tr_source(lane, r)
                    token, n = 16 * jt + tr_tok(src), 16 * q + 4 * tr_quad(src) + e
                    assert (token, n) == (16 * jt + 4 * grp + r, 16 * q + col)


def test_the_model_catches_cross_wave_rewrites():
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
    # the masked long-block kernel without its barriers: waves read images other waves write
    m = mask_model(32, 8, False)
    merged = new_model(m.arrays)
    for (iv, arr, b), lst in m.acc.items():
        merged.acc[(0, arr, b)].extend(lst)
    assert any(p[0] == "cross-wave access to a written byte" for p in merged.check())


def test_the_model_catches_planted_hazards():
    """The checks are live: a model with a missing barrier, a colliding write, an index
    past the end, a stale read or a mismatched slot is flagged."""
    m = seg_out_model(32, 0)
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
