"""CPU model of the attention kernel's addressing and load/wait schedule.

Test infrastructure.  It restates, in plain Python, the index arithmetic of
attn_fwd in paper_2505_22918_amd/csrc/attn.hip (per-lane DMA and LDS offsets,
the work-item order, the kept-chunk walk with its 64-entry offset table and
the caching walk's complement generator, the residual rows carried by the K
ring) and the program order of its vector-memory issues, waits and LDS reads.
Two families of checks run on it:

* addresses: for every work item, every global access falls inside its buffer
  resource's record range or wholly past it (the hardware returns zeros there),
  every plain store and statistic lands inside its tensor, and every LDS access
  lies inside the workgroup's allocation;
* schedule: replaying the issues and waits in program order with the in-order
  completion rule of the vector-memory counter, every LDS read of a stage finds
  the chunk (or residual tile) it expects, already landed and not yet
  overwritten.

It has no GPU dependency and shares nothing with the HIP sources beyond the
formulas it restates.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

K_OOB = 0x40000000  # buffer offset past every record: reads zero


@dataclass(frozen=True)
class Geometry:
    D: int
    BS: int

    @property
    def DK(self):  # Q K^T contraction width
        return 64 if self.D == 64 else 80

    @property
    def DV(self):  # rows of O^T
        return 64 if self.D == 64 else 96

    @property
    def SLOTS(self):  # 16-byte slots per token row
        return 8 if self.D == 64 else 9

    @property
    def SWZ(self):
        return self.D == 64

    @property
    def QT(self):
        return self.BS // 32

    @property
    def DS(self):
        return self.DK // 16

    @property
    def DT(self):
        return self.DV // 32

    @property
    def DC(self):
        return self.D // 8

    @property
    def ROWB(self):
        return self.SLOTS * 16

    @property
    def TILE(self):
        return 32 * self.ROWB

    @property
    def NSLOT(self):
        return 32 * self.SLOTS

    @property
    def NDMA(self):
        return (self.NSLOT + 63) // 64

    @property
    def SMEM(self):
        return 5 * self.TILE + (0 if self.D == 64 else 256)

    def kswz(self, r):
        return (r & 7) if self.SWZ else 0 * r

    def vswz(self, r):
        return (((r & 2) << 1) | (r & 1)) if self.SWZ else 0 * r


def lane_constants(g: Geometry):
    """Per-lane constants of the kernel, as arrays over the 64 lanes."""
    lane = np.arange(64)
    l32, hi = lane & 31, lane >> 5
    kdma = np.zeros((g.NDMA, 64), np.int64)
    vdma = np.zeros((g.NDMA, 64), np.int64)
    active = np.zeros((g.NDMA, 64), bool)
    for n in range(g.NDMA):
        slot = n * 64 + lane
        r, s = slot // g.SLOTS, slot % g.SLOTS
        kdma[n] = r * (2 * g.D) + (s ^ g.kswz(r)) * 16
        vdma[n] = r * (2 * g.D) + (s ^ g.vswz(r)) * 16
        active[n] = (g.NSLOT % 64 == 0) | (slot < g.NSLOT)
    k_rd = np.zeros((g.DS, 64), np.int64)
    for s in range(g.DS):
        ch = np.minimum(2 * s + hi, g.DC - 1)
        k_rd[s] = l32 * g.ROWB + (ch ^ g.kswz(l32)) * 16
    G4, L = lane >> 4, lane & 15
    r = 4 * hi + (L >> 2)
    v_rd = np.zeros((g.DT, 64), np.int64)
    for dt in range(g.DT):
        d = 32 * dt + 16 * (L & 1) + 8 * (G4 & 1) + 4 * ((L >> 1) & 1)
        v_rd[dt] = r * g.ROWB + ((d >> 3) ^ g.vswz(r)) * 16 + (d & 7) * 2
    return dict(lane=lane, l32=l32, hi=hi, kdma=kdma, vdma=vdma, dma_active=active, k_rd=k_rd, v_rd=v_rd)


@dataclass
class Launch:
    """One attention launch: shape, block, mode and the CSR (host copies)."""

    B: int
    H: int
    T: int
    D: int
    BS: int
    reshape: bool = False
    cache: bool = False
    dense: bool = False
    row_ptr: np.ndarray | None = None  # [n_masks][n_blk + 1]
    col_idx: np.ndarray | None = None
    n_masks: int = 1
    errors: list = field(default_factory=list)

    @property
    def n_blk(self):
        return -(-self.T // self.BS)

    @property
    def n_items(self):
        return self.B * self.H * self.n_blk

    @property
    def per_xcd(self):
        return -(-self.n_items // 8)

    @property
    def nnz(self):
        return 0 if self.col_idx is None else int(self.col_idx.size)


def item_order(L: Launch):
    """Work item of each hardware workgroup g (None for the ones that exit)."""
    g = np.arange(8 * L.per_xcd)
    item = (g & 7) * L.per_xcd + (g >> 3)
    return np.where(item < L.n_items, item, -1)


def kept_range(L: Launch, bh: int, qb: int):
    """[e_beg, e_end) of the query block's CSR row, clamped as the kernel does."""
    if L.dense:
        return 0, L.n_blk
    mid = 0 if L.n_masks <= 1 else (bh % L.H if L.n_masks == L.H else bh)
    rp = L.row_ptr.reshape(-1)[mid * (L.n_blk + 1):(mid + 1) * (L.n_blk + 1)]
    e_beg, e_end = int(rp[qb]), int(rp[qb + 1])
    e_beg = min(max(e_beg, 0), L.nnz)
    e_end = min(max(e_end, e_beg), L.nnz)
    return e_beg, e_end


def chunk_offsets(L: Launch, g: Geometry, e_beg: int, e_end: int):
    """Byte offset (or K_OOB) of every chunk the walk visits, in walk order, and
    the number of kept chunks n_in."""
    hpb = g.BS // 32
    n_in = (e_end - e_beg) * hpb
    if L.cache:
        kept = [int(c) for c in L.col_idx[e_beg:e_end]] if not L.dense else []
        kb_list = []
        for j in range(e_end - e_beg):
            kb_list += [kept[j]] * hpb
        halves = [i % hpb for i in range(n_in)]
        # complement walk: the blocks not in the (ascending) kept list
        gen_kb, gen_e = -1, 0
        for i in range(L.n_blk * hpb - n_in):
            half = i % hpb
            if half == 0:
                c = gen_kb + 1
                while gen_e < len(kept):
                    kk = kept[gen_e]
                    if kk < c:
                        gen_e += 1
                    elif kk == c:
                        c += 1
                        gen_e += 1
                    else:
                        break
                gen_kb = c
            kb_list.append(gen_kb)
            halves.append(half)
        n_chunk = L.n_blk * hpb
    else:
        n_chunk = n_in
        if L.dense:
            kb_list = [i // hpb for i in range(n_chunk)]
        else:
            kb_list = [int(L.col_idx[e_beg + i // hpb]) for i in range(n_chunk)]
        halves = [i % hpb for i in range(n_chunk)]
    kb = np.array(kb_list, np.int64).reshape(-1)
    half = np.array(halves, np.int64).reshape(-1)
    base = kb * g.BS + 32 * half
    ok = (kb >= 0) & (kb < L.n_blk) & (base < L.T)
    off = np.where(ok, base * 2 * g.D, K_OOB)
    return off, n_in, n_chunk


def _check(L: Launch, cond, what):
    if not np.all(cond):
        L.errors.append(what)


def check_buffer_access(L, offs, record, what):
    """16-byte buffer accesses: inside [0, record) or wholly at or past it, and
    below 2^31 (the offset register is 32-bit)."""
    offs = np.asarray(offs, np.int64)
    inside = (offs >= 0) & (offs + 16 <= record)
    past = offs >= record
    _check(L, inside | past, f"{what}: access straddles the record end {record}")
    _check(L, offs < 2 ** 31, f"{what}: offset overflows 32 bits")


def check_addresses(L: Launch, items=None, guard_rows=True, smem=None):
    """Address checks of every (or the given) work item of a launch.  The knobs
    exist for tests that plant a mistake: guard_rows=False drops the row < T
    guard of the stores, smem overrides the LDS allocation."""
    g = Geometry(L.D, L.BS)
    SMEM = g.SMEM if smem is None else smem
    c = lane_constants(g)
    order = item_order(L)
    hit = np.bincount(order[order >= 0], minlength=L.n_items)
    _check(L, hit == 1, "every work item runs exactly once")
    record = L.T * L.D * 2
    _check(L, record <= 2 ** 30, "one head fits a buffer resource")
    lds_dst = []
    for n in range(g.NDMA):
        lds_dst.append(n * 1024 + 16 * c["lane"][c["dma_active"][n]])
    lds_dst = np.concatenate(lds_dst)
    for stage in range(5):
        _check(L, stage * g.TILE + lds_dst + 16 <= SMEM, "DMA destination inside LDS")
    for st in range(3):
        _check(L, st * g.TILE + c["k_rd"] + 16 <= SMEM, "K operand read inside LDS")
    for st in (3, 4):
        for ks in range(2):
            for second in (0, 8):
                a = st * g.TILE + c["v_rd"] + (16 * ks + second) * g.ROWB
                _check(L, (a >= 0) & (a + 8 <= SMEM), "V^T transpose read inside LDS")
    tensor_elems = L.B * L.H * L.T * L.D
    ids = range(L.n_items) if items is None else items
    for item in ids:
        bh, qb = divmod(int(item), L.n_blk)
        row0 = qb * g.BS
        nrow = min(L.T - row0, g.BS)
        e_beg, e_end = kept_range(L, bh, qb)
        off, n_in, n_chunk = chunk_offsets(L, g, e_beg, e_end)
        real = off != K_OOB
        _check(L, (off[real] % (2 * g.D) == 0) & (off[real] < record), "chunk offset is a row inside the head")
        # K and V chunk DMAs (kOob chunks read zeros); every lane of every instruction
        for n in range(g.NDMA):
            act = c["dma_active"][n]
            for tab in (c["kdma"][n][act], c["vdma"][n][act]):
                check_buffer_access(L, off[:, None] + tab[None, :], record, "K/V chunk DMA")
        # residual rows through the K ring (fused reshape)
        if L.reshape:
            for j in range(g.QT):
                for n in range(g.NDMA):
                    act = c["dma_active"][n]
                    check_buffer_access(L, j * 32 * 2 * g.D + c["kdma"][n][act], nrow * 2 * g.D, "residual DMA")
        # Q (and the caching walk's O_s read-back): rows of the block
        for qt in range(g.QT):
            for s in range(g.DS):
                ch = 2 * s + c["hi"]
                q_off = np.where(ch < g.DC, (qt * 32 + c["l32"]) * 2 * g.D + ch * 16, K_OOB)
                check_buffer_access(L, q_off, nrow * 2 * g.D, "Q row load")
        # the rescale path re-reads the lane's K row of the current chunk
        for s in range(g.DS):
            ch = 2 * s + c["hi"]
            kr = np.where(real[:, None] & (ch < g.DC)[None, :], off[:, None] + c["l32"][None, :] * 2 * g.D + ch * 16,
                          K_OOB)
            check_buffer_access(L, kr, record, "rescale K row reload")
        # plain stores: O (and R in the caching walk) rows below T, statistics
        for qt in range(g.QT):
            row = row0 + qt * 32 + c["l32"]
            for dt in range(g.DT):
                for u in range(2):
                    ch = 4 * dt + 2 * c["hi"] + u
                    m = (ch < g.DC) & ((row < L.T) if guard_rows else True)
                    e = bh * L.T * L.D + row[m] * L.D + 8 * ch[m]
                    _check(L, (e >= 0) & (e + 8 <= tensor_elems), "O / R store inside the tensor")
            si = bh * L.T + row[(c["hi"] == 0) & ((row < L.T) if guard_rows else True)]
            _check(L, si < L.B * L.H * L.T, "statistic store inside [B,H,T]")
        # the offset table: steps read lanes t + 3 - tb in [0, 64)
        if not L.cache and n_chunk > 1:
            tb, t = 3, 1
            while True:
                t_end = min(n_chunk - 1, tb + 61)
                _check(L, (t_end - 1) + 3 - tb <= 63 if t < t_end else True, "table lane in range")
                t = max(t, t_end)
                if t >= n_chunk - 1:
                    break
                tb = t + 3
    return L.errors


# ---- schedule -------------------------------------------------------------------


class Schedule:
    """Replays vector-memory issues, waits and LDS reads in program order."""

    def __init__(self, name):
        self.name = name
        self.issued = []  # tags, in issue order
        self.done = 0  # issued[:done] have landed
        self.stage = {}  # LDS stage -> (tag, index into issued)
        self.errors = []

    def issue(self, tag, stage=None, count=1):
        for _ in range(count):
            self.issued.append(tag)
        if stage is not None:
            self.stage[stage] = (tag, len(self.issued) - 1)

    def wait(self, n):  # s_waitcnt vmcnt(n): all but the last n issued have landed
        self.done = max(self.done, len(self.issued) - n)

    def read(self, stage, tag):
        got = self.stage.get(stage)
        if got is None:
            self.errors.append(f"{self.name}: read of {tag} from stage {stage} that no load filled")
            return
        if got[0] != tag:
            self.errors.append(f"{self.name}: read of {tag} from stage {stage} finds {got[0]}")
        if got[1] >= self.done:
            self.errors.append(f"{self.name}: read of {tag} from stage {stage} before its load landed")


def schedule(g: Geometry, n_chunk: int, n_in: int, reshape: bool, cache: bool, dense: bool,
             waits=(3, 2, 3), v_into_current=False):
    """The kernel's program order for one work item with n_chunk chunks.  The
    knobs exist for tests that plant a mistake: `waits` are the multiples of
    NDMA in the steady step, the first / last step and the prologue;
    v_into_current sends V(t+1) into V(t)'s stage.  Stores (the caching walk's
    O_s rows) and the full drains of long-row table refills and the rare
    rescale only make later waits stricter, so they are left out."""
    S = Schedule(f"D{g.D} BS{g.BS} n={n_chunk} reshape={reshape} cache={cache}")
    NDMA = g.NDMA
    kst = lambda st: ("K", st)
    vst = lambda st: ("V", st)

    def k_tag(c):
        rj = c - n_chunk
        if reshape and 0 <= rj < g.QT:
            return ("R", rj)
        return ("K", c) if c < n_chunk else ("zero",)

    def v_tag(c):
        return ("Vc", c) if c < n_chunk else ("zero",)

    if not dense:
        S.issue(("cols",))  # the lane's CSR entries
        S.wait(0)
    S.issue(("Q",), count=g.QT * g.DS)
    S.issue(k_tag(0), kst(0), NDMA)
    S.issue(v_tag(0), vst(0), NDMA)
    S.issue(k_tag(1), kst(1), NDMA)
    S.issue(k_tag(2), kst(2), NDMA)
    S.wait(waits[2] * NDMA)
    if n_chunk > 0:
        S.read(kst(0), ("K", 0))
    k3, vo = 0, 0  # stage of K(t) and V(t)

    def step(t, has_qk, has_pv):
        nonlocal k3, vo
        vp = vo ^ 1
        kn = (k3 + 1) % 3
        if has_qk:
            S.issue(k_tag(t + 3), kst(k3), NDMA)
        if has_qk and has_pv:
            S.wait(waits[0] * NDMA)
        elif has_qk or has_pv:
            S.wait(waits[1] * NDMA)
        if has_pv:
            S.read(vst(vp), ("Vc", t - 1))
        if has_qk:
            S.read(kst(kn), ("K", t + 1))
        if t + 1 < n_chunk:
            S.issue(v_tag(t + 1), vst(vo if v_into_current else vp), NDMA)
        k3, vo = kn, vp

    if n_chunk == 1:
        step(0, False, False)
    elif n_chunk > 1:
        step(0, True, False)
        tb, t = 3, 1
        while True:
            t_end = n_chunk - 1 if cache else min(n_chunk - 1, tb + 61)
            while t < t_end:
                step(t, True, True)
                t += 1
            if t >= n_chunk - 1:
                break
            tb = t + 3
        step(n_chunk - 1, False, True)
    S.wait(0)
    if n_chunk > 0:
        S.read(vst(vo ^ 1), ("Vc", n_chunk - 1))
    if reshape:
        for qt in range(g.QT):
            S.read(kst((n_chunk + qt) % 3), ("R", qt))
    return S.errors
