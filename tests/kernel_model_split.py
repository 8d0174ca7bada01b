"""CPU model of a two-wave shared-ring layout of the attention kernel.

Test infrastructure.  The library's attention kernel runs one wavefront per
64-row query block.  A layout with two waves per block was built once: each
wave owned 32 query rows, both shared three K and three V stages in LDS (24 KB
at D = 64, 64-row blocks), each wave loaded half of every 32-key chunk (key
rows 16w .. 16w+15, two 16-byte loads per lane into LDS offsets
stage + 2048w + 1024n + 16 lane), one workgroup barrier per step ordered the
waves, and the residual rows came into registers in the last step.  Its only
GPU run faulted and it was removed; this model restates its index arithmetic
and program order so that any kernel of that layout is checked on the CPU
before it runs:

* addresses: per wave, the row base and clamped row count, every Q, residual
  and K/V chunk buffer access against its record range (or wholly past it),
  every LDS DMA destination and operand read against the 24 KB allocation,
  the two waves' DMA halves disjoint and together covering the chunk, and the
  plain stores below T;
* barriers: both waves reach the same number of workgroup barriers, and none
  sits on a path only one wave takes;
* schedule: each wave's loads complete in issue order (the vector-memory
  counter), the waves order only through barriers, and every LDS read of a
  stage finds both halves of the chunk it expects landed, with no load into
  that stage from the other wave in the same barrier phase.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

import kernel_model as km

D, BS = 64, 64
ROWB = 2 * D  # 128 bytes per K / V row
TILE = 32 * ROWB  # 4 KB per 32-key chunk
SMEM = 6 * TILE  # three K stages, three V stages
HALF = TILE // 2  # one wave's share of a chunk
NDMA_W = 2  # 16-byte loads per lane and chunk, per wave
QT, DS, DT, DC = 1, D // 16, D // 32, D // 8


def k_off(st):
    return st * TILE


def v_off(st):
    return (3 + st) * TILE


def lane_constants():
    g = km.Geometry(D, BS)
    return km.lane_constants(g)


def dma_targets(w, dst, voff, lane):
    """(LDS byte, buffer offset) of wave w's two loads per lane: the
    instruction offset n*1024 moves source and destination together."""
    lds, src = [], []
    for n in range(NDMA_W):
        lds.append(dst + HALF * w + 1024 * n + 16 * lane)
        src.append(voff + HALF * w + 1024 * n)
    return np.concatenate(lds), np.concatenate(src)


def check_addresses(L: km.Launch, items=None, half=HALF, smem=SMEM):
    """Address checks of the two-wave layout over every (or the given) item.
    `half` and `smem` exist for tests that plant a mistake."""
    assert L.D == D and L.BS == BS
    c = lane_constants()
    lane, l32, hi = c["lane"], c["l32"], c["hi"]
    kdma0, vdma0 = c["kdma"][0], c["vdma"][0]
    record = L.T * D * 2
    order = km.item_order(L)
    hit = np.bincount(order[order >= 0], minlength=L.n_items)
    km._check(L, hit == 1, "every work item runs exactly once")
    # LDS: DMA destinations of both waves, per stage, inside the allocation and
    # disjoint; operand reads inside the stage's 4 KB
    for st in range(6):
        dst = st * TILE
        cover = []
        for w in (0, 1):
            lds = np.concatenate([dst + half * w + 1024 * n + 16 * lane for n in range(NDMA_W)])
            km._check(L, (lds >= 0) & (lds + 16 <= smem), "DMA destination inside LDS")
            cover.append(lds)
        both = np.concatenate(cover)
        km._check(L, np.unique(both).size == both.size, "the waves' DMA halves are disjoint")
        km._check(L, np.array_equal(np.sort(both), dst + 16 * np.arange(TILE // 16)),
                  "the two halves cover the chunk")
    for st in range(3):
        km._check(L, k_off(st) + c["k_rd"] + 16 <= k_off(st) + TILE, "K operand read inside its stage")
    for st in range(3):
        for ks in range(2):
            for second in (0, 8):
                a = v_off(st) + c["v_rd"] + (16 * ks + second) * ROWB
                km._check(L, (a >= v_off(st)) & (a + 8 <= v_off(st) + TILE), "V^T read inside its stage")
    # the two waves' source rows: wave w's loads cover key rows 16w .. 16w+15
    for w in (0, 1):
        _, src = dma_targets(w, 0, kdma0, lane)
        rows = src // ROWB
        km._check(L, (rows >= 16 * w) & (rows < 16 * w + 16), "wave loads its own 16 key rows")
    tensor_elems = L.B * L.H * L.T * D
    g = km.Geometry(D, BS)
    ids = range(L.n_items) if items is None else items
    for item in ids:
        bh, qb = divmod(int(item), L.n_blk)
        e_beg, e_end = km.kept_range(L, bh, qb)
        off, n_in, n_chunk = km.chunk_offsets(L, g, e_beg, e_end)
        real = off != km.K_OOB
        for w in (0, 1):
            row0 = qb * BS + 32 * w
            nrow = min(max(L.T - row0, 0), 32)  # the scalar clamp
            # chunk DMAs, K and V, both offset tables (every lane, every chunk)
            for tab in (kdma0, vdma0):
                _, src = dma_targets(w, 0, tab, lane)
                km.check_buffer_access(L, off[:, None] + src[None, :], record, "K/V chunk DMA (two waves)")
            # Q rows and residual rows of this wave (record = its rows below T)
            for s in range(DS):
                ch = 2 * s + hi
                q_off = np.where(ch < DC, l32 * 2 * D + ch * 16, km.K_OOB)
                km.check_buffer_access(L, q_off, nrow * 2 * D, "Q row load (two waves)")
            if L.reshape:
                for dt in range(DT):
                    for u in range(2):
                        ch = 4 * dt + 2 * hi + u
                        r_off = np.where(ch < DC, l32 * 2 * D + ch * 16, km.K_OOB)
                        km.check_buffer_access(L, r_off, nrow * 2 * D, "residual load (two waves)")
            # rescale path: the lane's K row of the current chunk
            for s in range(DS):
                ch = 2 * s + hi
                kr = np.where(real[:, None] & (ch < DC)[None, :],
                              off[:, None] + l32[None, :] * 2 * D + ch * 16, km.K_OOB)
                km.check_buffer_access(L, kr, record, "rescale K row reload (two waves)")
            # stores: rows below T of this wave
            row = row0 + l32
            for dt in range(DT):
                for u in range(2):
                    ch = 4 * dt + 2 * hi + u
                    m = (ch < DC) & (row < L.T)
                    e = bh * L.T * D + row[m] * D + 8 * ch[m]
                    km._check(L, (e >= 0) & (e + 8 <= tensor_elems), "O store inside the tensor (two waves)")
            si = bh * L.T + row[(hi == 0) & (row < L.T)]
            km._check(L, si < L.B * L.H * L.T, "statistic store inside [B,H,T]")
    return L.errors


# ---- program order and schedule --------------------------------------------------


@dataclass
class Ev:
    kind: str  # "issue", "wait", "barrier", "read"
    stage: tuple = None  # ("K"|"V", index)
    tag: tuple = None
    n: int = 0  # wait: vmcnt
    count: int = 1  # issue: loads


def program(n_chunk: int, reshape: bool, dense: bool, barrier_in_rescale=False, v_into=None):
    """The program order of one wave for one item.  The knobs exist for tests
    that plant a mistake: barrier_in_rescale puts a barrier on the wave-uniform
    rescale path (taken by one wave only); v_into(t) overrides the stage V(t+1)
    is loaded into."""
    ev = []

    def tagk(c):
        return ("K", c) if c < n_chunk else ("zero",)

    def tagv(c):
        return ("Vc", c) if c < n_chunk else ("zero",)

    if not dense:
        ev.append(Ev("issue", tag=("cols",)))
        ev.append(Ev("wait", n=0))
    ev.append(Ev("issue", tag=("Q",), count=QT * DS))
    ev.append(Ev("issue", ("K", 0), tagk(0), count=NDMA_W))
    ev.append(Ev("issue", ("K", 1), tagk(1), count=NDMA_W))
    ev.append(Ev("issue", ("V", 0), tagv(0), count=NDMA_W))
    ev.append(Ev("issue", ("K", 2), tagk(2), count=NDMA_W))
    ev.append(Ev("wait", n=3 * NDMA_W))
    ev.append(Ev("barrier"))
    if reshape and n_chunk == 0:
        ev.append(Ev("issue", tag=("R",), count=QT * DT * 2))
    if n_chunk > 0:
        ev.append(Ev("read", ("K", 0), ("K", 0)))
    k3, vo, vpv = 0, 0, 2  # stages of K(t), V(t), V(t-1)

    def step(t, has_qk, has_pv):
        nonlocal k3, vo, vpv
        vp = vpv
        vn = 3 - vo - vpv  # the third V stage: V(t-2)'s
        kn = (k3 + 1) % 3
        if has_qk or has_pv:
            ev.append(Ev("wait", n=2 * NDMA_W))
        ev.append(Ev("barrier"))
        if has_qk:
            ev.append(Ev("issue", ("K", k3), tagk(t + 3), count=NDMA_W))
            target = vn if v_into is None else v_into(t, vo, vp, vn)
            ev.append(Ev("issue", ("V", target), tagv(t + 1), count=NDMA_W))
        if not has_qk and reshape:
            ev.append(Ev("issue", tag=("R",), count=QT * DT * 2))
        if has_pv:
            ev.append(Ev("read", ("V", vp), ("Vc", t - 1)))
        if barrier_in_rescale and t == 1:
            ev.append(Ev("barrier", tag=("rescale",)))
        if has_qk:
            ev.append(Ev("read", ("K", kn), ("K", t + 1)))
        k3, vpv, vo = kn, vo, vn

    if n_chunk == 1:
        step(0, False, False)
    elif n_chunk > 1:
        step(0, True, False)
        for t in range(1, n_chunk - 1):
            step(t, True, True)
        step(n_chunk - 1, False, True)
    if n_chunk > 0:
        ev.append(Ev("wait", n=QT * DT * 2 if reshape else 0))
        ev.append(Ev("barrier"))
        ev.append(Ev("read", ("V", vpv), ("Vc", n_chunk - 1)))
    ev.append(Ev("wait", n=0))
    return ev


def check_schedule(n_chunk, reshape=False, dense=False, rescale_wave=None, **knobs):
    """Replays both waves' programs.  rescale_wave (0 or 1) is the wave that
    takes the rescale path when a planted barrier sits on it."""
    errors = []
    progs = []
    for w in (0, 1):
        kw = dict(knobs)
        if kw.get("barrier_in_rescale") and w != rescale_wave:
            kw["barrier_in_rescale"] = False
        progs.append(program(n_chunk, reshape, dense, **kw))
    # phases and per-wave issue indices
    info = []
    for w in (0, 1):
        phase, issued, done = 0, 0, 0
        dmas, reads, done_at_barrier = [], [], []
        for e in progs[w]:
            if e.kind == "issue":
                first = issued
                issued += e.count
                if e.stage is not None:
                    dmas.append(dict(stage=e.stage, tag=e.tag, phase=phase, last=issued - 1, seq=first))
            elif e.kind == "wait":
                done = max(done, issued - e.n)
            elif e.kind == "barrier":
                done_at_barrier.append(done)
                phase += 1
            elif e.kind == "read":
                reads.append(dict(stage=e.stage, tag=e.tag, phase=phase, done=done, seq=issued))
        info.append(dict(dmas=dmas, reads=reads, n_barriers=phase, done_at_barrier=done_at_barrier))
    if info[0]["n_barriers"] != info[1]["n_barriers"]:
        errors.append(f"barrier counts differ: {info[0]['n_barriers']} vs {info[1]['n_barriers']}")
        return errors
    for w in (0, 1):
        for r in info[w]["reads"]:
            for h in (0, 1):  # half h is loaded by wave h
                if h == w:
                    cand = [d for d in info[h]["dmas"] if d["stage"] == r["stage"] and d["seq"] < r["seq"]]
                    landed = lambda d: d["last"] < r["done"]
                else:
                    cand = [d for d in info[h]["dmas"] if d["stage"] == r["stage"] and d["phase"] < r["phase"]]
                    # wave h's own waits before the barrier that opens this phase
                    landed = lambda d: d["last"] < info[h]["done_at_barrier"][r["phase"] - 1]
                    racing = [d for d in info[h]["dmas"] if d["stage"] == r["stage"] and d["phase"] == r["phase"]]
                    if racing:
                        errors.append(f"wave {w} reads {r['stage']} while wave {h} loads {racing[0]['tag']} into it")
                if not cand:
                    errors.append(f"wave {w} reads {r['stage']} (expects {r['tag']}): half {h} never loaded")
                    continue
                last = max(cand, key=lambda d: d["seq"])
                if last["tag"] != r["tag"]:
                    errors.append(f"wave {w} reads {r['stage']} expecting {r['tag']}, half {h} holds {last['tag']}")
                elif not landed(last):
                    errors.append(f"wave {w} reads {r['stage']} before half {h} of {r['tag']} landed")
    return errors
