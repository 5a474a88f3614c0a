"""Host model of the first version of the fused trainer at the excluded shape
(groups PX = 1, workgroups per group PR = 4, rows R = 16, units U = 256).

That version (the persistent trainer as first committed, runtime-shaped,
one kernel per (unit tiles, row tiles) per wave) was chosen for a 64-row batch
of the 32-256-1 net; on the GPU its gradient sums went wrong from the second
SGD step on and one run faulted the GPU, and the shape was taken out of the
next version's shape table. The shape cannot be instantiated today (the owner
waves hold at most 16 owned units per workgroup).

This model replays, thread by thread, every LDS and exchange-buffer index that
version computes at this shape, with the sizes it allocated, phase by phase
between its workgroup barriers, and checks (1) every index in bounds and (2) no
LDS word touched by two threads in one phase unless both only read it, or the
two are lanes of one wave whose reads are ordered before the write by program
order. Result: both hold, for every workgroup and both step parities. The
indexing of that version is not what failed at this shape; the cause remains
unexplained, and no run of this shape is made on the GPU.
"""
import itertools

PX, PR, R, U = 1, 4, 16, 256
NR, NU = R // 16, U // 16
WR = 4 if NR >= 4 else (2 if NR >= 2 else 1)
WU = 4 // WR
NUW, RTW = NU // WU, -(-NR // WR)
UPW = U // PR
XS, XTS, PS = 36, R + 4, U + 1
RS_STRIDE = (U * 32 + 1 + 31) // 32 * 32
HIDDEN = PX * U

# the LDS carve-up of that version, in floats
O_XS = 0
O_XT = O_XS + R * XS
O_Y = O_XT + 32 * XTS
O_YP = O_Y + R
O_G = O_YP + WU * R
O_R2 = O_G + R
O_P = O_R2 + R
O_WO = O_P + WR * 32 * PS
O_SSE = O_WO + UPW * 33
LDS_USED = O_SSE + 8
# its plan's LDS request: the same terms (one R too many), at least 84 KB
LDS_FLOATS = max((R * 36 + 32 * (R + 4) + R * (4 + WU) + WR * 32 * (U + 1) + UPW * 33 + 8),
                 84 * 1024 // 4)
# its exchange buffers, in 64-bit words
RS_WORDS = 2 * 32 * (HIDDEN * 32 + 8 * 32)
AG_WORDS = 2 * HIDDEN * 33


def lanes():
    for tid in range(256):
        lane, wave = tid & 63, tid >> 6
        yield tid, wave, lane, lane >> 4, lane & 15


def phases(gx, gb, first_wg):
    """LDS accesses per barrier-delimited phase: lists of (address, tid, 'r'|'w')."""
    wr_of = lambda wave: wave % WR
    wu_of = lambda wave: wave // WR
    P = {}
    # 1: stage rows (X tile, X^T tile, Y)
    acc = []
    for tid in range(256):
        for i in range(tid, R * 8, 256):
            r, c4 = i >> 3, (i & 7) * 4
            acc += [(O_XS + r * XS + c4 + j, tid, "w") for j in range(4)]
            acc += [(O_XT + (c4 + j) * XTS + r, tid, "w") for j in range(4)]
        for r in range(tid, R, 256):
            acc.append((O_Y + r, tid, "w"))
    P["stage"] = acc
    # 2: forward operands, partial outputs per unit wave
    acc = []
    for tid, wave, lane, lq, li in lanes():
        wr, wu = wr_of(wave), wu_of(wave)
        for rt in range(RTW):
            rtile = wr + rt * WR
            if rtile * 16 < R:
                acc += [(O_XS + (rtile * 16 + li) * XS + 8 * lq + t, tid, "r") for t in range(8)]
                if li == 0:
                    acc += [(O_YP + wu * R + rtile * 16 + 4 * lq + v, tid, "w") for v in range(4)]
    P["forward"] = acc
    # 3: row sums, residual (thread r owns row r)
    acc = []
    for tid in range(256):
        for r in range(tid, R, 256):
            acc += [(O_YP + w * R + r, tid, "r") for w in range(WU)]
            acc += [(O_G + r, tid, "w"), (O_G + r, tid, "r"), (O_Y + r, tid, "r"),
                    (O_R2 + r, tid, "w")]
    P["residual"] = acc
    # 4: SSE of the rows (wave 0), backward into the P partials
    acc = []
    for tid, wave, lane, lq, li in lanes():
        if wave == 0:
            acc += [(O_R2 + r, tid, "r") for r in range(lane, R, 64)]
            if lane == 0:
                acc.append((O_SSE + 0, tid, "w"))
        wr, wu = wr_of(wave), wu_of(wave)
        for rt in range(RTW):
            rtile = wr + rt * WR
            if rtile * 16 < R:
                rb = rtile * 16 + 4 * lq
                acc += [(O_G + rb + v, tid, "r") for v in range(4)]
                for kt in range(2):
                    acc += [(O_XT + (kt * 16 + li) * XTS + rb + v, tid, "r") for v in range(4)]
        for kt, u, v in itertools.product(range(2), range(NUW), range(4)):
            ul = (wu + u * WU) * 16 + li
            acc.append((O_P + (wr * 32 + kt * 16 + 4 * lq + v) * PS + ul, tid, "w"))
    P["backward"] = acc
    # 5: this workgroup's exchange-B words from the P partials
    acc = []
    for tid in range(256):
        for i in range(tid, 32 * U, 256):
            ul, k = i // 32, i % 32
            acc += [(O_P + (w * 32 + k) * PS + ul, tid, "r") for w in range(WR)]
        if tid == 0:
            acc.append((O_SSE + 0, tid, "r"))
    P["b_store"] = acc
    # 6: the owned units' P columns summed over the group's workgroups
    acc = []
    for tid in range(256):
        for i in range(tid, UPW * 32, 256):
            jl, k = i // 32, i % 32
            acc.append((O_P + jl * 32 + k, tid, "w"))
        if tid == 0 and first_wg:
            acc.append((O_SSE + 1, tid, "w"))
    P["b_reduce"] = acc
    # 7: update of the owned units
    acc = []
    for tid in range(256):
        for i in range(tid, UPW * 32, 256):
            jl, k = i // 32, i % 32
            acc += [(O_P + jl * 32 + k, tid, "r"), (O_WO + jl * 33 + k, tid, "r"),
                    (O_WO + jl * 33 + 32, tid, "r"), (O_WO + jl * 33 + k, tid, "w")]
            if k == 0:
                acc.append((O_WO + jl * 33 + 32, tid, "w"))
        if tid == 0 and first_wg:
            acc.append((O_SSE + 1, tid, "r"))
    P["update"] = acc
    # 8: exchange-C stores read the owned master words
    acc = []
    for tid in range(256):
        for i in range(tid, UPW * 33, 256):
            acc.append((O_WO + i, tid, "r"))
    P["c_store"] = acc
    return P


def global_indices(gx, gb, par):
    """Every exchange-buffer word index that workgroup (gx, gb) touches in a step
    of parity par: (buffer, index)."""
    out = []
    rsw = ((par * PX + gx) * PR + gb) * RS_STRIDE
    rsg = ((par * PX + gx) * PR) * RS_STRIDE
    out += [("rs", rsw + i) for i in range(32 * U)] + [("rs", rsw + U * 32)]
    out += [("rs", rsg + t * RS_STRIDE + U * 32) for t in range(PR)]
    for i in range(UPW * 32):
        jl, k = i // 32, i % 32
        ul = gb * UPW + jl
        out += [("rs", rsg + b2 * RS_STRIDE + ul * 32 + k) for b2 in range(PR)]
    agg = (par * PX + gx) * U * 33
    for i in range(UPW * 33):
        jl, k = i // 33, i % 33
        out.append(("ag", agg + (gb * UPW + jl) * 33 + k))
    out += [("ag", agg + (t * UPW) * 33) for t in range(PR)]
    for ul in range(U):
        out += [("ag", agg + ul * 33 + k) for k in range(33)]
    return out


def test_shape_parameters_of_that_version():
    assert (WR, WU, NUW, RTW, UPW) == (1, 4, 4, 1, 64)
    assert LDS_USED <= LDS_FLOATS <= 160 * 1024 // 4


def test_lds_indices_in_bounds_and_race_free():
    for gb in range(PR):
        for name, acc in phases(0, gb, gb == 0).items():
            by_addr = {}
            for addr, tid, kind in acc:
                assert 0 <= addr < LDS_USED, (name, addr, tid)
                by_addr.setdefault(addr, []).append((tid, kind))
            for addr, uses in by_addr.items():
                writers = {t for t, k in uses if k == "w"}
                others = {t for t, k in uses} - writers
                if not writers:
                    continue
                # one writer; other threads may read it only within the writer's wave
                # (their read instructions precede the write in program order)
                assert len(writers) == 1, (name, addr, sorted(writers))
                w = next(iter(writers))
                assert all(t >> 6 == w >> 6 for t in others), (name, addr, w, sorted(others))


def test_exchange_indices_in_bounds():
    for gb, par in itertools.product(range(PR), range(2)):
        for buf, i in global_indices(0, gb, par):
            limit = RS_WORDS if buf == "rs" else AG_WORDS
            assert 0 <= i < limit, (buf, i, gb, par)


def test_exchange_slots_disjoint_between_writers():
    """No two workgroups write the same exchange word in one step."""
    for par in range(2):
        written = {}
        for gb in range(PR):
            rsw = ((par * PX + 0) * PR + gb) * RS_STRIDE
            for i in list(range(32 * U)) + [U * 32]:
                key = ("rs", rsw + i)
                assert key not in written, key
                written[key] = gb
            agg = (par * PX + 0) * U * 33
            for i in range(UPW * 33):
                jl, k = i // 33, i % 33
                key = ("ag", agg + (gb * UPW + jl) * 33 + k)
                assert key not in written, key
                written[key] = gb
