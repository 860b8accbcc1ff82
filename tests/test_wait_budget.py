"""Host-side check of the explicit vmcnt waits of the GEMM's late-barrier
schedule (the MXFP4 forward, dX and dS; paper §3, the products whose values
depend on every stage having landed).

The kernel issues its global -> LDS copies as raw instructions that the
compiler does not track, so the counts in `wait_vm_lgkm0<N>` are derived by
hand: before the barrier that publishes stage kt + 1, a thread may leave at
most the N youngest loads in flight, and those must all belong to later
stages.  This test replays, for every tile configuration the launchers
instantiate with the late schedule, each wave's order of copies (in DMA
quarters), code-slice copies, scale-chunk loads and W loads, the waits and
the barriers, for every stage count from 1 to 40, and checks:

  (a) at each barrier, every copy of the stage read right after it has
      completed under the wait that precedes it (vmcnt counts in issue order:
      `wait<N>` completes everything but the N youngest loads);
  (b) a copy into a stage buffer is issued only after a barrier that follows
      every read of the stage the buffer held before;
  (c) dX's W tile of stage s is written only after a barrier that follows
      every read of stage s - 2's tile (two W buffers), converted from items
      that a wait has already completed, and published by a barrier before
      the first read of stage s.  The step that loads stage s's items (step
      s - 2) converts them right after its barrier in the 256 x 256 tile;
      smaller tiles convert them in the middle of step s - 1, after its first
      slice's MFMAs.

The replay mirrors the body of `step2` and the prologue in
csrc/sq_gemm.hip; `test_model_follows_the_kernel_source` compares the
sequence of schedule calls the model assumes with the ones in the source, so
an edit to the schedule that the model does not know about fails here.
"""

import os
import re

import pytest

from conftest import ROOT

SRC = os.path.join(ROOT, "paper_2609_04526_amd", "csrc", "sq_gemm.hip")
VMCNT_MAX = 63


def source():
    with open(SRC) as f:
        return f.read()


def configs():
    """The SQ_CFG_* tile configurations: name -> (BM, BN, WGM, WGN, STAGES, BK)."""
    cfg = {}
    for name, val in re.findall(r"^#define (SQ_CFG_\w+) (.+)$", source(), flags=re.M):
        val = val.strip()
        cfg[name] = val
    out = {}
    for name, val in cfg.items():
        while val in cfg:                       # an alias of another config
            val = cfg[val]
        out[name] = tuple(int(x) for x in val.split(","))
    return out


# Tile configurations each late-schedule product can run with (single and
# grouped launches, the small tile, the two half tiles of a split grid).
LATE = {
    "fwdc": ["SQ_CFG_FWDC", "SQ_CFG_SMALL_FWDC", "SQ_CFG_HALF_N_FWDC", "SQ_CFG_HALF_M", "SQ_CFG_GROUPED_FWDC",
             "SQ_CFG_GROUPED_FWDC_LONG"],
    "dx": ["SQ_CFG_DX", "SQ_CFG_SMALL", "SQ_CFG_HALF_N", "SQ_CFG_HALF_M", "SQ_CFG_GROUPED_THIN"],
    "ds": ["SQ_CFG_DS", "SQ_CFG_SMALL", "SQ_CFG_HALF_N_DS", "SQ_CFG_HALF_M_DS"],
}


def quarter_counts(n):
    """Loads of each DMA quarter of an operand with n loads per stage
    (issue_part<P*n/4, (P+1)*n/4>)."""
    return [(n * (p + 1)) // 4 - (n * p) // 4 for p in range(4)]


def dma_plan(mode, BM, BN, WGM, WGN, STAGES, BK, wave):
    """Per-thread copies of one stage, by quarter, for this wave."""
    NT = 64 * WGM * WGN
    waves = NT // 64
    q = [0, 0, 0, 0]
    if mode in ("fwdc", "dx"):
        assert BM % 8 == 0 and (BM // 8) % waves == 0
        a = BM // 8 // waves                                   # DmaKC<BM, NT>::kInst
        q = quarter_counts(a)
        if mode == "fwdc":
            wave_inst = BN // 32                               # DmaCodes<BN, NT>
            if wave_inst >= waves:
                assert wave_inst % waves == 0
                codes = wave_inst // waves
            else:
                assert waves % wave_inst == 0
                codes = 1 if wave < wave_inst else 0
            q[0] += codes                                      # the code slice goes out with quarter 0
    else:
        for R in (BM, BN):                                     # DmaNat<R, NT, BK>
            tot = BK * (R // 8) // 64
            assert tot % waves == 0
            for p, c in enumerate(quarter_counts(tot // waves)):
                q[p] += c
    return q


def kernel_constants(mode, BM, BN, WGM, WGN, STAGES, BK):
    """kDma, kAhead, kAheadLow and the codes-wave split as the kernel derives them."""
    NT = 64 * WGM * WGN
    waves = NT // 64
    k_dma = sum(dma_plan(mode, BM, BN, WGM, WGN, STAGES, BK, 0))
    split = mode == "fwdc" and BN // 32 < waves
    k_dma_low = k_dma - 1 if split else k_dma
    ahead = min((STAGES - 2) * k_dma, VMCNT_MAX)
    ahead_low = min((STAGES - 2) * k_dma_low, VMCNT_MAX)
    return k_dma, ahead, ahead_low, split, (BN // 32 if split else waves)


class Wave:
    """One wave's loads in issue order and the events that order them."""

    def __init__(self):
        self.loads = []            # [tag, done]
        self.barriers = 0
        self.last_read_barrier = {}     # stage -> barrier count when its last read happened
        self.w_last_read = {}

    def issue(self, tag, n=1):
        for _ in range(n):
            self.loads.append([tag, False])

    def wait(self, n):
        assert 0 <= n <= VMCNT_MAX
        out = [l for l in self.loads if not l[1]]
        for l in out[:max(0, len(out) - n)]:
            l[1] = True

    def pending(self, tag):
        return [l for l in self.loads if l[0] == tag and not l[1]]


def replay(mode, cfg, nk, wave):
    BM, BN, WGM, WGN, STAGES, BK = cfg
    TN = (BN // WGN) // 32
    k_dma, ahead, ahead_low, split, code_waves = kernel_constants(mode, *cfg)
    codes_wave = (not split) or wave < code_waves
    q = dma_plan(mode, *cfg, wave)
    NT = 64 * WGM * WGN
    w_items = 64 * (BN // 8) // NT if mode == "dx" else 0       # kWPer
    mid = mode == "dx" and BM * BN < 256 * 256                 # kWMid
    w = Wave()
    holder = {}                                                # buffer -> stage it holds
    w_published = {}                                           # W tile stage -> barrier count at its write

    def dma_half(stage, first):
        buf = stage % STAGES
        prev = holder.get(buf)
        if prev is not None and prev != stage:
            # (b) the previous stage of this buffer was last read before a barrier already passed
            assert w.last_read_barrier.get(prev, -1) < w.barriers, (mode, cfg, nk, wave, stage, prev)
        holder[buf] = stage
        parts = (0, 1) if first else (2, 3)
        for p in parts:
            w.issue(("dma", stage), q[p])

    def read(stage):
        # every copy of this stage must have completed before a read (a)
        assert not w.pending(("dma", stage)), (mode, cfg, nk, wave, stage, "read before landing")
        w.last_read_barrier[stage] = w.barriers
        if mode == "dx":
            # (c) the stage's W tile was written before a barrier already passed
            assert w_published.get(stage, w.barriers) < w.barriers, (mode, cfg, nk, wave, stage, "W tile unpublished")
            w.w_last_read[stage] = w.barriers

    def commit_w(stage, in_loop):
        prev = stage - 2
        if prev >= 0:
            assert w.w_last_read.get(prev, -1) < w.barriers, (mode, cfg, nk, wave, stage, "W tile reuse")
        if in_loop:
            # converted after the barrier whose wait completed the items
            assert not w.pending(("w", stage)), (mode, cfg, nk, wave, stage, "W items still in flight")
        # (the prologue's compiler wait completes the items and, loads
        # completing in order, everything older)
        ws = [i for i, l in enumerate(w.loads) if l[0] == ("w", stage)]
        for l in w.loads[:ws[-1] + 1]:
            l[1] = True
        w_published[stage] = w.barriers

    def load_sc(chunk):
        w.issue(("sc", chunk), 2 * TN)          # two 8-byte halves per row slice

    whole = mode == "fwdc"             # the forward issues each stage's DMA whole, after the barrier
    # prologue
    if nk > 0:
        if mode == "dx":
            w.issue(("w", 0), 2 * w_items)
            commit_w(0, False)
            if 1 < nk:
                w.issue(("w", 1), 2 * w_items)
                if not mid:
                    commit_w(1, False)
        if mode == "fwdc":
            load_sc(0)
        dma_half(0, True)
        dma_half(0, False)
        w.wait(0)
        w.barriers += 1
        read(0)
        for s in range(1, STAGES - 1):
            if s < nk:
                dma_half(s, True)
                dma_half(s, False)
        if STAGES - 1 < nk:
            dma_half(STAGES - 1, True)
            if whole:
                dma_half(STAGES - 1, False)
    for kt in range(nk):
        if mode == "fwdc" and kt % 8 == 7 and kt + 1 < nk:
            load_sc((kt + 1) // 8)
        if mode == "dx" and kt + 2 < nk:
            w.issue(("w", kt + 2), 2 * w_items)
        read(kt)                                               # slice 1
        if not whole and kt + STAGES - 1 < nk:
            dma_half(kt + STAGES - 1, False)
        if mid and kt + 1 < nk:
            commit_w(kt + 1, True)                             # after slice 0's MFMAs
        read(kt)                                               # slices 2, 3
        read(kt)
        if kt + STAGES - 1 < nk:
            w.wait(ahead if codes_wave else ahead_low)
        else:
            w.wait(0)
        w.barriers += 1
        if kt + 1 < nk:
            read(kt + 1)                                       # slice 0 of the next stage (a)
        if kt + STAGES < nk:
            dma_half(kt + STAGES, True)
            if whole:
                dma_half(kt + STAGES, False)
        if mode == "dx" and not mid and kt + 2 < nk:
            commit_w(kt + 2, True)
    w.wait(0)
    assert all(l[1] for l in w.loads)
    return w


def cases():
    cfg = configs()
    out = []
    for mode, names in LATE.items():
        for name in names:
            assert name in cfg, name
            c = cfg[name]
            if c not in [x[2] for x in out if x[0] == mode]:
                out.append((mode, name, c))
    return out


@pytest.mark.parametrize("mode,name,cfg", cases(), ids=lambda x: str(x))
def test_waits_cover_every_stage(mode, name, cfg):
    BM, BN, WGM, WGN, STAGES, BK = cfg
    waves = WGM * WGN
    for nk in range(1, 41):
        for wave in range(waves):
            replay(mode, cfg, nk, wave)


def test_a_shorter_wait_budget_is_caught(monkeypatch):
    """The replay fails for a budget one load larger than the kernel's on a
    three-stage dS half tile (the budget the check guards)."""
    import sys
    cfg = configs()["SQ_CFG_HALF_N_DS"]
    assert cfg[4] == 3
    k_dma, ahead, _, _, _ = kernel_constants("ds", *cfg)
    monkeypatch.setattr(sys.modules[__name__], "kernel_constants",
                        lambda *a: (k_dma, ahead + 1, ahead + 1, False, 8))
    with pytest.raises(AssertionError):
        for nk in range(1, 12):
            replay("ds", cfg, nk, 0)


def test_a_larger_forward_budget_is_caught(monkeypatch):
    """The same for the forward's four-stage grouped tile, whose stages go
    out whole after the barrier: one load more in flight at the wait fails."""
    import sys
    cfg = configs()["SQ_CFG_GROUPED_FWDC"]
    assert cfg[4] == 4
    k_dma, ahead, ahead_low, split, cw = kernel_constants("fwdc", *cfg)
    monkeypatch.setattr(sys.modules[__name__], "kernel_constants",
                        lambda *a: (k_dma, ahead + 1, ahead_low + 1, split, cw))
    with pytest.raises(AssertionError):
        for nk in range(1, 12):
            for wave in range(cfg[2] * cfg[3]):
                replay("fwdc", cfg, nk, wave)


def _calls(body):
    pat = (r"\b(take_scales|read|dma_half|load_w|commit_w|mma|wait_vm_lgkm0<\w+>|"
           r"__builtin_amdgcn_s_barrier)\s*\(")
    return [m.group(1) for m in re.finditer(pat, body)]


def test_model_follows_the_kernel_source():
    """The order of schedule calls in step2 and in the late prologue is the
    one the replay above models."""
    s = source()
    i = s.index("auto step2 = [&](auto SC, int kt) {")
    j = s.index("// prologue: stage 0 in LDS", i)
    step2 = _calls(s[i:j])
    # (dX below 256 x 256 loads into the set of the stage's parity and
    # converts after slice 0's MFMAs; the 256 x 256 tile after the barrier)
    assert step2 == ["take_scales", "load_w", "load_w", "read", "dma_half", "mma", "commit_w", "read", "mma",
                     "read", "mma", "wait_vm_lgkm0<kAhead>", "wait_vm_lgkm0<kAheadLow>", "wait_vm_lgkm0<0>",
                     "__builtin_amdgcn_s_barrier", "read", "dma_half", "dma_half", "mma", "commit_w"], step2
    k = s.index("for (int kt0 = 0; kt0 < nk; kt0 += STAGES)", j)
    pro = _calls(s[j:k])
    assert pro == ["load_w", "commit_w", "load_w", "load_w", "commit_w", "load_w", "commit_w", "wait_vm_lgkm0<0>",
                   "__builtin_amdgcn_s_barrier", "read", "dma_half", "dma_half"], pro
    assert "constexpr bool kWMid = MODE == kDx && BM * BN < 256 * 256;" in s
    assert "if (kt + 2 < nk) load_w(kt + 2, std::integral_constant<int, S % 2>{});" in s[i:j]
    assert "if (kt + 1 < nk) commit_w(kt + 1, std::integral_constant<int, (S + 1) % 2>{});" in s[i:j]
    assert "if (1 < nk) load_w(1, I1{});" in s[j:k]
    # the forward issues a stage's second half with its first (after the
    # barrier, and in the prologue), the others one step later
    assert "constexpr bool kWhole = MODE == kFwdC;" in s
    assert "if (!kWhole && kt + STAGES - 1 < nk) dma_half(SP{}, kt + STAGES - 1, I2{});" in s[i:j]
    assert "if (kWhole) dma_half(SC, kt + STAGES, I2{});" in s[i:j]
    assert "if (kWhole) dma_half(std::integral_constant<int, STAGES - 1>{}, STAGES - 1, I2{});" in s[j:k]
    # the W items of stage kt + 2 are loaded before the barrier's wait and
    # converted after it
    assert "if (kt + 2 < nk) load_w(kt + 2, I0{});" in s and "if (kt + 2 < nk) commit_w(kt + 2, I0{});" in s
    # the budgets and the code-slice split as the replay derives them
    assert "constexpr int kAhead = (STAGES - 2) * kDma < 63 ? (STAGES - 2) * kDma : 63;" in s
    assert "constexpr int kDmaLow = kCodesSplit ? kDma - DC::kInst : kDma;" in s
    assert "if ((kt & 7) == 7 && kt + 1 < nk) load_sc((kt + 1) >> 3);" in s
    assert "if constexpr (MODE == kFwdC && P == 0) dC.template issue_part<0, DC::kInst>" in s


# ---------------------------------------------------------------- streamed dS
# ds_stream_kernel runs a workgroup's tiles back to back as one pipeline of
# two stage buffers: a DMA cursor and a compute cursor walk the same list of
# (tile, stage) pairs, every barrier is preceded by a wait for all loads.

def stream_replay(nks):
    """Replay one wave of the streamed dS over tiles with nks[t] stages each;
    returns the (tile, stage) sequences the two cursors walked."""
    seq = [(t, k) for t, nk in enumerate(nks) for k in range(nk)]
    w = Wave()
    holder = {}
    reads = {}                 # global stage -> barrier count of its last read
    dma_walk, mma_walk = [], []
    cur = {"d": 0}             # DMA cursor: index into seq

    def dma_half(buf, first):
        g = cur["d"]
        prev = holder.get(buf)
        if first and prev is not None and prev != g:
            assert reads.get(prev, -1) < w.barriers, ("buffer reused before its reads were fenced", nks, g, prev)
        holder[buf] = g
        w.issue(("dma", g), 2)
        if not first:
            dma_walk.append(seq[g])
            cur["d"] += 1

    def read(g):
        assert not w.pending(("dma", g)), ("read before landing", nks, g)
        assert holder[g % 2] == g
        reads[g] = w.barriers

    # prologue
    dma_half(0, True)
    dma_half(0, False)
    w.wait(0)
    w.barriers += 1
    read(0)
    if cur["d"] < len(seq):
        dma_half(1, True)
        dma_half(1, False)
    g = 0
    while True:
        read(g)                                   # slices 1, 2, 3
        read(g)
        read(g)
        mma_walk.append(seq[g])
        w.wait(0)
        w.barriers += 1
        more = g + 1 < len(seq)
        if more:
            read(g + 1)                           # slice 0 of the next stage
        if cur["d"] < len(seq):                   # the whole stage after it
            dma_half(g % 2, True)
            dma_half(g % 2, False)
        if not more:
            break
        g += 1
    w.wait(0)
    assert all(l[1] for l in w.loads)
    return dma_walk, mma_walk, seq


def test_stream_cursors_cover_every_stage():
    import random
    rnd = random.Random(5)
    cases = [[1], [1, 1], [1, 1, 1, 1], [4], [2, 1, 3], [1, 5, 1, 1, 2]]
    cases += [[rnd.randint(1, 6) for _ in range(rnd.randint(1, 14))] for _ in range(300)]
    for nks in cases:
        dma_walk, mma_walk, seq = stream_replay(nks)
        assert dma_walk == seq and mma_walk == seq, nks


def test_stream_model_follows_the_kernel_source():
    """The calls of ds_stream_kernel's stage_step and prologue in the order
    stream_replay models."""
    s = source()
    i = s.index("auto stage_step = [&](SQ_LDS uint8_t* cur, SQ_LDS uint8_t* nxt) -> bool {")
    j = s.index("// prologue: the first stage whole", i)
    pat = r"\b(read|dma_half|dma_advance|mma|wait_vm_lgkm0<\w+>|__builtin_amdgcn_s_barrier|ds_store<FMT, TM, TN, (?:true|false)>|tile_codes|locate)\s*\("
    body = [m.group(1) for m in re.finditer(pat, s[i:j])]
    assert body == ["read", "mma", "read", "mma", "read", "mma", "wait_vm_lgkm0<0>",
                    "__builtin_amdgcn_s_barrier", "read", "dma_half", "dma_half", "dma_advance", "mma",
                    "ds_store<FMT, TM, TN, true>", "ds_store<FMT, TM, TN, false>", "locate", "tile_codes"], body
    k = s.index("while (stage_step(cur, nxt))", j)
    pro = [m.group(1) for m in re.finditer(pat, s[j:k])]
    assert pro == ["dma_half", "dma_half", "dma_advance", "tile_codes", "wait_vm_lgkm0<0>",
                   "__builtin_amdgcn_s_barrier", "read", "dma_half", "dma_half", "dma_advance"], pro
    # both halves of the stage after next go into the buffer just read, after the barrier
    assert "dma_half(cur, I0{});\n      dma_half(cur, I2{});\n      dma_advance();" in s[i:j]
    assert "const bool more = !last || cpos + step < end;" in s[i:j]
