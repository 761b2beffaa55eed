"""Generates spmm_asm_gen.h: the inner loops of the gfx950 panel kernel as inline
assembly.  One consumer routine per panel height RW and tile layout, and one producer
routine per staging kind.  The description below is that of the 256-column layout
(`WIDE`); the 128-column layout (`NARROW`, class Layout) differs only where stated there:
2 columns per lane, 512-byte ring rows and their field at bit 9 of the address words,
two producers that stage two rows per DMA, and 32-row panels beside the others.

Why generated assembly: the consumer keeps a wavefront's RW x 4 output tile in fixed
VGPRs and selects the row of each nonzero with VGPR index mode (s_set_gpr_idx_*), and
it software-pipelines scalar loads of the weight stream, LDS reads of B and FMAs
across rotating register sets.  Compiled code can express neither the indexed
accumulator nor the rotation.

Workgroup roles.  Waves 0..nc-1 are consumers (one panel each); waves nc..nc+NPROD-1
are producers.  B is staged through a ring of RING slots of CHUNK rows (1 KB per row:
64 lanes x 16 bytes) at LDS byte address 0; chunk c of B goes to slot c % RING, and
producer p stages rows [p, p + 1) * CHUNK/NPROD of every chunk.  There is no
workgroup barrier inside the loops: the roles synchronise through LDS words
    ready[p]    number of chunks whose rows producer p has landed in the ring
    progress[w] lowest chunk consumer w may still read (consumer w writes; the slots
                of absent consumers hold 0x7fffffff)
A producer stages its part of chunk c once c < min(progress) + RING (slot c % RING no
longer read by anyone; it re-reads the progress words only when it reaches the limit
it last computed), keeps up to PMAX chunks in flight, and advances its ready word as
each lands.  A consumer publishes progress and re-reads the ready words only at
groups whose sync bit is set; chunk c is there once every ready word exceeds c.
Several producer waves split each chunk so that its loads go out in parallel and the
per-chunk handshake of any one wave stays short.

Every group reads chunks c_lo..c_hi with c_hi - c_lo < RING and publishes
progress = c_lo before waiting for c_hi, so the slowest consumer's next chunk can
always be staged: the loops cannot deadlock.  Each wait is also bounded by
a per-wave poll budget (a launch argument), after which the wave goes on without
waiting, so the kernel always ends.  Going on is never silent: a producer that stages
past the ring limit first sets the workgroup's overrun word, and a consumer whose
budget ran out, or that finds the overrun word set when it finishes, replaces its
whole panel's results with NaN.

Stream consumed (see sdnn_internal.h): per panel, groups of 16 dwords (64 bytes,
one scalar load, one scalar-cache line) [w0..w7 a0..a7]; w = fp32 weight bits;
a = (ring row << 10) | row, plus c_lo in a6 >> 17, c_hi in a7 >> 18, the sync flag in
a7 bit 17 and the end-of-panel flag in a7 bit 9.  The ring row field is bits 10..16,
so (a & 0x1fc00) | (16 * lane) is the LDS address of the lane's 4 B values; VGPR
index mode uses only a's low 8 bits.

Consumer register plan of the 256-column layout (pinned in the asm statement; the
128-column one keeps v[32:47] / v[48:63] for B and v[64 + k*RW + r], k = 0..1, for the
accumulators, and reads only the two ready words v[26:27]):
  v31 0x1fc00 (ring-row mask), v28 zero offset and v29 sink of the L2 touch loads,
  v[24:27] ready words, v30 temp, v[32:63] / v[64:95] B values of the group being multiplied /
  fetched, v[96 + k*RW + r] accumulator of row r, column 4*lane + k (k = 0..3);
  s[36:83] ring of NSLOT = 3 stream groups (16 SGPRs each), s[84:85] next group to
  fetch, s86 chunks known ready, s87 temp, s88 poll budget, s89 saved m0, s[90:91]
  saved exec, s92 temp.
Per group g:
  wait until B of g and stream group g+1 have arrived
  if g+1 carries the sync bit: publish c_lo(g+1), wait until c_hi(g+1) < ready;
      if g+1 ends the panel: fetch its B, multiply g and g+1, finish
  s_load of stream group g+NSLOT-1 into the slot that group g-1 used
  vector touch TOUCH_AHEAD bytes ahead (pulls the stream into L2 for the scalar loads)
  address + ds_read_b128 of the 8 B rows of group g+1      (index mode off)
  for each entry: s_set_gpr_idx_* row; 4 v_fma_f32 into the row's accumulators
  (index mode DST|SRC2: only the accumulator operand is offset by the row)
The ring and the touch read up to kStreamTailGroups groups past a panel's last
group; the stream carries that many zero groups at its end.

Producer: issues one 16-byte (or four 4-byte) direct global->LDS load per B row,
addressed by a scalar pointer plus a per-lane VGPR offset, with M0 holding the LDS
row address; rows past K re-stage row K-1 into LDS rows no entry reads.

Hazards the hand-written code must respect (the compiler handles them for compiled
code): a VALU write of a VGPR followed at once by v_readfirstlane of that VGPR reads
the old value, so the ready words go from the LDS result straight to SGPRs; a
VALU-written vcc is read by SALU only after s_nop; an SALU write of M0 is followed by
at least one instruction before an LDS DMA that uses it.
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "spmm_asm_gen.h")

G = 8                                         # entries per group (64 bytes)
NSLOT = 3
E = tuple(36 + 2 * G * i for i in range(NSLOT))  # SGPR bases of the stream-group ring
LOW, HIW = 2 * G - 2, 2 * G - 1               # slot offsets of the c_lo / c_hi words
UNROLL = 6                                    # multiple of NSLOT and of 2
RW_VARIANTS = (4, 8, 12, 16)
RW_VARIANTS_NARROW = (4, 8, 12, 16, 32)  # 32-row panels: 128-column tiles only
SYNC_BIT, LO_SHIFT, HI_SHIFT = 17, 17, 18
CHUNK, RING = 32, 4
PMAX_VEC, PMAX_DWORD = 2, 1                   # chunks in flight per producer variant
TOUCH_AHEAD = 512  # bytes of stream pulled into L2 ahead of the scalar ring
GROUP_BYTES = 8 * G
INF = 0x7FFFFFFF
MAX_CONS = 14      # consumer waves a workgroup can have
PROFILE = False    # scratch builds only: time consumers spend waiting (%[twait])


class Layout:
    """Tile layout of a kernel variant.  V columns per lane (a tile is 64 V columns), so a
    staged B row segment is ROW_BYTES = 256 V bytes and the ring row of an entry sits at
    bit ROW_SHIFT of its address word (the LDS address of the lane's V values is then
    (a & RING_MASK) | (4 V lane)); the end-of-panel flag sits below the ring-row field,
    above the 8 bits that VGPR index mode reads.  NPROD producer waves; producer p stages
    rows [p, p+1) * CHUNK/NPROD of every chunk."""

    def __init__(self, name, v, nprod, row_shift, end_bit, scalars):
        self.name, self.V, self.NPROD = name, v, nprod
        # consumer SGPRs besides the stream ring: next group to fetch (64-bit), chunks
        # known ready, temp, poll budget, saved m0, saved exec (64-bit), temp
        (self.PTR, self.SREADY, self.STMP, self.SPOLL, self.M0S, self.SEXEC,
         self.SREADY1) = scalars
        self.ROW_SHIFT, self.END_BIT = row_shift, end_bit
        self.ROW_BYTES = 1 << row_shift
        assert self.ROW_BYTES == 256 * v and end_bit >= 8 and end_bit < row_shift
        self.RING_MASK = (RING * CHUNK - 1) << row_shift
        self.VB = (32, 32 + v * G)                # VGPR bases of the two B-value sets
        self.ACC = 32 + 2 * v * G                 # first accumulator VGPR
        self.prefix = "" if name == "wide" else "n_"


# 256-column tiles (4 columns per lane, ds_read_b128, 1 KB ring rows, 128 KB ring: one
# workgroup per CU) and 128-column tiles (2 columns per lane, ds_read_b64, 512-byte ring
# rows, 64 KB ring and two producers: two workgroups per CU)
# (both kernels run at most 6 waves per SIMD, which leaves 102 SGPRs a wave)
WIDE = Layout("wide", 4, 4, 10, 9, (84, 86, 87, 88, 89, 90, 92))
NARROW = Layout("narrow", 2, 2, 9, 8, (84, 86, 87, 88, 89, 90, 92))
# the wide layout's names, used by the producers and the header
VB, ACC, END_BIT, RING_MASK = WIDE.VB, WIDE.ACC, WIDE.END_BIT, WIDE.RING_MASK
TILE_BYTES = WIDE.ROW_BYTES  # bytes of one B row segment of a 256-column tile (the next tile's start)
NPROD = WIDE.NPROD


def address_phase(slot, vb, lay=WIDE):
    L = []
    v = lay.V
    for j in range(G):
        L.append(f"v_and_or_b32 v{vb + v * j}, s{slot + G + j}, v31, %[vl]")
        L.append(f"ds_read_b{32 * v} v[{vb + v * j}:{vb + v * j + v - 1}], v{vb + v * j}")
    return L


def fmas(slot, vb, rw, lay=WIDE):
    L = []
    v = lay.V
    for j in range(G):
        if j == 0:
            L.append(f"s_set_gpr_idx_on s{slot + G}, gpr_idx(DST,SRC2)")
        else:
            L.append(f"s_set_gpr_idx_idx s{slot + G + j}")
        for k in range(v):
            p = lay.ACC + k * rw
            L.append(f"v_fma_f32 v{p}, s{slot + j}, v{vb + v * j + k}, v{p}")
    L.append("s_set_gpr_idx_off")
    return L


def lane0_write(addr, vdata, lay=WIDE):
    """ds_write_b32 from lane 0 only (all lanes hold the same value)."""
    SEXEC = lay.SEXEC
    return [f"s_mov_b64 s[{SEXEC}:{SEXEC + 1}], exec", "s_mov_b64 exec, 1",
            f"ds_write_b32 {addr}, {vdata}", f"s_mov_b64 exec, s[{SEXEC}:{SEXEC + 1}]"]


def ready_regs(nprod=NPROD):
    """VGPRs that receive the producers' ready words: v27 | v[26:27] | v[24:27]."""
    assert nprod in (1, 2, 4)
    width = {1: "b32", 2: "b64", 4: "b128"}[nprod]
    words = [f"v{24 + 4 - nprod + k}" for k in range(nprod)]
    rng = words[0] if nprod == 1 else f"v[{24 + 4 - nprod}:27]"
    return width, words, rng


def fold_ready(lay=WIDE):
    """SREADY = min of the ready words in ready_regs().  Each word goes from the LDS
    result straight to an SGPR: a VALU write of a VGPR followed at once by
    v_readfirstlane of it reads the old value on gfx950."""
    SREADY, SREADY1 = lay.SREADY, lay.SREADY1
    _, words, _ = ready_regs(lay.NPROD)
    L = [f"v_readfirstlane_b32 s{SREADY}, {words[0]}"]
    for w in words[1:]:
        L += [f"v_readfirstlane_b32 s{SREADY1}, {w}", f"s_min_u32 s{SREADY}, s{SREADY}, s{SREADY1}"]
    return L


def sync(slot, tag, lay=WIDE):
    """Publish progress = c_lo of the group in `slot`, then wait until its c_hi has
    landed (c_hi < min of the producers' ready words), polling while the budget
    lasts.  Wave priority: a consumer enters each sync point at priority 1 and drops to
    0 when it has to poll, until its next sync point.  The ring lets no wave run more than
    four chunks ahead of the slowest, so a wave that waits is ahead of its workgroup, and
    the SIMD's issue then favours the waves that hold the ring back."""
    STMP, SREADY, SPOLL, SEXEC = lay.STMP, lay.SREADY, lay.SPOLL, lay.SEXEC
    width, _, rng = ready_regs(lay.NPROD)
    L = ["s_setprio 1", f"s_lshr_b32 s{STMP}, s{slot + LOW}, {LO_SHIFT}",
         f"s_add_u32 s{STMP}, s{STMP}, %[cbase]", f"v_mov_b32 v30, s{STMP}"]
    L += lane0_write("%[pa]", "v30", lay)
    L += [f"s_lshr_b32 s{STMP}, s{slot + HIW}, {HI_SHIFT}", f"s_add_u32 s{STMP}, s{STMP}, %[cbase]"]
    if PROFILE:
        L += [f"s_memtime s[{SEXEC}:{SEXEC + 1}]", "s_waitcnt lgkmcnt(0)"]
    L += [
        f".L%=_poll{tag}:",
        f"s_cmp_lt_u32 s{STMP}, s{SREADY}",
        f"s_cbranch_scc1 .L%=_ready{tag}",
        f"s_cmp_eq_u32 s{SPOLL}, 0",
        f"s_cbranch_scc1 .L%=_ready{tag}",
        f"s_sub_u32 s{SPOLL}, s{SPOLL}, 1",
        "s_setprio 0",
        f"ds_read_{width} {rng}, %[ra]",
        "s_waitcnt lgkmcnt(0)",
    ]
    L += fold_ready(lay)
    L += [
        f"s_cmp_lt_u32 s{STMP}, s{SREADY}",
        f"s_cbranch_scc1 .L%=_ready{tag}",
        "s_sleep 1",
        f"s_branch .L%=_poll{tag}",
        f".L%=_ready{tag}:",
    ]
    if PROFILE:  # scratch builds also pin s[94:95]
        L += ["s_memtime s[94:95]", "s_waitcnt lgkmcnt(0)",
              f"s_sub_u32 s94, s94, s{SEXEC}", "s_add_u32 %[twait], %[twait], s94"]
    return L


def consumer(rw, limit=False, lay=WIDE):
    """The FMA loop for RW-row panels of the tile layout `lay`.  limit: stop before a sync
    group whose c_lo reaches the chunk limit (K-split launches; the plain loop leaves that
    test out)."""
    VB, ACC, END_BIT, V = lay.VB, lay.ACC, lay.END_BIT, lay.V
    PTR, SREADY, STMP, SPOLL, M0S = lay.PTR, lay.SREADY, lay.STMP, lay.SPOLL, lay.M0S
    L = [
        f"s_mov_b32 s{M0S}, m0",
        f"v_mov_b32 v31, {hex(lay.RING_MASK)}",
        "v_mov_b32 v28, 0",
        f"s_mov_b32 s{SREADY}, 0",
        f"s_mov_b32 s{SPOLL}, %[budget]",
    ]
    if PROFILE:
        L.append("s_mov_b32 %[twait], 0")
    for g in range(NSLOT - 1):
        L.append(f"s_load_dwordx16 s[{E[g]}:{E[g] + 2 * G - 1}], %[sp], {hex(GROUP_BYTES * g)}")
    L += [
        f"s_mov_b64 s[{PTR}:{PTR + 1}], %[sp]",
        f"s_add_u32 s{PTR}, s{PTR}, {GROUP_BYTES * (NSLOT - 1)}",
        f"s_addc_u32 s{PTR + 1}, s{PTR + 1}, 0",
        "s_waitcnt lgkmcnt(0)",
    ]
    L += sync(E[0], "e", lay)   # a panel's first group always carries the sync bit
    L += address_phase(E[0], VB[0], lay)
    L += [f"s_bitcmp1_b32 s{E[0] + HIW}, {END_BIT}", "s_cbranch_scc0 .L%=_iter0",
          "s_waitcnt lgkmcnt(0)"]   # the panel is one group
    L += fmas(E[0], VB[0], rw, lay)
    L.append("s_branch .L%=_finish")
    for i in range(UNROLL):
        cur, nxt, pre = E[i % NSLOT], E[(i + 1) % NSLOT], E[(i + NSLOT - 1) % NSLOT]
        vbc, vbn = VB[i % 2], VB[(i + 1) % 2]
        L += [f".L%=_iter{i}:", "s_waitcnt lgkmcnt(0)",
              f"s_bitcmp1_b32 s{nxt + HIW}, {SYNC_BIT}", f"s_cbranch_scc1 .L%=_sync{i}",
              f".L%=_ret{i}:"]
        # the next scalar load goes out first, so it has the whole iteration to land
        L.append(f"s_load_dwordx16 s[{pre}:{pre + 2 * G - 1}], s[{PTR}:{PTR + 1}], 0x0")
        if TOUCH_AHEAD:  # pull the stream line TOUCH_AHEAD bytes ahead into L2
            L.append(f"global_load_dword v29, v28, s[{PTR}:{PTR + 1}] offset:{TOUCH_AHEAD}")
        L += [f"s_add_u32 s{PTR}, s{PTR}, {GROUP_BYTES}", f"s_addc_u32 s{PTR + 1}, s{PTR + 1}, 0"]
        L += address_phase(nxt, vbn, lay)
        L += fmas(cur, vbc, rw, lay)
    L.append("s_branch .L%=_iter0")
    for i in range(UNROLL):
        cur, nxt = E[i % NSLOT], E[(i + 1) % NSLOT]
        vbc, vbn = VB[i % 2], VB[(i + 1) % 2]
        L.append(f".L%=_sync{i}:")
        if limit:
            # a group starting at or past the chunk limit belongs to the next workgroup's
            # K-segments: finish with the current group
            L += [f"s_lshr_b32 s{STMP}, s{nxt + LOW}, {LO_SHIFT}",
                  f"s_cmp_ge_u32 s{STMP}, %[climit]", f"s_cbranch_scc1 .L%=_stop{i}"]
        L += sync(nxt, i, lay)
        L += [f"s_bitcmp1_b32 s{nxt + HIW}, {END_BIT}", f"s_cbranch_scc0 .L%=_ret{i}"]
        L += address_phase(nxt, vbn, lay)  # group g+1 ends the panel
        L += fmas(cur, vbc, rw, lay)
        L.append("s_waitcnt lgkmcnt(0)")
        L += fmas(nxt, vbn, rw, lay)
        L.append("s_branch .L%=_finish")
        if limit:
            L.append(f".L%=_stop{i}:")       # the current group's reads have landed
            L += fmas(cur, vbc, rw, lay)
            L.append("s_branch .L%=_finish")
    # a wave that went on without waiting, or whose chunks a producer may have
    # overwritten, leaves NaN instead of unchecked values
    L += [".L%=_finish:",
          f"s_cmp_eq_u32 s{SPOLL}, 0", "s_cbranch_scc1 .L%=_poison",
          "ds_read_b32 v30, %[ov]", "s_waitcnt lgkmcnt(0)",
          f"v_readfirstlane_b32 s{STMP}, v30",
          f"s_cmp_eq_u32 s{STMP}, 0", "s_cbranch_scc1 .L%=_clean",
          ".L%=_poison:"]
    L += [f"v_mov_b32 v{ACC + x}, 0x7fc00000" for x in range(V * rw)]
    L += [".L%=_clean:", "v_mov_b32 v30, %[next]"]
    L += lane0_write("%[pa]", "v30", lay)
    L += ["s_waitcnt vmcnt(0) lgkmcnt(0)", f"s_mov_b32 m0, s{M0S}"]
    body = "\n".join('      "' + x + '\\n\\t"' for x in L)
    planes = ", ".join(f'"+{{v[{ACC + k * rw}:{ACC + k * rw + rw - 1}]}}"(p{k})' for k in range(V))
    lo, hi = min(E[0], PTR), max(E[-1] + 2 * G - 1, lay.SREADY1)
    sregs = [f"s{x}" for x in range(lo, (95 if PROFILE else hi) + 1)]
    # v24..v31 minus the ready words a narrow consumer does not read, then the B sets
    vregs = [f"v{x}" for x in range(24 + 4 - lay.NPROD, ACC)]
    clob = ", ".join(f'"{r}"' for r in sregs + vregs + ["scc", "memory"])
    name = f"consume_{lay.prefix}rw{rw}" + ("_limit" if limit else "")
    operands = ('[sp] "s"(a.stream), [vl] "v"(a.vlane), [pa] "v"(a.prog_addr), '
                '[ra] "v"(a.ready_addr),\n        [budget] "s"(a.poll_budget), '
                '[ov] "v"(a.overrun_addr), [cbase] "s"(a.chunk_base), [next] "s"(a.next_progress)'
                + (', [climit] "s"(a.chunk_limit)' if limit else ''))
    params = ", ".join(f"acc_plane_t<{rw}>& p{k}" for k in range(V))
    return f"""// Consumer, RW = {rw}, {64 * V}-column tiles{', stopping at the chunk limit' if limit else ''}: accumulator planes p0..p{V - 1}
__device__ __forceinline__ void {name}({params},
    {'' if PROFILE else 'const '}ConsumerArgs& a) {{
  asm volatile(
{body}
      : {planes}{', [twait] "=&s"(a.twait)' if PROFILE else ''}
      : {operands}
      : {clob});
}}
"""


# producer SGPRs
PISS, PSIG, PINF, PLIM, PTMP, PPOLL, PROW, PM0 = 40, 41, 42, 43, 44, 45, 46, 47
PADDR, PEX, PBASE, PCS = 48, 50, 52, 54       # 64-bit each
PCM = 56                                       # column masks (1 or 4 pairs)
PKM1, PLAST = 64, 65
PCI, PB0, PRB = 78, 80, 79                     # chunk within the item; the item's first chunk
                                               # address; the item's row-block (tile-major items)
PTB = 82                                       # the item's tile base, B + n0 (64-bit)
# producer VGPRs: row offsets of the fast path, progress words, min tree
VO, VP, VMIN = 32, 40, 56


def producer_poll():
    """Read the 16 progress words and set PLIM = min(progress) + RING: chunks below
    PLIM have a free slot (every consumer has moved past the chunk that used it)."""
    L = [f"s_mov_b64 s[{PEX}:{PEX + 1}], exec", "s_mov_b64 exec, 1"]
    for k in range(4):
        L.append(f"ds_read_b128 v[{VP + 4 * k}:{VP + 4 * k + 3}], %[pg] offset:{16 * k}")
    L += ["s_waitcnt lgkmcnt(0)",
          f"v_min3_u32 v{VMIN}, v{VP}, v{VP + 1}, v{VP + 2}",
          f"v_min3_u32 v{VMIN + 1}, v{VP + 3}, v{VP + 4}, v{VP + 5}",
          f"v_min3_u32 v{VMIN + 2}, v{VP + 6}, v{VP + 7}, v{VP + 8}",
          f"v_min3_u32 v{VMIN + 3}, v{VP + 9}, v{VP + 10}, v{VP + 11}",
          f"v_min3_u32 v{VMIN + 4}, v{VP + 12}, v{VP + 13}, v{VP + 14}",
          f"v_min3_u32 v{VMIN}, v{VMIN}, v{VMIN + 1}, v{VMIN + 2}",
          f"v_min3_u32 v{VMIN + 1}, v{VMIN + 3}, v{VMIN + 4}, v{VP + 15}",
          f"v_min_u32 v{VMIN}, v{VMIN}, v{VMIN + 1}",
          "s_nop 4",                           # VALU write, then v_readfirstlane of it
          f"v_readfirstlane_b32 s{PTMP}, v{VMIN}",
          f"s_mov_b64 exec, s[{PEX}:{PEX + 1}]",
          f"s_add_u32 s{PLIM}, s{PTMP}, {RING}"]
    return L


def issue_rows_clamped(vec, half):
    """Stage rows PROW .. PROW+half-1 of B (each clamped to K-1) at LDS m0, m0+1KB, ..."""
    L = []
    pieces = 1 if vec else 4
    if vec:
        L.append(f"s_mov_b64 exec, s[{PCM}:{PCM + 1}]")
    for r in range(half):
        L += [
            f"s_min_u32 s{PTMP}, s{PROW}, s{PKM1}",
            f"s_mul_i32 s{PADDR}, s{PTMP}, %[rs]",
            f"s_mul_hi_u32 s{PADDR + 1}, s{PTMP}, %[rs]",
            f"s_add_u32 s{PADDR}, s{PADDR}, s{PTB}",
            f"s_addc_u32 s{PADDR + 1}, s{PADDR + 1}, s{PTB + 1}",
        ]
        if vec:
            L += [f"global_load_lds_dwordx4 %[vl], s[{PADDR}:{PADDR + 1}]",
                  "s_add_u32 m0, m0, 0x400"]
        else:
            for q in range(pieces):
                m = PCM + 2 * q
                if q:
                    L += [f"s_add_u32 s{PADDR}, s{PADDR}, 0x100",
                          f"s_addc_u32 s{PADDR + 1}, s{PADDR + 1}, 0"]
                L += [f"s_mov_b64 exec, s[{m}:{m + 1}]", "s_nop 0",
                      f"global_load_lds_dword %[vl], s[{PADDR}:{PADDR + 1}]",
                      "s_add_u32 m0, m0, 0x100"]
        L.append(f"s_add_u32 s{PROW}, s{PROW}, 1")
    return L


def issue_rows_clamped_narrow(half):
    """128-column tiles: stage rows PROW .. PROW+half-1 of B (each clamped to K-1) two per
    1 KB of LDS at m0, m0+1KB, ...: row r to lanes 0-31 (bytes 0-511 of the pair), row r+1
    to lanes 32-63, each half its own DMA with its own clamped row (%[vl] = 16 (lane % 32))."""
    L = []
    for r in range(half):
        L += [
            f"s_min_u32 s{PTMP}, s{PROW}, s{PKM1}",
            f"s_mul_i32 s{PADDR}, s{PTMP}, %[rs]",
            f"s_mul_hi_u32 s{PADDR + 1}, s{PTMP}, %[rs]",
            f"s_add_u32 s{PADDR}, s{PADDR}, s{PTB}",
            f"s_addc_u32 s{PADDR + 1}, s{PADDR + 1}, s{PTB + 1}",
        ]
        m = PCM + 2 + 2 * (r % 2)       # lanes 0-31, then lanes 32-63 (column-masked)
        L += [f"s_mov_b64 exec, s[{m}:{m + 1}]",
              f"global_load_lds_dwordx4 %[vl], s[{PADDR}:{PADDR + 1}]"]
        if r % 2:
            L.append("s_add_u32 m0, m0, 0x400")
        L.append(f"s_add_u32 s{PROW}, s{PROW}, 1")
    return L


# conv producer SGPRs: row bases (X + ic * plane + (ky - 1) * row_step, 64-bit, ky = 0..2),
# LDS row address, rows of the chunk below K, mask temp
RB, PRL, PNV, PMT, PXB = (66, 68, 70), 72, 73, 74, 76   # PXB: X itself (64-bit)
VZ, VA, VN = 36, 32, 33  # v[36:39] zeros, v32 zero-fill address, v33..v35 column offsets (the
                         # progress poll uses v40 and up)
CONV_OPERANDS = (
    ',\n        [rstep] "s"(a.row_step), [cstep] "s"(a.col_step), [plane] "s"(a.plane_bytes),\n'
    '        [vn] "v"(a.col_bytes), [dummy] "s"(a.dummy_lds),\n'
    '        [r0] "s"(a.rowmask[0]), [r1] "s"(a.rowmask[1]), [r2] "s"(a.rowmask[2]),\n'
    '        [c0] "s"(a.colmask[0]), [c1] "s"(a.colmask[1]), [c2] "s"(a.colmask[2])')


def issue_rows_conv(half):
    """Stage rows k0 .. k0+half-1 of the virtual B of a 3x3 convolution (stride 1,
    padding 1).  Row k is input channel k / 9 shifted by tap t = k % 9, (ky, kx) =
    (t / 3, t % 3): lane l's four columns n = n0 + 4l .. n0 + 4l + 3 are four images of
    one pixel (y, x), so they are the 16 bytes at
        RB[ky] + 4 n + (kx - 1) * NB * 4,   RB[ky] = X + ic * plane + (ky - 1) * W * NB * 4
    when (y + ky - 1, x + kx - 1) lies in the image, and zero otherwise.  The taps of a
    chunk's rows follow from t0 = k0 % 9, so the rows are generated once per t0 with
    static taps: the lane mask is rowmask[ky] & colmask[kx], the address is a row base
    plus one of three per-lane offsets, and the channel (the three row bases) advances
    after tap 8.  In-image lanes get the DMA, live lanes outside the image get zeros
    written to LDS; every row issues exactly one DMA (a one-lane load into a scratch
    LDS word when the row has no in-image lane or lies past K), so a chunk is always
    `half` loads and two chunks can be in flight."""
    lg_chunk = CHUNK.bit_length() - 1
    L = [
        f"s_mov_b32 s{PRL}, m0",
        # k0 = issued * CHUNK + prow0; rows of the chunk below K
        f"s_lshl_b32 s{PTMP}, s{PISS}, {lg_chunk}",
        f"s_add_u32 s{PTMP}, s{PTMP}, %[prow0]",
        f"s_sub_i32 s{PNV}, %[K], s{PTMP}",
        f"s_max_i32 s{PNV}, s{PNV}, 0",
        f"s_min_i32 s{PNV}, s{PNV}, {half}",
        # ic0 = k0 / 9 (multiply-high), t0 = k0 - 9 ic0
        f"s_mul_hi_u32 s{PROW}, s{PTMP}, 0x38e38e39",
        f"s_lshr_b32 s{PROW}, s{PROW}, 1",
        f"s_mul_i32 s{PADDR}, s{PROW}, 9",
        f"s_sub_u32 s{PTMP}, s{PTMP}, s{PADDR}",
        # row bases of channel ic0
        f"s_mul_i32 s{RB[1]}, s{PROW}, %[plane]",
        f"s_mul_hi_u32 s{RB[1] + 1}, s{PROW}, %[plane]",
        f"s_add_u32 s{RB[1]}, s{RB[1]}, %[bb_lo]",
        f"s_addc_u32 s{RB[1] + 1}, s{RB[1] + 1}, %[bb_hi]",
        f"s_sub_u32 s{RB[0]}, s{RB[1]}, %[rstep]",
        f"s_subb_u32 s{RB[0] + 1}, s{RB[1] + 1}, 0",
        f"s_add_u32 s{RB[2]}, s{RB[1]}, %[rstep]",
        f"s_addc_u32 s{RB[2] + 1}, s{RB[1] + 1}, 0",
    ]
    for t0 in range(9):
        L += [f"s_cmp_eq_u32 s{PTMP}, {t0}", f"s_cbranch_scc1 .L%=_cv{t0}"]
    L.append("s_branch .L%=_issued")          # unreachable: t0 < 9
    for t0 in range(9):
        L.append(f".L%=_cv{t0}:")
        for r in range(half):
            t = (t0 + r) % 9
            ky, kx = t // 3, t % 3
            tag = f"{t0}_{r}"
            L += [
                f"s_cmp_lt_u32 s{PNV}, {r + 1}",           # row past K
                f"s_cbranch_scc1 .L%=_cy{tag}",
                f"s_and_b64 s[{PMT}:{PMT + 1}], %[r{ky}], %[c{kx}]",
                f"s_andn2_b64 exec, s[{PCM}:{PCM + 1}], s[{PMT}:{PMT + 1}]",
                f"s_cbranch_execz .L%=_cz{tag}",
                f"v_add_u32 v{VA}, s{PRL}, %[vl]",
                f"ds_write_b128 v{VA}, v[{VZ}:{VZ + 3}]",
                f".L%=_cz{tag}:",
                f"s_mov_b64 exec, s[{PMT}:{PMT + 1}]",
                f"s_cbranch_execz .L%=_cy{tag}",
                f"global_load_lds_dwordx4 v{VN + kx}, s[{RB[ky]}:{RB[ky] + 1}]",
                f"s_branch .L%=_cn{tag}",
                f".L%=_cy{tag}:",                          # one-lane load to scratch LDS
                "s_mov_b32 m0, %[dummy]",
                "s_mov_b64 exec, 1",
                "s_nop 0",
                f"global_load_lds_dwordx4 %[vl], s[{PXB}:{PXB + 1}]",
                f".L%=_cn{tag}:",
                f"s_add_u32 s{PRL}, s{PRL}, 0x400",
                f"s_mov_b32 m0, s{PRL}",
            ]
            if t == 8 and r < half - 1:                    # next channel
                for b in RB:
                    L += [f"s_add_u32 s{b}, s{b}, %[plane]", f"s_addc_u32 s{b + 1}, s{b + 1}, 0"]
        L.append("s_branch .L%=_issued")
    return L


def producer(kind):
    """Producer loop (kind: "vec" 16-byte rows, "dword" 4-byte pieces, "conv" the virtual
    B of a 3x3 convolution, "vecn" 16-byte rows of 128-column tiles: two 512-byte rows
    per DMA, lanes 0-31 the first).  State: issued (chunks whose loads went out), landed
    (chunks published in the ready word), in flight = issued - landed <= PMAX, and the
    cached issue limit PLIM (re-read from the progress words only when issued reaches
    it).  vec: chunks below PLAST take the fast path: the chunk's base address advances
    by CHUNK rows per chunk and row r adds the lane's precomputed VGPR offset
    16 * lane + r * row_bytes, so each row is one DMA and one m0 step.  The last chunk
    when K is not a multiple of CHUNK, and every chunk of the 4-byte variant, take the
    clamped path, which re-stages row K-1 for rows past K (LDS rows no entry reads).
    conv: rows as in issue_rows_conv, `half` loads per chunk like vec."""
    narrow = kind == "vecn"
    lay = NARROW if narrow else WIDE
    vec = kind in ("vec", "conv", "vecn")
    conv = kind == "conv"
    half = CHUNK // lay.NPROD
    pmax = PMAX_VEC if vec else PMAX_DWORD
    # loads of a fast-path chunk (the clamped path of a narrow chunk issues twice as many,
    # which only makes the vmcnt waits below wait longer)
    loads_per_chunk = half // 2 if narrow else half if vec else 4 * half
    assert loads_per_chunk * (pmax - 1) <= 63
    lg_chunk = CHUNK.bit_length() - 1
    rs_lg = lay.ROW_SHIFT
    L = [
        f"s_mov_b32 s{PM0}, m0",
        f"s_mov_b32 s{PISS}, %[fc]",
        f"s_mov_b32 s{PSIG}, %[fc]",
        f"s_mov_b32 s{PINF}, 0",
        f"s_add_u32 s{PLIM}, %[fc], {RING}",
        f"s_mov_b32 s{PPOLL}, %[budget]",
        f"s_sub_u32 s{PKM1}, %[K], 1",
        # fast-path state: chunk base B + (c0 * CHUNK + prow0) * row_bytes, chunk stride
        # CHUNK * row_bytes
        f"s_lshl_b32 s{PTMP}, %[fc], {lg_chunk}",
        f"s_add_u32 s{PTMP}, s{PTMP}, %[prow0]",
        f"s_mul_i32 s{PBASE}, s{PTMP}, %[rs]",
        f"s_mul_hi_u32 s{PBASE + 1}, s{PTMP}, %[rs]",
        f"s_add_u32 s{PBASE}, s{PBASE}, %[bb_lo]",
        f"s_addc_u32 s{PBASE + 1}, s{PBASE + 1}, %[bb_hi]",
        f"s_lshl_b32 s{PCS}, %[rs], {lg_chunk}",
        f"s_lshr_b32 s{PCS + 1}, %[rs], {32 - lg_chunk}",
        f"s_mov_b64 s[{PB0}:{PB0 + 1}], s[{PBASE}:{PBASE + 1}]",
        f"s_mov_b32 s{PCI}, %[fc]",
        f"s_mov_b32 s{PRB}, %[rb0]",
        f"s_mov_b32 s{PTB}, %[bb_lo]",
        f"s_mov_b32 s{PTB + 1}, %[bb_hi]",
    ]
    if kind == "vec":  # PLAST = K / CHUNK: chunks below it hold CHUNK rows of B
        L += [f"s_lshr_b32 s{PLAST}, %[K], {lg_chunk}",
              f"v_mov_b32 v{VO}, %[vl]"]
        for r in range(1, half):
            L.append(f"v_add_u32 v{VO + r}, %[rs], v{VO + r - 1}")
    elif narrow:  # v[VO + j] = %[vf] + 2 j row_bytes (%[vf]: lanes 32-63 one row on)
        L += [f"s_lshr_b32 s{PLAST}, %[K], {lg_chunk}",
              f"v_mov_b32 v{VO}, %[vf]",
              f"s_lshl_b32 s{PTMP}, %[rs], 1"]
        for r in range(1, half // 2):
            L.append(f"v_add_u32 v{VO + r}, s{PTMP}, v{VO + r - 1}")
    else:
        L.append(f"s_mov_b32 s{PLAST}, 0")
    if conv:
        L += [f"v_mov_b32 v{VZ + q}, 0" for q in range(4)]
        L += [f"v_subrev_u32 v{VN}, %[cstep], %[vn]",      # 4 n - NB * 4 (kx = 0)
              f"v_mov_b32 v{VN + 1}, %[vn]",                # 4 n           (kx = 1)
              f"v_add_u32 v{VN + 2}, %[cstep], %[vn]",      # 4 n + NB * 4  (kx = 2)
              f"s_mov_b32 s{PXB}, %[bb_lo]",
              f"s_mov_b32 s{PXB + 1}, %[bb_hi]"]
    # column masks: vec -> lanes whose 4 columns exist (lane < ncol / 4);
    # dword -> piece q of a row: lanes with 64 q + lane < ncol;
    # vecn -> lanes with lane % 32 < ncol / 4 (both rows of a pair), then the lanes 0-31
    # and the lanes 32-63 of that mask
    pieces = 3 if narrow else 1 if vec else 4
    if narrow:
        L += [
            f"s_lshr_b32 s{PTMP}, %[ncol], 2",
            f"s_min_u32 s{PTMP}, s{PTMP}, 32",
            f"s_bfm_b64 s[{PCM}:{PCM + 1}], s{PTMP}, 0",
            f"s_mov_b32 s{PCM + 1}, s{PCM}",
            f"s_mov_b32 s{PCM + 2}, s{PCM}",
            f"s_mov_b32 s{PCM + 3}, 0",
            f"s_mov_b32 s{PCM + 4}, 0",
            f"s_mov_b32 s{PCM + 5}, s{PCM}",
        ]
    for q in range(0 if narrow else pieces):
        m = PCM + 2 * q
        if vec:
            L.append(f"s_lshr_b32 s{PTMP}, %[ncol], 2")
        else:
            L += [f"s_sub_i32 s{PTMP}, %[ncol], {64 * q}", f"s_max_i32 s{PTMP}, s{PTMP}, 0"]
        L += [
            f"s_min_u32 s{PTMP}, s{PTMP}, 64",
            f"s_bfm_b64 s[{m}:{m + 1}], s{PTMP}, 0",
            f"s_cmp_ge_u32 s{PTMP}, 64",
            f"s_cselect_b64 s[{m}:{m + 1}], -1, s[{m}:{m + 1}]",
        ]
    L += [
        ".L%=_loop:",
        f"s_cmp_ge_u32 s{PSIG}, %[nch]",
        "s_cbranch_scc1 .L%=_done",
        f"s_cmp_ge_u32 s{PISS}, %[nch]",
        "s_cbranch_scc1 .L%=_land",
        f"s_cmp_ge_u32 s{PINF}, {pmax}",
        "s_cbranch_scc1 .L%=_land",
        f"s_cmp_lt_u32 s{PISS}, s{PLIM}",
        "s_cbranch_scc1 .L%=_issue",
    ]
    L += producer_poll()
    L += [
        f"s_cmp_lt_u32 s{PISS}, s{PLIM}",
        "s_cbranch_scc1 .L%=_issue",
        f"s_cmp_eq_u32 s{PINF}, 0",
        "s_cbranch_scc0 .L%=_land",
        f"s_cmp_eq_u32 s{PPOLL}, 0",          # budget spent: stage anyway
        "s_cbranch_scc1 .L%=_overrun",
        f"s_sub_u32 s{PPOLL}, s{PPOLL}, 1",
        "s_sleep 1",
        "s_branch .L%=_loop",
        # staging past the limit may overwrite a slot still being read: say so in the
        # overrun word (landed before the load goes out) and go on to issue
        ".L%=_overrun:",
        "v_mov_b32 v27, 1",
        f"s_mov_b64 s[{PEX}:{PEX + 1}], exec",
        "s_mov_b64 exec, 1",
        "ds_write_b32 %[ov], v27",
        "s_waitcnt lgkmcnt(0)",
        f"s_mov_b64 exec, s[{PEX}:{PEX + 1}]",
        # LDS row of the producer's first row of chunk `issued`:
        # (issued % RING) * CHUNK + prow0
        ".L%=_issue:",
        f"s_and_b32 s{PTMP}, s{PISS}, {RING - 1}",
        f"s_lshl_b32 s{PTMP}, s{PTMP}, {lg_chunk + rs_lg}",
        f"s_lshl_b32 m0, %[prow0], {rs_lg}",
        f"s_add_u32 m0, m0, s{PTMP}",
        f"s_mov_b64 s[{PEX}:{PEX + 1}], exec",
    ]
    if conv:
        L += issue_rows_conv(half)
    else:
        L += [f"s_cmp_lt_u32 s{PCI}, s{PLAST}", "s_cbranch_scc0 .L%=_clamped"]
        if vec:
            L.append(f"s_mov_b64 exec, s[{PCM}:{PCM + 1}]")   # also spaces the m0 write from the DMA
            for r in range(loads_per_chunk):
                if r:
                    L.append("s_nop 0")                       # m0 write, then a DMA reading it
                L += [f"global_load_lds_dwordx4 v{VO + r}, s[{PBASE}:{PBASE + 1}]",
                      "s_add_u32 m0, m0, 0x400"]
            L.append("s_branch .L%=_issued")
        L += [".L%=_clamped:",
              f"s_lshl_b32 s{PROW}, s{PCI}, {lg_chunk}",
              f"s_add_u32 s{PROW}, s{PROW}, %[prow0]"]
        L += issue_rows_clamped_narrow(half) if narrow else issue_rows_clamped(vec, half)
    L += [
        ".L%=_issued:",
        f"s_mov_b64 exec, s[{PEX}:{PEX + 1}]",
        f"s_add_u32 s{PBASE}, s{PBASE}, s{PCS}",
        f"s_addc_u32 s{PBASE + 1}, s{PBASE + 1}, s{PCS + 1}",
        f"s_add_u32 s{PISS}, s{PISS}, 1",
        f"s_add_u32 s{PINF}, s{PINF}, 1",
        # the next item restages its tile's rows from the start: the same tile (the
        # tile's next row-block), or, for tile-major items, dtile tiles on plus one more
        # when the row-block index wraps past the tile's row-blocks
        f"s_add_u32 s{PCI}, s{PCI}, 1",
        f"s_cmp_lt_u32 s{PCI}, %[nci]",
        "s_cbranch_scc1 .L%=_loop",
        f"s_mov_b32 s{PCI}, 0",
        f"s_add_u32 s{PRB}, s{PRB}, %[drb]",
        f"s_cmp_lt_u32 s{PRB}, %[nrb]",
        "s_cbranch_scc1 .L%=_samerb",
        f"s_sub_u32 s{PRB}, s{PRB}, %[nrb]",
        f"s_add_u32 s{PB0}, s{PB0}, {lay.ROW_BYTES}",
        f"s_addc_u32 s{PB0 + 1}, s{PB0 + 1}, 0",
        f"s_add_u32 s{PTB}, s{PTB}, {lay.ROW_BYTES}",
        f"s_addc_u32 s{PTB + 1}, s{PTB + 1}, 0",
        ".L%=_samerb:",
        f"s_add_u32 s{PB0}, s{PB0}, %[dtb]",
        f"s_addc_u32 s{PB0 + 1}, s{PB0 + 1}, 0",
        f"s_add_u32 s{PTB}, s{PTB}, %[dtb]",
        f"s_addc_u32 s{PTB + 1}, s{PTB + 1}, 0",
        f"s_mov_b64 s[{PBASE}:{PBASE + 1}], s[{PB0}:{PB0 + 1}]",
        "s_branch .L%=_loop",
        # wait for the oldest chunk in flight (loads complete in order), publish it
        ".L%=_land:",
    ]
    for n in range(pmax, 1, -1):
        L += [f"s_cmp_eq_u32 s{PINF}, {n}", f"s_cbranch_scc0 .L%=_land{n}",
              f"s_waitcnt vmcnt({loads_per_chunk * (n - 1)})", "s_branch .L%=_landed",
              f".L%=_land{n}:"]
    L += [
        "s_waitcnt vmcnt(0)",
        ".L%=_landed:",
        f"s_add_u32 s{PSIG}, s{PSIG}, 1",
        f"s_sub_u32 s{PINF}, s{PINF}, 1",
        f"v_mov_b32 v27, s{PSIG}",
        f"s_mov_b64 s[{PEX}:{PEX + 1}], exec",
        "s_mov_b64 exec, 1",
        "ds_write_b32 %[ra], v27",
        f"s_mov_b64 exec, s[{PEX}:{PEX + 1}]",
        "s_branch .L%=_loop",
        ".L%=_done:",
        "s_waitcnt vmcnt(0) lgkmcnt(0)",
        f"s_mov_b32 m0, s{PM0}",
    ]
    body = "\n".join('      "' + x + '\\n\\t"' for x in L)
    sregs = [f"s{x}" for x in list(range(PISS, PCM + 2 * pieces)) + [PKM1, PLAST, PCI, PRB, PB0, PB0 + 1,
                                                                    PTB, PTB + 1]]
    if conv:
        sregs += [f"s{x}" for x in range(RB[0], PXB + 2)]
    vregs = ["v27"] + [f"v{x}" for x in range(VO, VMIN + 5)]
    clob = ", ".join(f'"{r}"' for r in sregs + vregs + ["vcc", "scc", "memory"])
    title = {"vec": "16-byte staging", "dword": "4-byte staging",
             "conv": "the virtual B of a 3x3 convolution",
             "vecn": "16-byte staging of 128-column tiles"}[kind]
    return f"""// Producer, {title}
__device__ __forceinline__ void produce_{kind}(const ProducerArgs& a) {{
  asm volatile(
{body}
      :
      : [nch] "s"(a.nchunks), [K] "s"(a.K), [rs] "s"(a.row_bytes), [bb_lo] "s"(a.bbase_lo),
        [bb_hi] "s"(a.bbase_hi), [ncol] "s"(a.ncol), [prow0] "s"(a.first_row),
        [vl] "v"(a.vlane), [pg] "v"(a.prog_addr), [ra] "v"(a.ready_addr),
        [budget] "s"(a.poll_budget), [ov] "v"(a.overrun_addr), [fc] "s"(a.first_chunk),
        [nci] "s"(a.item_chunks), [rb0] "s"(a.item_rb), [drb] "s"(a.item_drb),
        [nrb] "s"(a.item_nrb), [dtb] "s"(a.item_dtile_bytes){CONV_OPERANDS if conv else ""}{', [vf] "v"(a.vlane_fast)' if narrow else ""}
      : {clob});
}}
"""


def generate() -> str:
    parts = ["// Generated by gen_spmm_asm.py -- do not edit by hand.",
             "#pragma once", "",
             "// zero groups the stream must carry past its last panel: the scalar ring runs",
             "// NSLOT-1 groups ahead and the L2 touch a further TOUCH_AHEAD bytes",
             f"constexpr int kStreamTailGroups = {NSLOT - 1 + (TOUCH_AHEAD + GROUP_BYTES - 1) // GROUP_BYTES + 1};",
             "// stream and ring layout the loops assume",
             f"constexpr int kAsmChunk = {CHUNK}, kAsmRing = {RING}, kAsmProducers = {NPROD};",
             f"constexpr int kAsmTileBytes = {TILE_BYTES};",
             f"constexpr int kAsmMaxConsumers = {MAX_CONS};",
             f"constexpr int kAsmGroup = {G}, kAsmAccBase = {ACC};",
             f"constexpr int kAsmEndBit = {END_BIT}, kAsmSyncBit = {SYNC_BIT};",
             f"constexpr int kAsmLoShift = {LO_SHIFT}, kAsmHiShift = {HI_SHIFT};",
             f"constexpr uint32_t kAsmRingMask = {hex(RING_MASK)}u;",
             "// the same for 128-column tiles",
             f"constexpr int kAsmProducersN = {NARROW.NPROD}, kAsmTileBytesN = {NARROW.ROW_BYTES};",
             f"constexpr int kAsmAccBaseN = {NARROW.ACC}, kAsmEndBitN = {NARROW.END_BIT};",
             f"constexpr uint32_t kAsmRingMaskN = {hex(NARROW.RING_MASK)}u;",
             f"constexpr uint32_t kProgressDone = {hex(INF)}u;",
             ""]
    for rw in RW_VARIANTS:
        parts.append(consumer(rw))
        parts.append(consumer(rw, limit=True))
    for rw in RW_VARIANTS_NARROW:
        parts.append(consumer(rw, lay=NARROW))
        parts.append(consumer(rw, limit=True, lay=NARROW))
    for kind in ("vec", "dword", "conv", "vecn"):
        parts.append(producer(kind))
    return "\n".join(parts)


def main(check: bool = False) -> int:
    text = generate()
    if check:
        return 0 if os.path.exists(OUT) and open(OUT).read() == text else 1
    with open(OUT, "w") as f:
        f.write(text)
    return 0


if __name__ == "__main__":
    sys.exit(main(check="--check" in sys.argv))
