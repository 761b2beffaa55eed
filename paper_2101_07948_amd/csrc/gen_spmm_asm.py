"""Generates spmm_asm_gen.h: the K-loop of the gfx950 panel kernel as inline assembly,
one function per (panel height RW, staging width).

Why generated assembly: the loop keeps a wavefront's RW x 4 output tile in fixed VGPRs
and selects the row of each nonzero with VGPR index mode (s_set_gpr_idx_*), and it
software-pipelines scalar loads of the weight stream, LDS reads of B and FMAs across
rotating register sets that must keep their state across K-chunks.  Compiled code can
express neither the indexed accumulator nor the persistent rotation.

Stream consumed (see sdnn_internal.h): for each panel, the segments of chunks
0..nchunks-1 back to back; a segment is >= 1 group; a group is 8 dwords
[w0 w1 w2 w3 a0 a1 a2 a3], w = fp32 weight bits, a = (column in chunk << 10) | row,
and bit 9 of a3 marks the last group of a segment.

Register plan (pinned in the asm statement):
  v30             LDS byte address of this lane's 16 bytes in the current B buffer
  v31             0xfc00 (column-offset mask)
  v[32:47]        B values of the group being multiplied / being fetched (2 sets of 4 x 4)
  v[48:63]
  v[64 + k*RW + r]  accumulator of row r, column 4*lane + k   (k = 0..3)
  v25             N * 4 (B row stride in bytes); v[26:27] B row address being staged
  v28, v29        zero offset / sink of the L2 touch loads
  s[40:79]        ring of NSLOT = 5 stream groups (8 SGPRs each)
  s[80:81]        address of the next group to fetch
  s82 phase (position in the unrolled loop), s83 saved m0, s84 next chunk to compute,
  s85 chunk being staged, s[86:87] column mask, s88 LDS buffer being staged, s89 row,
  s90 temp, s[92:93] saved exec
The staging buffers are at LDS byte addresses 0 and 64 KB (the kernel checks this).
A wave without a panel passes a null stream address: it stages B and takes part in
every barrier but runs no FMAs.

Per group g:
  wait until B of g and stream group g+1 have arrived
  address + ds_read_b128 of the 4 B rows of group g+1      (index mode off)
  s_load of stream group g+NSLOT-1 into the slot that group g-1 used
  for each entry: s_set_gpr_idx_* row; 4 v_fma_f32 into the row's accumulators
  (index mode DST|SRC2: only the accumulator operand is offset by the row)
  if g ends its segment: leave to the chunk transition, remembering the phase
Chunk transition (every wave, active or not, executes it once per chunk):
  wait for this wave's B DMA, s_barrier (all DMA of the chunk landed; every wave is done
  with the other buffer), DMA of the chunk after the one about to be computed into the
  free buffer, switch the LDS read base, re-issue the LDS reads of the current group
  from the new buffer, and re-enter the unrolled loop at the saved phase.
Scalar loads run NSLOT-2 groups ahead of their first use and continue across chunks.
Each iteration also issues a vector load (result unused, waited for only at the next
barrier) TOUCH_AHEAD bytes ahead of the ring pointer: it brings the stream into L2, so
scalar-cache misses are served from L2 instead of the memory-side cache or HBM.
The ring and the touch read up to kStreamTailGroups groups past a panel's last
segment; the stream carries that many zero groups at its end so those reads stay
inside it, and LDS reads stay inside the B buffer because every column offset is < 64.
"""
import math
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "spmm_asm_gen.h")

NSLOT = 5
E = tuple(40 + 8 * i for i in range(NSLOT))  # SGPR bases of the stream-group ring
PTR, PHASE, M0S, KNEXT, DCH, CMASK = 80, 82, 83, 84, 85, 86
DBUF, DROW, DTMP, DEXEC = 88, 89, 90, 92
SLAST = 93
VB = (32, 48)                                 # VGPR bases of the two B-value sets
ACC = 64                                      # first accumulator VGPR
UNROLL = NSLOT * 2 // math.gcd(NSLOT, 2)
RW_VARIANTS = (4, 8, 12, 16)
END_BIT = 9
TOUCH_AHEAD = 512  # bytes of stream pulled into L2 ahead of the scalar ring
PROFILE = False    # scratch builds only: time spent in chunk transitions (%[tbar])


def address_phase(slot, vb):
    L = []
    for j in range(4):
        L.append(f"v_and_or_b32 v{vb + 4 * j}, s{slot + 4 + j}, v31, v30")
        L.append(f"ds_read_b128 v[{vb + 4 * j}:{vb + 4 * j + 3}], v{vb + 4 * j}")
    return L


def iteration(i, rw):
    cur, nxt, pre = E[i % NSLOT], E[(i + 1) % NSLOT], E[(i + NSLOT - 1) % NSLOT]
    vbc, vbn = VB[i % 2], VB[(i + 1) % 2]
    L = [f".L%=_iter{i}:", "s_waitcnt lgkmcnt(0)"]
    L += address_phase(nxt, vbn)
    L.append(f"s_load_dwordx8 s[{pre}:{pre + 7}], s[{PTR}:{PTR + 1}], 0x0")
    if TOUCH_AHEAD:  # pull the stream line TOUCH_AHEAD bytes ahead into L2 (vector path)
        L.append(f"global_load_dword v29, v28, s[{PTR}:{PTR + 1}] offset:{TOUCH_AHEAD}")
    L.append(f"s_add_u32 s{PTR}, s{PTR}, 32")
    L.append(f"s_addc_u32 s{PTR + 1}, s{PTR + 1}, 0")
    for j in range(4):
        if j == 0:
            L.append(f"s_set_gpr_idx_on s{cur + 4}, gpr_idx(DST,SRC2)")
        else:
            L.append(f"s_set_gpr_idx_idx s{cur + 4 + j}")
        for k in range(4):
            p = ACC + k * rw
            L.append(f"v_fma_f32 v{p}, s{cur + j}, v{vbc + 4 * j + k}, v{p}")
    L.append("s_set_gpr_idx_off")
    L.append(f"s_bitcmp1_b32 s{cur + 7}, {END_BIT}")
    L.append(f"s_cbranch_scc1 .L%=_exit{i}")
    return L


def dma(tag, vec):
    """Stage chunk DCH (if < nch) into buffer DCH & 1: rows wave, wave+nw, ... < 64.
    The B row address is formed in v[26:27] from the tile base %[vb] (64-bit) and the
    row stride v25 (one v_mad_u64_u32 per row)."""
    L = [
        f"s_cmp_ge_u32 s{DCH}, %[nch]",
        f"s_cbranch_scc1 .L%=_dmadone{tag}",
        f"s_and_b32 s{DBUF}, s{DCH}, 1",
        f"s_lshl_b32 s{DBUF}, s{DBUF}, 16",
        f"s_mov_b32 s{DROW}, %[wave]",
        f".L%=_dmaloop{tag}:",
        f"s_cmp_ge_u32 s{DROW}, 64",
        f"s_cbranch_scc1 .L%=_dmadone{tag}",
        f"s_lshl_b32 s{DTMP}, s{DCH}, 6",
        f"s_add_u32 s{DTMP}, s{DTMP}, s{DROW}",
        f"s_cmp_ge_u32 s{DTMP}, %[K]",
        f"s_cbranch_scc1 .L%=_dmadone{tag}",
        f"v_mad_u64_u32 v[26:27], vcc, s{DTMP}, v25, %[vb]",
        f"s_lshl_b32 m0, s{DROW}, 10",
        f"s_add_u32 m0, m0, s{DBUF}",
    ]
    if vec:
        L += [
            f"s_and_saveexec_b64 s[{DEXEC}:{DEXEC + 1}], s[{CMASK}:{CMASK + 1}]",
            "s_nop 0",
            "global_load_lds_dwordx4 v[26:27], off",
            f"s_mov_b64 exec, s[{DEXEC}:{DEXEC + 1}]",
        ]
    else:
        for q in range(4):
            if q:
                L += ["s_add_u32 m0, m0, 0x100", "v_add_co_u32 v26, vcc, 0x100, v26",
                      "v_addc_co_u32 v27, vcc, 0, v27, vcc"]
            L += [
                f"s_sub_i32 s{DTMP}, %[ncol], {64 * q}",
                f"v_cmp_gt_i32 vcc, s{DTMP}, %[lanev]",
                f"s_and_saveexec_b64 s[{DEXEC}:{DEXEC + 1}], vcc",
                "s_nop 0",
                "global_load_lds_dword v[26:27], off",
                f"s_mov_b64 exec, s[{DEXEC}:{DEXEC + 1}]",
            ]
    L += [
        f"s_add_u32 s{DROW}, s{DROW}, %[nw]",
        f"s_branch .L%=_dmaloop{tag}",
        f".L%=_dmadone{tag}:",
    ]
    return L


def function(rw, vec):
    L = [
        f"s_mov_b32 s{M0S}, m0",
        "v_mov_b32 v31, 0xfc00",
        "v_mov_b32 v28, 0",
        "v_mov_b32 v25, %[rs]",
        f"s_mov_b32 s{KNEXT}, 0",
        f"s_mov_b32 s{PHASE}, 0",
    ]
    if vec:  # lanes whose 4 columns lie inside N: lane < ncol / 4
        L += [
            f"s_lshr_b32 s{DTMP}, %[ncol], 2",
            f"s_min_u32 s{DTMP}, s{DTMP}, 64",
            f"s_bfm_b64 s[{CMASK}:{CMASK + 1}], s{DTMP}, 0",
            f"s_cmp_ge_u32 s{DTMP}, 64",
            f"s_cselect_b64 s[{CMASK}:{CMASK + 1}], -1, s[{CMASK}:{CMASK + 1}]",
        ]
    L += [
        "s_cmp_eq_u64 %[sp], 0",
        "s_cbranch_scc1 .L%=_pro_idle",
    ]
    for g in range(NSLOT - 1):
        L.append(f"s_load_dwordx8 s[{E[g]}:{E[g] + 7}], %[sp], {hex(32 * g)}")
    L += [
        f"s_mov_b64 s[{PTR}:{PTR + 1}], %[sp]",
        f"s_add_u32 s{PTR}, s{PTR}, {32 * (NSLOT - 1)}",
        f"s_addc_u32 s{PTR + 1}, s{PTR + 1}, 0",
        ".L%=_pro_idle:",
        f"s_mov_b32 s{DCH}, 0",
    ]
    L += dma("p", vec)
    # chunk transition
    L += [
        ".L%=_trans:",
        f"s_cmp_ge_u32 s{KNEXT}, %[nch]",
        "s_cbranch_scc1 .L%=_finish",
    ]
    if PROFILE:  # cycles spent waiting for the DMA and the barrier
        L += [f"s_memtime s[{DEXEC}:{DEXEC + 1}]", "s_waitcnt lgkmcnt(0)"]
    L += [
        "s_waitcnt vmcnt(0)",
        "s_barrier",
    ]
    if PROFILE:  # scratch builds also pin s[94:95]
        L += ["s_memtime s[94:95]", "s_waitcnt lgkmcnt(0)",
              f"s_sub_u32 s94, s94, s{DEXEC}", "s_add_u32 %[tbar], %[tbar], s94"]
    L += [f"s_add_u32 s{DCH}, s{KNEXT}, 1"]
    L += dma("t", vec)
    L += [
        f"s_bitcmp1_b32 s{KNEXT}, 0",
        "s_cselect_b64 vcc, -1, 0",
        "v_cndmask_b32 v30, %[vl0], %[vl1], vcc",
        f"s_add_u32 s{KNEXT}, s{KNEXT}, 1",
        "s_cmp_eq_u64 %[sp], 0",
        "s_cbranch_scc1 .L%=_trans",
    ]
    for p in range(UNROLL):
        L += [f"s_cmp_eq_u32 s{PHASE}, {p}", f"s_cbranch_scc1 .L%=_entry{p}"]
    L.append("s_branch .L%=_finish")  # unreachable: phase is always < UNROLL
    for p in range(UNROLL):
        L.append(f".L%=_entry{p}:")
        L.append("s_waitcnt lgkmcnt(0)")
        L += address_phase(E[p % NSLOT], VB[p % 2])
        L.append(f"s_branch .L%=_iter{p}")
    for i in range(UNROLL):
        L += iteration(i, rw)
    L.append("s_branch .L%=_iter0")
    for i in range(UNROLL):
        L += [f".L%=_exit{i}:", f"s_mov_b32 s{PHASE}, {(i + 1) % UNROLL}", "s_branch .L%=_trans"]
    L += [
        ".L%=_finish:",
        "s_waitcnt vmcnt(0) lgkmcnt(0)",
        f"s_mov_b32 m0, s{M0S}",
    ]
    if PROFILE:
        L.insert(0, "s_mov_b32 %[tbar], 0")
    body = "\n".join('      "' + x + '\\n\\t"' for x in L)
    planes = ", ".join(f'"+{{v[{ACC + k * rw}:{ACC + k * rw + rw - 1}]}}"(p{k})' for k in range(4))
    sregs = [f"s{x}" for x in range(E[0], (95 if PROFILE else SLAST) + 1)]
    vregs = [f"v{x}" for x in range(25, 64)]
    # exec is changed only around each DMA and restored right after it
    clob = ", ".join(f'"{r}"' for r in sregs + vregs + ["vcc", "scc"])
    suffix = "vec" if vec else "dword"
    return f"""// RW = {rw}, {"16-byte" if vec else "4-byte"} staging: accumulator planes p0..p3
__device__ __forceinline__ void kloop_{suffix}(acc_plane_t<{rw}>& p0, acc_plane_t<{rw}>& p1,
                                         acc_plane_t<{rw}>& p2, acc_plane_t<{rw}>& p3,
                                         const KloopArgs& a) {{
  asm volatile(
{body}
      : {planes}{', [tbar] "=&s"(a.tbar)' if PROFILE else ''}
      : [sp] "s"(a.stream), [nch] "s"(a.nchunks), [rs] "s"(a.row_bytes), [K] "s"(a.K),
        [wave] "s"(a.wave), [nw] "s"(a.nwaves), [ncol] "s"(a.ncol), [vb] "v"(a.vbase),
        [vl0] "v"(a.vl0), [vl1] "v"(a.vl1), [lanev] "v"(a.lane)
      : {clob});
}}
"""


def generate() -> str:
    parts = ["// Generated by gen_spmm_asm.py -- do not edit by hand.",
             "#pragma once", "",
             "// zero groups the stream must carry past its last segment: the scalar ring runs",
             "// NSLOT-1 groups ahead and the L2 touch a further TOUCH_AHEAD bytes",
             f"constexpr int kStreamTailGroups = {NSLOT - 1 + (TOUCH_AHEAD + 31) // 32 + 1};",
             "// bit of a group's last column word that marks the end of a segment",
             f"constexpr uint32_t kSegmentEndBit = 1u << {END_BIT};", ""]
    for rw in RW_VARIANTS:
        for vec in (True, False):
            parts.append(function(rw, vec))
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
