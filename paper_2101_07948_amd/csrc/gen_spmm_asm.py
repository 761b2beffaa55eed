"""Generates spmm_asm_gen.h: the per-K-chunk inner loop of the gfx950 panel kernel as
inline assembly, one function per panel height RW.

Why generated assembly: the loop keeps a wavefront's RW x 4 output tile in fixed
VGPRs and selects the row of each nonzero with VGPR index mode (s_set_gpr_idx_*),
and it software-pipelines three kinds of latency (scalar loads of the weight stream,
LDS reads of B, FMAs) across rotating register sets.  Compiled code cannot express the
indexed accumulator and re-orders/copies the rotating sets.

Stream consumed (see sdnn_internal.h): a segment of `ng` groups; a group is 8 dwords
[w0 w1 w2 w3 a0 a1 a2 a3] with w = fp32 weight bits and a = (column in chunk << 10) | row.

Register plan (all pinned in the asm statement):
  v31             0xfc00 (column-offset mask)
  v[32:47]        B values of the group being multiplied / being fetched (2 sets of 4 x 4)
  v[48:63]
  v[64 + 4*k ...] accumulator plane k (k = 0..3, column 4*lane + k), RW VGPRs each:
                  plane k, row r lives in v[64 + k*RW + r]
  s[40:79]        ring of NSLOT = 5 stream groups (8 SGPRs each)
  s[80:81]        pointer to the next group to fetch, s82 groups left, s83 saved m0

Per group g (all rows of the wavefront's panel are interleaved in one flat stream):
  wait until B of g and stream group g+1 have arrived
  address + ds_read_b128 of the 4 B rows of group g+1      (index mode off)
  s_load of stream group g+NSLOT-1 into the slot group g-1 used
  for each entry: s_set_gpr_idx_* row; 4 v_fma_f32 into the row's accumulators
  (index mode DST|SRC2: only the accumulator operand is offset by the row)
Scalar loads run NSLOT-2 groups ahead of their first use (the address phase), so an L2
miss of the scalar cache is hidden behind several groups of FMAs.  The loop body is
unrolled over lcm(NSLOT, 2) groups so that every register set is named statically.
The last iterations prefetch up to NSLOT-1 groups past the segment; the stream carries
that many zero groups at its end so those reads stay inside it, and LDS reads stay
inside the chunk buffer because every column offset is < 64.
"""
import math
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(HERE, "spmm_asm_gen.h")

NSLOT = 5
E = tuple(40 + 8 * i for i in range(NSLOT))  # SGPR bases of the stream-group ring
SPTR, SCNT, SM0 = 80, 82, 83
VB = (32, 48)     # VGPR bases of the two B-value sets
ACC = 64          # first accumulator VGPR
RW_VARIANTS = (4, 8, 12, 16)


def iteration(i, rw):
    cur, nxt, pre = E[i % NSLOT], E[(i + 1) % NSLOT], E[(i + NSLOT - 1) % NSLOT]
    vbc, vbn = VB[i % 2], VB[(i + 1) % 2]
    L = ["s_waitcnt lgkmcnt(0)"]
    for j in range(4):
        L.append(f"v_and_or_b32 v{vbn + 4 * j}, s{nxt + 4 + j}, v31, %[vl]")
        L.append(f"ds_read_b128 v[{vbn + 4 * j}:{vbn + 4 * j + 3}], v{vbn + 4 * j}")
    L.append(f"s_load_dwordx8 s[{pre}:{pre + 7}], s[{SPTR}:{SPTR + 1}], 0x0")
    L.append(f"s_add_u32 s{SPTR}, s{SPTR}, 32")
    L.append(f"s_addc_u32 s{SPTR + 1}, s{SPTR + 1}, 0")
    for j in range(4):
        if j == 0:
            L.append(f"s_set_gpr_idx_on s{cur + 4}, gpr_idx(DST,SRC2)")
        else:
            L.append(f"s_set_gpr_idx_idx s{cur + 4 + j}")
        for k in range(4):
            p = ACC + k * rw
            L.append(f"v_fma_f32 v{p}, s{cur + j}, v{vbc + 4 * j + k}, v{p}")
    L.append("s_set_gpr_idx_off")
    L.append(f"s_sub_u32 s{SCNT}, s{SCNT}, 1")
    L.append(f"s_cmp_eq_u32 s{SCNT}, 0")
    L.append("s_cbranch_scc1 .L%=_done")
    return L


def function(rw):
    L = [
        f"s_mov_b32 s{SM0}, m0",
        "v_mov_b32 v31, 0xfc00",
        "s_cmp_eq_u32 %[ng], 0",
        "s_cbranch_scc1 .L%=_end",
    ]
    # groups 0 .. NSLOT-2 into slots 0 .. NSLOT-2
    for g in range(NSLOT - 1):
        L.append(f"s_load_dwordx8 s[{E[g]}:{E[g] + 7}], %[seg], {hex(32 * g)}")
    L += [
        f"s_mov_b64 s[{SPTR}:{SPTR + 1}], %[seg]",
        f"s_add_u32 s{SPTR}, s{SPTR}, {32 * (NSLOT - 1)}",
        f"s_addc_u32 s{SPTR + 1}, s{SPTR + 1}, 0",
        f"s_mov_b32 s{SCNT}, %[ng]",
        "s_waitcnt lgkmcnt(0)",
    ]
    for j in range(4):
        L.append(f"v_and_or_b32 v{VB[0] + 4 * j}, s{E[0] + 4 + j}, v31, %[vl]")
        L.append(f"ds_read_b128 v[{VB[0] + 4 * j}:{VB[0] + 4 * j + 3}], v{VB[0] + 4 * j}")
    L.append(".L%=_loop:")
    unroll = NSLOT * 2 // math.gcd(NSLOT, 2)
    for i in range(unroll):
        L.extend(iteration(i, rw))
    L.append("s_branch .L%=_loop")
    L.append(".L%=_done:")
    L.append("s_waitcnt lgkmcnt(0)")
    L.append(".L%=_end:")
    L.append(f"s_mov_b32 m0, s{SM0}")
    body = "\n".join('      "' + x + '\\n\\t"' for x in L)
    planes = ", ".join(f'"+{{v[{ACC + k * rw}:{ACC + k * rw + rw - 1}]}}"(p{k})' for k in range(4))
    sregs = [f"s{x}" for x in range(E[0], SM0 + 1)]
    vregs = [f"v{x}" for x in range(31, 64)]
    clob = ", ".join(f'"{r}"' for r in sregs + vregs + ["scc"])
    return f"""// RW = {rw}: accumulator planes p0..p3 (column 4*lane + k, rows 0..{rw - 1})
__device__ __forceinline__ void chunk_fma_asm(acc_plane_t<{rw}>& p0, acc_plane_t<{rw}>& p1,
                                              acc_plane_t<{rw}>& p2, acc_plane_t<{rw}>& p3,
                                              const uint32_t* seg, int32_t ng, uint32_t vl) {{
  asm volatile(
{body}
      : {planes}
      : [seg] "s"(seg), [ng] "s"(ng), [vl] "v"(vl)
      : {clob});
}}
"""


def generate() -> str:
    parts = ["// Generated by gen_spmm_asm.py -- do not edit by hand.",
             "#pragma once", "",
             f"// zero groups the stream must carry past its last segment",
             f"constexpr int kStreamTailGroups = {NSLOT - 1};", ""]
    for rw in RW_VARIANTS:
        parts.append(function(rw))
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
