// gfx950 kernels of the sparse-weight x dense-activation product (SparseDNN, arXiv
// 2101.07948, Sec. 3.2.2) and the dense FP32 comparison GEMM (Sec. 3.2.1).
//
// Sparse kernel ("panel kernel").  The paper's microkernel walks the nonzeros of a
// slice of the sparse matrix, broadcasts each nonzero into vector registers and
// multiplies it with a row slice of the dense matrix held in registers, accumulating
// into an output tile kept in registers; the register that a nonzero accumulates into
// is fixed by generated code per matrix (Sec. 3.2.2, Fig. 3).  On CDNA4:
//   * a consumer wavefront owns a panel of RW rows of the permuted W and a tile of 256
//     columns of C; lane l holds columns 4l..4l+3 of all RW rows in VGPRs (or, on the
//     128-column tiles that a call takes when they suit its grid, columns 2l and 2l+1,
//     with half the LDS ring, so that two workgroups share a CU or 32-row panels fit);
//   * the panel's nonzeros form one flat stream of (weight, ring row, row) entries
//     read with scalar loads, so weights sit in SGPRs; the output row of each entry
//     selects the accumulator through VGPR index mode instead of per-matrix generated
//     code;
//   * the rows of B the workgroup needs are staged in LDS (the paper's split-K tiling
//     of the dense operand) by producer wavefronts, through a ring of 32-row slots
//     filled by direct global->LDS 16-byte DMA; a lane reads its 4 columns of a B row
//     with one ds_read_b128;
//   * producers and consumers synchronise through LDS words (chunks landed, lowest
//     chunk each consumer still reads), so no wave ever waits at a workgroup barrier
//     for the slowest one; the loops are generated inline assembly (spmm_asm_gen.h);
//   * the bias + activation epilogue is fused and C is written once, coalesced, to
//     the original (unpermuted) row, or to the permuted position when the plan keeps
//     rows permuted for the next layer (Sec. 3.1.2);
//   * the same kernel computes a sparse 3x3 convolution (Sec. 3.2.3, direct
//     convolution): a third producer kind stages the rows of the virtual dense operand
//     (input channel x filter tap) straight from the input activations.
// Plain FP32 FMA is used throughout (no MFMA: the work is not a dense contraction).
//
// Workgroups: one column tile x one row-block of nc consecutive panels, plus the
// producer waves.  All panels of a row-block share the staged B rows.  The flat block
// id is remapped so that all row-blocks of a tile land on one XCD (blocks are dealt
// to the 8 XCDs round robin), letting them share that XCD's L2 copy of the B tile.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "sdnn_internal.h"

namespace sdnn {
namespace {

template <int RW>
using acc_plane_t = float __attribute__((ext_vector_type(RW)));

// Operands of the assembly loops (wave-uniform values go to SGPRs, the rest to VGPRs).
struct ConsumerArgs {
  const uint32_t* stream;  // the panel's first group
  uint32_t vlane;          // 16 * lane: the lane's byte offset in a staged B row
  uint32_t prog_addr;      // LDS address of this consumer's progress word
  uint32_t ready_addr;     // LDS address of the ready word
  uint32_t poll_budget;    // failed readiness checks the wave may poll through in total
  uint32_t overrun_addr;   // LDS address of the workgroup's overrun word
  uint32_t chunk_limit;    // the wave stops before a sync group whose c_lo reaches this chunk
  uint32_t chunk_base;     // ring chunk number of the item's chunk 0 (added to c_lo, c_hi)
  uint32_t next_progress;  // progress word written when the panel is done
};
struct ProducerArgs {
  int32_t nchunks, K;      // nchunks: one past the last ring chunk to stage
  int32_t first_chunk;     // first chunk to stage
  int32_t item_chunks;     // chunks per item: ring chunk g stages chunk g % item_chunks of B
                           // (a persistent workgroup's row-blocks restage the same rows)
  // the item's tile after each item: item_rb += item_drb, wrapping at item_nrb with one
  // more tile, and item_dtile_bytes more of B (0, 0: every item is on the same tile)
  int32_t item_rb, item_drb, item_nrb;
  uint32_t item_dtile_bytes;
  uint32_t row_bytes;      // N * 4
  uint32_t bbase_lo, bbase_hi;  // address of B[0][n0]
  int32_t ncol;            // N - n0 (columns of the tile that exist)
  uint32_t first_row;      // first row of each chunk this producer stages
  uint32_t vlane;          // the lane's byte offset in a B row segment (16 or 4 * lane;
                           // 128-column tiles: 16 * (lane % 32))
  uint32_t vlane_fast;     // 128-column tiles: 16 * (lane % 32) + (lane / 32) * N * 4, the
                           // lane's offset from a row pair's first row
  uint32_t prog_addr;      // LDS address of the 16 progress words
  uint32_t ready_addr;     // LDS address of this producer's ready word
  uint32_t poll_budget;    // failed ring-limit checks the wave may poll through in total
  uint32_t overrun_addr;   // LDS address of the workgroup's overrun word
  // virtual B of a 3x3 convolution (bbase is then X itself)
  uint32_t row_step, col_step;  // bytes between image rows (W * NB * 4), columns (NB * 4)
  uint32_t plane_bytes;         // bytes per input channel (H * W * NB * 4)
  uint32_t col_bytes;           // 4 * (n0 + 4 * lane): the lane's first column in a plane
  uint32_t dummy_lds;           // 16 bytes of LDS no one reads (one-lane filler loads)
  uint64_t rowmask[3];          // lanes whose pixel row y + ky - 1 lies in the image
  uint64_t colmask[3];          // lanes whose pixel column x + kx - 1 lies in the image
};

#include "spmm_asm_gen.h"
static_assert(kStreamTailGroups <= kTailGroups, "stream tail shorter than the prefetch");
static_assert(kAsmChunk == kChunk && kAsmRing == kRing, "ring layout mismatch");
static_assert(kAsmGroup == kGroup, "group size mismatch");
static_assert(kAsmTileBytes == kTileCols * 4, "tile width mismatch");
constexpr int kProducers = kAsmProducers;
static_assert(kAsmEndBit == kEndBit && kAsmSyncBit == kSyncBit && kAsmLoShift == kLoShift &&
                  kAsmHiShift == kHiShift,
              "stream fields mismatch");
static_assert(kAsmRingMask == (uint32_t)(kRing * kChunk - 1) << kRingRowShift,
              "ring-row mask mismatch");
static_assert(kAsmTileBytesN == kNarrowTileCols * 4 && kAsmEndBitN == kEndBitNarrow &&
                  kAsmRingMaskN == (uint32_t)(kRing * kChunk - 1) << kRingRowShiftNarrow,
              "128-column layout mismatch");

// Tile layouts (TW columns per tile): 256 columns, 4 per lane, one workgroup per CU; or
// 128 columns, 2 per lane, a 64 KB ring and two producer waves, two workgroups per CU.
template <int TW>
constexpr int ring_bytes() { return kRing * kChunk * TW * 4; }
template <int TW>
constexpr int producers_of() { return TW == kTileCols ? kAsmProducers : kAsmProducersN; }
// Failed checks a wave may poll through before it goes on without waiting (results then
// turn to NaN, never silently wrong); SDNN_POLL_BUDGET overrides it (tests only).
constexpr int kPollBudget = 1 << 22;
// Threads per workgroup a panel height allows: the accumulators sit above the loop's
// pinned VGPRs and end at v[kAsmAccBase + 4 * RW - 1], so RW <= 8 fits the 128 VGPRs
// that 16 waves per CU leave each wave, and RW >= 12 needs 12 waves per CU.
template <int RW>
constexpr int max_threads() { return kAsmAccBase + 4 * RW <= 128 ? 1024 : 768; }
// 128-column tiles: the accumulators end at v[kAsmAccBaseN + 2 * RW - 1]; VGPRs are
// granted in blocks of 8 from 512 per SIMD lane, and a workgroup takes half the waves a
// CU then holds, so that two workgroups (2 x 65 KB of LDS) share each CU: 6 waves per SIMD
// at RW = 4 and 8 (10 consumers per workgroup), 5 at RW = 12 and 16 (8).  (7 waves at RW = 4
// would leave the compiler 88 SGPRs, too few beside the loop's 58: it then reserves a
// stack frame.)  32-row panels (128 VGPRs, 4 waves per SIMD) take a whole CU: 16 waves, 14
// consumers, 448 rows sharing each staged 512-byte row of B.
template <int RW>
constexpr int narrow_waves_per_simd() {
  return 512 / ((kAsmAccBaseN + 2 * RW + 7) / 8 * 8) < 6 ? 512 / ((kAsmAccBaseN + 2 * RW + 7) / 8 * 8)
                                                          : 6;
}
template <int RW>
constexpr int narrow_threads() {
  return RW >= 32 ? 64 * 4 * narrow_waves_per_simd<RW>() : 64 * (4 * narrow_waves_per_simd<RW>() / 2);
}
template <int RW, int TW>
constexpr int threads_of() { return TW == kTileCols ? max_threads<RW>() : narrow_threads<RW>(); }
template <int RW, int TW>
constexpr int min_waves_of() { return TW == kTileCols ? 1 : narrow_waves_per_simd<RW>(); }
// LDS control words after the ring: ready[kProducers] at +0, progress[16] at +64, the
// overrun word at +128 (nonzero once a producer staged past the ring limit), and 16
// bytes per producer at +512 that the convolution producer's filler loads write.
constexpr int kCtlWords = 256;
static_assert(512 + 16 * kProducers <= kCtlWords * 4, "filler words outside the control area");
static_assert(kAsmProducersN <= kProducers, "ready words overlap the progress words");
static_assert(kProducers <= 16, "ready words overlap the progress words");

// GELU(x) = x Phi(x) = 0.5 x (1 + erf(x / sqrt 2)) (the exact erf form).  erf(z) for
// z >= 0 comes from Abramowitz & Stegun 7.1.26 (Hastings' approximation, absolute error
// at most 1.5e-7): erf(z) = 1 - q, q = t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) e^(-z^2),
// t = 1 / (1 + p z); with erf(-z) = -erf(z), GELU(x) = 0.5 x (2 - q) for x >= 0 and
// 0.5 x q for x < 0 (no cancellation on the negative side).  The reciprocal and the
// exponential are the hardware's (v_rcp_f32, v_exp_f32, about 1 ulp); the result is within
// 0.5 |x| * 4e-7 of the exact GELU, far inside the 1e-6 floor of the parity bar at the
// |x| these layers reach, and costs about a third of the library erff's instructions.
__device__ __forceinline__ float gelu(float x) {
  const float z = fabsf(x) * 0.70710678118654752f;
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, z, 1.0f));
  float poly = fmaf(t, 1.061405429f, -1.453152027f);
  poly = fmaf(t, poly, 1.421413741f);
  poly = fmaf(t, poly, -0.284496736f);
  poly = fmaf(t, poly, 0.254829592f);
  poly *= t;
  const float q = poly * __builtin_amdgcn_exp2f(-z * z * 1.4426950408889634f);
  return 0.5f * x * (x >= 0.0f ? 2.0f - q : q);
}

// C is written once and not read again by the kernel: its stores are non-temporal, so the
// output stream does not evict the B tiles and the packed stream from L2 (the stores of the
// 201 MB output of the 3072 x 768 layer at N = 16384 otherwise push the 0.57 MB stream out
// between tiles).
typedef float nt_float4 __attribute__((ext_vector_type(4)));
typedef float nt_float2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void store_c4(float* p, float x, float y, float z, float w) {
  const nt_float4 v = {x, y, z, w};
  __builtin_nontemporal_store(v, reinterpret_cast<nt_float4*>(p));
}
__device__ __forceinline__ void store_c2(float* p, float x, float y) {
  const nt_float2 v = {x, y};
  __builtin_nontemporal_store(v, reinterpret_cast<nt_float2*>(p));
}
__device__ __forceinline__ void store_c1(float* p, float x) { __builtin_nontemporal_store(x, p); }

__device__ __forceinline__ float activation(float x, int epi) {
  if (epi == SDNN_EPI_RELU) return fmaxf(x, 0.0f);
  if (epi == SDNN_EPI_GELU) return gelu(x);
  return x;
}

// Scalar launch parameters (the pointers are separate __restrict__ kernel arguments so
// the compiler may read them through the scalar cache).
struct SpmmArgs {
  int32_t K, N, nchunks, npanels;
  int32_t n_rb;      // row-blocks per column tile
  int32_t total_wg;  // real workgroups (n_tiles * n_rb)
  int32_t per_xcd;   // launched grid / 8
  int32_t epi;
  int32_t out_permuted;  // store permuted row i at row i instead of at its source row
  int32_t H, W, NB;      // image geometry of a 3x3 convolution (B is then the input X)
  uint32_t poll_budget;  // failed readiness / ring-limit checks a wave may poll through
  // split-K: nsplit > 1 gives each run of seg_per_split consecutive K-segments (of
  // split_chunks chunks each; nseg in all) of each tile and row-block its own workgroup,
  // which writes its partial product, without bias or activation, to C + run * M * N
  // (C is then the workspace)
  int32_t M, nsplit, seg_per_split, nseg, split_chunks;
  // persistent workgroups (unsplit launches): wg_per_tile workgroups per column tile,
  // workgroup g of a tile taking row-blocks g, g + wg_per_tile, ... in turn (wg_per_tile =
  // n_rb: one row-block each); or, tile_major, workgroup w taking the items (tile, row-
  // block) numbered w, w + total_wg, ... in tile-major order, so that at any time the
  // workgroups of one XCD (consecutive w) work on consecutive items, mostly of one tile
  int32_t wg_per_tile, tile_major, n_tiles;
};

// Producer kinds: 4-byte staging (any N), 16-byte staging (N % 4 == 0, aligned), the
// virtual B of a 3x3 convolution (16-byte segments of an IC x H x W x NB input).
enum { kStageDword = 0, kStageVec = 1, kStageConv = 2 };

// RW: rows per panel; STAGE: the producer kind (16-byte kinds also store C as float4:
// N % 4 == 0 and B, C 16-byte aligned); TW: columns per tile (256, or 128 with 16-byte
// staging only).  blockDim.x = 64 * (consumers + producers_of<TW>()).
template <int RW, int STAGE, int TW>
__global__ __launch_bounds__((threads_of<RW, TW>()), (min_waves_of<RW, TW>())) void spmm_panel_kernel(
    const uint32_t* __restrict__ entries, const int32_t* __restrict__ panel_start,
    const int32_t* __restrict__ panel_rows, const int32_t* __restrict__ panel_out,
    const int32_t* __restrict__ seg_start, const float* __restrict__ B, float* __restrict__ C,
    const float* __restrict__ bias, SpmmArgs a) {
  // the ring ([0, kRingBytes)) and the control words; the ring must start at LDS 0
  // (the loops form LDS addresses from the ring-row field alone), which holds because
  // this is the kernel's only LDS object
  static_assert(TW == kTileCols || (TW == kNarrowTileCols && STAGE == kStageVec),
                "128-column tiles stage 16-byte rows");
  constexpr int NP = producers_of<TW>();
  constexpr int V = TW / 64;  // columns per lane
  constexpr int kRingB = ring_bytes<TW>();
  __shared__ __attribute__((aligned(16))) uint32_t lds[kRingB / 4 + kCtlWords];

  const int bid = blockIdx.x;
  const int lin = (bid & 7) * a.per_xcd + (bid >> 3);
  if (lin >= a.total_wg) return;  // whole workgroup leaves before the barrier
  // workgroups of one tile and run of K-segments are consecutive (they stage the same rows)
  const int per_tile = a.nsplit * a.wg_per_tile;
  const int tile0 = a.tile_major ? lin / a.n_rb : lin / per_tile;
  const int split = a.tile_major ? 0 : (lin - tile0 * per_tile) / a.wg_per_tile;
  const int g = a.tile_major ? lin - tile0 * a.n_rb : lin - tile0 * per_tile - split * a.wg_per_tile;
  // items: row-blocks g + i * wg_per_tile of tile0, or (tile-major) items lin + i * total_wg
  const int nitems = a.tile_major
                         ? (a.n_tiles * a.n_rb - lin + a.total_wg - 1) / a.total_wg
                         : (a.n_rb - g + a.wg_per_tile - 1) / a.wg_per_tile;
  const bool splitk = a.nsplit > 1;
  const int s0 = split * a.seg_per_split, s1 = min(s0 + a.seg_per_split, a.nseg);
  const int c0 = splitk ? s0 * a.split_chunks : 0;
  const int c1 = splitk ? min(s1 * a.split_chunks, a.nchunks) : a.nchunks;
  const int nc = (blockDim.x >> 6) - NP;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int prod = wave - nc;  // >= 0: producer index

  const uint32_t lds_base = (uint32_t)(uintptr_t)((__attribute__((address_space(3))) uint32_t*)lds);
  if (lds_base != 0) return;  // never taken: see above
  const uint32_t ready_addr = lds_base + kRingB;
  const uint32_t prog0 = ready_addr + 64;
  const uint32_t overrun_addr = ready_addr + 128;
  uint32_t* ctl = lds + kRingB / 4;
  if (prod >= 0) {
    if (lane == 0) ctl[prod] = (uint32_t)c0;                                 // nothing landed
    if (prod == 0 && lane == 0) ctl[32] = 0u;                                // no overrun
    if (prod == 0 && lane >= nc && lane < 16) ctl[16 + lane] = kProgressDone;  // absent consumers
  } else if (lane == 0) {
    ctl[16 + wave] = (uint32_t)c0;  // reads the first item from its first chunk on
  }
  __syncthreads();

  if (prod >= 0) {
    ProducerArgs pa;
    // ring chunks: the items' chunk ranges back to back (split runs: one item, [c0, c1))
    pa.nchunks = splitk ? c1 : nitems * a.nchunks;
    pa.first_chunk = c0;
    pa.item_chunks = splitk ? c1 : a.nchunks;
    pa.item_rb = a.tile_major ? g : 0;
    pa.item_drb = a.tile_major ? a.total_wg % a.n_rb : 0;
    pa.item_nrb = a.tile_major ? a.n_rb : 1;
    pa.item_dtile_bytes = a.tile_major ? (uint32_t)(a.total_wg / a.n_rb) * (TW * 4u) : 0u;
    const int n0 = tile0 * TW;
    pa.K = a.K;
    pa.row_bytes = (uint32_t)a.N * 4u;
    const uint64_t bb = (uint64_t)(uintptr_t)(B + n0);
    pa.bbase_lo = (uint32_t)bb;
    pa.bbase_hi = (uint32_t)(bb >> 32);
    pa.ncol = a.N - n0;
    pa.first_row = (uint32_t)(prod * (kChunk / NP));
    if constexpr (TW == kTileCols) {
      pa.vlane = (uint32_t)lane * (STAGE != kStageDword ? 16u : 4u);
      pa.vlane_fast = pa.vlane;
    } else {  // lanes 32-63 stage the second row of each pair
      pa.vlane = (uint32_t)(lane & 31) * 16u;
      pa.vlane_fast = pa.vlane + (uint32_t)(lane >> 5) * pa.row_bytes;
    }
    pa.prog_addr = prog0;
    pa.ready_addr = ready_addr + 4u * (uint32_t)prod;
    pa.poll_budget = a.poll_budget;
    pa.overrun_addr = overrun_addr;
    if constexpr (STAGE == kStageConv) {
      // lane l's columns n0 + 4l .. + 3: four images of pixel (y, x)
      const uint64_t xb = (uint64_t)(uintptr_t)B;
      pa.bbase_lo = (uint32_t)xb;
      pa.bbase_hi = (uint32_t)(xb >> 32);
      pa.row_step = (uint32_t)a.W * (uint32_t)a.NB * 4u;
      pa.col_step = (uint32_t)a.NB * 4u;
      pa.plane_bytes = (uint32_t)a.H * pa.row_step;
      pa.dummy_lds = ready_addr + 512u + 16u * (uint32_t)prod;
      const int n = n0 + 4 * lane;
      pa.col_bytes = 4u * (uint32_t)n;
      const bool live = n < a.N;
      const int q = n / a.NB, y = q / a.W, x = q - y * a.W;
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        pa.rowmask[t] = __ballot(live && (unsigned)(y + t - 1) < (unsigned)a.H);
        pa.colmask[t] = __ballot(live && (unsigned)(x + t - 1) < (unsigned)a.W);
      }
      produce_conv(pa);
    } else if constexpr (STAGE == kStageVec) {
      if constexpr (TW == kTileCols) produce_vec(pa);
      else produce_vecn(pa);
    } else {
      produce_dword(pa);
    }
    return;
  }

  for (int it = 0; it < nitems; ++it) {
    int tile = tile0, rb = g + it * a.wg_per_tile;
    if (a.tile_major) {
      const int k = lin + it * a.total_wg;
      tile = k / a.n_rb;
      rb = k - tile * a.n_rb;
    }
    const int ncol = tile * TW + lane * V;
    const int panel = rb * nc + wave;
    const uint32_t cbase = splitk ? 0u : (uint32_t)(it * a.nchunks);
    const uint32_t next = it + 1 < nitems ? (uint32_t)((it + 1) * a.nchunks) : kProgressDone;
    int gstart = -1;  // the wave's first group: the first of its panel in the run
    if (panel < a.npanels) {
      if (!splitk) {
        gstart = panel_start[panel];
      } else {
        for (int sg = s0; sg < s1 && gstart < 0; ++sg) gstart = seg_start[(size_t)panel * a.nseg + sg];
      }
    }
    if (panel >= a.npanels) {  // no panel in this row-block (tile-major: maybe in later ones)
      if (lane == 0) ctl[16 + wave] = next;
      continue;
    }

    acc_plane_t<RW> p0 = {}, p1 = {}, p2 = {}, p3 = {};  // p2, p3: 256-column tiles only
    if (gstart >= 0) {  // a panel without entries only writes epi(bias)
      ConsumerArgs ca;
      ca.stream = entries + (size_t)gstart * (2 * kGroup);
      ca.vlane = (uint32_t)lane * (4u * V);
      ca.prog_addr = prog0 + 4u * (uint32_t)wave;
      ca.ready_addr = ready_addr;
      ca.poll_budget = a.poll_budget;
      ca.overrun_addr = overrun_addr;
      ca.chunk_limit = (uint32_t)c1;
      ca.chunk_base = cbase;
      ca.next_progress = next;
      if constexpr (TW != kTileCols) {
        if (splitk) {
          if constexpr (RW == 4) consume_n_rw4_limit(p0, p1, ca);
          if constexpr (RW == 8) consume_n_rw8_limit(p0, p1, ca);
          if constexpr (RW == 12) consume_n_rw12_limit(p0, p1, ca);
          if constexpr (RW == 16) consume_n_rw16_limit(p0, p1, ca);
          if constexpr (RW == 32) consume_n_rw32_limit(p0, p1, ca);
        } else {
          if constexpr (RW == 4) consume_n_rw4(p0, p1, ca);
          if constexpr (RW == 8) consume_n_rw8(p0, p1, ca);
          if constexpr (RW == 12) consume_n_rw12(p0, p1, ca);
          if constexpr (RW == 16) consume_n_rw16(p0, p1, ca);
          if constexpr (RW == 32) consume_n_rw32(p0, p1, ca);
        }
      } else if (splitk) {  // runs of K-segments: the loop also stops at the run's last chunk
        if constexpr (RW == 4) consume_rw4_limit(p0, p1, p2, p3, ca);
        if constexpr (RW == 8) consume_rw8_limit(p0, p1, p2, p3, ca);
        if constexpr (RW == 12) consume_rw12_limit(p0, p1, p2, p3, ca);
        if constexpr (RW == 16) consume_rw16_limit(p0, p1, p2, p3, ca);
      } else {
        if constexpr (RW == 4) consume_rw4(p0, p1, p2, p3, ca);
        if constexpr (RW == 8) consume_rw8(p0, p1, p2, p3, ca);
        if constexpr (RW == 12) consume_rw12(p0, p1, p2, p3, ca);
        if constexpr (RW == 16) consume_rw16(p0, p1, p2, p3, ca);
      }
    } else if (lane == 0) {
      ctl[16 + wave] = next;  // nothing to read in this row-block
    }

#pragma unroll
    for (int r = 0; r < RW; ++r) {
      const int orig = panel_rows[panel * RW + r];
      if (orig < 0) continue;
      const int row = panel_out[panel * RW + r];
      const float v[4] = {p0[r], p1[r], p2[r], p3[r]};
      if constexpr (TW != kTileCols) {
        if (splitk) {  // raw partial sums (16-byte aligned workspace, N % 4 == 0)
          float* prow = C + ((size_t)split * a.M + row) * a.N;
          if (ncol + 2 <= a.N) *reinterpret_cast<float2*>(prow + ncol) = make_float2(v[0], v[1]);
          else if (ncol < a.N) prow[ncol] = v[0];
          continue;
        }
        const float bb = bias ? bias[orig] : 0.0f;
        float* crow = C + (size_t)row * a.N;
        if (ncol + 2 <= a.N) {
          store_c2(crow + ncol, activation(v[0] + bb, a.epi), activation(v[1] + bb, a.epi));
        } else if (ncol < a.N) {
          store_c1(crow + ncol, activation(v[0] + bb, a.epi));
        }
        continue;
      }
      if (splitk) {  // raw partial sums; the reduction adds the bias and applies epi
        float* prow = C + ((size_t)split * a.M + row) * a.N;
        if (STAGE != kStageDword && ncol + 4 <= a.N) {
          *reinterpret_cast<float4*>(prow + ncol) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (ncol + i < a.N) prow[ncol + i] = v[i];
        }
        continue;
      }
      const float bb = bias ? bias[orig] : 0.0f;
      float* crow = C + (size_t)row * a.N;
      if (STAGE != kStageDword && ncol + 4 <= a.N) {
        store_c4(crow + ncol, activation(v[0] + bb, a.epi), activation(v[1] + bb, a.epi),
                 activation(v[2] + bb, a.epi), activation(v[3] + bb, a.epi));
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (ncol + i < a.N) store_c1(crow + ncol + i, activation(v[i] + bb, a.epi));
      }
    }
  }
}

struct SpmmPtrs {
  const uint32_t* entries;
  const int32_t* panel_start;
  const int32_t* panel_rows;
  const int32_t* panel_out;
  const int32_t* seg_start;
  const float* B;
  float* C;
  const float* bias;
};

template <int RW, int STAGE, int TW>
hipError_t launch_variant(const SpmmPtrs& p, const SpmmArgs& args, int waves, int grid,
                          hipStream_t stream) {
  hipLaunchKernelGGL((spmm_panel_kernel<RW, STAGE, TW>), dim3(grid),
                     dim3(64 * (waves + producers_of<TW>())), 0, stream,
                     p.entries, p.panel_start, p.panel_rows, p.panel_out, p.seg_start, p.B, p.C,
                     p.bias, args);
  return hipGetLastError();
}

template <int STAGE, int TW = kTileCols>
hipError_t launch_rw(int RW, const SpmmPtrs& p, const SpmmArgs& args, int waves, int grid,
                     hipStream_t stream) {
  switch (RW) {
    case 4: return launch_variant<4, STAGE, TW>(p, args, waves, grid, stream);
    case 8: return launch_variant<8, STAGE, TW>(p, args, waves, grid, stream);
    case 12: return launch_variant<12, STAGE, TW>(p, args, waves, grid, stream);
    case 16: return launch_variant<16, STAGE, TW>(p, args, waves, grid, stream);
    case 32:
      if constexpr (TW == kNarrowTileCols) return launch_variant<32, STAGE, TW>(p, args, waves, grid, stream);
      break;
  }
  return hipErrorInvalidValue;
}

// Consumer waves a workgroup can hold at panel height RW and tile width TW (the register
// limit of the accumulators, less the producers).
int max_consumers(int RW, int TW = kTileCols) {
  int threads;
  if (TW == kTileCols)
    threads = RW == 4 ? max_threads<4>() : RW == 8 ? max_threads<8>()
            : RW == 12 ? max_threads<12>() : max_threads<16>();
  else
    threads = RW == 4 ? narrow_threads<4>() : RW == 8 ? narrow_threads<8>()
            : RW == 12 ? narrow_threads<12>() : RW == 16 ? narrow_threads<16>()
            : narrow_threads<32>();
  const int c = threads / 64 - (TW == kTileCols ? kAsmProducers : kAsmProducersN);
  return c < kAsmMaxConsumers ? c : kAsmMaxConsumers;
}

int env_int(const char* name, int dflt) {
  const char* s = getenv(name);
  return s ? atoi(s) : dflt;
}

struct LaunchCfg {
  int waves, n_tiles, n_rb;  // waves: consumer waves per workgroup (the producers come on top)
};

// Workgroups a grid is sized for: one per CU.  Two workgroups with 128-column tiles fit a CU
// (65 KB of LDS each), but on the layers whose launch takes those tiles a grid of one per CU
// with more consumer waves each was the faster (C2's 768 x 768 layer at N = 1024: 14.1 against
// 15.4 us; the 768 x 3072 layer at N = 1024: 43.8 against 51.6 us).
int slots_of(int num_cus) { return num_cus > 0 ? num_cus : 256; }

// Waves per SIMD the kernel for panel height RW and tile width tw allows (its VGPRs).
int waves_per_simd(int RW, int tw) {
  if (tw == kTileCols) {
    const int vgprs = (kAsmAccBase + 4 * RW + 7) / 8 * 8;
    return std::min(8, 512 / vgprs);
  }
  return RW == 4 ? narrow_waves_per_simd<4>() : RW == 8 ? narrow_waves_per_simd<8>()
       : RW == 12 ? narrow_waves_per_simd<12>() : RW == 16 ? narrow_waves_per_simd<16>()
       : narrow_waves_per_simd<32>();
}

// Workgroups the device holds at once (the persistent launches' grid): per CU, at most one
// with 256-column tiles (129 KB of LDS each) and two with 128-column tiles (65 KB), and no
// more than the CU's waves at the kernel's occupancy allow (a 14-consumer workgroup of
// 32-row panels takes a whole CU).
int resident_of(int num_cus, int tw, int RW, int waves) {
  const int cus = num_cus > 0 ? num_cus : 256;
  const int per_wg = waves + (tw == kTileCols ? kAsmProducers : kAsmProducersN);
  const int by_waves = std::max(1, 4 * waves_per_simd(RW, tw) / per_wg);
  return cus * std::min(tw == kTileCols ? 1 : 2, by_waves);
}

// The 129 KB of ring and control LDS allow one workgroup per CU, so a grid of G
// workgroups runs in ceil(G / CUs) rounds, and a partly filled last round costs as
// much as a full one.
int64_t rounds_of(int64_t n_tiles, int npanels, int waves, int target) {
  const int64_t wgs = n_tiles * ((npanels + waves - 1) / waves);
  return (wgs + target - 1) / target;
}

// Consumer waves per workgroup: the fewest rounds that the register-limited consumer
// count allows, and within that many rounds the smallest workgroups (fewest panels
// each, so the most workgroups share the work).  SDNN_FORCE_WAVES fixes the count.
LaunchCfg choose_cfg(const DevPacking& pk, int num_cus, int N, int nseg = 1, int tw = kTileCols) {
  const int target = slots_of(num_cus);
  int cap = max_consumers(pk.RW, tw);
  if (cap > pk.npanels) cap = pk.npanels;
  if (cap < 1) cap = 1;
  const int forceW = env_int("SDNN_FORCE_WAVES", 0);
  LaunchCfg c;
  c.n_tiles = (N + tw - 1) / tw;
  const int64_t units = (int64_t)c.n_tiles * nseg;  // (tile, K-segment) pairs
  if (forceW > 0) {
    c.waves = forceW < cap ? forceW : cap;
  } else {
    const int64_t fewest = rounds_of(units, pk.npanels, cap, target);
    c.waves = cap;
    for (int w = 1; w < cap; ++w)
      if (rounds_of(units, pk.npanels, w, target) == fewest) {
        c.waves = w;
        break;
      }
  }
  c.n_rb = (pk.npanels + c.waves - 1) / c.waves;
  return c;
}

// The packing a call runs on (a default plan holds 4-, 12-, 8- and 16-row packings): among
// the packings, the 4-row one left out when its panels average fewer than 8 entries per
// 32-row chunk (a group of 8 then spans a chunk or more, which starves the ring's
// lookahead, and the workgroups' staging chains outweigh their arithmetic) and another
// exists, those needing the fewest rounds of workgroups over the
// tiles (times the K-runs of a split launch) at their full consumer count; among those,
// the ones keeping the most CUs busy in those rounds (within 5 %); among those, the
// shortest panels averaging at least 8 entries per chunk, else the tallest.  Measured on
// MI355X for products (M = K = 512-2048 at 80-98 %, N = 1024-16384, the W0 and C2-C5
// layers) and for the 3x3 convolutions of the benchmark, whose staging differs but
// follows the same trade.
// The 32-row packing with kDeepWaves consumer waves per workgroup (128-column tiles: 384
// rows share each staged 512-byte B row, against 128 rows per 1 KB row on 256-column tiles
// with 16-row panels), taken for an unsplit product when W holds under 20 entries per 16
// rows and 32 columns (so the other packings' workgroups stage many B rows for few entries)
// and its grid fills the CUs; null otherwise.  Measured on MI355X at 97 % and N = 16384:
// the 768 x 3072 layer 119.2 -> 87.5 us, the 768 x 768 layer 40.2 -> 32.0 us, the 3072 x 768
// layer 130.4 -> 122.5 us (at N = 4096 40.2 -> 33.6 us); with fewer items than CUs (the
// 768-row layers at N = 8192) or at 94 % and denser it was slower.
constexpr int kDeepWaves = 12;
const DevPacking* deep_packing(const sdnn_plan_s* p, int N, int nseg) {
  if (nseg != 1 || p->npack < 5 || p->pk[4].RW != kDeepPanel || !p->pk[4].entries_n) return nullptr;
  const double density = (double)p->nnz / ((double)p->M * (double)p->K);
  if (kTallestPanel * kChunk * density >= 20.0) return nullptr;
  const int64_t tiles = (N + kNarrowTileCols - 1) / kNarrowTileCols;
  const int64_t rbs = (p->pk[4].npanels + kDeepWaves - 1) / kDeepWaves;
  return tiles * rbs >= (p->num_cus > 0 ? p->num_cus : 256) ? &p->pk[4] : nullptr;
}

const DevPacking& choose_packing(const sdnn_plan_s* p, int N, int nseg = 1, int tw = kTileCols) {
  if (p->npack < 2) return p->pk[0];
  if (tw == kNarrowTileCols)
    if (const DevPacking* d = deep_packing(p, N, nseg)) return *d;
  const int64_t n_tiles = (int64_t)((N + tw - 1) / tw) * nseg;
  const int cus = slots_of(p->num_cus);
  const double density = (double)p->nnz / ((double)p->M * (double)p->K);
  auto per_chunk = [&](const DevPacking& pk) { return pk.RW * kChunk * density; };
  int64_t rounds[kMaxPackings];
  double util[kMaxPackings];
  bool live[kMaxPackings];
  int64_t best_rounds = -1;
  for (int k = 0; k < p->npack; ++k) {
    const DevPacking& pk = p->pk[k];
    live[k] = !(pk.RW == 4 && per_chunk(pk) < 8.0) && pk.RW <= kTallestPanel;
    const int waves = std::max(1, std::min(max_consumers(pk.RW, tw), pk.npanels));
    const int64_t wgs = n_tiles * ((pk.npanels + waves - 1) / waves);
    rounds[k] = (wgs + cus - 1) / cus;
    util[k] = (double)wgs / ((double)rounds[k] * cus);
  }
  bool any = false;
  for (int k = 0; k < p->npack; ++k) any |= live[k];
  if (!any)
    for (int k = 0; k < p->npack; ++k) live[k] = p->pk[k].RW <= kTallestPanel;
  for (int k = 0; k < p->npack; ++k)
    if (live[k] && (best_rounds < 0 || rounds[k] < best_rounds)) best_rounds = rounds[k];
  double best_util = 0.0;
  for (int k = 0; k < p->npack; ++k)
    if (live[k] && rounds[k] == best_rounds) best_util = std::max(best_util, util[k]);
  int pick = -1, tallest = -1;
  for (int k = 0; k < p->npack; ++k) {
    if (!live[k] || rounds[k] != best_rounds || util[k] < 0.95 * best_util) continue;
    if (tallest < 0 || p->pk[k].RW > p->pk[tallest].RW) tallest = k;
    if (per_chunk(p->pk[k]) >= 8.0 && (pick < 0 || p->pk[k].RW < p->pk[pick].RW)) pick = k;
  }
  return p->pk[pick >= 0 ? pick : tallest];
}

}  // namespace

namespace {
// Workgroups along K for a K-split call that leaves the choice to the library: the
// count that minimises a small cost model, in microseconds,
//     rounds * chunks_per_workgroup * t_chunk                  (staging of B)
//   + (splits > 1) * (t_launch + (splits + 1) * 4 M N / bw)    (reduction kernel)
// where rounds counts full waves of workgroups on the CUs at the launch shape the call
// would use, and a chunk costs a workgroup the longer of the staging latency (0.45 us;
// 0.75 us for the convolution's staging) and its consumers' LDS reads of that chunk
// (waves * RW * 32 rows * density / fill entries of 1 KB at 434 KB/us, the measured
// ds_read_b128 rate of one CU).  t_launch = 4 us, bw = 4 TB/s (the partials mostly sit
// in the Infinity Cache); all measured on MI355X.  A count is tried only if runs of
// ceil(nseg / count) segments give exactly it, and replaces a smaller one only if it
// costs at least 10 % less (the model's error on MI355X is about that size).
constexpr int kMaxAutoSplits = 32;  // more runs than this never paid for their partials

int choose_splits(const sdnn_plan_s* p, int N, bool conv) {
  const int total_seg = p->pk[0].nseg;
  const int cus = p->num_cus > 0 ? p->num_cus : 256;
  const int64_t n_tiles = (N + kTileCols - 1) / kTileCols;
  const double t_lat = conv ? 0.75 : 0.45, t_launch = 4.0, bw = 4.0e6;  // bytes per us
  const double lds_per_us = 434.0e3;
  const double density = (double)p->nnz / ((double)p->M * (double)p->K);
  int best = 1;
  double best_cost = 0.0;
  for (int splits = 1; splits <= std::min(total_seg, kMaxAutoSplits); ++splits) {
    const int per = (total_seg + splits - 1) / splits;
    if ((total_seg + per - 1) / per != splits) continue;
    const DevPacking& pk = choose_packing(p, N, splits);
    const LaunchCfg cfg = choose_cfg(pk, cus, N, splits);
    const int64_t rounds = rounds_of(n_tiles * splits, pk.npanels, cfg.waves, cus);
    const int64_t chunks = std::min<int64_t>((int64_t)per * p->split_chunks, p->nchunks);
    const double reads = (double)cfg.waves * pk.RW * kChunk * density / std::max(pk.fill, 0.05);
    const double t_chunk = std::max(t_lat, reads * 1024.0 / lds_per_us);
    double cost = (double)rounds * (double)chunks * t_chunk;
    if (splits > 1) cost += t_launch + (splits + 1) * 4.0 * (double)p->M * (double)N / bw;
    if (splits == 1 || cost < 0.9 * best_cost) {  // a larger count must win clearly
      best_cost = cost;
      best = splits;
    }
  }
  return best;
}

// Split-K reduction: C[i][n] = act(sum_s ws[s][i][n] + bias[rowmap[i]]) over the nseg
// partial products of an M x N output (rowmap: NULL for the identity).  Each thread
// takes four consecutive columns of one row; vec: N % 4 == 0 and 16-byte aligned
// buffers, so the four are one float4.
template <bool VEC>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ ws,
                                                            float* __restrict__ C,
                                                            const float* __restrict__ bias,
                                                            const int32_t* __restrict__ rowmap,
                                                            int32_t M, int32_t N, int32_t nseg,
                                                            int32_t epi) {
  const int64_t nq = (N + 3) / 4, total = (int64_t)M * nq, plane = (int64_t)M * N;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total;
       q += (int64_t)gridDim.x * 256) {
    const int32_t i = (int32_t)(q / nq);
    const int32_t n = (int32_t)(q - (int64_t)i * nq) * 4;
    const int64_t at = (int64_t)i * N + n;
    const float bb = bias ? bias[rowmap ? rowmap[i] : i] : 0.0f;
    if (VEC) {
      float4 acc = *reinterpret_cast<const float4*>(ws + at);
      for (int s = 1; s < nseg; ++s) {
        const float4 v = *reinterpret_cast<const float4*>(ws + s * plane + at);
        acc.x += v.x;
        acc.y += v.y;
        acc.z += v.z;
        acc.w += v.w;
      }
      store_c4(C + at, activation(acc.x + bb, epi), activation(acc.y + bb, epi),
               activation(acc.z + bb, epi), activation(acc.w + bb, epi));
    } else {
      for (int c = 0; c < 4 && n + c < N; ++c) {
        float acc = ws[at + c];
        for (int s = 1; s < nseg; ++s) acc += ws[s * plane + at + c];
        store_c1(C + at + c, activation(acc + bb, epi));
      }
    }
  }
}

hipError_t launch_reduce(const float* ws, float* C, const float* bias, const int32_t* rowmap,
                         int32_t M, int32_t N, int32_t nseg, int epi, hipStream_t stream) {
  const int64_t total = (int64_t)M * ((N + 3) / 4);
  const int64_t blocks = std::min<int64_t>((total + 255) / 256, 8 * 1024);
  const bool vec = N % 4 == 0 && ((uintptr_t)ws & 15) == 0 && ((uintptr_t)C & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(splitk_reduce_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       ws, C, bias, rowmap, M, N, nseg, epi);
  else
    hipLaunchKernelGGL(splitk_reduce_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       ws, C, bias, rowmap, M, N, nseg, epi);
  return hipGetLastError();
}

// `shape` (packing index and consumer waves) overrides the plan's tuned or heuristic
// choice when non-null.  Tuned shapes were timed on unsplit products, so a convolution,
// whose staging differs, and a K-split launch keep the heuristic.  ws non-null (a plan
// with K-segments): `splits` workgroups along K (0: choose_splits), so every (tile, run
// of segments, row-block) is a workgroup that writes its partial product to ws, and a
// reduction kernel forms C.
// Workgroups along K of a K-split launch (each taking a run of *seg_per_split
// consecutive segments) for a requested count (0: choose_splits).
int split_runs_of(const sdnn_plan_s* p, int32_t N, int splits, bool conv, int* seg_per_split) {
  const int total_seg = p->pk[0].nseg;
  if (splits <= 0 && !conv)  // the count sdnn_plan_tune measured fastest at this N
    for (int i = 0; i < p->ntuned; ++i)
      if (p->tuned[i].N == N && p->tuned[i].splits > 0) splits = p->tuned[i].splits;
  if (splits <= 0) splits = choose_splits(p, N, conv);
  splits = std::min(std::max(splits, 1), total_seg);
  const int per = (total_seg + splits - 1) / splits;
  if (seg_per_split) *seg_per_split = per;
  return (total_seg + per - 1) / per;
}

// Whether a call may run on 128-column tiles: a product (not a convolution) with N % 4 == 0
// and 16-byte aligned B and output (C, or a K-split call's workspace: the 16-byte staging),
// on a plan that holds the 128-column stream, with per-lane staging offsets
// 16 (lane % 32) + (lane / 32 + 2 j) 4N (j < 8) below 2^31.
bool narrow_allowed(const sdnn_plan_s* p, int N, bool aligned, bool conv) {
  return aligned && !conv && p->pk[0].entries_n != nullptr &&
         (uint64_t)N * 4u * (kChunk / kAsmProducersN) < ((uint64_t)1 << 31);
}

// Tile width of a call that may use either: the plan's tile_cols option, else 128 columns
// when the 256-column launch would give its workgroups at most 4 consumer waves (few tiles
// and rows per CU: each workgroup's time is then the staging chain of its tile's K rows, and
// half-width rows halve the staged bytes per chunk), else 256 (the 128-column loop issues an
// LDS read and an address op per two FMAs instead of four, which the loaded layers pay for).
// Measured on MI355X over 68 layers and batch widths (the benchmark's layers, C2-C5 and W0 at
// N = 256-4096, M = K = 256-2048 at 70-95 % with N = 128-2048): every launch of 1-4 waves
// was 7-30 % faster on 128 columns (C1 8.9 -> 6.6 us, C2 16.6 -> 13.8 us, the 768 x 3072
// layer at N = 1024 53.5 -> 43.4 us, M = K = 2048 at 90 % with N = 128 34.8 -> 26.3 us); from
// 6 waves on 256 columns was as fast or faster (W0 at N = 4096 67.0 against 82.7 us, C5's
// 3072 x 768 layer 130.5 against 185.5 us).
// A K-split launch of nk workgroups along K follows the same rule on its own grid.
constexpr int kNarrowMaxWaves = 4;
int choose_tile(const sdnn_plan_s* p, int N, int nk = 1) {
  if (p->tile_cols != 0) return p->tile_cols;
  if (deep_packing(p, N, nk)) return kNarrowTileCols;
  const DevPacking& pk = choose_packing(p, N, nk);
  return choose_cfg(pk, p->num_cus, N, nk).waves <= kNarrowMaxWaves ? kNarrowTileCols : kTileCols;
}

// tile: a tile width to use where the call allows it (0: the tuned or the rule's).
hipError_t launch_panels(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                         const float* bias, int epi, const int32_t* conv_hwn,
                         const TunedShape* shape, float* ws, int splits, hipStream_t stream,
                         int tile = 0) {
  // nk: workgroups along K, each taking a run of seg_per_split consecutive segments
  int seg_per_split = 1, nk = 1;
  if (ws) {
    nk = split_runs_of(p, N, splits, conv_hwn != nullptr, &seg_per_split);
    if (splits <= 0 && !tile)  // a tuned count comes with its tile width
      for (int i = 0; i < p->ntuned; ++i)
        if (p->tuned[i].N == N && p->tuned[i].splits == nk && nk > 1) tile = p->tuned[i].split_tile;
  }
  if (!shape && !conv_hwn && nk == 1)
    for (int i = 0; i < p->ntuned; ++i)
      if (p->tuned[i].N == N) shape = &p->tuned[i];
  float* out = nk > 1 ? ws : C;
  const bool aligned = (N % 4 == 0) && (((uintptr_t)B & 15) == 0) && (((uintptr_t)out & 15) == 0);
  int tw = kTileCols;
  if (narrow_allowed(p, N, aligned, conv_hwn != nullptr))
    tw = shape ? shape->tile : tile ? tile : choose_tile(p, N, nk);
  // a tuned shape on a packing that 256-column tiles cannot run (32-row panels), for a call
  // that cannot use 128 columns: the rule decides instead
  if (shape && p->pk[shape->pack].RW > kTallestPanel && tw != kNarrowTileCols) shape = nullptr;
  const DevPacking& pk =
      shape ? p->pk[shape->pack] : choose_packing(p, N, nk, tw);
  if (pk.RW > 16 && tw != kNarrowTileCols) return hipErrorInvalidValue;  // 128-column only
  LaunchCfg cfg = choose_cfg(pk, p->num_cus, N, nk, tw);
  if (shape) {
    cfg.waves = std::min(shape->waves, max_consumers(pk.RW, tw));
    cfg.n_rb = (pk.npanels + cfg.waves - 1) / cfg.waves;
  }
  const SpmmPtrs ptrs{tw == kTileCols ? pk.entries : pk.entries_n, pk.panel_start, pk.panel_rows,
                      pk.panel_out, pk.seg_start, B, out, bias};
  SpmmArgs args;
  args.K = p->K;
  args.N = N;
  args.nchunks = p->nchunks;
  args.npanels = pk.npanels;
  args.n_rb = cfg.n_rb;
  args.M = p->M;
  args.nsplit = nk;
  args.seg_per_split = seg_per_split;
  args.nseg = pk.nseg;
  args.split_chunks = nk > 1 ? p->split_chunks : 0;
  // Persistent workgroups: when an unsplit product has more (tile, row-block) items than
  // CUs, each tile gets wg_per_tile = CUs / tiles workgroups (at least one) that take its
  // row-blocks in turn; the producers stage the next row-block's chunks into the ring
  // while the consumers finish the current one, so a workgroup's start-up (first chunks
  // in flight) and wind-down (epilogue, stores) overlap its neighbours' work instead of
  // recurring per row-block.  Ring chunk numbers run on across row-blocks, so a
  // row-block's chunk c sits in ring slot (base + c) % kRing: the row-blocks' chunk
  // counts must be multiples of kRing, as the stream's ring rows assume c % kRing.
  // When every tile is full (N a multiple of the tile width) the items go to the
  // workgroups in tile-major order instead (workgroup w takes items w, w + CUs, ...):
  // the consecutive workgroups of one XCD then share one or a few tiles at a time, whose
  // B rows stay in that XCD's L2 across the row-blocks, where CUs / tiles workgroups per
  // tile would spread each XCD over many tiles (C5's 3072 x 768 layer: 8 tiles of 768 KB
  // per XCD against a 4 MB L2).
  const int cus = resident_of(p->num_cus, tw, pk.RW, cfg.waves);  // workgroups resident at once
  const int64_t items = (int64_t)cfg.n_tiles * cfg.n_rb;
  const bool can_persist = nk == 1 && !conv_hwn && p->nchunks % kRing == 0;
  int wg_per_tile = cfg.n_rb, tile_major = 0;
  int64_t total = (int64_t)cfg.n_tiles * nk * cfg.n_rb;
  if (can_persist && items > cus) {
    if (N % tw == 0) {
      tile_major = 1;
      total = cus;
    } else {
      wg_per_tile = std::max(1, std::min(cfg.n_rb, cus / std::max(1, cfg.n_tiles)));
      total = (int64_t)cfg.n_tiles * wg_per_tile;
    }
  }
  if (can_persist) {  // forced shapes (tests)
    const int forced = env_int("SDNN_FORCE_WG_PER_TILE", 0);
    const int forced_tm = env_int("SDNN_FORCE_TILE_MAJOR_WGS", 0);
    if (forced > 0) {
      tile_major = 0;
      wg_per_tile = std::min(forced, cfg.n_rb);
      total = (int64_t)cfg.n_tiles * wg_per_tile;
    } else if (forced_tm > 0 && N % tw == 0) {
      tile_major = 1;
      wg_per_tile = cfg.n_rb;
      total = std::min<int64_t>(forced_tm, items);
    }
  }
  args.wg_per_tile = wg_per_tile;
  args.tile_major = tile_major;
  args.n_tiles = cfg.n_tiles;
  if (total > (int64_t)1 << 30) return hipErrorInvalidValue;
  const int64_t grid = (total + 7) / 8 * 8;
  args.total_wg = (int32_t)total;
  args.per_xcd = (int32_t)(grid / 8);
  args.epi = epi;
  args.out_permuted = p->out_permuted;
  args.H = conv_hwn ? conv_hwn[0] : 0;
  args.W = conv_hwn ? conv_hwn[1] : 0;
  args.NB = conv_hwn ? conv_hwn[2] : 0;
  {
    const int budget = env_int("SDNN_POLL_BUDGET", kPollBudget);
    args.poll_budget = budget > 0 ? (uint32_t)budget : 0u;
  }
  hipError_t err;
  if (conv_hwn) {
    err = launch_rw<kStageConv>(pk.RW, ptrs, args, cfg.waves, (int)grid, stream);
  } else if (tw == kNarrowTileCols) {
    err = launch_rw<kStageVec, kNarrowTileCols>(pk.RW, ptrs, args, cfg.waves, (int)grid, stream);
  } else {
    // the 16-byte producer addresses a chunk's rows with 32-bit per-lane offsets
    // 16 * lane + r * 4N (r < kChunk / kProducers)
    const bool vec = aligned && (uint64_t)N * 4u * (kChunk / kProducers) < ((uint64_t)1 << 31);
    err = vec ? launch_rw<kStageVec>(pk.RW, ptrs, args, cfg.waves, (int)grid, stream)
              : launch_rw<kStageDword>(pk.RW, ptrs, args, cfg.waves, (int)grid, stream);
  }
  if (err != hipSuccess || nk == 1) return err;
  return launch_reduce(ws, C, bias, p->out_permuted ? p->d_perm : nullptr, p->M, N, nk, epi,
                       stream);
}
}  // namespace

void launch_shape(const sdnn_plan_s* p, int32_t N, int32_t* panel_rows, int32_t* waves,
                  int32_t* tile_cols) {
  const TunedShape* shape = nullptr;
  for (int i = 0; i < p->ntuned; ++i)
    if (p->tuned[i].N == N) shape = &p->tuned[i];
  int tw = kTileCols;
  if (narrow_allowed(p, N, N % 4 == 0, false)) tw = shape ? shape->tile : choose_tile(p, N);
  const DevPacking& pk = shape ? p->pk[shape->pack] : choose_packing(p, N, 1, tw);
  *panel_rows = pk.RW;
  *waves = shape ? std::min(shape->waves, max_consumers(pk.RW, tw))
                 : choose_cfg(pk, p->num_cus, N, 1, tw).waves;
  *tile_cols = tw;
}

hipError_t launch_spmm(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                       const float* bias, int epi, hipStream_t stream) {
  return launch_panels(p, B, C, N, bias, epi, nullptr, nullptr, nullptr, 0, stream);
}

hipError_t launch_spmm_split(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                             const float* bias, int epi, int splits, float* ws,
                             hipStream_t stream) {
  return launch_panels(p, B, C, N, bias, epi, nullptr, nullptr, ws, splits, stream);
}

hipError_t tune_spmm(sdnn_plan_s* p, const float* B, float* C, int32_t N, hipStream_t stream,
                     TunedShape* chosen) {
  // candidates: every tile width the call and the plan's tile_cols option allow and every
  // packing, each with its register-limited consumer count and three fewer-wave shapes,
  // plus the heuristic's own choice
  std::vector<TunedShape> cands;
  const bool aligned = (N % 4 == 0) && (((uintptr_t)B & 15) == 0) && (((uintptr_t)C & 15) == 0);
  std::vector<int> tiles;
  if (!narrow_allowed(p, N, aligned, false) || p->tile_cols != kNarrowTileCols)
    tiles.push_back(kTileCols);
  if (narrow_allowed(p, N, aligned, false)) tiles.push_back(kNarrowTileCols);
  for (int tw : tiles)
    for (int k = 0; k < p->npack; ++k) {
      if (p->pk[k].RW > kTallestPanel && tw != kNarrowTileCols) continue;  // 128-column only
      const int cap = std::min(max_consumers(p->pk[k].RW, tw), p->pk[k].npanels);
      const int heur = choose_cfg(p->pk[k], p->num_cus, N, 1, tw).waves;
      for (int w : {cap, (3 * cap) / 4, cap / 2, cap / 4, heur}) {
        if (w < 1) continue;
        bool dup = false;
        for (const TunedShape& t : cands) dup |= (t.pack == k && t.waves == w && t.tile == tw);
        if (!dup) cands.push_back(TunedShape{N, k, w, tw});
      }
    }
  if (cands.empty()) return hipErrorInvalidValue;  // no packing runs at this call's tile width
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t err = hipEventCreate(&e0);
  if (err == hipSuccess) err = hipEventCreate(&e1);
  // two passes over the candidates, each keeping its faster pass, so that a clock
  // change or a noisy pass does not decide alone
  std::vector<float> ms_best(cands.size(), -1.0f);
  for (int pass = 0; pass < 2; ++pass) {
    for (size_t i = 0; i < cands.size() && err == hipSuccess; ++i) {
      for (int r = 0; r < 2 && err == hipSuccess; ++r)   // warm-up
        err = launch_panels(p, B, C, N, nullptr, 0, nullptr, &cands[i], nullptr, 0, stream);
      if (err == hipSuccess) err = hipEventRecord(e0, stream);
      for (int r = 0; r < 8 && err == hipSuccess; ++r)
        err = launch_panels(p, B, C, N, nullptr, 0, nullptr, &cands[i], nullptr, 0, stream);
      if (err == hipSuccess) err = hipEventRecord(e1, stream);
      if (err == hipSuccess) err = hipEventSynchronize(e1);
      float ms = 0.0f;
      if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
      if (err == hipSuccess && (ms_best[i] < 0.0f || ms < ms_best[i])) ms_best[i] = ms;
    }
  }
  float best = -1.0f;
  for (size_t i = 0; i < cands.size() && err == hipSuccess; ++i)
    if (best < 0.0f || ms_best[i] < best) {
      best = ms_best[i];
      *chosen = cands[i];
    }
  int slot = -1;
  if (err == hipSuccess) {
    for (int i = 0; i < p->ntuned; ++i)
      if (p->tuned[i].N == N) slot = i;
    if (slot < 0) slot = p->ntuned < kTunedSlots ? p->ntuned++ : (int)(N % kTunedSlots);
    chosen->splits = 0;
    p->tuned[slot] = *chosen;
  }
  // K-segmented plans: the split-K tiling factor, i.e. the workgroups along K of
  // sdnn_spmm_split (each count whose runs of ceil(nseg / count) segments give exactly it, up
  // to kMaxAutoSplits, on each tile width the call allows, at the launch's own packing and
  // consumer count), timed into a workspace allocated for the search; one workgroup along K
  // is the unsplit call just tuned
  const int nseg = p->pk[0].nseg;
  if (err == hipSuccess && p->split_chunks > 0 && nseg > 1) {
    float* ws = nullptr;
    const size_t ws_bytes = (size_t)nseg * (size_t)p->M * (size_t)N * sizeof(float);
    if (hipMalloc(&ws, ws_bytes) == hipSuccess) {
      int best_runs = 1, best_tile = 0;
      float best_ms = best;
      for (int r = 2; r <= std::min(nseg, kMaxAutoSplits) && err == hipSuccess; ++r) {
        const int per = (nseg + r - 1) / r;
        if ((nseg + per - 1) / per != r) continue;
        for (int tw : tiles) {
          float ms_r = -1.0f;
          for (int pass = 0; pass < 2 && err == hipSuccess; ++pass) {
            for (int w = 0; w < 2 && err == hipSuccess; ++w)
              err = launch_panels(p, B, C, N, nullptr, 0, nullptr, nullptr, ws, r, stream, tw);
            if (err == hipSuccess) err = hipEventRecord(e0, stream);
            for (int w = 0; w < 8 && err == hipSuccess; ++w)
              err = launch_panels(p, B, C, N, nullptr, 0, nullptr, nullptr, ws, r, stream, tw);
            if (err == hipSuccess) err = hipEventRecord(e1, stream);
            if (err == hipSuccess) err = hipEventSynchronize(e1);
            float ms = 0.0f;
            if (err == hipSuccess) err = hipEventElapsedTime(&ms, e0, e1);
            if (err == hipSuccess && (ms_r < 0.0f || ms < ms_r)) ms_r = ms;
          }
          if (err == hipSuccess && ms_r < best_ms) {
            best_ms = ms_r;
            best_runs = r;
            best_tile = tw;
          }
        }
      }
      (void)hipStreamSynchronize(stream);
      (void)hipFree(ws);
      if (err == hipSuccess) {
        p->tuned[slot].splits = best_runs;
        p->tuned[slot].split_tile = best_tile;
      }
    } else {
      (void)hipGetLastError();  // no room for the search: the cost model keeps deciding
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return err;
}

int split_runs(const sdnn_plan_s* p, int32_t N, int32_t splits) {
  return p->split_chunks > 0 ? split_runs_of(p, N, splits, false, nullptr) : 1;
}

// Partial products of the non-allocating K-split call (sdnn_spmm_split_noalloc): a
// file-scope device array, so each GPU the library runs on holds its own copy at its own
// address until the process ends.  In host code `scratch` names a host-side stand-in,
// never the device memory: host code uses only the address hipGetSymbolAddress returns
// for the current device, kept per device below.
static __device__ __align__(256) float scratch[kScratchFloats];

namespace {
std::mutex g_scratch_mu;
float* g_scratch_at[kMaxScratchDevices] = {};
}  // namespace

hipError_t scratch_address(int device, float** out) {
  if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_at[device]) {
    void* at = nullptr;
    const hipError_t e = hipGetSymbolAddress(&at, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!at) return hipErrorInvalidSymbol;
    g_scratch_at[device] = static_cast<float*>(at);
  }
  *out = g_scratch_at[device];
  return hipSuccess;
}

hipError_t launch_conv3x3(const sdnn_plan_s* p, const float* X, float* C, int32_t H, int32_t W,
                          int32_t NB, const float* bias, int epi, hipStream_t stream) {
  const int32_t hwn[3] = {H, W, NB};
  return launch_panels(p, X, C, H * W * NB, bias, epi, hwn, nullptr, nullptr, 0, stream);
}

hipError_t launch_conv3x3_split(const sdnn_plan_s* p, const float* X, float* C, int32_t H,
                                int32_t W, int32_t NB, const float* bias, int epi, int splits,
                                float* ws, hipStream_t stream) {
  const int32_t hwn[3] = {H, W, NB};
  return launch_panels(p, X, C, H * W * NB, bias, epi, hwn, nullptr, ws, splits, stream);
}

// ---------------------------------------------------------------------------------
// Dense FP32 comparison GEMM: C = act(W B + bias), W M x K, B K x N, row-major.  A
// measurement aid in the role of the paper's dense comparators (Sec. 3.2.1: outer-product
// microkernel, register blocking, cache tiling), written for the FP32 matrix cores:
//   * workgroup tile BM x BN of C (128 x 128, 96 x 128, 96 x 64 or 64 x 64, the one that
//     needs the fewest tile-rounds over the CUs), 8 waves (two per SIMD) arranged as
//     (8 / (BN / 16)) row bands x (BN / 16) column strips of 16, each wave owning its band
//     of its strip as tiles of v_mfma_f32_16x16x4_f32 (a 16 x 16 accumulator tile in 4
//     VGPRs per lane; one 16 x 4 slice of W times one 4 x 16 slice of B per issue), so each
//     B slice a wave reads serves all of its band's tiles;
//   * K is walked in stages of 32 through double-buffered LDS: the next stage's W and B
//     tiles are loaded into registers while the current one is multiplied;
//   * W's stage is stored as [k % 4][m][k / 4] so that a lane's eight values of its row
//     over the stage's eight MFMA steps are 32 contiguous bytes (two ds_read_b128), and
//     B's as [k][n] so that a lane's value of each step is one conflict-free ds_read_b32;
//   * the same fused bias + activation epilogue and a single store of C.
// Operand layouts of v_mfma_f32_16x16x4_f32 (lane l): A[i = l % 16][k = l / 16],
// B[k = l / 16][j = l % 16]; accumulator register r holds D[4 (l / 16) + r][l % 16].
namespace {
constexpr int kDenseBK = 32, kDenseWaves = 8;
constexpr int kDenseThreads = 64 * kDenseWaves;
typedef float float4_t __attribute__((ext_vector_type(4)));

template <int BM, int BN>
__global__ __launch_bounds__(kDenseThreads) void dense_gemm_kernel(
    const float* __restrict__ W, const float* __restrict__ B, float* __restrict__ C, int M, int K,
    int N, const float* __restrict__ bias, int epi) {
  constexpr int WC = BN / 16, WR = kDenseWaves / WC;  // waves along N and along M
  constexpr int TM = BM / (16 * WR);          // 16-row MFMA tiles per wave
  static_assert(WC * WR == kDenseWaves && TM * 16 * WR == BM, "tile shape");
  constexpr int S = kDenseBK / 4;             // MFMA steps (4 k each) per stage
  constexpr int A_F4 = BM * kDenseBK / 4;     // float4 loads of one W stage
  constexpr int B_F4 = kDenseBK * BN / 4;
  constexpr int A_PER = (A_F4 + kDenseThreads - 1) / kDenseThreads;
  constexpr int B_PER = (B_F4 + kDenseThreads - 1) / kDenseThreads;
  // rows padded so that the four k-groups of lanes (l / 16) read distinct LDS banks
  __shared__ __attribute__((aligned(16))) float As[2][4][BM + 2][S];
  __shared__ __attribute__((aligned(16))) float Bs[2][kDenseBK][BN + 16];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wc = wave % WC, wr = wave / WC;   // this wave's 16-column strip and row band
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int li = lane & 15, lk = lane >> 4;

  float4 ra[A_PER], rb[B_PER];
  // interior tiles (every row, column and k of the stage in range, rows 16-byte aligned)
  // take unconditional float4 loads; edge tiles check each element
  const bool rows_in = m0 + BM <= M && n0 + BN <= N && (K & 3) == 0 && (N & 3) == 0 &&
                       (((uintptr_t)W | (uintptr_t)B) & 15) == 0;
  auto load_stage = [&](int k0) {
    if (rows_in && k0 + kDenseBK <= K) {
#pragma unroll
      for (int t = 0; t < A_PER; ++t) {
        const int idx = tid + kDenseThreads * t;
        const int m = idx / (kDenseBK / 4), q = idx % (kDenseBK / 4);
        if (A_F4 % kDenseThreads == 0 || idx < A_F4)
          ra[t] = *reinterpret_cast<const float4*>(W + (size_t)(m0 + m) * K + k0 + 4 * q);
      }
#pragma unroll
      for (int t = 0; t < B_PER; ++t) {
        const int idx = tid + kDenseThreads * t;
        const int kr = idx / (BN / 4), c = idx % (BN / 4);
        if (B_F4 % kDenseThreads == 0 || idx < B_F4)
          rb[t] = *reinterpret_cast<const float4*>(B + (size_t)(k0 + kr) * N + n0 + 4 * c);
      }
      return;
    }
#pragma unroll
    for (int t = 0; t < A_PER; ++t) {
      const int idx = tid + kDenseThreads * t;
      const int m = idx / (kDenseBK / 4), q = idx % (kDenseBK / 4);
      const int gm = m0 + m, gk = k0 + 4 * q;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (idx < A_F4 && gm < M) {
        const float* src = W + (size_t)gm * K + gk;
        if (gk + 0 < K) v.x = src[0];
        if (gk + 1 < K) v.y = src[1];
        if (gk + 2 < K) v.z = src[2];
        if (gk + 3 < K) v.w = src[3];
      }
      ra[t] = v;
    }
#pragma unroll
    for (int t = 0; t < B_PER; ++t) {
      const int idx = tid + kDenseThreads * t;
      const int kr = idx / (BN / 4), c = idx % (BN / 4);
      const int gk = k0 + kr, gn = n0 + 4 * c;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (idx < B_F4 && gk < K) {
        const float* src = B + (size_t)gk * N + gn;
        if (gn + 0 < N) v.x = src[0];
        if (gn + 1 < N) v.y = src[1];
        if (gn + 2 < N) v.z = src[2];
        if (gn + 3 < N) v.w = src[3];
      }
      rb[t] = v;
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int t = 0; t < A_PER; ++t) {
      const int idx = tid + kDenseThreads * t;
      if (idx < A_F4) {
        // k = 4q + c goes to (k % 4, k / 4) = (c, q)
        const int m = idx / (kDenseBK / 4), q = idx % (kDenseBK / 4);
        As[buf][0][m][q] = ra[t].x;
        As[buf][1][m][q] = ra[t].y;
        As[buf][2][m][q] = ra[t].z;
        As[buf][3][m][q] = ra[t].w;
      }
    }
#pragma unroll
    for (int t = 0; t < B_PER; ++t) {
      const int idx = tid + kDenseThreads * t;
      if (idx < B_F4) {
        const int kr = idx / (BN / 4), c = idx % (BN / 4);
        *reinterpret_cast<float4*>(&Bs[buf][kr][4 * c]) = rb[t];
      }
    }
  };

  float4_t acc[TM];
#pragma unroll
  for (int t = 0; t < TM; ++t) acc[t] = float4_t{0.f, 0.f, 0.f, 0.f};

  const int nstages = (K + kDenseBK - 1) / kDenseBK;
  if (nstages > 0) {
    load_stage(0);
    store_stage(0);
  }
  __syncthreads();
  for (int st = 0; st < nstages; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstages) load_stage((st + 1) * kDenseBK);
    // this wave's B column (wave * 16 + li) at k = 4 s + lk, and each tile's W row
    float fb[S];
#pragma unroll
    for (int s2 = 0; s2 < S; ++s2) fb[s2] = Bs[buf][4 * s2 + lk][wc * 16 + li];
    float fa[TM][S];
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
      for (int q = 0; q < S / 4; ++q) {
        const float4 v =
            *reinterpret_cast<const float4*>(&As[buf][lk][(wr * TM + t) * 16 + li][4 * q]);
        fa[t][4 * q] = v.x;
        fa[t][4 * q + 1] = v.y;
        fa[t][4 * q + 2] = v.z;
        fa[t][4 * q + 3] = v.w;
      }
#pragma unroll
    for (int s2 = 0; s2 < S; ++s2)
#pragma unroll
      for (int t = 0; t < TM; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[t][s2], fb[s2], acc[t], 0, 0, 0);
    if (st + 1 < nstages) store_stage(buf ^ 1);
    __syncthreads();
  }

  const int j = n0 + wc * 16 + li;
  if (j >= N) return;
#pragma unroll
  for (int t = 0; t < TM; ++t) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = m0 + (wr * TM + t) * 16 + 4 * lk + r;
      if (i < M) C[(size_t)i * N + j] = activation(acc[t][r] + (bias ? bias[i] : 0.0f), epi);
    }
  }
}

template <int BM, int BN>
hipError_t launch_dense_tile(const float* W, const float* B, float* C, int32_t M, int32_t K,
                             int32_t N, const float* bias, int epi, hipStream_t stream) {
  const dim3 grid((N + BN - 1) / BN, (M + BM - 1) / BM);
  if (grid.y > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL((dense_gemm_kernel<BM, BN>), grid, dim3(kDenseThreads), 0, stream, W, B, C, M,
                     K, N, bias, epi);
  return hipGetLastError();
}
}  // namespace

// The workgroup tile: the one that minimises rounds of workgroups on the CUs times the
// work of one workgroup; among equals, first one that gives every CU at least two
// workgroups (the second hides the first one's load and barrier latency), then the
// largest tile (less operand traffic per product).
hipError_t launch_dense(const float* W, const float* B, float* C, int32_t M, int32_t K, int32_t N,
                        const float* bias, int epi, hipStream_t stream) {
  int cus = 256, dev = 0;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  struct Tile { int bm, bn; };
  const Tile tiles[] = {{128, 128}, {96, 128}, {96, 64}, {64, 64}};
  int best = 0;
  int64_t best_cost = -1;
  bool best_two = false;
  for (int c = 0; c < 4; ++c) {
    const int64_t wgs = (int64_t)((N + tiles[c].bn - 1) / tiles[c].bn) * ((M + tiles[c].bm - 1) / tiles[c].bm);
    const int64_t cost = (wgs + cus - 1) / cus * tiles[c].bm * tiles[c].bn;
    const bool two = wgs >= 2 * (int64_t)cus;
    if (best_cost < 0 || cost < best_cost || (cost == best_cost && two && !best_two)) {
      best_cost = cost;
      best = c;
      best_two = two;
    }
  }
  switch (best) {
    case 0: return launch_dense_tile<128, 128>(W, B, C, M, K, N, bias, epi, stream);
    case 1: return launch_dense_tile<96, 128>(W, B, C, M, K, N, bias, epi, stream);
    case 2: return launch_dense_tile<96, 64>(W, B, C, M, K, N, bias, epi, stream);
    default: return launch_dense_tile<64, 64>(W, B, C, M, K, N, bias, epi, stream);
  }
}

}  // namespace sdnn
