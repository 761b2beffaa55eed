// gfx950 kernels of the sparse-weight x dense-activation product (SparseDNN, arXiv
// 2101.07948, Sec. 3.2.2) and the dense FP32 comparison GEMM (Sec. 3.2.1).
//
// Sparse kernel ("panel kernel").  The paper's microkernel walks the nonzeros of a
// slice of the sparse matrix, broadcasts each nonzero into vector registers and
// multiplies it with a row slice of the dense matrix held in registers, accumulating
// into an output tile kept in registers (Sec. 3.2.2, Fig. 3).  On CDNA4 this becomes:
//   * a wavefront owns a panel of RW rows of the permuted W and an N-tile of 64*V
//     columns; each lane holds V consecutive columns of all RW output rows in VGPRs;
//   * every nonzero (weight, column) is wave-uniform: it is read by scalar loads from
//     the plan's traversal-ordered stream, so the weight lives in an SGPR;
//   * the rows of B that the workgroup's panels touch in the current K-chunk are
//     staged in LDS (the paper's split-K tiling of the dense operand), double
//     buffered, by direct global->LDS 16-byte DMA so staging of chunk k+1 overlaps the
//     FMAs of chunk k; a lane reads its V columns of a B row with one ds_read;
//   * the bias + activation epilogue is fused and C is written once, coalesced, to
//     the original (unpermuted) row.
// Plain FP32 FMA is used throughout (no MFMA: the work is not a dense contraction).
//
// Workgroups: one N-tile x one row-block of `waves` consecutive panels.  All panels of
// a row-block share the staged B chunk, so each B element fetched from L2 feeds every
// nonzero of its column inside the row-block.  The flat block id is remapped so that
// all row-blocks of an N-tile land on one XCD (blocks are dealt to the 8 XCDs round
// robin), letting them share that XCD's L2 copy of the B tile.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>

#include "sdnn_internal.h"

namespace sdnn {
namespace {

template <int V>
struct VecT;
template <>
struct VecT<1> {
  using T = float;
};
template <>
struct VecT<2> {
  using T = float2;
};
template <>
struct VecT<4> {
  using T = float4;
};

__device__ __forceinline__ void fma_acc(float& a, float w, float b) { a = fmaf(w, b, a); }
__device__ __forceinline__ void fma_acc(float2& a, float w, float2 b) {
  a.x = fmaf(w, b.x, a.x);
  a.y = fmaf(w, b.y, a.y);
}
__device__ __forceinline__ void fma_acc(float4& a, float w, float4 b) {
  a.x = fmaf(w, b.x, a.x);
  a.y = fmaf(w, b.y, a.y);
  a.z = fmaf(w, b.z, a.z);
  a.w = fmaf(w, b.w, a.w);
}

__device__ __forceinline__ float lane_get(float v, int) { return v; }
__device__ __forceinline__ float lane_get(float2 v, int i) { return i == 0 ? v.x : v.y; }
__device__ __forceinline__ float lane_get(float4 v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}
__device__ __forceinline__ void lane_set(float& v, int, float x) { v = x; }
__device__ __forceinline__ void lane_set(float2& v, int i, float x) {
  if (i == 0) v.x = x; else v.y = x;
}
__device__ __forceinline__ void lane_set(float4& v, int i, float x) {
  if (i == 0) v.x = x; else if (i == 1) v.y = x; else if (i == 2) v.z = x; else v.w = x;
}

__device__ __forceinline__ float activation(float x, int epi) {
  if (epi == SDNN_EPI_RELU) return fmaxf(x, 0.0f);
  if (epi == SDNN_EPI_GELU) return 0.5f * x * (1.0f + erff(x * 0.70710678118654752f));
  return x;
}

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Direct global -> LDS copy of `size` bytes per active lane: lane i's bytes land at
// lds_base + i * size (lds_base is wave-uniform).  The compiler tracks these as LDS
// writes to the named buffer only, so reads of the other staging buffer are not held
// behind them; the kernel waits for them (vmcnt(0)) right before the barrier that
// publishes the buffer.
__device__ __forceinline__ void dma16(const float* gptr, lds_ptr_t lds_base) {
  __builtin_amdgcn_global_load_lds(gptr, lds_base, 16, 0, 0);
}
__device__ __forceinline__ void dma4(const float* gptr, lds_ptr_t lds_base) {
  __builtin_amdgcn_global_load_lds(gptr, lds_base, 4, 0, 0);
}
// s_waitcnt vmcnt(0) (gfx9 encoding: expcnt and lgkmcnt fields left at their maximum)
__device__ __forceinline__ void wait_vmcnt0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Scalar launch parameters (the pointers are separate __restrict__ kernel arguments so
// the compiler may read the plan stream through the scalar cache).
struct SpmmArgs {
  int32_t K, N, nchunks, npanels;
  int32_t n_rb;      // row-blocks per N-tile
  int32_t total_wg;  // real workgroups (n_tiles * n_rb)
  int32_t per_xcd;   // launched grid / 8
  int32_t epi;
};

// Stages rows [k*kChunk, k*kChunk + kChunk) x columns [n0, n0 + 64*V) of B into an LDS
// buffer laid out row-major with 64*V floats per row.  Out-of-range rows and columns
// are skipped: no stream entry refers to such a row, and such columns are never stored.
template <int V, bool VEC>
__device__ __forceinline__ void stage_chunk(const float* __restrict__ B, int K, int N, int n0,
                                            int k, float* buf, int wave, int nwaves, int lane) {
  constexpr int COLS = 64 * V;
  constexpr int CHUNK_FLOATS = kChunk * COLS;
  const int k0 = k * kChunk;
  if (VEC) {
    // 16-byte pieces, 64 per instruction (1 KB of LDS)
    constexpr int PIECES_PER_ROW = COLS / 4;
    constexpr int INSTS = CHUNK_FLOATS / 4 / 64;
    for (int j = wave; j < INSTS; j += nwaves) {
      const int q = j * 64 + lane;
      const int row = q / PIECES_PER_ROW;
      const int col = n0 + (q - row * PIECES_PER_ROW) * 4;
      const int krow = k0 + row;
      if (krow < K && col < N) dma16(B + (size_t)krow * N + col, (lds_ptr_t)(buf + j * 256));
    }
  } else {
    constexpr int INSTS = CHUNK_FLOATS / 64;
    for (int j = wave; j < INSTS; j += nwaves) {
      const int q = j * 64 + lane;
      const int row = q / COLS;
      const int col = n0 + (q - row * COLS);
      const int krow = k0 + row;
      if (krow < K && col < N) dma4(B + (size_t)krow * N + col, (lds_ptr_t)(buf + j * 64));
    }
  }
}

// FMAs of one K-chunk for one panel: for each of the RW rows (static register tile),
// walk its entries in this chunk; each entry is (weight, column offset in the chunk),
// read with scalar loads; the lane's V columns of that B row come from one ds_read.
// The RW 16-bit counts of a segment are read as RW/2 dwords (scalar loads are dword
// granular); RW is even and each segment's counts start 4-byte aligned.
template <int V, int RW>
__device__ __forceinline__ void panel_chunk(typename VecT<V>::T (&acc)[RW],
                                            const uint2* __restrict__ ep,
                                            const uint32_t* __restrict__ cnt2, const float* buf,
                                            int lane) {
  using VT = typename VecT<V>::T;
  const VT* lb = reinterpret_cast<const VT*>(buf) + lane;
  uint32_t packed[RW / 2];
#pragma unroll
  for (int i = 0; i < RW / 2; ++i) packed[i] = cnt2[i];
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int c = (packed[r >> 1] >> ((r & 1) * 16)) & 0xffff;
    for (int j = 0; j < c; ++j) {
      const uint2 e = ep[j];
      const VT b = lb[e.y * 64];
      fma_acc(acc[r], __uint_as_float(e.x), b);
    }
    ep += c;
  }
}

// V: columns per lane; RW: rows per panel; VEC: B rows are 16-byte aligned (N % 4 == 0
// and B 16-byte aligned), so staging uses 16-byte DMA and C stores are vectorised.
template <int V, int RW, bool VEC>
__global__ __launch_bounds__(1024) void spmm_panel_kernel(
    const uint2* __restrict__ entries, const int32_t* __restrict__ segs,
    const uint32_t* __restrict__ counts, const int32_t* __restrict__ panel_rows,
    const float* __restrict__ B, float* __restrict__ C, const float* __restrict__ bias,
    SpmmArgs a) {
  using VT = typename VecT<V>::T;
  constexpr int COLS = 64 * V;
  constexpr int CHUNK_FLOATS = kChunk * COLS;
  // two staging buffers as two arrays, so the compiler can tell them apart
  __shared__ __attribute__((aligned(16))) float buf0[CHUNK_FLOATS];
  __shared__ __attribute__((aligned(16))) float buf1[CHUNK_FLOATS];

  const int bid = blockIdx.x;
  const int lin = (bid & 7) * a.per_xcd + (bid >> 3);
  if (lin >= a.total_wg) return;  // whole workgroup leaves before any barrier
  const int tile = lin / a.n_rb;
  const int rb = lin - tile * a.n_rb;
  const int nwaves = blockDim.x >> 6;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int panel = rb * nwaves + wave;
  const bool active = panel < a.npanels;
  const int n0 = tile * COLS;
  const int nchunks = a.nchunks;

  VT acc[RW];
#pragma unroll
  for (int r = 0; r < RW; ++r) acc[r] = VT{};

  const int seg0 = panel * nchunks;
  if (nchunks > 0) stage_chunk<V, VEC>(B, a.K, a.N, n0, 0, buf0, wave, nwaves, lane);
  // two chunks per trip so that each buffer is named statically
  for (int k = 0; k < nchunks; k += 2) {
    wait_vmcnt0();
    __syncthreads();  // chunk k is in buf0; every wave is done reading buf1
    if (k + 1 < nchunks) stage_chunk<V, VEC>(B, a.K, a.N, n0, k + 1, buf1, wave, nwaves, lane);
    if (active)
      panel_chunk<V, RW>(acc, entries + segs[seg0 + k], counts + (size_t)(seg0 + k) * (RW / 2),
                         buf0, lane);
    if (k + 1 >= nchunks) break;
    wait_vmcnt0();
    __syncthreads();  // chunk k+1 is in buf1; every wave is done reading buf0
    if (k + 2 < nchunks) stage_chunk<V, VEC>(B, a.K, a.N, n0, k + 2, buf0, wave, nwaves, lane);
    if (active)
      panel_chunk<V, RW>(acc, entries + segs[seg0 + k + 1],
                         counts + (size_t)(seg0 + k + 1) * (RW / 2), buf1, lane);
  }

  if (!active) return;
  const int ncol = n0 + lane * V;
#pragma unroll
  for (int r = 0; r < RW; ++r) {
    const int orig = panel_rows[panel * RW + r];
    if (orig < 0) continue;
    const float bb = bias ? bias[orig] : 0.0f;
    float* crow = C + (size_t)orig * a.N;
    if (VEC && ncol + V <= a.N) {
      VT out;
#pragma unroll
      for (int i = 0; i < V; ++i) lane_set(out, i, activation(lane_get(acc[r], i) + bb, a.epi));
      *reinterpret_cast<VT*>(crow + ncol) = out;
    } else {
#pragma unroll
      for (int i = 0; i < V; ++i)
        if (ncol + i < a.N) crow[ncol + i] = activation(lane_get(acc[r], i) + bb, a.epi);
    }
  }
}

struct SpmmPtrs {
  const uint2* entries;
  const int32_t* seg;
  const uint32_t* counts;
  const int32_t* panel_rows;
  const float* B;
  float* C;
  const float* bias;
};

template <int V, int RW, bool VEC>
hipError_t launch_variant(const SpmmPtrs& p, const SpmmArgs& args, int waves, int grid,
                          hipStream_t stream) {
  hipLaunchKernelGGL((spmm_panel_kernel<V, RW, VEC>), dim3(grid), dim3(64 * waves), 0, stream,
                     p.entries, p.seg, p.counts, p.panel_rows, p.B, p.C, p.bias, args);
  return hipGetLastError();
}

template <int V, bool VEC>
hipError_t launch_rw(int RW, const SpmmPtrs& p, const SpmmArgs& args, int waves, int grid,
                     hipStream_t stream) {
  switch (RW) {
    case 4: return launch_variant<V, 4, VEC>(p, args, waves, grid, stream);
    case 8: return launch_variant<V, 8, VEC>(p, args, waves, grid, stream);
    case 16: return launch_variant<V, 16, VEC>(p, args, waves, grid, stream);
  }
  return hipErrorInvalidValue;
}

int env_int(const char* name, int dflt) {
  const char* s = getenv(name);
  return s ? atoi(s) : dflt;
}

struct LaunchCfg {
  int V, waves, n_tiles, n_rb;
};

// Chooses columns per lane (V) and panels per workgroup so that the grid covers the
// chip about once: wider N-tiles need fewer instructions per FMA (one address add
// per nonzero is shared by V FMAs), more panels per workgroup re-read less of B.
LaunchCfg choose_cfg(const sdnn_plan_s* p, int N) {
  const int target = p->num_cus > 0 ? p->num_cus : 256;
  const int forceV = env_int("SDNN_FORCE_V", 0);
  const int forceW = env_int("SDNN_FORCE_WAVES", 0);
  LaunchCfg best{1, 1, 1, 1};
  for (int V : {4, 2, 1}) {
    if (forceV && V != forceV) continue;
    LaunchCfg c;
    c.V = V;
    c.n_tiles = (N + 64 * V - 1) / (64 * V);
    if (forceW > 0) {
      c.waves = forceW < p->npanels ? forceW : p->npanels;
    } else {
      int n_rb = (target + c.n_tiles - 1) / c.n_tiles;
      if (n_rb > p->npanels) n_rb = p->npanels;
      c.waves = (p->npanels + n_rb - 1) / n_rb;
    }
    if (c.waves > 16) c.waves = 16;
    if (c.waves < 1) c.waves = 1;
    c.n_rb = (p->npanels + c.waves - 1) / c.waves;
    best = c;
    if (forceV || (int64_t)c.n_tiles * c.n_rb >= (int64_t)target * 9 / 10) break;
  }
  return best;
}

}  // namespace

hipError_t launch_spmm(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                       const float* bias, int epi, hipStream_t stream) {
  const LaunchCfg cfg = choose_cfg(p, N);
  const SpmmPtrs ptrs{p->d_entries, p->d_seg, reinterpret_cast<const uint32_t*>(p->d_counts),
                      p->d_panel_rows, B, C, bias};
  SpmmArgs args;
  args.K = p->K;
  args.N = N;
  args.nchunks = p->nchunks;
  args.npanels = p->npanels;
  args.n_rb = cfg.n_rb;
  const int64_t total = (int64_t)cfg.n_tiles * cfg.n_rb;
  if (total > (int64_t)1 << 30) return hipErrorInvalidValue;
  const int64_t grid = (total + 7) / 8 * 8;
  args.total_wg = (int32_t)total;
  args.per_xcd = (int32_t)(grid / 8);
  args.epi = epi;
  const bool vec = (N % 4 == 0) && (((uintptr_t)B & 15) == 0) && (((uintptr_t)C & 15) == 0);
  switch (cfg.V) {
    case 4:
      return vec ? launch_rw<4, true>(p->RW, ptrs, args, cfg.waves, (int)grid, stream)
                 : launch_rw<4, false>(p->RW, ptrs, args, cfg.waves, (int)grid, stream);
    case 2:
      return vec ? launch_rw<2, true>(p->RW, ptrs, args, cfg.waves, (int)grid, stream)
                 : launch_rw<2, false>(p->RW, ptrs, args, cfg.waves, (int)grid, stream);
    default:
      return vec ? launch_rw<1, true>(p->RW, ptrs, args, cfg.waves, (int)grid, stream)
                 : launch_rw<1, false>(p->RW, ptrs, args, cfg.waves, (int)grid, stream);
  }
}

// ---------------------------------------------------------------------------------
// Dense FP32 comparison GEMM: C = act(W B + bias), W M x K, B K x N, row-major.
// 64 x 64 output tile per 256-thread workgroup, 4 x 4 per thread, K tiled by 16
// through LDS.  A measurement aid only.
namespace {
constexpr int DT = 64, DK = 16;

__global__ __launch_bounds__(256) void dense_gemm_kernel(const float* __restrict__ W,
                                                         const float* __restrict__ B,
                                                         float* __restrict__ C, int M, int K,
                                                         int N, const float* __restrict__ bias,
                                                         int epi) {
  __shared__ float As[DK][DT + 4];
  __shared__ float Bs[DK][DT + 4];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * DT, n0 = blockIdx.x * DT;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += DK) {
    for (int i = threadIdx.x; i < DT * DK; i += 256) {
      const int mm = i / DK, kk = i % DK;
      const int gm = m0 + mm, gk = k0 + kk;
      As[kk][mm] = (gm < M && gk < K) ? W[(size_t)gm * K + gk] : 0.0f;
      const int kb = i / DT, nn = i % DT;
      const int gkb = k0 + kb, gn = n0 + nn;
      Bs[kb][nn] = (gkb < K && gn < N) ? B[(size_t)gkb * N + gn] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < DK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int gm = m0 + ty * 4 + i;
    if (gm >= M) continue;
    const float bb = bias ? bias[gm] : 0.0f;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int gn = n0 + tx * 4 + j;
      if (gn < N) C[(size_t)gm * N + gn] = activation(acc[i][j] + bb, epi);
    }
  }
}
}  // namespace

hipError_t launch_dense(const float* W, const float* B, float* C, int32_t M, int32_t K, int32_t N,
                        const float* bias, int epi, hipStream_t stream) {
  dim3 grid((N + DT - 1) / DT, (M + DT - 1) / DT);
  if (grid.y > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(dense_gemm_kernel, grid, dim3(256), 0, stream, W, B, C, M, K, N, bias, epi);
  return hipGetLastError();
}

}  // namespace sdnn
