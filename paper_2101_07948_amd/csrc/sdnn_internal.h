// Internal declarations shared by the host-side plan code and the HIP kernels.
// Not part of the public ABI (see include/sdnn.h).
#ifndef SDNN_INTERNAL_H_
#define SDNN_INTERNAL_H_

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/sdnn.h"

namespace sdnn {

// Rows of B staged in LDS per pass over the reduction dimension (the paper's split-K
// tiling of the dense operand, Sec. 3.2.2).  The packed stream is cut at these
// boundaries, so the value is fixed at plan creation.
constexpr int kChunk = 64;
// Stream entries are consumed in groups of kGroup.
constexpr int kGroup = 4;
// Columns of C per workgroup tile: 64 lanes x 4 consecutive columns.
constexpr int kTileCols = 256;
// Zero groups appended after the last segment: the kernel's stream prefetch may read
// this many groups past the end of a panel's stream.
constexpr int kTailGroups = 24;
// Marks the last group of a segment (in the group's last column word).
constexpr int kSegEndBit = 9;

// Host-side packed form of W in the kernel's traversal order (Sec. 3.2.2: each
// matrix stored in its own format, read sequentially).
//
//   Panels of RW consecutive rows of the permuted matrix.  For panel p and chunk k the
//   segment holds the entries of rows 0..RW-1 of the panel (row by row, each row in
//   ascending column order) whose column lies in [k*kChunk, (k+1)*kChunk), padded at
//   its end with zero entries to whole groups, and at least one group long.  A group
//   of kGroup entries is stored as 2*kGroup dwords: the kGroup fp32 weight bits, then
//   kGroup words (column offset inside the chunk << 10) | r; bit kSegEndBit of the
//   group's last word is set on the last group of a segment.  A panel's segments are
//   stored back to back in chunk order, panels in order, and the stream ends with
//   kTailGroups zero groups so that a kernel may prefetch that many groups past it.
struct Packed {
  int32_t M = 0, K = 0, RW = 0, nchunks = 0, npanels = 0;
  int64_t nnz = 0, stored = 0;     // structural entries, stored entries (with padding)
  std::vector<int32_t> perm;        // [M]   original row at permuted position
  std::vector<int32_t> panel_rows;  // [npanels*RW] original row or -1 (padding)
  std::vector<int32_t> seg_start;   // [npanels*nchunks + 1] first group of each segment
  std::vector<uint16_t> counts;     // [npanels*nchunks*RW] real entries per (panel, chunk, row)
                                    // (host-side only, used by the self-check)
  std::vector<uint32_t> entries;    // [2*(stored + kTailGroups*kGroup)] dwords
  double rho = 1.0;                 // nnz / sum_p |union of the panel's column sets|
};

// CSR validation; returns SDNN_OK or SDNN_ERR_*.
sdnn_status validate_csr(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K);
// Algorithm 1 on 64-bit column bitsets (inputs already validated).
sdnn_status reorder_bitset(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K,
                           int32_t* perm_out);
// Builds the packed stream (inputs already validated, perm is a permutation of 0..M-1).
sdnn_status pack(const int32_t* row_ptr, const int32_t* col_idx, const float* values, int32_t M,
                 int32_t K, int32_t RW, const int32_t* perm, Packed* out);

}  // namespace sdnn

// The plan handle.
struct sdnn_plan_s {
  int device = -1;
  int num_cus = 0;
  int32_t M = 0, K = 0, RW = 0, nchunks = 0, npanels = 0;
  int64_t nnz = 0, packed_bytes = 0;
  double rho = 1.0, fill = 1.0;
  std::vector<int32_t> perm;
  void* d_mem = nullptr;             // one device allocation holding the three arrays
  const uint32_t* d_entries = nullptr;  // [2*(stored + kTailGroups*kGroup)] dwords
  const int32_t* d_seg = nullptr;    // [npanels*nchunks + 1] (in groups)
  const int32_t* d_panel_rows = nullptr;  // [npanels*RW]
};

namespace sdnn {
// Kernel launchers (sdnn_kernels.hip).  Arguments are already checked.
hipError_t launch_spmm(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                       const float* bias, int epi, hipStream_t stream);
hipError_t launch_dense(const float* W, const float* B, float* C, int32_t M, int32_t K, int32_t N,
                        const float* bias, int epi, hipStream_t stream);
}  // namespace sdnn

#endif  // SDNN_INTERNAL_H_
