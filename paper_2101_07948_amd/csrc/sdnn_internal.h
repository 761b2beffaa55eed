// Internal declarations shared by the host-side plan code and the HIP kernels.
// Not part of the public ABI (see include/sdnn.h).
#ifndef SDNN_INTERNAL_H_
#define SDNN_INTERNAL_H_

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/sdnn.h"

namespace sdnn {

// Rows of B per LDS staging slot (the paper's split-K tiling of the dense operand,
// Sec. 3.2.2) and slots in the workgroup's LDS ring.  Chunk c of B (rows
// [c*kChunk, (c+1)*kChunk)) lives in slot c % kRing while it is in use.
constexpr int kChunk = 32;
constexpr int kRing = 4;
// Stream entries are consumed in groups of kGroup: one group is 64 bytes, one scalar
// load and one scalar-cache line.
constexpr int kGroup = 8;
// Columns of C per workgroup tile: 64 lanes x 4 consecutive columns; or, for the
// 128-column tiles, 64 lanes x 2 (the narrow layout, two workgroups per CU).
constexpr int kTileCols = 256;
constexpr int kNarrowTileCols = 128;
// Zero groups appended after the last panel: the kernel's stream prefetch may read
// this many groups past the end of a panel's stream.
constexpr int kTailGroups = 16;
// Fields of a group's address words a_0..a_7 (see Packed); L = kGroup - 1.
constexpr int kRowBits = 8;         // a_j & 0xff: row inside the panel
constexpr int kEndBit = 9;          // a_L: last group of the panel
constexpr int kRingRowShift = 10;   // (a_j >> 10) & 0x7f: row of the LDS ring
constexpr int kSyncBit = 17;        // a_L: publish progress / check readiness first
constexpr int kLoShift = 17;        // a_{L-1} >> 17: lowest chunk the group reads
constexpr int kHiShift = 18;        // a_L >> 18: highest chunk the group reads
constexpr int kLoWord = kGroup - 2, kHiWord = kGroup - 1;
constexpr int kMaxChunks = 1 << 14; // chunk numbers must fit a3's high bits
// The stream of the 128-column tiles carries the same groups with 512-byte ring rows:
// the ring-row field one bit lower and the end flag at bit 8 (narrow_stream).
constexpr int kRingRowShiftNarrow = 9;  // (a_j >> 9) & 0x7f
constexpr int kEndBitNarrow = 8;
// A row of B or C must stay below 2^31 bytes (N < 2^29): the staging and the stores
// address within a row with 32-bit byte offsets.
constexpr int64_t kMaxRowBytes = (int64_t)1 << 31;
static_assert(kRing * kChunk <= 128, "ring rows must fit 7 bits");

// Host-side packed form of W in the kernel's traversal order (Sec. 3.2.2: each
// matrix stored in its own format, read sequentially).
//
//   Panels of RW consecutive rows of the permuted matrix.  A panel's entries are
//   ordered by K-chunk, then by row inside the panel, then by column, and cut into
//   groups of kGroup.  A group never spans more than kRing chunks: the entry that
//   would make it do so starts a new group, and a group cut short this way or by the
//   end of the panel is filled with zero-weight copies of its first entry.  A group
//   is 2*kGroup dwords: the kGroup fp32 weight bits, then kGroup words
//       a_j = ((c_j % kRing) * kChunk + col_j - c_j * kChunk) << 10 | row_j
//   (c_j = chunk of the entry; the shifted part is the entry's B row in the LDS
//   ring) with extra fields in the last two words
//       a6 |= c_lo << 17, a7 |= c_hi << 18 | sync << 17 | end << 9
//   where c_lo / c_hi are the lowest / highest chunk the group reads, end marks the
//   panel's last group and sync is set on a panel's first and last groups and
//   whenever c_lo or c_hi differs from the previous group's.  Panels are stored back
//   to back; panel_start holds each panel's first group (-1: the panel has no
//   entries).  The stream ends with kTailGroups zero groups.
//
//   K-segments (split_chunks = S > 0): chunks [s*S, (s+1)*S) form segment s, no group
//   holds entries of two segments (an entry of the next segment starts a new group,
//   like one too far ahead), so each segment's first group carries the sync bit (its
//   c_lo differs from the previous group's), and seg_start[p][s] is the panel's first
//   group in segment s (-1: none).  A launch may then give each run of consecutive
//   segments to its own workgroup, which starts at the run's first group and stops at
//   the first sync group whose c_lo lies past the run.
struct Packed {
  int32_t M = 0, K = 0, RW = 0, nchunks = 0, npanels = 0;
  int64_t nnz = 0, stored = 0;     // structural entries, stored entries (with padding)
  std::vector<int32_t> perm;        // [M]   original row at permuted position (reported order)
  std::vector<int32_t> panel_rows;  // [npanels*RW] original row or -1 (padding), in the
                                    // grouping order (the row order, or balanced panels)
  std::vector<int32_t> panel_out;   // [npanels*RW] row of C each panel row is stored to
                                    // (its original row, or its position in perm for
                                    // out_permuted plans), -1 for padding
  int32_t grouping = 1;             // 1: panels are consecutive rows of perm; 2: balanced
  int32_t out_permuted = 0;         // panel_out holds positions in perm
  std::vector<int32_t> panel_start; // [npanels] first group of the panel, or -1
  std::vector<int32_t> panel_order; // [npanels] panels by stored groups, heaviest first
  std::vector<uint32_t> entries;    // [2*(stored + kTailGroups*kGroup)] dwords
  double rho = 1.0;                 // nnz / sum_p |union of the panel's column sets|
  int32_t split_chunks = 0;         // chunks per K-segment (0: one segment, no table)
  int32_t nseg = 1;                 // K-segments
  std::vector<int32_t> seg_start;   // [npanels*nseg] (split_chunks > 0 only)
};

// Panel heights of the packings a default plan holds (in this order): short panels keep
// enough waves busy when a tile has few rows per CU; taller ones carry more entries per
// K-chunk (so a group spans fewer chunks of the ring) and stage each B tile for more rows.
// The fifth, 32-row panels, serves 128-column tiles only (a plan holds it when it holds
// their stream): 14 such panels share each staged B row.  The launch picks one per call
// (choose_packing).
constexpr int kShortPanel = 4, kTallPanel = 12, kMidPanel = 8, kTallestPanel = 16;
constexpr int kDeepPanel = 32;
constexpr int kMaxPackings = 5;

// CSR validation; returns SDNN_OK or SDNN_ERR_*.
sdnn_status validate_csr(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K);
// Algorithm 1 on 64-bit column bitsets (inputs already validated).
sdnn_status reorder_bitset(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K,
                           int32_t* perm_out);
// Builds the packed stream (inputs already validated): panel p holds rows
// group[p*RW .. p*RW+RW-1] (group is a permutation of 0..M-1; out->perm is left to the
// caller).
sdnn_status pack(const int32_t* row_ptr, const int32_t* col_idx, const float* values, int32_t M,
                 int32_t K, int32_t RW, const int32_t* group, int32_t split_chunks, Packed* out);

// The stream of the 128-column tiles: each address word a_j of P.entries re-encoded with
// the ring row at bit kRingRowShiftNarrow and the end flag at kEndBitNarrow (weights,
// row, chunk and sync fields unchanged).
std::vector<uint32_t> narrow_stream(const std::vector<uint32_t>& entries);
// True if `narrow` is narrow_stream(entries) field by field (decoded independently).
bool check_narrow_stream(const std::vector<uint32_t>& entries, const std::vector<uint32_t>& narrow);

// A launch shape sdnn_plan_tune measured fastest for one N: which packing, how many
// consumer waves per workgroup and which tile width; and, for plans with K-segments, the
// workgroups along K and the tile width of the fastest K-split call (0: not measured).
struct TunedShape {
  int32_t N = 0, pack = 0, waves = 0, tile = 256, splits = 0, split_tile = 0;
};
constexpr int kTunedSlots = 8;

// One packing of the plan in device memory.
struct DevPacking {
  int32_t RW = 0, npanels = 0;
  double rho = 1.0, fill = 1.0;
  const uint32_t* entries = nullptr;      // [2*(stored + kTailGroups*kGroup)] dwords
  const uint32_t* entries_n = nullptr;    // the same groups for 128-column tiles (or null)
  const int32_t* panel_start = nullptr;   // [npanels] (in groups, -1: empty panel)
  const int32_t* panel_rows = nullptr;    // [npanels*RW] original rows (bias)
  const int32_t* panel_out = nullptr;     // [npanels*RW] rows of C the panel rows go to
  const int32_t* seg_start = nullptr;     // [npanels*nseg] in slot order (split plans)
  int32_t nseg = 1;                       // K-segments
  // (panel_start, panel_rows and panel_out are uploaded in slot order: slot j holds the
  // j-th heaviest panel; workgroups take consecutive slots)
};

}  // namespace sdnn

// The plan handle.
struct sdnn_plan_s {
  int device = -1;
  int num_cus = 0;
  int32_t M = 0, K = 0, nchunks = 0;
  int64_t nnz = 0, packed_bytes = 0;
  std::vector<int32_t> perm;
  void* d_mem = nullptr;       // one device allocation holding every packing's arrays
  int npack = 0;               // 1 (explicit panel height), 4 (short, tall, mid, tallest) or
                               // 5 (and deep, with the 128-column stream)
  int32_t out_permuted = 0;    // C rows stored in the permuted order
  int32_t in_permuted = 0;     // W's columns renamed to a caller-given order of B's rows
  int32_t split_chunks = 0;    // chunks per K-segment (0: the packings have one segment)
  int32_t grouping = 1;        // panel grouping the packings use (1: perm order, 2: balanced)
  int32_t tile_cols = 0;       // 0: the launch picks 256 or 128 columns per tile; else fixed
  const int32_t* d_perm = nullptr;  // [M] perm on the device (K-segmented plans only)
  sdnn::DevPacking pk[sdnn::kMaxPackings];
  sdnn::TunedShape tuned[sdnn::kTunedSlots];  // filled by sdnn_plan_tune
  int32_t ntuned = 0;
};

namespace sdnn {
// Kernel launchers (sdnn_kernels.hip).  Arguments are already checked.
hipError_t launch_spmm(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                       const float* bias, int epi, hipStream_t stream);
hipError_t launch_conv3x3(const sdnn_plan_s* p, const float* X, float* C, int32_t H, int32_t W,
                          int32_t NB, const float* bias, int epi, hipStream_t stream);
// K-split variants: `splits` workgroups along K (0: the library's choice; clamped to
// 1..nseg, nseg = p->pk[0].nseg), ws holds at least nseg * M * N floats; with one
// workgroup along K they are the plain launches and ws is not touched.
hipError_t launch_spmm_split(const sdnn_plan_s* p, const float* B, float* C, int32_t N,
                             const float* bias, int epi, int splits, float* ws,
                             hipStream_t stream);
hipError_t launch_conv3x3_split(const sdnn_plan_s* p, const float* X, float* C, int32_t H,
                                int32_t W, int32_t NB, const float* bias, int epi, int splits,
                                float* ws, hipStream_t stream);
// Workgroups along K that launch_spmm_split runs for `splits` (0: the library's
// choice) at N; 1 for a plan without K-segments (host only).
int split_runs(const sdnn_plan_s* p, int32_t N, int32_t splits);
// The non-allocating K-split call keeps its partial products in a fixed device array of
// kScratchFloats floats per device; scratch_address gives its address on `device`,
// which must be the current device (looked up once per device, then cached).
constexpr int64_t kScratchFloats = (int64_t)16 << 20;  // 64 MiB
constexpr int kMaxScratchDevices = 64;
hipError_t scratch_address(int device, float** out);
// The packing height, consumer waves and tile width launch_spmm uses at N for B and C
// that allow 16-byte staging (host only).
void launch_shape(const sdnn_plan_s* p, int32_t N, int32_t* panel_rows, int32_t* waves,
                  int32_t* tile_cols);
// Times every candidate launch shape of the plan at N on the given buffers (blocking)
// and records the fastest in p->tuned.
hipError_t tune_spmm(sdnn_plan_s* p, const float* B, float* C, int32_t N, hipStream_t stream,
                     TunedShape* chosen);
hipError_t launch_dense(const float* W, const float* B, float* C, int32_t M, int32_t K, int32_t N,
                        const float* bias, int epi, hipStream_t stream);
}  // namespace sdnn

#endif  // SDNN_INTERNAL_H_
