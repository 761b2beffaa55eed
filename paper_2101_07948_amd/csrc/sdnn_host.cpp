// Host side of the C ABI: CSR validation, the greedy weight-row permutation
// (Sec. 3.1.2, Algorithm 1) on column bitsets, packing of W into the kernel's
// traversal-ordered stream (Sec. 3.2.2), plan lifetime and argument checks.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <utility>
#include <new>
#include <vector>

#include "sdnn_internal.h"

namespace sdnn {

sdnn_status validate_csr(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K) {
  if (M < 0 || K < 0) return SDNN_ERR_DIM;
  if (!row_ptr) return SDNN_ERR_NULL;
  if (row_ptr[0] != 0) return SDNN_ERR_CSR;
  for (int32_t i = 0; i < M; ++i)
    if (row_ptr[i + 1] < row_ptr[i]) return SDNN_ERR_CSR;
  const int32_t nnz = row_ptr[M];
  if (nnz > 0 && !col_idx) return SDNN_ERR_NULL;
  for (int32_t i = 0; i < M; ++i) {
    for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p) {
      const int32_t c = col_idx[p];
      if (c < 0 || c >= K) return SDNN_ERR_CSR;
      if (p > row_ptr[i] && c <= col_idx[p - 1]) return SDNN_ERR_CSR;  // unsorted or duplicate
    }
  }
  return SDNN_OK;
}

// Algorithm 1 with each row's column set held as ceil(K/64) 64-bit words; the overlap
// |cols(prev) ∩ cols(x)| is a popcount of the AND.  Picks: first the densest row;
// then, repeatedly, the remaining row with the largest overlap with the row placed
// last.  Ties: more nonzeros first, then the lower original index.
sdnn_status reorder_bitset(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K,
                           int32_t* perm_out) {
  if (M == 0) return SDNN_OK;
  const int64_t words = (K + 63) / 64;
  std::vector<uint64_t> bits;
  std::vector<int32_t> remaining;
  try {
    bits.assign((size_t)M * (size_t)std::max<int64_t>(words, 1), 0);
    remaining.resize(M);
  } catch (const std::bad_alloc&) {
    return SDNN_ERR_ALLOC;
  }
  for (int32_t i = 0; i < M; ++i) {
    uint64_t* row = bits.data() + (size_t)i * words;
    for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
      row[col_idx[p] >> 6] |= 1ull << (col_idx[p] & 63);
  }
  auto nnz = [&](int32_t x) { return row_ptr[x + 1] - row_ptr[x]; };

  int32_t first = 0;
  for (int32_t x = 1; x < M; ++x)
    if (nnz(x) > nnz(first)) first = x;
  perm_out[0] = first;

  // remaining rows, kept in ascending index order so equal keys resolve to the lower index
  int32_t nrem = 0;
  for (int32_t x = 0; x < M; ++x)
    if (x != first) remaining[nrem++] = x;

  for (int32_t i = 1; i < M; ++i) {
    const uint64_t* prev = bits.data() + (size_t)perm_out[i - 1] * words;
    int32_t best_pos = 0, best_ov = -1, best_nnz = -1;
    for (int32_t j = 0; j < nrem; ++j) {
      const int32_t x = remaining[j];
      const uint64_t* row = bits.data() + (size_t)x * words;
      int32_t ov = 0;
      for (int64_t w = 0; w < words; ++w) ov += __builtin_popcountll(prev[w] & row[w]);
      const int32_t nx = nnz(x);
      if (ov > best_ov || (ov == best_ov && nx > best_nnz)) {
        best_pos = j;
        best_ov = ov;
        best_nnz = nx;
      }
    }
    perm_out[i] = remaining[best_pos];
    // erase while keeping ascending order
    memmove(remaining.data() + best_pos, remaining.data() + best_pos + 1,
            sizeof(int32_t) * (size_t)(nrem - best_pos - 1));
    --nrem;
  }
  return SDNN_OK;
}

namespace {
struct Entry {
  uint32_t w;      // weight bits
  uint32_t a;      // ring row << 10 | row
  int32_t chunk;
};

// Writes one group (n <= kGroup real entries from e) with its fields.
void emit_group(std::vector<uint32_t>& out, const Entry* e, int n, bool first, bool last,
                int32_t* prev_lo, int32_t* prev_hi) {
  uint32_t w[kGroup], a[kGroup];
  for (int j = 0; j < kGroup; ++j) {
    w[j] = j < n ? e[j].w : 0u;            // zero-weight copies of the first entry
    a[j] = j < n ? e[j].a : e[0].a;
  }
  const int32_t lo = e[0].chunk, hi = e[n - 1].chunk;
  const bool sync = first || last || lo != *prev_lo || hi != *prev_hi;
  a[kLoWord] |= (uint32_t)lo << kLoShift;
  a[kHiWord] |= (uint32_t)hi << kHiShift | (uint32_t)sync << kSyncBit | (uint32_t)last << kEndBit;
  *prev_lo = lo;
  *prev_hi = hi;
  for (int j = 0; j < kGroup; ++j) out.push_back(w[j]);
  for (int j = 0; j < kGroup; ++j) out.push_back(a[j]);
}
}  // namespace

sdnn_status pack(const int32_t* row_ptr, const int32_t* col_idx, const float* values, int32_t M,
                 int32_t K, int32_t RW, const int32_t* group, int32_t split_chunks, Packed* out) {
  try {
    Packed& P = *out;
    P.M = M;
    P.K = K;
    P.RW = RW;
    P.nnz = M ? row_ptr[M] : 0;
    P.nchunks = (K + kChunk - 1) / kChunk;
    if (P.nchunks > kMaxChunks) return SDNN_ERR_DIM;
    P.npanels = (M + RW - 1) / RW;
    P.panel_rows.assign((size_t)P.npanels * RW, -1);
    for (int32_t i = 0; i < M; ++i) P.panel_rows[i] = group[i];
    P.panel_start.assign((size_t)P.npanels, -1);
    P.split_chunks = split_chunks;
    P.nseg = split_chunks > 0 ? std::max(1, (P.nchunks + split_chunks - 1) / split_chunks) : 1;
    if (split_chunks > 0) P.seg_start.assign((size_t)P.npanels * P.nseg, -1);
    auto seg_of = [&](int32_t c) { return split_chunks > 0 ? c / split_chunks : 0; };
    P.entries.clear();
    P.entries.reserve((size_t)(P.nnz + P.nnz / 8 + 64) * 2);

    std::vector<int32_t> cursor(RW);
    std::vector<int32_t> mark((size_t)std::max(K, 1), -1);
    std::vector<Entry> ent;
    int64_t union_total = 0;
    for (int32_t p = 0; p < P.npanels; ++p) {
      ent.clear();
      for (int32_t r = 0; r < RW; ++r) {
        const int32_t orig = P.panel_rows[(size_t)p * RW + r];
        cursor[r] = orig >= 0 ? row_ptr[orig] : 0;
        if (orig >= 0)
          for (int32_t q = row_ptr[orig]; q < row_ptr[orig + 1]; ++q)
            if (mark[col_idx[q]] != p) {
              mark[col_idx[q]] = p;
              ++union_total;
            }
      }
      // the panel's entries in (chunk, row, column) order
      for (int32_t c = 0; c < P.nchunks; ++c) {
        const int32_t hi = (c + 1) * kChunk;
        const uint32_t ring_base = (uint32_t)((c % kRing) * kChunk);
        for (int32_t r = 0; r < RW; ++r) {
          const int32_t orig = P.panel_rows[(size_t)p * RW + r];
          if (orig < 0) continue;
          int32_t q = cursor[r];
          const int32_t end = row_ptr[orig + 1];
          for (; q < end && col_idx[q] < hi; ++q) {
            Entry e;
            memcpy(&e.w, &values[q], 4);
            e.a = (ring_base + (uint32_t)(col_idx[q] - c * kChunk)) << kRingRowShift | (uint32_t)r;
            e.chunk = c;
            ent.push_back(e);
          }
          cursor[r] = q;
        }
      }
      if (ent.empty()) continue;
      P.panel_start[p] = (int32_t)(P.entries.size() / (2 * kGroup));
      int32_t prev_lo = -1, prev_hi = -1;
      size_t i = 0;
      bool first = true;
      while (i < ent.size()) {
        // a group never reads more than kRing chunks, nor two K-segments
        const int32_t seg = seg_of(ent[i].chunk);
        int n = 1;
        while (n < kGroup && i + n < ent.size() && ent[i + n].chunk - ent[i].chunk < kRing &&
               seg_of(ent[i + n].chunk) == seg)
          ++n;
        const bool last = i + n == ent.size();
        // a segment's first group differs from the group before it in c_lo, so it
        // carries the sync bit, where a workgroup ending at that segment stops
        const bool seg_first = first || seg_of(ent[i - 1].chunk) != seg;
        if (split_chunks > 0 && seg_first)
          P.seg_start[(size_t)p * P.nseg + seg] = (int32_t)(P.entries.size() / (2 * kGroup));
        emit_group(P.entries, &ent[i], n, first, last, &prev_lo, &prev_hi);
        first = false;
        i += n;
      }
    }
    P.stored = (int64_t)(P.entries.size() / 2);
    if (P.stored > INT32_MAX - kTailGroups * kGroup) return SDNN_ERR_DIM;
    for (int i = 0; i < kTailGroups * kGroup; ++i) {  // tail padding for the prefetch
      P.entries.push_back(0u);
      P.entries.push_back(0u);
    }
    P.rho = union_total ? (double)P.nnz / (double)union_total : 1.0;
    // workgroup order: panels by stored groups, heaviest first (ties: lower panel), so
    // that consecutive panels -- one workgroup's -- carry similar work and the heaviest
    // workgroups are dispatched first
    std::vector<int64_t> groups((size_t)P.npanels, 0);
    for (int32_t p = 0; p < P.npanels; ++p) {
      if (P.panel_start[p] < 0) continue;
      int64_t g = P.panel_start[p];
      while (!((P.entries[(size_t)g * 2 * kGroup + kGroup + kHiWord] >> kEndBit) & 1u)) ++g;
      groups[p] = g + 1 - P.panel_start[p];
    }
    P.panel_order.resize((size_t)P.npanels);
    for (int32_t p = 0; p < P.npanels; ++p) P.panel_order[p] = p;
    std::stable_sort(P.panel_order.begin(), P.panel_order.end(),
                     [&](int32_t a, int32_t b) { return groups[a] > groups[b]; });
  } catch (const std::bad_alloc&) {
    return SDNN_ERR_ALLOC;
  }
  return SDNN_OK;
}

// Independent re-walk of a packed stream.  Decoding each panel's groups must give
// back exactly the CSR entries of the panel's rows (weight bits unchanged) in (chunk,
// row, column) order; every field of every group must be consistent (chunk range at
// most kRing wide and inside it every entry's chunk, sync and end flags set exactly
// where the format says, unused bits clear); zero-weight filler copies of a group's
// first entry may only close a group that ends the panel or that the next entry
// could not join; and the stream must end with kTailGroups zero groups.
static bool check_packed(const int32_t* row_ptr, const int32_t* col_idx, const float* values,
                         const Packed& P) {
  if ((int64_t)P.entries.size() != 2 * (P.stored + kTailGroups * kGroup)) return false;
  if (P.stored % kGroup != 0) return false;
  if ((int64_t)P.panel_start.size() != P.npanels) return false;
  const bool split = P.split_chunks > 0;
  auto seg_of = [&](int32_t c) { return split ? c / P.split_chunks : 0; };
  if (split ? (P.nseg != std::max(1, (P.nchunks + P.split_chunks - 1) / P.split_chunks) ||
               (int64_t)P.seg_start.size() != (int64_t)P.npanels * P.nseg)
            : (P.nseg != 1 || !P.seg_start.empty()))
    return false;
  const int64_t ngroups = P.stored / kGroup;
  std::vector<char> seen((size_t)P.nnz, 0);
  int64_t expect_group = 0;  // panels are stored back to back
  for (int32_t p = 0; p < P.npanels; ++p) {
    // the panel's CSR entries in (chunk, row, column) order
    std::vector<int64_t> want;
    for (int32_t c = 0; c < P.nchunks; ++c)
      for (int32_t r = 0; r < P.RW; ++r) {
        const int32_t orig = P.panel_rows[(size_t)p * P.RW + r];
        if (orig < 0) continue;
        for (int32_t q = row_ptr[orig]; q < row_ptr[orig + 1]; ++q)
          if (col_idx[q] / kChunk == c) want.push_back(q);
      }
    if (want.empty()) {
      if (P.panel_start[p] != -1) return false;
      for (int32_t sg = 0; split && sg < P.nseg; ++sg)
        if (P.seg_start[(size_t)p * P.nseg + sg] != -1) return false;
      continue;
    }
    std::vector<int64_t> seg_first(split ? (size_t)P.nseg : 0, -1);
    if (P.panel_start[p] != expect_group) return false;
    size_t k = 0;  // next wanted entry
    int32_t prev_lo = -1, prev_hi = -1;
    for (int64_t g = P.panel_start[p];; ++g) {
      if (g >= ngroups) return false;
      const uint32_t* w = &P.entries[(size_t)g * 2 * kGroup];
      const uint32_t* a = w + kGroup;
      const int32_t lo = (int32_t)(a[kLoWord] >> kLoShift), hi = (int32_t)(a[kHiWord] >> kHiShift);
      const bool sync = (a[kHiWord] >> kSyncBit) & 1u, last = (a[kHiWord] >> kEndBit) & 1u;
      if (lo > hi || hi - lo >= kRing || hi >= P.nchunks || lo < prev_lo) return false;
      if (seg_of(hi) != seg_of(lo)) return false;
      const bool first = g == P.panel_start[p];
      if (sync != (first || last || lo != prev_lo || hi != prev_hi)) return false;
      if (split && seg_first[seg_of(lo)] < 0) {
        if (!sync) return false;  // a workgroup's run of segments stops at this group
        seg_first[seg_of(lo)] = g;
      }
      prev_lo = lo;
      prev_hi = hi;
      int nreal = 0;
      int32_t max_chunk = -1;
      for (int j = 0; j < kGroup; ++j) {
        uint32_t fields = a[j] & ((1u << kLoShift) - 1);
        if (j == kHiWord) fields &= ~(1u << kEndBit);
        if ((fields >> kRowBits) & ((1u << (kRingRowShift - kRowBits)) - 1)) return false;
        if (j < kLoWord && (a[j] >> kLoShift) != 0u) return false;
        const uint32_t row = fields & ((1u << kRowBits) - 1);
        const uint32_t ring_row = fields >> kRingRowShift;
        if (row >= (uint32_t)P.RW || ring_row >= (uint32_t)(kRing * kChunk)) return false;
        const int32_t slot = (int32_t)ring_row / kChunk;
        const int32_t chunk = lo + ((slot - lo % kRing) % kRing + kRing) % kRing;
        const int32_t col = chunk * kChunk + (int32_t)ring_row % kChunk;
        const bool filler = j > 0 && w[j] == 0u && (fields == (a[0] & ((1u << kLoShift) - 1)));
        if (filler) {
          if (nreal == 0) return false;
          continue;
        }
        if (nreal != j) return false;  // fillers only after the real entries
        ++nreal;
        if (k >= want.size()) return false;
        const int64_t q = want[k++];
        const int32_t orig = P.panel_rows[(size_t)p * P.RW + row];
        if (orig < 0 || q < row_ptr[orig] || q >= row_ptr[orig + 1]) return false;
        if (col_idx[q] != col || chunk > hi || seen[q]) return false;
        uint32_t vbits;
        memcpy(&vbits, &values[q], 4);
        if (vbits != w[j]) return false;
        seen[q] = 1;
        max_chunk = std::max(max_chunk, chunk);
      }
      if (max_chunk != hi) return false;
      if (last != (k == want.size())) return false;
      // cut short: the next entry is too far ahead or in the next K-segment
      const int32_t next_chunk = last ? -1 : col_idx[want[k]] / kChunk;
      if (nreal < kGroup && !last && next_chunk - lo < kRing && seg_of(next_chunk) == seg_of(lo))
        return false;
      if (last) {
        expect_group = g + 1;
        break;
      }
    }
    for (int32_t sg = 0; split && sg < P.nseg; ++sg)
      if (P.seg_start[(size_t)p * P.nseg + sg] != seg_first[sg]) return false;
  }
  if (expect_group != ngroups) return false;
  // panel_order: a permutation of the panels, by stored groups (descending)
  if ((int64_t)P.panel_order.size() != P.npanels) return false;
  {
    std::vector<char> used((size_t)std::max(P.npanels, 1), 0);
    int64_t prev = INT64_MAX;
    for (int32_t j = 0; j < P.npanels; ++j) {
      const int32_t p = P.panel_order[j];
      if (p < 0 || p >= P.npanels || used[p]) return false;
      used[p] = 1;
      int64_t g = 0;
      if (P.panel_start[p] >= 0) {
        int64_t e = P.panel_start[p];
        while (!((P.entries[(size_t)e * 2 * kGroup + kGroup + kHiWord] >> kEndBit) & 1u)) ++e;
        g = e + 1 - P.panel_start[p];
      }
      if (g > prev) return false;
      prev = g;
    }
  }
  for (int64_t q = 0; q < P.nnz; ++q)
    if (!seen[q]) return false;
  for (size_t d = (size_t)(2 * P.stored); d < P.entries.size(); ++d)
    if (P.entries[d] != 0u) return false;
  std::vector<char> used((size_t)std::max(P.M, 1), 0);
  std::vector<int32_t> pos((size_t)std::max(P.M, 1), -1);
  for (int32_t i = 0; i < P.M; ++i) {
    const int32_t x = P.perm[i];
    if (x < 0 || x >= P.M || used[x]) return false;
    used[x] = 1;
    pos[x] = i;
  }
  // every panel row is stored to its original row, or to its position in perm
  if (P.panel_out.size() != P.panel_rows.size()) return false;
  std::fill(used.begin(), used.end(), 0);
  for (size_t j = 0; j < P.panel_rows.size(); ++j) {
    const int32_t orig = P.panel_rows[j], out = P.panel_out[j];
    if (orig < 0) {
      if (out != -1) return false;
      continue;
    }
    if (orig >= P.M || used[orig]) return false;
    used[orig] = 1;
    if (out != (P.out_permuted ? pos[orig] : orig)) return false;
  }
  for (int32_t i = 0; i < P.M; ++i)
    if (!used[i]) return false;
  return true;
}

// Resolved plan options.
struct Options {
  std::vector<int32_t> rws;      // panel heights to pack
  int32_t permute = 1;           // row order: Algorithm 1 (see row_order)
  int32_t grouping = 0;          // panel grouping: 0 the library's (balanced), 1 the row order's, 2 balanced
  int32_t out_permuted = 0;      // store C in the permuted row order
  int32_t split_chunks = 0;      // chunks per K-segment (0: no K-segments)
  const int32_t* in_perm = nullptr;  // order of B's rows (NULL: original)
  int32_t tile_cols = 0;         // 0: both tile widths; 256: 256-column tiles only; 128: 128 where the call allows
};

// Panel heights to pack: the explicit option, or the five defaults (the 32-row one only
// for plans that hold the 128-column stream).
static sdnn_status resolve_opts(const sdnn_plan_opts* opts, int32_t K, Options* o) {
  o->rws = {kShortPanel, kTallPanel, kMidPanel, kTallestPanel, kDeepPanel};
  if (!opts) return SDNN_OK;
  if (opts->panel_rows != 0) {
    if (opts->panel_rows != 4 && opts->panel_rows != 8 && opts->panel_rows != 12 &&
        opts->panel_rows != 16 && opts->panel_rows != 32)
      return SDNN_ERR_DIM;
    // 32-row panels exist for 128-column tiles only (their 64 accumulators per lane)
    if (opts->panel_rows == 32 && opts->tile_cols != kNarrowTileCols) return SDNN_ERR_DIM;
    o->rws = {opts->panel_rows};
  }
  if (opts->permute < 0 || opts->permute > 5) return SDNN_ERR_DIM;
  if (opts->out_permuted != 0 && opts->out_permuted != 1) return SDNN_ERR_DIM;
  if (opts->split_chunks < 0) return SDNN_ERR_DIM;
  if (opts->grouping < 0 || opts->grouping > 2) return SDNN_ERR_DIM;
  if (opts->tile_cols != 0 && opts->tile_cols != kTileCols && opts->tile_cols != kNarrowTileCols)
    return SDNN_ERR_DIM;
  o->grouping = opts->grouping;
  o->tile_cols = opts->tile_cols;
  // the 32-row packing serves 128-column tiles only
  if (opts->panel_rows == 0 && opts->tile_cols == kTileCols) o->rws.pop_back();
  o->split_chunks = opts->split_chunks;
  o->permute = opts->permute;
  o->out_permuted = opts->out_permuted;
  o->in_perm = opts->in_perm;
  if (o->in_perm) {  // must be a permutation of 0..K-1
    std::vector<char> seen((size_t)std::max(K, 1), 0);
    for (int32_t i = 0; i < K; ++i) {
      const int32_t x = o->in_perm[i];
      if (x < 0 || x >= K || seen[x]) return SDNN_ERR_DIM;
      seen[x] = 1;
    }
  }
  return SDNN_OK;
}

// Row order that balances the panels' work (plan option permute = 2): rows are taken
// by nonzero count (descending, ties by index) and each goes to the 4-row panel with
// the fewest nonzeros so far among those with room (ties: lower panel), the greedy
// longest-first rule for equal-size bins.  Position p * kShortPanel + r holds panel
// p's r-th row, so a tall panel (kTallPanel = 3 * kShortPanel consecutive positions)
// is three balanced short panels.
static void balanced_order(const int32_t* row_ptr, int32_t M, int32_t* perm_out) {
  std::vector<int32_t> rows((size_t)M);
  for (int32_t i = 0; i < M; ++i) rows[i] = i;
  std::stable_sort(rows.begin(), rows.end(), [&](int32_t a, int32_t b) {
    return row_ptr[a + 1] - row_ptr[a] > row_ptr[b + 1] - row_ptr[b];
  });
  const int32_t P = (M + kShortPanel - 1) / kShortPanel;
  std::vector<int32_t> fill((size_t)std::max(P, 1), 0);
  // min-heap of (nonzeros so far, panel) over panels with room
  std::vector<std::pair<int64_t, int32_t>> heap;
  heap.reserve((size_t)P);
  for (int32_t p = 0; p < P; ++p) heap.emplace_back(0, p);
  auto greater = [](const std::pair<int64_t, int32_t>& a, const std::pair<int64_t, int32_t>& b) {
    return a > b;
  };
  std::make_heap(heap.begin(), heap.end(), greater);
  for (int32_t j = 0; j < M; ++j) {
    std::pop_heap(heap.begin(), heap.end(), greater);
    std::pair<int64_t, int32_t> top = heap.back();
    heap.pop_back();
    const int32_t p = top.second, r = rows[j];
    perm_out[(size_t)p * kShortPanel + fill[p]] = r;
    ++fill[p];
    const int32_t cap = (p == P - 1) ? M - (P - 1) * kShortPanel : kShortPanel;
    if (fill[p] < cap) {
      heap.emplace_back(top.first + (row_ptr[r + 1] - row_ptr[r]), p);
      std::push_heap(heap.begin(), heap.end(), greater);
    }
  }
}

// The CSR a plan packs: the caller's, or (with in_perm) the same rows with column c
// renamed to its position in B's row order, pos[c] (in_perm[pos[c]] = c), re-sorted
// within each row.  W'[r][pos[c]] = W[r][c] makes W' * B_given = W * B when
// B_given[i] = B[in_perm[i]] (Sec. 3.1.2: the next layer's columns absorb the previous
// layer's row permutation).
struct CsrView {
  const int32_t* row_ptr = nullptr;
  const int32_t* col_idx = nullptr;
  const float* values = nullptr;
  std::vector<int32_t> cols;     // storage when relabelled
  std::vector<float> vals;
};

static void relabel_columns(const int32_t* row_ptr, const int32_t* col_idx, const float* values,
                            int32_t M, int32_t K, const int32_t* in_perm, CsrView* v) {
  std::vector<int32_t> pos((size_t)std::max(K, 1));
  for (int32_t i = 0; i < K; ++i) pos[in_perm[i]] = i;
  const int64_t nnz = M ? row_ptr[M] : 0;
  v->cols.resize((size_t)nnz);
  v->vals.resize((size_t)nnz);
  std::vector<std::pair<int32_t, float>> row;
  for (int32_t r = 0; r < M; ++r) {
    row.clear();
    for (int32_t q = row_ptr[r]; q < row_ptr[r + 1]; ++q)
      row.emplace_back(pos[col_idx[q]], values ? values[q] : 0.0f);
    std::sort(row.begin(), row.end(),
              [](const std::pair<int32_t, float>& a, const std::pair<int32_t, float>& b) {
                return a.first < b.first;
              });
    for (size_t k = 0; k < row.size(); ++k) {
      v->cols[(size_t)row_ptr[r] + k] = row[k].first;
      v->vals[(size_t)row_ptr[r] + k] = row[k].second;
    }
  }
  v->row_ptr = row_ptr;
  v->col_idx = v->cols.data();
  v->values = v->vals.data();
}

// Panel-union greedy order (plan option permute = 3), a panel-aware variant of
// Algorithm 1: positions are filled one 4-row panel at a time; a panel's first row is
// the remaining row with the most nonzeros, and each further row is the remaining row
// whose column set overlaps most with the union of the column sets already in the
// panel (Algorithm 1 compares with the previous row only).  Ties: more nonzeros, then
// the lower original index.  A tall panel is three consecutive short panels.
static sdnn_status panel_union_order(const int32_t* row_ptr, const int32_t* col_idx, int32_t M,
                                     int32_t K, int32_t* perm_out) {
  if (M == 0) return SDNN_OK;
  const int64_t words = std::max<int64_t>((K + 63) / 64, 1);
  std::vector<uint64_t> bits, uni;
  std::vector<int32_t> remaining;
  try {
    bits.assign((size_t)M * (size_t)words, 0);
    uni.assign((size_t)words, 0);
    remaining.resize(M);
  } catch (const std::bad_alloc&) {
    return SDNN_ERR_ALLOC;
  }
  for (int32_t i = 0; i < M; ++i) {
    uint64_t* row = bits.data() + (size_t)i * words;
    for (int32_t p = row_ptr[i]; p < row_ptr[i + 1]; ++p)
      row[col_idx[p] >> 6] |= 1ull << (col_idx[p] & 63);
  }
  auto nnz = [&](int32_t x) { return row_ptr[x + 1] - row_ptr[x]; };
  // remaining rows in ascending index order, so a strict improvement keeps the lower
  // index among equal keys
  int32_t nrem = M;
  for (int32_t x = 0; x < M; ++x) remaining[x] = x;
  for (int32_t i = 0; i < M; ++i) {
    const bool head = i % kShortPanel == 0;
    if (head) std::fill(uni.begin(), uni.end(), 0ull);
    int32_t best_pos = 0, best_ov = -1, best_nnz = -1;
    for (int32_t j = 0; j < nrem; ++j) {
      const int32_t x = remaining[j];
      int32_t ov = 0;
      if (!head) {
        const uint64_t* row = bits.data() + (size_t)x * words;
        for (int64_t w = 0; w < words; ++w) ov += __builtin_popcountll(uni[w] & row[w]);
      }
      const int32_t nx = nnz(x);
      if (ov > best_ov || (ov == best_ov && nx > best_nnz)) {
        best_pos = j;
        best_ov = ov;
        best_nnz = nx;
      }
    }
    const int32_t pick = remaining[best_pos];
    perm_out[i] = pick;
    const uint64_t* row = bits.data() + (size_t)pick * words;
    for (int64_t w = 0; w < words; ++w) uni[w] |= row[w];
    memmove(remaining.data() + best_pos, remaining.data() + best_pos + 1,
            sizeof(int32_t) * (size_t)(nrem - best_pos - 1));
    --nrem;
  }
  return SDNN_OK;
}

// MurmurHash3's 32-bit finalizer (Appleby): a bijective avalanche mix of one word.
static uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85ebca6bu;
  h ^= h >> 13;
  h *= 0xc2b2ae35u;
  h ^= h >> 16;
  return h;
}

// MinHash clustering order (plan option permute = 4), a locality-sensitive-hashing
// order: row r's signature is (m_0(r), .., m_3(r)) with m_t(r) = min over its columns c
// of fmix32(c ^ kMinHashSeed[t]) (0xffffffff for an empty row); two rows agree on each
// m_t with probability equal to the Jaccard similarity of their column sets, so sorting
// rows by signature (then nonzeros descending, then index) places rows with similar
// column sets together, and rows with equal column sets consecutively.
static const uint32_t kMinHashSeed[4] = {0x9e3779b9u, 0x7f4a7c15u, 0x94d049bbu, 0xbf58476du};

static void minhash_order(const int32_t* row_ptr, const int32_t* col_idx, int32_t M,
                          int32_t* perm_out) {
  std::vector<std::array<uint32_t, 4>> sig((size_t)M);
  for (int32_t r = 0; r < M; ++r) {
    std::array<uint32_t, 4> m = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
    for (int32_t q = row_ptr[r]; q < row_ptr[r + 1]; ++q)
      for (int t = 0; t < 4; ++t) m[t] = std::min(m[t], fmix32((uint32_t)col_idx[q] ^ kMinHashSeed[t]));
    sig[r] = m;
  }
  for (int32_t i = 0; i < M; ++i) perm_out[i] = i;
  std::sort(perm_out, perm_out + M, [&](int32_t a, int32_t b) {
    if (sig[a] != sig[b]) return sig[a] < sig[b];
    const int32_t na = row_ptr[a + 1] - row_ptr[a], nb = row_ptr[b + 1] - row_ptr[b];
    return na != nb ? na > nb : a < b;
  });
}

// Bin-then-greedy order (plan option permute = 5): rows are binned by nonzero count,
// bin floor(log2(nnz + 1)), the densest bin first, and Algorithm 1 orders the rows of
// each bin among themselves (first the bin's densest row, then repeatedly the bin's
// remaining row with the largest overlap with the row placed last; ties: more
// nonzeros, then the lower index).  Panels then hold rows of similar length.
static sdnn_status bin_greedy_order(const int32_t* row_ptr, const int32_t* col_idx, int32_t M,
                                    int32_t K, int32_t* perm_out) {
  auto bin_of = [&](int32_t r) {
    uint32_t n = (uint32_t)(row_ptr[r + 1] - row_ptr[r]) + 1u;
    int b = 0;
    while (n >>= 1) ++b;
    return b;
  };
  std::vector<std::vector<int32_t>> bins(33);
  for (int32_t r = 0; r < M; ++r) bins[bin_of(r)].push_back(r);
  int32_t at = 0;
  std::vector<int32_t> sub_ptr, sub_col, sub_perm;
  for (int b = 32; b >= 0; --b) {
    const std::vector<int32_t>& rows = bins[b];
    if (rows.empty()) continue;
    // the bin's rows as a CSR of their own (ascending original index), Algorithm 1 on it
    sub_ptr.assign(1, 0);
    sub_col.clear();
    for (int32_t r : rows) {
      sub_col.insert(sub_col.end(), col_idx + row_ptr[r], col_idx + row_ptr[r + 1]);
      sub_ptr.push_back((int32_t)sub_col.size());
    }
    sub_perm.resize(rows.size());
    sdnn_status st = reorder_bitset(sub_ptr.data(), sub_col.data(), (int32_t)rows.size(), K,
                                    sub_perm.data());
    if (st != SDNN_OK) return st;
    for (int32_t x : sub_perm) perm_out[at++] = rows[x];
  }
  return SDNN_OK;
}

// The row order of plan option `permute` (0 identity, 1 Algorithm 1, 2 panel-balancing,
// 3 panel-union greedy, 4 MinHash clustering, 5 bin-then-greedy) for a validated CSR.
static sdnn_status row_order(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K,
                             int32_t permute, int32_t* perm_out) {
  switch (permute) {
    case 1:
      return reorder_bitset(row_ptr, col_idx, M, K, perm_out);
    case 2:
      balanced_order(row_ptr, M, perm_out);
      return SDNN_OK;
    case 3:
      return panel_union_order(row_ptr, col_idx, M, K, perm_out);
    case 4:
      minhash_order(row_ptr, col_idx, M, perm_out);
      return SDNN_OK;
    case 5:
      return bin_greedy_order(row_ptr, col_idx, M, K, perm_out);
    default:
      for (int32_t i = 0; i < M; ++i) perm_out[i] = i;
      return SDNN_OK;
  }
}

// Validation, column relabelling (with in_perm), the row order (once: its keys do not
// depend on column names) and one packing per panel height.  *csr is what was packed.
static sdnn_status prepare(const int32_t* row_ptr, const int32_t* col_idx, const float* values,
                           int32_t M, int32_t K, const sdnn_plan_opts* opts,
                           std::vector<Packed>* packs, CsrView* csr, Options* o) {
  sdnn_status st = resolve_opts(opts, K, o);
  if (st != SDNN_OK) return st;
  st = validate_csr(row_ptr, col_idx, M, K);
  if (st != SDNN_OK) return st;
  if (M > 0 && row_ptr[M] > 0 && !values) return SDNN_ERR_NULL;
  std::vector<int32_t> perm;
  try {
    perm.resize(M);
    packs->assign(o->rws.size(), Packed());
    if (o->in_perm) {
      relabel_columns(row_ptr, col_idx, values, M, K, o->in_perm, csr);
    } else {
      csr->row_ptr = row_ptr;
      csr->col_idx = col_idx;
      csr->values = values;
    }
  } catch (const std::bad_alloc&) {
    return SDNN_ERR_ALLOC;
  }
  st = row_order(csr->row_ptr, csr->col_idx, M, K, o->permute, perm.data());
  if (st != SDNN_OK) return st;
  // the panels: consecutive rows of the order, or balanced ones (the order stays the
  // plan's reported permutation either way, and fixes the stored row order of
  // out_permuted plans).  The library's choice is the balanced grouping: a workgroup's
  // panels advance together through the staged chunks, so the heaviest panel and the one
  // whose entries bunch into the fewest chunks set the pace, and the loop reads B once per
  // stored entry whatever the panel's column overlap.  Measured on MI355X against the
  // permutation's own panels on W0 and C2-C5: never slower, 2-8 % faster on the uniform
  // and block-correlated layers, 1.3-1.8x on the lognormal ones.
  std::vector<int32_t> balanced, pos;
  int32_t grouping = o->grouping == 0 ? 2 : o->grouping;
  try {
    if (grouping == 2) {
      balanced.resize(M);
      balanced_order(csr->row_ptr, M, balanced.data());
    }
    pos.assign((size_t)std::max(M, 1), 0);
    for (int32_t i = 0; i < M; ++i) pos[perm[i]] = i;
  } catch (const std::bad_alloc&) {
    return SDNN_ERR_ALLOC;
  }
  const int32_t* group = grouping == 2 ? balanced.data() : perm.data();
  for (size_t i = 0; i < o->rws.size(); ++i) {
    Packed& P = (*packs)[i];
    st = pack(csr->row_ptr, csr->col_idx, csr->values, M, K, o->rws[i], group, o->split_chunks, &P);
    if (st != SDNN_OK) return st;
    try {
      P.perm = perm;
      P.grouping = grouping;
      P.out_permuted = o->out_permuted;
      P.panel_out.assign(P.panel_rows.size(), -1);
      for (size_t j = 0; j < P.panel_rows.size(); ++j) {
        const int32_t orig = P.panel_rows[j];
        if (orig >= 0) P.panel_out[j] = o->out_permuted ? pos[orig] : orig;
      }
    } catch (const std::bad_alloc&) {
      return SDNN_ERR_ALLOC;
    }
  }
  return SDNN_OK;
}

static double fill_of(const Packed& P) {
  return P.stored ? (double)P.nnz / (double)P.stored : 1.0;
}

// Statistics of the first packing, plus the tall and mid ones' if there are.
static void fill_info(const std::vector<Packed>& packs, int64_t packed_bytes,
                      const Options& o, sdnn_plan_info_t* out) {
  const Packed& P = packs[0];
  out->M = P.M;
  out->K = P.K;
  out->nnz = P.nnz;
  out->panels = P.npanels;
  out->packed_bytes = packed_bytes;
  out->rho = P.rho;
  out->fill = fill_of(P);
  out->panel_rows = P.RW;
  out->k_chunk = kChunk;
  const bool tall = packs.size() > 1;
  out->tall_panel_rows = tall ? packs[1].RW : 0;
  out->splits = P.split_chunks > 0 ? P.nseg : 0;
  out->tall_rho = tall ? packs[1].rho : 0.0;
  out->tall_fill = tall ? fill_of(packs[1]) : 0.0;
  out->out_permuted = o.out_permuted;
  out->in_permuted = o.in_perm ? 1 : 0;
  const bool mid = packs.size() > 2;
  out->mid_panel_rows = mid ? packs[2].RW : 0;
  out->packings = (int32_t)packs.size();
  out->mid_rho = mid ? packs[2].rho : 0.0;
  out->mid_fill = mid ? fill_of(packs[2]) : 0.0;
  const bool tallest = packs.size() > 3;
  out->tallest_panel_rows = tallest ? packs[3].RW : 0;
  out->reserved2 = 0;
  out->tallest_rho = tallest ? packs[3].rho : 0.0;
  out->tallest_fill = tallest ? fill_of(packs[3]) : 0.0;
  const bool deep = packs.size() > 4;
  out->deep_panel_rows = deep ? packs[4].RW : 0;
  out->reserved3 = 0;
  out->deep_rho = deep ? packs[4].rho : 0.0;
  out->deep_fill = deep ? fill_of(packs[4]) : 0.0;
  out->grouping = P.grouping;
  out->tile_cols = o.tile_cols;
}

static int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }

// Device bytes of one packing's arrays (each 256-byte aligned), with the stream of the
// 128-column tiles when `narrow`.
static int64_t packing_bytes(const Packed& P, bool narrow) {
  return align256((int64_t)P.entries.size() * 4) * (narrow ? 2 : 1) +
         align256((int64_t)P.panel_start.size() * 4) + align256((int64_t)P.panel_rows.size() * 4) +
         align256((int64_t)P.panel_out.size() * 4) + align256((int64_t)P.seg_start.size() * 4);
}

// Plans serve 128-column tiles unless the option fixes 256.
static bool wants_narrow(const Options& o) { return o.tile_cols != kTileCols; }

std::vector<uint32_t> narrow_stream(const std::vector<uint32_t>& entries) {
  std::vector<uint32_t> out(entries);
  const size_t groups = entries.size() / (2 * kGroup);
  for (size_t g = 0; g < groups; ++g)
    for (int j = 0; j < kGroup; ++j) {
      uint32_t& a = out[g * 2 * kGroup + kGroup + j];
      const uint32_t ring = (a >> kRingRowShift) & (uint32_t)(kRing * kChunk - 1);
      const uint32_t end = (a >> kEndBit) & 1u;
      const uint32_t high = a & ~((1u << kSyncBit) - 1u);  // chunk and sync fields
      a = high | ring << kRingRowShiftNarrow | end << kEndBitNarrow | (a & ((1u << kRowBits) - 1u));
    }
  return out;
}

bool check_narrow_stream(const std::vector<uint32_t>& entries, const std::vector<uint32_t>& narrow) {
  if (narrow.size() != entries.size()) return false;
  for (size_t d = 0; d < entries.size(); ++d) {
    const uint32_t w = entries[d], n = narrow[d];
    if ((d / kGroup) % 2 == 0) {  // weight words are copied
      if (w != n) return false;
      continue;
    }
    // address words: row (bits 0-7), ring row, end flag, and bits 17 up
    if ((w & 0xffu) != (n & 0xffu)) return false;
    if (((w >> 10) & 0x7fu) != ((n >> 9) & 0x7fu)) return false;
    if (((w >> 9) & 1u) != ((n >> 8) & 1u)) return false;
    if ((w >> 17) != (n >> 17)) return false;
    if ((n >> 16) & 1u) return false;  // the narrow layout leaves bit 16 clear
  }
  return true;
}

}  // namespace sdnn

using namespace sdnn;

extern "C" {

const char* sdnn_status_str(sdnn_status s) {
  switch (s) {
    case SDNN_OK: return "SDNN_OK";
    case SDNN_ERR_NULL: return "SDNN_ERR_NULL: required pointer is NULL";
    case SDNN_ERR_DIM: return "SDNN_ERR_DIM: invalid size, option or overlapping buffers";
    case SDNN_ERR_CSR: return "SDNN_ERR_CSR: malformed CSR input";
    case SDNN_ERR_ALLOC: return "SDNN_ERR_ALLOC: allocation failed";
    case SDNN_ERR_HIP: return "SDNN_ERR_HIP: HIP runtime or launch error";
    case SDNN_ERR_DEVICE: return "SDNN_ERR_DEVICE: plan used on another device";
    case SDNN_ERR_INTERNAL: return "SDNN_ERR_INTERNAL: packed stream failed its self-check";
  }
  return "SDNN_ERR_UNKNOWN";
}

sdnn_status sdnn_row_order(const int32_t* row_ptr, const int32_t* col_idx, int32_t M, int32_t K,
                           int32_t permute, int32_t* perm_out) {
  if (M < 0 || K < 0 || permute < 0 || permute > 5) return SDNN_ERR_DIM;
  if (M > 0 && !perm_out) return SDNN_ERR_NULL;
  sdnn_status st = validate_csr(row_ptr, col_idx, M, K);
  if (st != SDNN_OK) return st;
  try {
    return row_order(row_ptr, col_idx, M, K, permute, perm_out);
  } catch (...) {
    return SDNN_ERR_ALLOC;
  }
}

sdnn_status sdnn_reorder_rows(const int32_t* row_ptr, const int32_t* col_idx, int32_t M,
                              int32_t K, int32_t* perm_out) {
  if (M < 0 || K < 0) return SDNN_ERR_DIM;
  if (M > 0 && !perm_out) return SDNN_ERR_NULL;
  sdnn_status st = validate_csr(row_ptr, col_idx, M, K);
  if (st != SDNN_OK) return st;
  try {
    return reorder_bitset(row_ptr, col_idx, M, K, perm_out);
  } catch (...) {
    return SDNN_ERR_ALLOC;
  }
}

sdnn_status sdnn_plan_check_host(const int32_t* row_ptr, const int32_t* col_idx,
                                 const float* values, int32_t M, int32_t K,
                                 const sdnn_plan_opts* opts, sdnn_plan_info_t* info) {
  try {
    std::vector<Packed> packs;
    CsrView csr;
    Options o;
    sdnn_status st = prepare(row_ptr, col_idx, values, M, K, opts, &packs, &csr, &o);
    if (st != SDNN_OK) return st;
    int64_t bytes = 0;
    for (const Packed& P : packs) {
      if (!check_packed(csr.row_ptr, csr.col_idx, csr.values, P)) return SDNN_ERR_INTERNAL;
      if (wants_narrow(o) && !check_narrow_stream(P.entries, narrow_stream(P.entries)))
        return SDNN_ERR_INTERNAL;
      bytes += packing_bytes(P, wants_narrow(o));
    }
    if (o.split_chunks > 0) bytes += align256((int64_t)M * 4);  // the device copy of perm
    if (info) fill_info(packs, bytes, o, info);
    return SDNN_OK;
  } catch (...) {
    return SDNN_ERR_ALLOC;
  }
}

sdnn_status sdnn_plan_create(const int32_t* row_ptr, const int32_t* col_idx, const float* values,
                             int32_t M, int32_t K, const sdnn_plan_opts* opts, sdnn_plan* out) {
  if (!out) return SDNN_ERR_NULL;
  *out = nullptr;
  sdnn_plan_s* plan = nullptr;
  try {
    std::vector<Packed> packs;
    CsrView csr;
    Options o;
    sdnn_status st = prepare(row_ptr, col_idx, values, M, K, opts, &packs, &csr, &o);
    if (st != SDNN_OK) return st;

    plan = new sdnn_plan_s();
    if (hipGetDevice(&plan->device) != hipSuccess) {
      delete plan;
      return SDNN_ERR_HIP;
    }
    if (hipDeviceGetAttribute(&plan->num_cus, hipDeviceAttributeMultiprocessorCount,
                              plan->device) != hipSuccess) {
      delete plan;
      return SDNN_ERR_HIP;
    }
    const Packed& P0 = packs[0];
    plan->M = P0.M;
    plan->K = P0.K;
    plan->nchunks = P0.nchunks;
    plan->nnz = P0.nnz;
    plan->perm = P0.perm;
    plan->npack = (int)packs.size();
    plan->out_permuted = o.out_permuted;
    plan->split_chunks = o.split_chunks;
    plan->in_permuted = o.in_perm ? 1 : 0;
    plan->grouping = P0.grouping;
    plan->tile_cols = o.tile_cols;
    const bool narrow = wants_narrow(o);

    int64_t total = 0;
    for (const Packed& P : packs) total += packing_bytes(P, narrow);
    // a K-segmented plan's reduction adds the bias through perm (out_permuted plans)
    const int64_t perm_off = total;
    if (o.split_chunks > 0) total += align256((int64_t)M * 4);
    plan->packed_bytes = total;
    if (total > 0) {
      if (hipMalloc(&plan->d_mem, (size_t)total) != hipSuccess) {
        (void)hipGetLastError();
        delete plan;
        return SDNN_ERR_ALLOC;
      }
      std::vector<char> host((size_t)total, 0);
      int64_t off = 0;
      for (size_t i = 0; i < packs.size(); ++i) {
        const Packed& P = packs[i];
        DevPacking& d = plan->pk[i];
        const int64_t b_ent = align256((int64_t)P.entries.size() * 4);
        const int64_t b_seg = align256((int64_t)P.panel_start.size() * 4);
        const int64_t b_rows = align256((int64_t)P.panel_rows.size() * 4);
        char* base = (char*)plan->d_mem + off;
        d.RW = P.RW;
        d.npanels = P.npanels;
        d.rho = P.rho;
        d.fill = fill_of(P);
        d.entries = (const uint32_t*)base;
        // the 128-column stream sits after the packing's other arrays
        const int64_t b_all = packing_bytes(P, false);
        d.entries_n = narrow ? (const uint32_t*)(base + b_all) : nullptr;
        d.panel_start = (const int32_t*)(base + b_ent);
        d.panel_rows = (const int32_t*)(base + b_ent + b_seg);
        d.panel_out = (const int32_t*)(base + b_ent + b_seg + b_rows);
        const int64_t b_pos = align256((int64_t)P.panel_out.size() * 4);
        d.nseg = P.nseg;
        d.seg_start = P.seg_start.empty() ? nullptr
                                          : (const int32_t*)(base + b_ent + b_seg + b_rows + b_pos);
        // panel tables in workgroup (slot) order: slot j is panel panel_order[j]
        char* h = host.data() + off;
        if (!P.entries.empty()) memcpy(h, P.entries.data(), P.entries.size() * 4);
        if (narrow && !P.entries.empty()) {
          const std::vector<uint32_t> nst = narrow_stream(P.entries);
          memcpy(h + b_all, nst.data(), nst.size() * 4);
        }
        int32_t* hs = (int32_t*)(h + b_ent);
        int32_t* hr = (int32_t*)(h + b_ent + b_seg);
        int32_t* hp = (int32_t*)(h + b_ent + b_seg + b_rows);
        for (int32_t j = 0; j < P.npanels; ++j) {
          const int32_t q = P.panel_order[j];
          hs[j] = P.panel_start[q];
          memcpy(hr + (size_t)j * P.RW, P.panel_rows.data() + (size_t)q * P.RW, 4 * (size_t)P.RW);
          memcpy(hp + (size_t)j * P.RW, P.panel_out.data() + (size_t)q * P.RW, 4 * (size_t)P.RW);
          if (!P.seg_start.empty())
            memcpy((int32_t*)(h + b_ent + b_seg + b_rows + b_pos) + (size_t)j * P.nseg,
                   P.seg_start.data() + (size_t)q * P.nseg, 4 * (size_t)P.nseg);
        }
        off += packing_bytes(P, narrow);
      }
      if (o.split_chunks > 0 && M > 0) {
        memcpy(host.data() + perm_off, P0.perm.data(), (size_t)M * 4);
        plan->d_perm = (const int32_t*)((char*)plan->d_mem + perm_off);
      }
      if (hipMemcpy(plan->d_mem, host.data(), (size_t)total, hipMemcpyHostToDevice) !=
          hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(plan->d_mem);
        delete plan;
        return SDNN_ERR_HIP;
      }
    } else {
      for (size_t i = 0; i < packs.size(); ++i) {
        plan->pk[i].RW = packs[i].RW;
        plan->pk[i].npanels = packs[i].npanels;
      }
    }
    *out = plan;
    return SDNN_OK;
  } catch (...) {
    if (plan) {
      if (plan->d_mem) (void)hipFree(plan->d_mem);
      delete plan;
    }
    return SDNN_ERR_ALLOC;
  }
}

sdnn_status sdnn_plan_get_perm(sdnn_plan p, int32_t* perm_out) {
  if (!p) return SDNN_ERR_NULL;
  if (p->M > 0 && !perm_out) return SDNN_ERR_NULL;
  if (p->M > 0) memcpy(perm_out, p->perm.data(), sizeof(int32_t) * (size_t)p->M);
  return SDNN_OK;
}

sdnn_status sdnn_plan_info(sdnn_plan p, sdnn_plan_info_t* out) {
  if (!p || !out) return SDNN_ERR_NULL;
  const DevPacking& d = p->pk[0];
  out->M = p->M;
  out->K = p->K;
  out->nnz = p->nnz;
  out->panels = d.npanels;
  out->packed_bytes = p->packed_bytes;
  out->rho = d.rho;
  out->fill = d.fill;
  out->panel_rows = d.RW;
  out->k_chunk = kChunk;
  const bool tall = p->npack > 1;
  out->tall_panel_rows = tall ? p->pk[1].RW : 0;
  out->splits = p->split_chunks > 0 ? d.nseg : 0;
  out->tall_rho = tall ? p->pk[1].rho : 0.0;
  out->tall_fill = tall ? p->pk[1].fill : 0.0;
  out->out_permuted = p->out_permuted;
  out->in_permuted = p->in_permuted;
  const bool mid = p->npack > 2;
  out->mid_panel_rows = mid ? p->pk[2].RW : 0;
  out->packings = p->npack;
  out->mid_rho = mid ? p->pk[2].rho : 0.0;
  out->mid_fill = mid ? p->pk[2].fill : 0.0;
  out->grouping = p->grouping;
  out->tile_cols = p->tile_cols;
  const bool tallest = p->npack > 3;
  out->tallest_panel_rows = tallest ? p->pk[3].RW : 0;
  out->reserved2 = 0;
  out->tallest_rho = tallest ? p->pk[3].rho : 0.0;
  out->tallest_fill = tallest ? p->pk[3].fill : 0.0;
  const bool deep = p->npack > 4;
  out->deep_panel_rows = deep ? p->pk[4].RW : 0;
  out->reserved3 = 0;
  out->deep_rho = deep ? p->pk[4].rho : 0.0;
  out->deep_fill = deep ? p->pk[4].fill : 0.0;
  return SDNN_OK;
}

void sdnn_plan_destroy(sdnn_plan p) {
  if (!p) return;
  if (p->d_mem) {
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (cur != p->device) (void)hipSetDevice(p->device);
    (void)hipFree(p->d_mem);
    if (cur != p->device && cur >= 0) (void)hipSetDevice(cur);
  }
  delete p;
}

static bool ranges_overlap(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
  if (!a || !b || abytes <= 0 || bbytes <= 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)bbytes && b0 < a0 + (uintptr_t)abytes;
}

// Checks of a K-split call's workspace: nseg * M * N floats, 16-byte aligned, clear of
// the call's other buffers.  A plan with one K-segment needs none.
static sdnn_status check_workspace(const sdnn_plan_s* p, int64_t N, const float* ws,
                                   int64_t ws_floats, const void* in, int64_t inbytes,
                                   const float* C, const float* bias) {
  if (p->split_chunks <= 0) return SDNN_ERR_DIM;
  const int64_t nseg = p->pk[0].nseg;
  if (nseg == 1) return SDNN_OK;
  if (!ws) return SDNN_ERR_NULL;
  const int64_t need = nseg * p->M * N;
  if (ws_floats < need || ((uintptr_t)ws & 15) != 0) return SDNN_ERR_DIM;
  const int64_t wbytes = need * 4;
  if (ranges_overlap(ws, wbytes, in, inbytes) || ranges_overlap(ws, wbytes, C, p->M * N * 4) ||
      ranges_overlap(ws, wbytes, bias, (int64_t)p->M * 4))
    return SDNN_ERR_DIM;
  return SDNN_OK;
}

// noalloc: a K-split call whose partial products go to the library's fixed scratch array
// (ws must then be NULL).
static sdnn_status spmm_entry(sdnn_plan p, const float* B, float* C, int32_t N, const float* bias,
                              sdnn_epilogue epi, int32_t splits, float* ws, int64_t ws_floats,
                              bool split, void* stream, bool noalloc = false) {
  if (!p) return SDNN_ERR_NULL;
  // the kernels address one row of B or C with 32-bit byte offsets
  if (N < 0 || (int64_t)N * 4 >= kMaxRowBytes) return SDNN_ERR_DIM;
  if (epi != SDNN_EPI_NONE && epi != SDNN_EPI_RELU && epi != SDNN_EPI_GELU) return SDNN_ERR_DIM;
  if (split && (p->split_chunks <= 0 || splits < 0)) return SDNN_ERR_DIM;
  if (p->M == 0 || N == 0) return SDNN_OK;
  if (!C) return SDNN_ERR_NULL;
  if (p->K > 0 && !B) return SDNN_ERR_NULL;
  const int64_t bbytes = (int64_t)p->K * N * 4, cbytes = (int64_t)p->M * N * 4;
  if (ranges_overlap(B, bbytes, C, cbytes)) return SDNN_ERR_DIM;
  if (ranges_overlap(bias, (int64_t)p->M * 4, C, cbytes)) return SDNN_ERR_DIM;
  if (split && !noalloc) {
    const sdnn_status st = check_workspace(p, N, ws, ws_floats, B, bbytes, C, bias);
    if (st != SDNN_OK) return st;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return SDNN_ERR_HIP;
  if (cur != p->device) return SDNN_ERR_DEVICE;
  // a plan of 32-row panels alone runs on 128-column tiles only (their 16-byte staging)
  if (p->npack == 1 && p->pk[0].RW > kTallestPanel &&
      (N % 4 != 0 || ((uintptr_t)B & 15) != 0 || ((uintptr_t)C & 15) != 0))
    return SDNN_ERR_DIM;
  if (noalloc) {
    const int64_t runs = split_runs(p, N, splits);
    if (runs > 1) {
      if (runs * p->M * (int64_t)N > kScratchFloats) return SDNN_ERR_DIM;
      if (scratch_address(cur, &ws) != hipSuccess) return SDNN_ERR_HIP;
    }
  }
  try {
    hipError_t e = split ? launch_spmm_split(p, B, C, N, bias, (int)epi, splits, ws,
                                             (hipStream_t)stream)
                         : launch_spmm(p, B, C, N, bias, (int)epi, (hipStream_t)stream);
    return e == hipSuccess ? SDNN_OK : SDNN_ERR_HIP;
  } catch (...) {
    return SDNN_ERR_HIP;
  }
}

sdnn_status sdnn_spmm(sdnn_plan p, const float* B, float* C, int32_t N, const float* bias,
                      sdnn_epilogue epi, void* stream) {
  return spmm_entry(p, B, C, N, bias, epi, 0, nullptr, 0, false, stream);
}

sdnn_status sdnn_spmm_split(sdnn_plan p, const float* B, float* C, int32_t N, const float* bias,
                            sdnn_epilogue epi, int32_t splits, float* workspace,
                            int64_t workspace_floats, void* stream) {
  return spmm_entry(p, B, C, N, bias, epi, splits, workspace, workspace_floats, true, stream);
}

sdnn_status sdnn_spmm_split_noalloc(sdnn_plan p, const float* B, float* C, int32_t N,
                                    const float* bias, sdnn_epilogue epi, int32_t splits,
                                    void* stream) {
  return spmm_entry(p, B, C, N, bias, epi, splits, nullptr, 0, true, stream, true);
}

sdnn_status sdnn_plan_launch_shape(sdnn_plan p, int32_t N, int32_t* panel_rows, int32_t* waves) {
  if (!p) return SDNN_ERR_NULL;
  if (N <= 0 || p->M == 0) return SDNN_ERR_DIM;
  int32_t rw = 0, w = 0, t = 0;
  launch_shape(p, N, &rw, &w, &t);
  if (panel_rows) *panel_rows = rw;
  if (waves) *waves = w;
  return SDNN_OK;
}

sdnn_status sdnn_plan_split_runs(sdnn_plan p, int32_t N, int32_t splits, int32_t* runs) {
  if (!p || !runs) return SDNN_ERR_NULL;
  if (N <= 0 || p->M == 0 || splits < 0) return SDNN_ERR_DIM;
  *runs = split_runs(p, N, splits);
  return SDNN_OK;
}

sdnn_status sdnn_plan_launch_tile(sdnn_plan p, int32_t N, int32_t* tile_cols) {
  if (!p || !tile_cols) return SDNN_ERR_NULL;
  if (N <= 0 || p->M == 0) return SDNN_ERR_DIM;
  int32_t rw = 0, w = 0;
  launch_shape(p, N, &rw, &w, tile_cols);
  return SDNN_OK;
}

sdnn_status sdnn_plan_tune(sdnn_plan p, const float* B, float* C, int32_t N, void* stream,
                           int32_t* panel_rows, int32_t* waves) {
  if (!p) return SDNN_ERR_NULL;
  if (N <= 0 || (int64_t)N * 4 >= kMaxRowBytes) return SDNN_ERR_DIM;
  if (p->M == 0) return SDNN_ERR_DIM;
  if (!C || (p->K > 0 && !B)) return SDNN_ERR_NULL;
  const int64_t bbytes = (int64_t)p->K * N * 4, cbytes = (int64_t)p->M * N * 4;
  if (ranges_overlap(B, bbytes, C, cbytes)) return SDNN_ERR_DIM;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return SDNN_ERR_HIP;
  if (cur != p->device) return SDNN_ERR_DEVICE;
  // a plan of 32-row panels alone has no shape for a call that cannot use 128-column tiles
  if (p->npack == 1 && p->pk[0].RW > kTallestPanel &&
      (N % 4 != 0 || ((uintptr_t)B & 15) != 0 || ((uintptr_t)C & 15) != 0))
    return SDNN_ERR_DIM;
  try {
    TunedShape chosen;
    if (tune_spmm(p, B, C, N, (hipStream_t)stream, &chosen) != hipSuccess) return SDNN_ERR_HIP;
    if (panel_rows) *panel_rows = p->pk[chosen.pack].RW;
    if (waves) *waves = chosen.waves;
    return SDNN_OK;
  } catch (...) {
    return SDNN_ERR_HIP;
  }
}

static sdnn_status conv_entry(sdnn_plan p, const float* X, float* C, int32_t H, int32_t W,
                              int32_t NB, const float* bias, sdnn_epilogue epi, int32_t splits,
                              float* ws, int64_t ws_floats, bool split, void* stream) {
  if (!p) return SDNN_ERR_NULL;
  if (H < 0 || W < 0 || NB < 0) return SDNN_ERR_DIM;
  if (epi != SDNN_EPI_NONE && epi != SDNN_EPI_RELU && epi != SDNN_EPI_GELU) return SDNN_ERR_DIM;
  if (p->K % 9 != 0 || p->K == 0 || p->in_permuted) return SDNN_ERR_DIM;
  if (p->npack == 1 && p->pk[0].RW > kTallestPanel) return SDNN_ERR_DIM;  // 128-column only
  if (NB % 4 != 0) return SDNN_ERR_DIM;
  if (split && (p->split_chunks <= 0 || splits < 0)) return SDNN_ERR_DIM;
  const int64_t N = (int64_t)H * W * NB;
  if (p->M == 0 || N == 0) return SDNN_OK;
  // 32-bit column and channel-plane byte offsets in the staging loop
  if (N * 4 >= kMaxRowBytes || (int64_t)(p->K / 9) * N * 4 >= ((int64_t)1 << 40))
    return SDNN_ERR_DIM;
  if (!X || !C) return SDNN_ERR_NULL;
  if ((((uintptr_t)X | (uintptr_t)C) & 15) != 0) return SDNN_ERR_DIM;
  const int64_t xbytes = (int64_t)(p->K / 9) * N * 4, cbytes = (int64_t)p->M * N * 4;
  if (ranges_overlap(X, xbytes, C, cbytes)) return SDNN_ERR_DIM;
  if (ranges_overlap(bias, (int64_t)p->M * 4, C, cbytes)) return SDNN_ERR_DIM;
  if (split) {
    const sdnn_status st = check_workspace(p, N, ws, ws_floats, X, xbytes, C, bias);
    if (st != SDNN_OK) return st;
  }
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return SDNN_ERR_HIP;
  if (cur != p->device) return SDNN_ERR_DEVICE;
  try {
    hipError_t e =
        split ? launch_conv3x3_split(p, X, C, H, W, NB, bias, (int)epi, splits, ws,
                                     (hipStream_t)stream)
              : launch_conv3x3(p, X, C, H, W, NB, bias, (int)epi, (hipStream_t)stream);
    return e == hipSuccess ? SDNN_OK : SDNN_ERR_HIP;
  } catch (...) {
    return SDNN_ERR_HIP;
  }
}

sdnn_status sdnn_conv3x3(sdnn_plan p, const float* X, float* C, int32_t H, int32_t W,
                         int32_t NB, const float* bias, sdnn_epilogue epi, void* stream) {
  return conv_entry(p, X, C, H, W, NB, bias, epi, 0, nullptr, 0, false, stream);
}

sdnn_status sdnn_conv3x3_split(sdnn_plan p, const float* X, float* C, int32_t H, int32_t W,
                               int32_t NB, const float* bias, sdnn_epilogue epi, int32_t splits,
                               float* workspace, int64_t workspace_floats, void* stream) {
  return conv_entry(p, X, C, H, W, NB, bias, epi, splits, workspace, workspace_floats, true,
                    stream);
}

sdnn_status sdnn_dense_gemm(const float* W, const float* B, float* C, int32_t M, int32_t K,
                            int32_t N, const float* bias, sdnn_epilogue epi, void* stream) {
  if (M < 0 || K < 0 || N < 0) return SDNN_ERR_DIM;
  if (epi != SDNN_EPI_NONE && epi != SDNN_EPI_RELU && epi != SDNN_EPI_GELU) return SDNN_ERR_DIM;
  if (M == 0 || N == 0) return SDNN_OK;
  if (!C) return SDNN_ERR_NULL;
  if (K > 0 && (!W || !B)) return SDNN_ERR_NULL;
  const int64_t cbytes = (int64_t)M * N * 4;
  if (ranges_overlap(B, (int64_t)K * N * 4, C, cbytes) ||
      ranges_overlap(W, (int64_t)M * K * 4, C, cbytes) ||
      ranges_overlap(bias, (int64_t)M * 4, C, cbytes))
    return SDNN_ERR_DIM;
  try {
    hipError_t e = launch_dense(W, B, C, M, K, N, bias, (int)epi, (hipStream_t)stream);
    return e == hipSuccess ? SDNN_OK : SDNN_ERR_HIP;
  } catch (...) {
    return SDNN_ERR_HIP;
  }
}

}  // extern "C"
