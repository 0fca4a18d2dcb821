// Sort / scan / de-duplication launchers (k_sort.hip).
#pragma once

#include "embc_internal.h"

namespace embc {

template <typename T>
hipError_t scan_exclusive(const T* in, T* out, int64_t n, const unsigned long long* dev_n, T* part, T* total,
                          hipStream_t s);

// Exclusive scans of two u32 arrays in one pass (out_a / out_b may alias a / b; the sums
// of a must stay below 2^32); *total = total(a) + total(b) * 2^32.
hipError_t scan_exclusive_pair(const uint32_t* a, const uint32_t* b, uint32_t* out_a, uint32_t* out_b, int64_t n,
                               const unsigned long long* dev_n, unsigned long long* part,
                               unsigned long long* total, hipStream_t s);

// Scratch of the radix sort, carved from the workspace.
struct SortScratch {
  uint32_t* ghist;      // [kMaxPasses][256] digit counts
  uint32_t* gbase;      // [kMaxPasses][256] their exclusive prefix sums
  uint32_t* tickets;    // [kMaxPasses] tile tickets
  uint32_t* status[2];  // [sort_status_words(n, T)] look-back status words, alternating by pass
};

// Scratch of the segmented mode (sort_seg_words(T) words).
struct SegSort {
  uint32_t* pos = nullptr;    // [T+1] first position of each table's lookups; pos[T] = n
  uint32_t* tbase = nullptr;  // [T+1] first tile of each table's segment; tbase[T] = tiles
  uint32_t* hist = nullptr;   // [T][kMaxPasses][256] local-key digit counts per table
  uint32_t* base = nullptr;   // [T][kMaxPasses][256] where each table's digit runs start
};

// Stable LSD radix sort of n < 2^30 (key, value) pairs over `passes` (<= kMaxPasses)
// 8-bit digits, ping-ponging between (kA, vA) and (kB, vB); *in_B tells where the
// result is.  A look-back that waits too long sets kErrSort in *err.
hipError_t sort_pairs(uint32_t* kA, uint32_t* vA, uint32_t* kB, uint32_t* vB, int64_t n, int passes,
                      const SortScratch& ss, int32_t* err, int* in_B, hipStream_t s);

// The counting of the per-table sort mode, when the expansion does it (launch_expand
// with an ExpandHist from seg_begin): per-table digit counts, skipped keys, and the
// first pass's status words.
struct ExpandHist {
  uint32_t* hist = nullptr;            // SegSort::hist
  const int64_t* key_base = nullptr;   // [T+1]
  uint32_t* n_skipped = nullptr;       // zeroed by seg_begin
  uint32_t* status = nullptr;          // status words of the first pass
  int64_t status_words = 0;
  int passes = 0;
};

// Clears the counts and writes the segment starts for n > 0 keys (the same checks as
// sort_pairs_segmented), and fills *eh for the expansion.
hipError_t seg_begin(int64_t n, int passes, const int32_t* off, int32_t B, int T, const int64_t* key_base,
                     const unsigned long long* ctr, const SortScratch& ss, const SegSort& sg, ExpandHist* eh,
                     hipStream_t s);

// The same order from `passes` (< kMaxPasses) digit passes over each table's segment
// of the stream (lookups of table t at [off[t*B], off[(t+1)*B])), sorted by the local
// key; every table's key range must be below 2^(8*passes).  One more pass and a copy
// run only when some key is kKeyInvalid.  The counting is done before: seg_begin, then
// launch_expand with its ExpandHist.
hipError_t sort_pairs_segmented(uint32_t* kA, uint32_t* vA, uint32_t* kB, uint32_t* vB, int64_t n, int passes,
                                const int32_t* off, int32_t B, int T, const int64_t* key_base,
                                const unsigned long long* ctr, const SortScratch& ss, const SegSort& sg, int32_t* err,
                                int* in_B, hipStream_t s);

// Offsets must be non-decreasing and inside [0, L]; otherwise set the error flag and
// ctr[kCBadOffsets].
__global__ void k_check_offsets(Dev dv, const int32_t* __restrict__ off, int64_t nbags, int64_t L,
                                unsigned long long* __restrict__ ctr);

// Lookups -> (set-major key, bag) pairs; every key is skipped when ctr[kCBadOffsets]
// is set (k_check_offsets must have run first on the same stream).  eh: nullptr, or the
// per-table counting to do on the way (seg_begin first).
hipError_t launch_expand(const Dev& dv, const int32_t* idx, int64_t L, const int32_t* off, int32_t B, uint32_t* keys,
                         uint32_t* vals, unsigned long long* ctr, const ExpandHist* eh, hipStream_t s);

// Unique rows of the sorted stream sk[0, n): their keys, first occurrences and tables, and
// the first unique row of each touched set (tile_cnt / tile_pre: uniq_tile_words(n) words each).
// thread_pre: 256 words per tile, each thread's offset inside its tile.
hipError_t launch_unique(const Dev& dv, const uint32_t* sk, int64_t n, unsigned long long* tile_cnt,
                         unsigned long long* tile_pre, unsigned long long* thread_pre, uint32_t* uk, uint32_t* seg,
                         uint32_t* set_first, int32_t* utab, unsigned long long* ctr,
                         hipStream_t s);

}  // namespace embc
