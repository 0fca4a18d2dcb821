// Internal declarations shared by the runtime and the HIP kernels of libembcache.
//
// Data layout in HBM (one caller-owned state buffer, 256-byte aligned pieces):
//   rec   [total_rows][row_bytes]   low-precision row records: codes, then scale, then bias
//                                   (INT4: two codes per byte, even column in the low nibble;
//                                   scale/bias FP32 pair, or FP16 pair packed in one dword),
//                                   then, under row-wise Adagrad, the row's FP32 accumulator
//                                   while the row is not cached (a miss reads it with the codes),
//                                   unless that would make the record cross one more 64-byte line
//                                   (FP16 tables): then it is in acc_rows
//   crow  [total_slots][dim] FP32   cache rows; slot = slot_base[t] + set*assoc + way
//   tag   [total_slots] int32       resident row id (table-local), -1 = empty way
//   ts    [total_slots] int32       LRU: step of last access (-1 = empty); absent under LFU
//   acc_rows [total_rows] FP32      row-wise Adagrad, accumulator not in the records: the
//                                   accumulators of the rows not cached
//   acc_slot [total_slots] FP32     row-wise Adagrad: the accumulator of the row cached in the
//                                   slot (it moves between record and slot with the row); absent
//                                   under SGD
//   cnt   [total_rows] int32        LFU: access counts; absent under LRU
//   desc  [T] TableDesc, key_base [T+1], stats [T][kNStat] u64, err flags
// Rows of all tables are concatenated (global row = row_base[t] + row), and so
// are cache slots, so one base pointer serves every table.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace embc {

constexpr uint32_t kKeyInvalid = 0xFFFFFFFFu;  // sort key of a skipped lookup (sorts last)
// Merged gradient of a row (its lookups in position order): up to kBlockAbove lookups
// in chunks of kSumChunk consecutive lookups; more by bag blocks of kBlockFloats/d
// bags (one block of FP32 gradient rows is 128 KiB, staged in LDS once for all rows).
constexpr int kSumChunk = 64;
constexpr uint32_t kBlockAbove = 512;
constexpr int kBlockFloats = 32768;
// A bag block is staged in LDS in kStages runs of kBlockFloats/kStages floats.
constexpr int kStages = 2;
constexpr int64_t bound_stride(int64_t max_nblk) { return kStages * max_nblk + 1; }
constexpr int kMaxAssoc = 64;

enum : int32_t { kActHitStay = 0, kActHitEvict = 1, kActInsert = 2, kActBypass = 3 };

enum : int {
  kStLookups = 0, kStHitLookups, kStBwdLookups, kStUnique, kStUniqueHits, kStInserts, kStBypasses,
  kStEvictions, kStEmptyFills, kStHitEvictions, kStInvalidFwd, kStInvalidBwd, kNStat
};

enum : int { kErrIndex = 1, kErrOffsets = 2, kErrSort = 4 };
constexpr int kMaxPasses = 4;  // 8-bit digits of a 32-bit sort key

// Per-table geometry.  Sort keys are set-major: key = key_base + set*Q + row/n_sets,
// with set = row % n_sets and Q = ceil(N/n_sets), so that one sort groups the
// lookups by row, the rows by set, and the rows of a set in ascending order.
// Unsigned 32-bit division by a constant 1 <= d < 2^31 as one high multiply, a
// subtract, an add and two shifts (Granlund and Montgomery, "Division by invariant
// integers using multiplication", PLDI 1994, Sec. 4): with l = ceil(log2 d),
// m = floor(2^32 (2^l - d) / d) + 1, t = mulhi(m, n):
// n / d = (t + ((n - t) >> s1)) >> s2, s1 = min(l, 1), s2 = max(l - 1, 0), exact for
// every 32-bit n.
struct DivConst {
  uint32_t d = 1, m = 1, s1 = 0, s2 = 0;
};
// Its magic numbers for 1 <= d < 2^31 (host).
DivConst div_const(uint32_t d);

struct TableDesc {
  int64_t N;
  int64_t row_base;
  int64_t n_sets;     // 0: no cache
  int64_t slot_base;
  int64_t Q;          // key stride of a set; N when there is no cache
  int64_t key_base;
  DivConst by_sets;   // division by n_sets (by 1 when there is no cache)
  DivConst by_Q;      // division by Q
};

// Device view of the state, passed by value to every kernel.
struct Dev {
  uint8_t* rec;
  float* crow;
  int32_t* tag;
  int32_t* ts;
  int32_t* cnt;
  float* acc_slot;
  float* acc_rows;    // nullptr when the accumulators of uncached rows are in the records
  const TableDesc* desc;
  const int64_t* key_base;       // [T+1], key_base[T] = total key space
  unsigned long long* stats;     // [T][kNStat]
  int32_t* err;
  int32_t T;
  int32_t dim;
  int32_t bits;
  int32_t sb16;
  int32_t assoc;
  int32_t rec_bytes;  // record stride (Rec<>::BYTES, plus the accumulator and padding under Adagrad)
  int32_t acc_offset; // byte of the accumulator in a record (Rec<>::BYTES)
  int32_t policy;     // 0 LRU, 1 LFU
  int32_t rounding;   // 0 nearest, 1 stochastic
  int32_t optimizer;  // 0 SGD, 1 row-wise Adagrad
  float lr;
  float eps;
  uint64_t seed;
  int64_t total_rows;
  int64_t total_slots;
};

// Per-call temporaries carved from the caller's workspace buffer.
struct Work {
  uint32_t* keysA;
  uint32_t* valsA;
  uint32_t* keysB;
  uint32_t* valsB;
  uint32_t* sort_small;  // radix sort: digit counts, their prefix sums, tile tickets
  uint32_t* sort_status[2];  // radix sort look-back status words
  uint32_t* sort_seg;    // radix sort, segmented mode: segment starts, first tiles, per-table digit counts
  unsigned long long* part;  // scan partials
  unsigned long long* tile_cnt;  // unique rows and touched sets per tile of sorted keys, packed (sets << 32 | rows)
  unsigned long long* tile_pre;  // their exclusive prefix sums
  unsigned long long* thread_pre;  // [256 per tile] each thread's offset inside its tile
  uint32_t* uniq_key;    // [L]
  uint32_t* seg;         // [L+1] start of each unique row's occurrences in the sorted stream
  uint32_t* set_first;   // [L+1] first unique row of each touched set
  int32_t* urow;         // [L] global row id
  int32_t* utab;         // [L] table
  int32_t* uslot;        // [L] global slot before the step, -1 = miss
  int32_t* uact;         // [L] action
  int32_t* udest;        // [L] destination slot of an insert
  uint32_t* nch;         // [L] chunk count (rows with > kSumChunk occurrences), then its prefix
  uint32_t* chunk_base;  // [L+1]
  int32_t* uvic_row;     // [L] insert: table-local row displaced from its way, -1 = empty way
  int32_t* uvic_u;       // [L] insert: unique index of that row if it was updated this step, else -1
  uint4* umeta;          // [L] per unique row, the inputs of the row update in one word (k_pack_meta)
  unsigned long long* ukey;  // [L] LFU: a missed row's rank key (count << 32 | ~row), 0 for a hit
  float* partial;        // [L/32 + 2][dim] chunk sums
  uint2* chunk_span;     // [L/32 + 2] occurrences [x, y) of the sorted stream summed by each chunk
  uint32_t* ubig;        // [L] 1 for a row with more than kBlockAbove lookups, then its exclusive prefix
  int32_t* big_rows;     // [max_big] unique row of each such row ("big row"), in unique-row order
  uint32_t* bbound;      // [max_big][bound_stride(max_nblk)] first occurrence of each stage of a big row
  float* bpart;          // [max_big][max_nblk][dim] block sums of the big rows
  int64_t max_big;
  int32_t max_nblk;
  int32_t* tab_first;    // [T+1] first unique row of each table (tab_first[T] = number of unique rows)
  int32_t* fwd_src;      // [L] forward: cache slot of each lookup, -2-row for a miss, -1 if skipped
  unsigned long long* ctr;  // counters, see kC*
  int64_t max_indices;
  int64_t max_partials;
};

enum : int {
  kCValid = 0,      // valid (sorted) lookups
  kCUnique = 1,     // unique rows
  kCSets = 2,       // touched sets (of cached tables)
  kCChunks = 3,     // chunk partials
  kCVictims = 4,
  kCInserts = 5,
  kCScanTotal = 6,  // scratch total of the last scan
  kCBadOffsets = 7, // offsets of this step failed validation
  kCBig = 8,        // big rows
  kCHitEv = 9,      // inserts displacing a resident updated this step
  kNCounters = 16
};

// ---- launchers (defined in the .hip sources) -------------------------------------------
hipError_t launch_fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s);
hipError_t launch_reset_state(const Dev& d, hipStream_t s);
hipError_t launch_init_uniform(const Dev& d, float lo, float hi, uint64_t init_seed, hipStream_t s);
// Row-wise Adagrad: the accumulators of the rows cached in global slots [slot0, slot0 + slots)
// (one table, whose rows start at row_base) from the slot array to the records (to_rec),
// or from the records to the slot array.
hipError_t launch_move_acc(const Dev& d, int64_t slot0, int64_t slots, int64_t row_base, bool to_rec, hipStream_t s);
hipError_t launch_forward(const Dev& d, const Work& w, const int32_t* idx, int64_t L, const int32_t* off,
                          int32_t B, float* out, hipStream_t s);
// The forward with its temporaries in the library's static scratch array instead of a
// workspace (L <= EMB_NOALLOC_MAX_INDICES); scratch_dev from noalloc_scratch.
hipError_t noalloc_scratch(uint8_t** out);
hipError_t launch_forward_noalloc(const Dev& d, uint8_t* scratch_dev, const int32_t* idx, int64_t L,
                                  const int32_t* off, int32_t B, float* out, hipStream_t s);
// A second stream of the handle and two events: the replacement decisions and the
// write-back of displaced residents run there while the merged gradients are summed
// on the caller's stream.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};

// update_events: nullptr, or two events recorded on `s` around the row-update kernel.
hipError_t launch_backward(const Dev& d, const Work& w, const int32_t* idx, int64_t L, const int32_t* off,
                           int32_t B, const float* grad, uint64_t step, int key_bits, int seg_passes, bool decay,
                           const hipEvent_t* update_events, const SideStream& side, hipStream_t s);

size_t sort_status_words(int64_t n, int T);
size_t sort_seg_words(int T);
constexpr size_t kSortSmallWords = 2 * kMaxPasses * 256 + 64;
size_t scan_partial_words(int64_t n);
size_t uniq_tile_words(int64_t n);

}  // namespace embc
