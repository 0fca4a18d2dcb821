// Host side of libembcache: the C ABI of include/emb_cache.h.
//
// Validates configurations, plans the layout of the caller's state and
// workspace buffers, keeps the step counter and launches the kernels.  The
// library never allocates device memory.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <tuple>
#include <utility>
#include <vector>

#include "emb_cache.h"
#include "embc_dispatch.h"
#include "embc_internal.h"

using embc::TableDesc;

namespace embc {

unsigned resident_grid(const void* kernel, int threads) {
  static std::mutex mu;
  static std::map<std::tuple<const void*, int, int>, unsigned> known;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  std::lock_guard<std::mutex> lock(mu);
  const auto key = std::make_tuple(kernel, dev, threads);
  const auto it = known.find(key);
  if (it != known.end()) return it->second;
  int per_cu = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess || per_cu < 1)
    per_cu = 1;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) cus = 8;
  unsigned n = (unsigned)per_cu * (unsigned)cus / 8u * 8u;
  if (n < 8) n = 8;
  known[key] = n;
  return n;
}

// Magic numbers of DivConst for 1 <= d < 2^31.
DivConst div_const(uint32_t d) {
  DivConst c;
  uint32_t l = 0;
  while (l < 32 && (1ull << l) < d) ++l;  // ceil(log2 d)
  c.d = d;
  c.m = (uint32_t)(((1ull << 32) * ((1ull << l) - d)) / d + 1);
  c.s1 = l < 1 ? l : 1;
  c.s2 = l > 1 ? l - 1 : 0;
  return c;
}

}  // namespace embc

namespace {
using embc::div_const;
}  // namespace

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int bit_length(uint64_t v) {
  int b = 0;
  while (v) {
    ++b;
    v >>= 1;
  }
  return b;
}

struct Plan {
  int64_t total_rows = 0, total_slots = 0, total_keys = 0;
  int rec_bytes = 0;
  int acc_offset = 0;  // byte of the Adagrad accumulator in a record (under row-wise Adagrad)
  bool acc_in_rec = false;  // the accumulators of uncached rows are in the records (else acc_rows)
  std::vector<TableDesc> desc;
  std::vector<int64_t> key_base;
  // state offsets
  size_t o_rec, o_crow, o_tag, o_ts, o_cnt, o_accs, o_accr, o_desc, o_keyb, o_stats, o_err, state_bytes, table_bytes;
  // workspace offsets
  size_t o_kA, o_vA, o_kB, o_vB, o_ssmall, o_sst0, o_sst1, o_sseg, o_part, o_tcnt, o_tpre, o_tthr, o_uk, o_seg, o_setf, o_urow, o_utab, o_uslot,
      o_uact, o_udest, o_umeta, o_ukey, o_nch, o_cbase, o_uvrow, o_uvu, o_partial, o_span, o_ubig, o_brows, o_bbound, o_bpart, o_tabf, o_src, o_ctr, ws_bytes;
  int64_t max_partials = 0;
  int64_t max_big = 0;
  int32_t max_nblk = 0;
};

bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

int plan_config(const emb_cache_config* c, Plan* p) {
  if (!c || !p) return EMB_EINVAL;
  if (c->num_tables < 1 || c->num_tables > 65535 || !c->rows) return EMB_EINVAL;
  if (c->dim != 16 && c->dim != 32 && c->dim != 64 && c->dim != 128 && c->dim != 256) return EMB_EINVAL;
  if (c->precision != EMB_FP16 && c->precision != EMB_INT8 && c->precision != EMB_INT4 && c->precision != EMB_INT2)
    return EMB_EINVAL;
  if (c->sb_dtype != EMB_SB_FP32 && c->sb_dtype != EMB_SB_FP16) return EMB_EINVAL;
  if (!(c->cache_fraction >= 0.0) || !std::isfinite(c->cache_fraction)) return EMB_EINVAL;
  if (!is_pow2(c->assoc) || c->assoc > embc::kMaxAssoc) return EMB_EINVAL;
  if (c->policy != EMB_LRU && c->policy != EMB_LFU) return EMB_EINVAL;
  if (c->lfu_decay_interval < 0) return EMB_EINVAL;
  if (c->rounding != EMB_ROUND_NEAREST && c->rounding != EMB_ROUND_STOCHASTIC) return EMB_EINVAL;
  if (c->optimizer != EMB_OPT_SGD && c->optimizer != EMB_OPT_ROWWISE_ADAGRAD) return EMB_EINVAL;
  if (!std::isfinite(c->lr) || !std::isfinite(c->eps) || c->eps < 0.0f) return EMB_EINVAL;
  if (c->max_batch < 1 || c->max_indices < 1 || c->max_indices >= ((int64_t)1 << 30)) return EMB_EINVAL;
  if ((int64_t)c->max_batch * c->num_tables >= (int64_t)UINT32_MAX) return EMB_EINVAL;

  const int T = c->num_tables;
  p->desc.assign(T, TableDesc{});
  p->key_base.assign(T + 1, 0);
  int64_t rows = 0, slots = 0, keys = 0;
  for (int t = 0; t < T; ++t) {
    const int64_t N = c->rows[t];
    if (N < 1 || N >= (int64_t)INT32_MAX) return EMB_EINVAL;
    int64_t n_sets = 0;
    if (c->cache_fraction > 0.0) {
      const double cr = std::floor(c->cache_fraction * (double)N);
      if (!(cr < 4.0e18)) return EMB_EINVAL;
      n_sets = (int64_t)cr / c->assoc;
      if (n_sets < 1) n_sets = 1;
    }
    TableDesc& d = p->desc[t];
    d.N = N;
    d.row_base = rows;
    d.n_sets = n_sets;
    d.slot_base = slots;
    d.Q = n_sets ? (N + n_sets - 1) / n_sets : N;
    d.by_sets = div_const(n_sets ? (uint32_t)n_sets : 1u);
    d.by_Q = div_const((uint32_t)d.Q);
    d.key_base = keys;
    p->key_base[t] = keys;
    rows += N;
    slots += n_sets * c->assoc;
    keys += n_sets ? n_sets * d.Q : N;
    if (rows >= (int64_t)INT32_MAX || slots >= (int64_t)INT32_MAX || keys >= (int64_t)UINT32_MAX - 1)
      return EMB_EINVAL;
  }
  p->key_base[T] = keys;
  p->total_rows = rows;
  p->total_slots = slots;
  p->total_keys = keys;
  // an FP16 table stores the elements alone; integer codes carry (s, b); under row-wise
  // Adagrad the row's FP32 accumulator follows, the record padded to the alignment of
  // its first part (at most 16 bytes), as Rec<> in the kernels lays it out -- unless
  // the record would then span one more 64-byte line than without it (an FP16 table of
  // d >= 32: its records fill whole lines), when the accumulators get an array of their own
  p->acc_offset = c->dim * c->precision / 8 + (c->precision == EMB_FP16 ? 0 : c->sb_dtype == EMB_SB_FP16 ? 4 : 8);
  p->rec_bytes = p->acc_offset;
  p->acc_in_rec = false;
  if (c->optimizer == EMB_OPT_ROWWISE_ADAGRAD) {
    const int a = std::min(p->acc_offset & -p->acc_offset, 16);
    const int with = (p->acc_offset + 4 + a - 1) / a * a;
    p->acc_in_rec = (with + 63) / 64 <= (p->acc_offset + 63) / 64;
    if (p->acc_in_rec) p->rec_bytes = with;
  }

  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  const bool lru = c->policy == EMB_LRU, lfu = c->policy == EMB_LFU;
  p->o_crow = take((size_t)slots * c->dim * 4);
  p->o_tag = take((size_t)slots * 4);
  p->o_ts = take(lru ? (size_t)slots * 4 : 0);
  p->o_cnt = take(lfu ? (size_t)rows * 4 : 0);
  p->o_accs = take(c->optimizer == EMB_OPT_ROWWISE_ADAGRAD ? (size_t)slots * 4 : 0);
  p->o_accr = take(c->optimizer == EMB_OPT_ROWWISE_ADAGRAD && !p->acc_in_rec ? (size_t)rows * 4 : 0);
  p->o_desc = take(sizeof(TableDesc) * T);
  p->o_keyb = take(sizeof(int64_t) * (T + 1));
  p->o_stats = take(sizeof(unsigned long long) * T * embc::kNStat);
  p->o_err = take(kAlign);
  // the low-precision table comes last: a caller may place it in a buffer of its own
  p->o_rec = take((size_t)rows * p->rec_bytes);
  p->table_bytes = o - p->o_rec;
  p->state_bytes = o;

  const size_t L = (size_t)c->max_indices;
  o = 0;
  p->o_kA = take(4 * L);
  p->o_vA = take(4 * L);
  p->o_kB = take(4 * L);
  p->o_vB = take(4 * L);
  p->o_ssmall = take(4 * embc::kSortSmallWords);
  p->o_sst0 = take(4 * embc::sort_status_words((int64_t)L, T));
  p->o_sst1 = take(4 * embc::sort_status_words((int64_t)L, T));
  p->o_sseg = take(4 * embc::sort_seg_words(T));
  p->o_part = take(8 * embc::scan_partial_words((int64_t)L + 256 * 64));
  p->o_tcnt = take(8 * embc::uniq_tile_words((int64_t)L));
  p->o_tpre = take(8 * embc::uniq_tile_words((int64_t)L));
  p->o_tthr = take(8 * 256 * embc::uniq_tile_words((int64_t)L));
  p->o_uk = take(4 * L);
  p->o_seg = take(4 * (L + 1));
  p->o_setf = take(4 * (L + 1));
  p->o_urow = take(4 * L);
  p->o_utab = take(4 * L);
  p->o_uslot = take(4 * L);
  p->o_uact = take(4 * L);
  p->o_udest = take(4 * L);
  p->o_umeta = take(16 * L);
  p->o_ukey = take(c->policy == EMB_LFU ? 8 * L : 0);
  p->o_nch = take(4 * L);
  p->o_cbase = take(4 * (L + 1));
  p->o_uvrow = take(4 * L);
  p->o_uvu = take(4 * L);
  p->max_partials = (int64_t)(L / (embc::kSumChunk / 2) + 2);
  p->o_partial = take((size_t)p->max_partials * c->dim * 4);
  p->o_span = take((size_t)p->max_partials * 8);
  p->o_ubig = take(4 * (L + 1));
  p->max_big = (int64_t)(L / (embc::kBlockAbove + 1) + 1);
  {
    const int64_t nb = embc::kBlockFloats / c->dim;
    p->max_nblk = (int32_t)((c->max_batch + nb - 1) / nb);
  }
  p->o_brows = take(4 * (size_t)p->max_big);
  p->o_bbound = take(4 * (size_t)p->max_big * (size_t)embc::bound_stride(p->max_nblk));
  p->o_bpart = take(4 * (size_t)p->max_big * (size_t)p->max_nblk * (size_t)c->dim);
  p->o_tabf = take(4 * (size_t)(T + 1));
  p->o_src = take(4 * L);
  p->o_ctr = take(8 * embc::kNCounters);
  p->ws_bytes = o;
  return EMB_OK;
}

}  // namespace

struct emb_cache {
  emb_cache_config cfg;
  std::vector<int64_t> rows;
  Plan plan;
  embc::Dev dev;
  embc::Work work;
  uint64_t step = 0;
  int key_bits = 1;
  int seg_passes = 0;  // digit passes of the per-table sort, 0 = sort the whole key
  // measurement: event pairs around the row-update kernel of the last kTimedCalls calls
  static constexpr int kTimedCalls = 64;
  bool timing = false;
  std::vector<hipEvent_t> tev;
  uint64_t timed = 0;
  embc::SideStream side;  // default priority, non-blocking; events without timing
  uint8_t* noalloc = nullptr;  // device address of the static scratch of emb_cache_forward_noalloc
  ~emb_cache() {
    for (hipEvent_t e : tev) (void)hipEventDestroy(e);
    if (side.fork) (void)hipEventDestroy(side.fork);
    if (side.join) (void)hipEventDestroy(side.join);
    if (side.s) (void)hipStreamDestroy(side.s);
  }
};

namespace {

hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

int hip_status(hipError_t e) { return e == hipSuccess ? EMB_OK : EMB_EHIP; }

// IEEE binary16 <-> binary32 on the host (exact widening; RNE narrowing).
float half_bits_to_float(uint16_t h) { return (float)*reinterpret_cast<const _Float16*>(&h); }
uint16_t float_to_half_bits(float f) {
  const _Float16 h = (_Float16)f;
  uint16_t b;
  std::memcpy(&b, &h, 2);
  return b;
}

}  // namespace

extern "C" {

int emb_cache_query_sizes(const emb_cache_config* cfg, emb_cache_sizes* out) {
  if (!out) return EMB_EINVAL;
  Plan p;
  const int st = plan_config(cfg, &p);
  if (st != EMB_OK) return st;
  out->state_bytes = p.state_bytes;
  out->workspace_bytes = p.ws_bytes;
  out->total_rows = p.total_rows;
  out->total_slots = p.total_slots;
  out->row_bytes = p.rec_bytes;
  out->pad = 0;
  out->table_bytes = p.table_bytes;
  return EMB_OK;
}

int emb_cache_table_geometry(const emb_cache_config* cfg, int32_t table, int64_t* n_sets, int64_t* slots) {
  Plan p;
  const int st = plan_config(cfg, &p);
  if (st != EMB_OK) return st;
  if (table < 0 || table >= cfg->num_tables || !n_sets || !slots) return EMB_EINVAL;
  *n_sets = p.desc[table].n_sets;
  *slots = p.desc[table].n_sets * cfg->assoc;
  return EMB_OK;
}

namespace {

// The device address of a caller's table buffer: device memory as it is, pinned host
// memory (hipHostMalloc) through its device mapping; anything else is refused, since
// a kernel could not reach it.
int table_device_address(void* table, uint8_t** dev) {
  hipPointerAttribute_t a{};
  if (hipPointerGetAttributes(&a, table) != hipSuccess) {
    (void)hipGetLastError();
    return EMB_EINVAL;
  }
  if (a.type == hipMemoryTypeDevice) {
    *dev = static_cast<uint8_t*>(table);
    return EMB_OK;
  }
  if (a.type == hipMemoryTypeHost && a.devicePointer) {
    *dev = static_cast<uint8_t*>(a.devicePointer);
    return EMB_OK;
  }
  return EMB_EINVAL;
}

int create_impl(const emb_cache_config* cfg, void* state, size_t state_bytes, void* table, size_t table_bytes,
                void* workspace, size_t workspace_bytes, void* stream, emb_cache_t* out);

}  // namespace

int emb_cache_create(const emb_cache_config* cfg, void* state, size_t state_bytes, void* workspace,
                     size_t workspace_bytes, void* stream, emb_cache_t* out) {
  return create_impl(cfg, state, state_bytes, nullptr, 0, workspace, workspace_bytes, stream, out);
}

int emb_cache_create_with_table(const emb_cache_config* cfg, void* state, size_t state_bytes, void* table,
                                size_t table_bytes, void* workspace, size_t workspace_bytes, void* stream,
                                emb_cache_t* out) {
  if (!table) {
    if (out) *out = nullptr;
    return EMB_EINVAL;
  }
  return create_impl(cfg, state, state_bytes, table, table_bytes, workspace, workspace_bytes, stream, out);
}

namespace {

int create_impl(const emb_cache_config* cfg, void* state, size_t state_bytes, void* table, size_t table_bytes,
                void* workspace, size_t workspace_bytes, void* stream, emb_cache_t* out) {
  if (!out) return EMB_EINVAL;
  *out = nullptr;
  emb_cache* h = new (std::nothrow) emb_cache();
  if (!h) return EMB_EINVAL;
  int st = plan_config(cfg, &h->plan);
  if (st != EMB_OK) {
    delete h;
    return st;
  }
  const Plan& p = h->plan;
  if (!state || !workspace || (reinterpret_cast<uintptr_t>(state) % kAlign) ||
      (reinterpret_cast<uintptr_t>(workspace) % kAlign) || (reinterpret_cast<uintptr_t>(table) % kAlign)) {
    delete h;
    return EMB_EINVAL;
  }
  // with a table buffer of its own, the state buffer holds everything before the table
  const size_t need_state = table ? p.o_rec : p.state_bytes;
  if (state_bytes < need_state || workspace_bytes < p.ws_bytes || (table && table_bytes < p.table_bytes)) {
    delete h;
    return EMB_ENOMEM;
  }
  uint8_t* table_dev = nullptr;
  if (table && table_device_address(table, &table_dev) != EMB_OK) {
    delete h;
    return EMB_EINVAL;
  }
  h->cfg = *cfg;
  h->rows.assign(cfg->rows, cfg->rows + cfg->num_tables);
  h->cfg.rows = h->rows.data();
  // every valid key is below 2^key_bits - 1, the skipped-lookup key truncated to key_bits
  h->key_bits = bit_length((uint64_t)p.total_keys);
  if (h->key_bits < 1) h->key_bits = 1;
  // the lookups come grouped by table: sorting each table's segment by its local key
  // takes fewer passes when every table's key range is much smaller than their sum
  {
    int64_t max_range = 1;
    for (int t = 0; t < cfg->num_tables; ++t) max_range = std::max(max_range, p.key_base[t + 1] - p.key_base[t]);
    const int seg = (bit_length((uint64_t)max_range) + 7) / 8;
    h->seg_passes = seg < (h->key_bits + 7) / 8 ? seg : 0;
  }

  uint8_t* sb = static_cast<uint8_t*>(state);
  embc::Dev& d = h->dev;
  d.rec = table ? table_dev : sb + p.o_rec;
  d.crow = reinterpret_cast<float*>(sb + p.o_crow);
  d.tag = reinterpret_cast<int32_t*>(sb + p.o_tag);
  d.ts = cfg->policy == EMB_LRU ? reinterpret_cast<int32_t*>(sb + p.o_ts) : nullptr;
  d.cnt = cfg->policy == EMB_LFU ? reinterpret_cast<int32_t*>(sb + p.o_cnt) : nullptr;
  d.acc_slot = cfg->optimizer == EMB_OPT_ROWWISE_ADAGRAD ? reinterpret_cast<float*>(sb + p.o_accs) : nullptr;
  d.acc_rows = cfg->optimizer == EMB_OPT_ROWWISE_ADAGRAD && !p.acc_in_rec ? reinterpret_cast<float*>(sb + p.o_accr)
                                                                          : nullptr;
  d.desc = reinterpret_cast<const TableDesc*>(sb + p.o_desc);
  d.key_base = reinterpret_cast<const int64_t*>(sb + p.o_keyb);
  d.stats = reinterpret_cast<unsigned long long*>(sb + p.o_stats);
  d.err = reinterpret_cast<int32_t*>(sb + p.o_err);
  d.T = cfg->num_tables;
  d.dim = cfg->dim;
  d.bits = cfg->precision;
  d.sb16 = cfg->precision != EMB_FP16 && cfg->sb_dtype == EMB_SB_FP16;  // an FP16 table has no (s, b)
  d.assoc = cfg->assoc;
  d.rec_bytes = p.rec_bytes;
  d.acc_offset = p.acc_offset;
  d.policy = cfg->policy;
  d.rounding = cfg->rounding;
  d.optimizer = cfg->optimizer;
  d.lr = cfg->lr;
  d.eps = cfg->eps;
  d.seed = cfg->seed;
  d.total_rows = p.total_rows;
  d.total_slots = p.total_slots;

  uint8_t* wb = static_cast<uint8_t*>(workspace);
  embc::Work& w = h->work;
  w.keysA = reinterpret_cast<uint32_t*>(wb + p.o_kA);
  w.valsA = reinterpret_cast<uint32_t*>(wb + p.o_vA);
  w.keysB = reinterpret_cast<uint32_t*>(wb + p.o_kB);
  w.valsB = reinterpret_cast<uint32_t*>(wb + p.o_vB);
  w.sort_small = reinterpret_cast<uint32_t*>(wb + p.o_ssmall);
  w.sort_status[0] = reinterpret_cast<uint32_t*>(wb + p.o_sst0);
  w.sort_status[1] = reinterpret_cast<uint32_t*>(wb + p.o_sst1);
  w.sort_seg = reinterpret_cast<uint32_t*>(wb + p.o_sseg);
  w.part = reinterpret_cast<unsigned long long*>(wb + p.o_part);
  w.tile_cnt = reinterpret_cast<unsigned long long*>(wb + p.o_tcnt);
  w.tile_pre = reinterpret_cast<unsigned long long*>(wb + p.o_tpre);
  w.thread_pre = reinterpret_cast<unsigned long long*>(wb + p.o_tthr);
  w.uniq_key = reinterpret_cast<uint32_t*>(wb + p.o_uk);
  w.seg = reinterpret_cast<uint32_t*>(wb + p.o_seg);
  w.set_first = reinterpret_cast<uint32_t*>(wb + p.o_setf);
  w.urow = reinterpret_cast<int32_t*>(wb + p.o_urow);
  w.utab = reinterpret_cast<int32_t*>(wb + p.o_utab);
  w.uslot = reinterpret_cast<int32_t*>(wb + p.o_uslot);
  w.uact = reinterpret_cast<int32_t*>(wb + p.o_uact);
  w.udest = reinterpret_cast<int32_t*>(wb + p.o_udest);
  w.umeta = reinterpret_cast<uint4*>(wb + p.o_umeta);
  w.ukey = reinterpret_cast<unsigned long long*>(wb + p.o_ukey);
  w.nch = reinterpret_cast<uint32_t*>(wb + p.o_nch);
  w.chunk_base = reinterpret_cast<uint32_t*>(wb + p.o_cbase);
  w.uvic_row = reinterpret_cast<int32_t*>(wb + p.o_uvrow);
  w.uvic_u = reinterpret_cast<int32_t*>(wb + p.o_uvu);
  w.partial = reinterpret_cast<float*>(wb + p.o_partial);
  w.ubig = reinterpret_cast<uint32_t*>(wb + p.o_ubig);
  w.big_rows = reinterpret_cast<int32_t*>(wb + p.o_brows);
  w.bbound = reinterpret_cast<uint32_t*>(wb + p.o_bbound);
  w.bpart = reinterpret_cast<float*>(wb + p.o_bpart);
  w.max_big = p.max_big;
  w.max_nblk = p.max_nblk;
  w.chunk_span = reinterpret_cast<uint2*>(wb + p.o_span);
  w.tab_first = reinterpret_cast<int32_t*>(wb + p.o_tabf);
  w.fwd_src = reinterpret_cast<int32_t*>(wb + p.o_src);
  w.ctr = reinterpret_cast<unsigned long long*>(wb + p.o_ctr);
  w.max_indices = cfg->max_indices;
  w.max_partials = p.max_partials;

  hipStream_t s = S(stream);
  hipError_t e = hipMemcpyAsync(sb + p.o_desc, p.desc.data(), sizeof(TableDesc) * p.desc.size(),
                                hipMemcpyHostToDevice, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(sb + p.o_keyb, p.key_base.data(), sizeof(int64_t) * p.key_base.size(), hipMemcpyHostToDevice,
                       s);
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&h->side.s, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&h->side.fork, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&h->side.join, hipEventDisableTiming);
  if (e == hipSuccess) e = embc::noalloc_scratch(&h->noalloc);  // once per device, this device current
  if (e == hipSuccess) e = embc::launch_reset_state(d, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) {
    delete h;
    return EMB_EHIP;
  }
  h->step = 0;
  *out = h;
  return EMB_OK;
}

}  // namespace

int emb_cache_destroy(emb_cache_t h) {
  delete h;
  return EMB_OK;
}

int emb_cache_init_uniform(emb_cache_t h, float lo, float hi, uint64_t init_seed, void* stream) {
  if (!h || !std::isfinite(lo) || !std::isfinite(hi)) return EMB_EINVAL;
  return hip_status(embc::launch_init_uniform(h->dev, lo, hi, init_seed, S(stream)));
}

int emb_cache_forward(emb_cache_t h, const int32_t* indices, int64_t num_indices, const int32_t* offsets,
                      int32_t batch, float* out, void* stream) {
  if (!h || batch < 0 || batch > h->cfg.max_batch || num_indices < 0 || num_indices > h->cfg.max_indices)
    return EMB_EINVAL;
  if ((num_indices > 0 && !indices) || !offsets || (batch > 0 && !out)) return EMB_EINVAL;
  return hip_status(embc::launch_forward(h->dev, h->work, indices, num_indices, offsets, batch, out, S(stream)));
}

int emb_cache_forward_noalloc(emb_cache_t h, const int32_t* indices, int64_t num_indices, const int32_t* offsets,
                              int32_t batch, float* out, void* stream) {
  if (!h || batch < 0 || batch > h->cfg.max_batch || num_indices < 0) return EMB_EINVAL;
  if ((num_indices > 0 && !indices) || !offsets || (batch > 0 && !out)) return EMB_EINVAL;
  if (num_indices > EMB_NOALLOC_MAX_INDICES) return EMB_ENOMEM;  // beyond the static scratch
  if (!h->noalloc) return EMB_EHIP;
  return hip_status(
      embc::launch_forward_noalloc(h->dev, h->noalloc, indices, num_indices, offsets, batch, out, S(stream)));
}

int emb_cache_backward_update(emb_cache_t h, const int32_t* indices, int64_t num_indices, const int32_t* offsets,
                              int32_t batch, const float* grad_out, void* stream) {
  if (!h || batch < 0 || batch > h->cfg.max_batch || num_indices < 0 || num_indices > h->cfg.max_indices)
    return EMB_EINVAL;
  if ((num_indices > 0 && !indices) || !offsets || (batch > 0 && !grad_out)) return EMB_EINVAL;
  const int K = h->cfg.lfu_decay_interval;
  const bool decay = h->cfg.policy == EMB_LFU && K > 0 && h->step > 0 && h->step % (uint64_t)K == 0;
  const hipEvent_t* tev = nullptr;
  if (h->timing) tev = &h->tev[2 * (h->timed % emb_cache::kTimedCalls)];
  const hipError_t e = embc::launch_backward(h->dev, h->work, indices, num_indices, offsets, batch, grad_out,
                                             h->step, h->key_bits, h->seg_passes, decay, tev, h->side, S(stream));
  if (e != hipSuccess) return EMB_EHIP;
  if (h->timing) h->timed += 1;
  h->step += 1;
  return EMB_OK;
}

int emb_cache_get_stats(emb_cache_t h, int32_t table, int64_t* out, void* stream) {
  if (!h || !out || table < 0 || table >= h->cfg.num_tables) return EMB_EINVAL;
  hipStream_t s = S(stream);
  unsigned long long tmp[embc::kNStat];
  hipError_t e = hipMemcpyAsync(tmp, h->dev.stats + (int64_t)table * embc::kNStat, sizeof(tmp), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return EMB_EHIP;
  for (int i = 0; i < embc::kNStat; ++i) out[i] = (int64_t)tmp[i];
  return EMB_OK;
}

int emb_cache_check(emb_cache_t h, void* stream) {
  if (!h) return EMB_EINVAL;
  hipStream_t s = S(stream);
  int32_t flag = 0;
  hipError_t e = hipMemcpyAsync(&flag, h->dev.err, sizeof(flag), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return EMB_EHIP;
  if (flag) {
    const int32_t zero = 0;
    e = hipMemcpyAsync(h->dev.err, &zero, sizeof(zero), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return EMB_EHIP;
    return (flag & embc::kErrSort) ? EMB_EHIP : EMB_EINDEX;
  }
  return EMB_OK;
}

namespace {
// Row-wise Adagrad: the accumulator of a cached row is in the slot array, not in its record.
// The tags and slot accumulators of `table` on the host (synchronizes s).
hipError_t table_slots(emb_cache_t h, int32_t table, hipStream_t s, std::vector<int32_t>* tags,
                       std::vector<float>* acc) {
  const TableDesc& td = h->plan.desc[table];
  const int64_t slots = td.n_sets * h->cfg.assoc;
  tags->assign((size_t)slots, -1);
  acc->assign((size_t)slots, 0.0f);
  if (slots == 0) return hipSuccess;
  hipError_t e = hipMemcpyAsync(tags->data(), h->dev.tag + td.slot_base, 4 * (size_t)slots, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(acc->data(), h->dev.acc_slot + td.slot_base, 4 * (size_t)slots, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return e;
}
}  // namespace

int emb_cache_export_rows(emb_cache_t h, int32_t table, int64_t row0, int64_t n, void* codes_out, float* scale,
                          float* bias, int32_t* lfu_count, float* adagrad, void* stream) {
  if (!h || table < 0 || table >= h->cfg.num_tables || row0 < 0 || n < 0) return EMB_EINVAL;
  const TableDesc& td = h->plan.desc[table];
  if (row0 + n > td.N) return EMB_EINVAL;
  if (n == 0) return EMB_OK;
  hipStream_t s = S(stream);
  const int d = h->cfg.dim, RB = h->plan.rec_bytes, bits = h->cfg.precision;
  const int64_t g0 = td.row_base + row0;
  const bool ada = h->cfg.optimizer == EMB_OPT_ROWWISE_ADAGRAD;
  const bool acc_rec = ada && h->plan.acc_in_rec;
  hipError_t e = hipSuccess;
  if (adagrad && ada && !acc_rec)
    e = hipMemcpyAsync(adagrad, h->dev.acc_rows + g0, 4 * (size_t)n, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess && (codes_out || scale || bias || (adagrad && acc_rec))) {
    std::vector<uint8_t> buf((size_t)n * RB);
    e = hipMemcpyAsync(buf.data(), h->dev.rec + g0 * RB, buf.size(), hipMemcpyDefault, s);  // device or pinned host table
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return EMB_EHIP;
    const int cb = d * bits / 8;
    uint8_t* codes = static_cast<uint8_t*>(codes_out);
    for (int64_t i = 0; i < n; ++i) {
      const uint8_t* r = buf.data() + i * RB;
      if (adagrad && acc_rec) std::memcpy(&adagrad[i], r + h->plan.acc_offset, 4);
      if (bits == EMB_FP16) {  // binary16 bit patterns as stored, no (s, b)
        if (codes) std::memcpy(codes + i * d * 2, r, 2 * (size_t)d);
        if (scale) scale[i] = 0.0f;
        if (bias) bias[i] = 0.0f;
        continue;
      }
      if (codes) {
        const int per = 8 / bits, mask = (1 << bits) - 1;  // codes per byte, column j in bits (j % per) * bits
        for (int j = 0; j < d; ++j) codes[i * d + j] = (uint8_t)((r[j / per] >> ((j % per) * bits)) & mask);
      }
      float sv, bv;
      if (h->cfg.sb_dtype == EMB_SB_FP16) {
        uint16_t hs, hb;
        std::memcpy(&hs, r + cb, 2);
        std::memcpy(&hb, r + cb + 2, 2);
        sv = half_bits_to_float(hs);
        bv = half_bits_to_float(hb);
      } else {
        std::memcpy(&sv, r + cb, 4);
        std::memcpy(&bv, r + cb + 4, 4);
      }
      if (scale) scale[i] = sv;
      if (bias) bias[i] = bv;
    }
  }
  if (lfu_count) {
    if (h->dev.cnt) e = hipMemcpyAsync(lfu_count, h->dev.cnt + g0, 4 * (size_t)n, hipMemcpyDeviceToHost, s);
    else std::memset(lfu_count, 0, 4 * (size_t)n);
  }
  if (adagrad && !ada) std::memset(adagrad, 0, 4 * (size_t)n);
  if (e == hipSuccess && adagrad && ada) {
    std::vector<int32_t> tags;
    std::vector<float> acc;
    e = table_slots(h, table, s, &tags, &acc);
    for (size_t i = 0; e == hipSuccess && i < tags.size(); ++i)
      if (tags[i] >= row0 && tags[i] < row0 + n) adagrad[tags[i] - row0] = acc[i];
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return hip_status(e);
}

int emb_cache_import_rows(emb_cache_t h, int32_t table, int64_t row0, int64_t n, const void* codes_in,
                          const float* scale, const float* bias, const int32_t* lfu_count, const float* adagrad,
                          void* stream) {
  if (!h || table < 0 || table >= h->cfg.num_tables || row0 < 0 || n < 0) return EMB_EINVAL;
  const TableDesc& td = h->plan.desc[table];
  if (row0 + n > td.N) return EMB_EINVAL;
  if (n == 0) return EMB_OK;
  hipStream_t s = S(stream);
  const int d = h->cfg.dim, RB = h->plan.rec_bytes, bits = h->cfg.precision;
  const int64_t g0 = td.row_base + row0;
  const bool ada = h->cfg.optimizer == EMB_OPT_ROWWISE_ADAGRAD;
  const uint8_t* codes = static_cast<const uint8_t*>(codes_in);
  const bool put_codes = bits == EMB_FP16 ? codes != nullptr : (codes || scale || bias);
  if (bits != EMB_FP16 && put_codes && (!codes || !scale || !bias)) return EMB_EINVAL;  // codes and (s, b) go together
  const bool put_acc = adagrad && ada;
  const bool acc_rec = ada && h->plan.acc_in_rec;
  hipError_t e = hipSuccess;
  if (put_acc && !acc_rec)
    e = hipMemcpyAsync(h->dev.acc_rows + g0, adagrad, 4 * (size_t)n, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && (put_codes || (put_acc && acc_rec))) {
    // the records as they are (what is not given stays), then the given parts
    std::vector<uint8_t> buf((size_t)n * RB);
    e = hipMemcpyAsync(buf.data(), h->dev.rec + g0 * RB, buf.size(), hipMemcpyDefault, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return EMB_EHIP;
    const int K = (1 << bits) - 1;
    const int cb = d * bits / 8;
    for (int64_t i = 0; i < n; ++i) {
      uint8_t* r = buf.data() + i * RB;
      if (put_codes && bits == EMB_FP16) {  // binary16 bit patterns as stored; scale and bias are not used
        std::memcpy(r, codes + i * d * 2, 2 * (size_t)d);
      } else if (put_codes) {
        const int per = 8 / bits;  // codes per byte, column j in bits (j % per) * bits
        std::memset(r, 0, (size_t)cb);
        for (int j = 0; j < d; ++j) {
          const uint8_t q = codes[i * d + j];
          if (q > K) return EMB_EINVAL;
          r[j / per] |= (uint8_t)(q << ((j % per) * bits));
        }
        if (h->cfg.sb_dtype == EMB_SB_FP16) {
          const uint16_t hs = float_to_half_bits(scale[i]), hb = float_to_half_bits(bias[i]);
          if (half_bits_to_float(hs) != scale[i] || half_bits_to_float(hb) != bias[i]) return EMB_EINVAL;
          std::memcpy(r + cb, &hs, 2);
          std::memcpy(r + cb + 2, &hb, 2);
        } else {
          std::memcpy(r + cb, &scale[i], 4);
          std::memcpy(r + cb + 4, &bias[i], 4);
        }
      }
      if (put_acc && acc_rec) std::memcpy(r + h->plan.acc_offset, &adagrad[i], 4);
    }
    e = hipMemcpyAsync(h->dev.rec + g0 * RB, buf.data(), buf.size(), hipMemcpyDefault, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);  // buf is released on return
  }
  if (e == hipSuccess && put_acc) {
    // a cached row's accumulator is in the slot array
    std::vector<int32_t> tags;
    std::vector<float> acc;
    e = table_slots(h, table, s, &tags, &acc);
    bool any = false;
    for (size_t i = 0; e == hipSuccess && i < tags.size(); ++i)
      if (tags[i] >= row0 && tags[i] < row0 + n) acc[i] = adagrad[tags[i] - row0], any = true;
    if (e == hipSuccess && any)
      e = hipMemcpyAsync(h->dev.acc_slot + td.slot_base, acc.data(), 4 * acc.size(), hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
  }
  if (e == hipSuccess && lfu_count && h->dev.cnt)
    e = hipMemcpyAsync(h->dev.cnt + g0, lfu_count, 4 * (size_t)n, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return hip_status(e);
}

int emb_cache_export_cache(emb_cache_t h, int32_t table, float* rows, int32_t* tags, int32_t* lru_stamp,
                           void* stream) {
  if (!h || table < 0 || table >= h->cfg.num_tables) return EMB_EINVAL;
  const TableDesc& td = h->plan.desc[table];
  const int64_t slots = td.n_sets * h->cfg.assoc;
  if (slots == 0) return EMB_OK;
  hipStream_t s = S(stream);
  const int d = h->cfg.dim;
  hipError_t e = hipSuccess;
  if (rows) e = hipMemcpyAsync(rows, h->dev.crow + td.slot_base * d, 4 * (size_t)(slots * d), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess && tags)
    e = hipMemcpyAsync(tags, h->dev.tag + td.slot_base, 4 * (size_t)slots, hipMemcpyDeviceToHost, s);
  if (e == hipSuccess && lru_stamp) {
    if (h->dev.ts) e = hipMemcpyAsync(lru_stamp, h->dev.ts + td.slot_base, 4 * (size_t)slots, hipMemcpyDeviceToHost, s);
    else
      for (int64_t i = 0; i < slots; ++i) lru_stamp[i] = -1;
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return hip_status(e);
}

int emb_cache_import_cache(emb_cache_t h, int32_t table, const float* rows, const int32_t* tags,
                           const int32_t* lru_stamp, void* stream) {
  if (!h || table < 0 || table >= h->cfg.num_tables) return EMB_EINVAL;
  const TableDesc& td = h->plan.desc[table];
  const int64_t slots = td.n_sets * h->cfg.assoc;
  if (slots == 0) return EMB_OK;
  if (tags) {
    for (int64_t i = 0; i < slots; ++i) {
      const int32_t tg = tags[i];
      if (tg < -1 || tg >= td.N) return EMB_EINVAL;
      if (tg >= 0 && (tg % td.n_sets) != (i / h->cfg.assoc)) return EMB_EINVAL;  // row must map to its set
    }
  }
  hipStream_t s = S(stream);
  const int d = h->cfg.dim;
  hipError_t e = hipSuccess;
  if (rows) e = hipMemcpyAsync(h->dev.crow + td.slot_base * d, rows, 4 * (size_t)(slots * d), hipMemcpyHostToDevice, s);
  // new residents: the accumulators of the rows leaving the cache go back to their
  // records, those of the rows entering it come from theirs
  if (e == hipSuccess && tags) e = embc::launch_move_acc(h->dev, td.slot_base, slots, td.row_base, true, s);
  if (e == hipSuccess && tags)
    e = hipMemcpyAsync(h->dev.tag + td.slot_base, tags, 4 * (size_t)slots, hipMemcpyHostToDevice, s);
  if (e == hipSuccess && tags) e = embc::launch_move_acc(h->dev, td.slot_base, slots, td.row_base, false, s);
  if (e == hipSuccess && lru_stamp && h->dev.ts)
    e = hipMemcpyAsync(h->dev.ts + td.slot_base, lru_stamp, 4 * (size_t)slots, hipMemcpyHostToDevice, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  return hip_status(e);
}

int emb_cache_set_update_timing(emb_cache_t h, int32_t enable) {
  if (!h) return EMB_EINVAL;
  if (enable && h->tev.empty()) {
    h->tev.assign(2 * emb_cache::kTimedCalls, nullptr);
    for (hipEvent_t& e : h->tev)
      if (hipEventCreate(&e) != hipSuccess) return EMB_EHIP;
  }
  h->timing = enable != 0;
  h->timed = 0;
  return EMB_OK;
}

int emb_cache_get_update_times(emb_cache_t h, float* ms, int32_t max, int32_t* n) {
  if (!h || !n || max < 0 || (max > 0 && !ms)) return EMB_EINVAL;
  uint64_t k = h->timed < (uint64_t)emb_cache::kTimedCalls ? h->timed : (uint64_t)emb_cache::kTimedCalls;
  if (k > (uint64_t)max) k = (uint64_t)max;
  for (uint64_t i = 0; i < k; ++i) {
    const uint64_t call = h->timed - k + i;
    hipEvent_t* ev = &h->tev[2 * (call % emb_cache::kTimedCalls)];
    if (hipEventSynchronize(ev[1]) != hipSuccess || hipEventElapsedTime(&ms[i], ev[0], ev[1]) != hipSuccess)
      return EMB_EHIP;
  }
  *n = (int32_t)k;
  return EMB_OK;
}

int emb_cache_get_step(emb_cache_t h, uint64_t* step) {
  if (!h || !step) return EMB_EINVAL;
  *step = h->step;
  return EMB_OK;
}

int emb_cache_set_step(emb_cache_t h, uint64_t step) {
  if (!h) return EMB_EINVAL;
  h->step = step;
  return EMB_OK;
}

const char* emb_cache_status_string(int status) {
  switch (status) {
    case EMB_OK: return "ok";
    case EMB_EINVAL: return "invalid argument or configuration";
    case EMB_ENOMEM: return "buffer smaller than required";
    case EMB_EINDEX: return "index outside the table, or malformed offsets";
    case EMB_EHIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

}  // extern "C"
