// C ABI of libmlkv: table manager (device allocation, index sizing, per-call
// scratch, error latch) and the launch sequence of each call.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <utility>
#include <string>
#include <vector>

#include "mlkv.h"
#include "mlkv_kernels.h"

using namespace mlkv;

// A set of scratch buffers replaced by a larger one; freed once `done` (an
// event recorded behind the last work that may use them) has completed.
struct ScratchSet {
  std::vector<void*> ptrs;
  hipEvent_t done = nullptr;
};

struct mlkv_table {
  int device = 0;
  int32_t dim = 0;
  int64_t capacity = 0;
  uint64_t seed = 0;
  float max_load = 0.75f;
  uint32_t nb_log2 = 0;
  uint64_t nb = 0;
  Bucket* idx = nullptr;
  float* rows = nullptr;   // all rows in HBM; for a tiered table the HBM row cache
  float* state = nullptr;
  // tiered table: rows at home in pinned host memory, cache_rows of them in HBM
  float* host_rows = nullptr;
  uint32_t* slot_of_row = nullptr;  // [capacity] cache slot or kNoSlot
  uint32_t* row_of_slot = nullptr;  // [cache_rows] row held or kNoSlot
  uint8_t* dirty = nullptr;         // [cache_rows]
  uint32_t* keep = nullptr;         // [cache_rows] lookahead call that asked for the slot's row
  int64_t cache_rows = 0;
  void* host_alloc = nullptr;       // the pinned allocation behind host_rows
  uint32_t tier_tag = 0;            // lookahead calls made (tags the rows each one keeps)
  uint64_t tier_calls = 0;          // the same count without wrapping: its parity picks the miss counter
  // lookahead scratch (tiered tables): misses and the copy plan, n entries each
  uint32_t* miss = nullptr;
  uint32_t* plan_slot = nullptr;
  Ctrl* ctrl = nullptr;
  // sequence number of calls that may change the table; starts at 1 because
  // the control block's epoch markers start at 0 ("no call")
  uint64_t epoch = 1;

  // bounded staleness: one word per row (count | get-call epoch), the bound,
  // and the epoch of the next get call (from 1: a cleared stamp is 0)
  unsigned long long* clock = nullptr;
  int64_t bound = -1;
  uint64_t cepoch = 1;

  // per-call scratch, grown on demand
  int64_t ws_n = 0;
  NewKey* newlist = nullptr;
  uint32_t* tile_cnt = nullptr;
  uint64_t* items = nullptr;
  uint32_t* meta = nullptr;
  uint64_t* spill = nullptr;
  uint64_t spill_words = 0;
  uint32_t* rs_cnt = nullptr;  // radix dedup: per-tile digit counts and the item total
  int dedup = kDedupHash;
  int rs_bits = 0;             // radix dedup: bits of the sort key
  double* partials = nullptr;
  uint64_t* pc_key = nullptr;  // the last get's present keys and rows by position
  uint32_t* pc_row = nullptr;
  bool pc_lookahead = false;   // they were last written by a lookahead (its gets usually follow)
  // key-range lists of a get that runs between a put's probe and its reduce
  // (mlkv_get_put_grad), apart from the put's items and metadata
  uint64_t* mid_xkey = nullptr;
  uint32_t* mid_xslot = nullptr;
  // new keys of a get filed by key range (RangeLists): the lists, the counts
  // of two consecutive calls (ping-pong on rl_calls) then the number of
  // ranges of the cut points, and the cut points
  NewKey* rl_list = nullptr;
  uint64_t rl_entries = 0;
  uint32_t* rl_cnt = nullptr;
  uint64_t* rl_cuts = nullptr;
  uint64_t rl_calls = 0;
  std::vector<ScratchSet> retired;  // replaced scratch, freed at sync / reserve / close
  int cus = 256;  // compute units of the device

  // optional per-launch timing: HIP events recorded around each kernel
  struct ProfRec {
    int kernel;
    hipEvent_t start, stop;
  };
  bool prof_on = false;
  std::vector<ProfRec> prof_recs;
  std::vector<hipEvent_t> prof_pool;
  hipEvent_t prof_open[K_COUNT] = {};
};

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  g_err = std::string(what) + ": " + hipGetErrorString(e);
  return e == hipErrorOutOfMemory ? MLKV_ENOMEM : MLKV_EDEVICE;
}

template <class T>
hipError_t dev_alloc(T** p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  return hipMalloc(reinterpret_cast<void**>(p), bytes);
}

// The scratch buffers of a table, as one set (grown as a whole).
void free_scratch_set(const ScratchSet& s) {
  for (void* p : s.ptrs) (void)hipFree(p);
}

ScratchSet current_set(mlkv_table* t) {
  ScratchSet s;
  s.ptrs = {t->newlist, t->tile_cnt, t->items, t->meta, t->spill, t->partials, t->pc_key, t->pc_row,
            t->rs_cnt, t->miss, t->plan_slot, t->mid_xkey, t->mid_xslot, t->rl_list, t->rl_cnt, t->rl_cuts};
  return s;
}

void clear_workspace_ptrs(mlkv_table* t) {
  t->miss = nullptr;
  t->plan_slot = nullptr;
  t->pc_key = nullptr;
  t->pc_row = nullptr;
  t->mid_xkey = nullptr;
  t->mid_xslot = nullptr;
  t->rl_list = nullptr;
  t->rl_cnt = nullptr;
  t->rl_cuts = nullptr;
  t->rl_entries = 0;
  t->partials = nullptr;
  t->newlist = nullptr;
  t->tile_cnt = nullptr;
  t->items = nullptr;
  t->meta = nullptr;
  t->spill = nullptr;
  t->rs_cnt = nullptr;
  t->ws_n = 0;
  t->spill_words = 0;
}

void free_workspace(mlkv_table* t) {
  free_scratch_set(current_set(t));
  clear_workspace_ptrs(t);
}

// Frees the scratch sets replaced by larger ones, once the work queued
// before each replacement has finished (their events have completed).
int release_retired(mlkv_table* t) {
  int rc = MLKV_OK;
  for (auto& r : t->retired) {
    if (r.done != nullptr) {
      hipError_t e = hipEventSynchronize(r.done);
      if (e != hipSuccess && rc == MLKV_OK) rc = hip_fail(e, "hipEventSynchronize");
      (void)hipEventDestroy(r.done);
    }
    free_scratch_set(r);
  }
  t->retired.clear();
  return rc;
}

// Partitions of a put call of n keys: a power of two, at most kMaxParts,
// with at most kPartTarget keys each on average before in-tile merging.
uint32_t part_bits(int64_t n) {
  uint32_t pb = 0;
  while ((1 << pb) < kMaxParts && ((int64_t)kPartTarget << pb) < n) ++pb;
  return pb;
}

// Partitions used by a put call: as part_bits (never more; the partition
// metadata holds kMaxParts per tile), but one partition per CU, up to twice
// the target each, when that keeps the grouping blocks to one round. A small
// batch keeps its few large partitions: a block's grouping costs about the
// same for fewer items, and more blocks measured slower.
uint32_t call_part_bits(int64_t n, int cus) {
  uint32_t pb = part_bits(n);
  if (pb > 0 && (1 << pb) > cus && (1 << (pb - 1)) >= cus && (int64_t)(2 * kPartTarget) * cus >= n) --pb;
  return pb;
}

// Scratch for calls of up to n keys: new-key lists, per-tile counts, the
// partitioned items, partition metadata, the spill area, in-tile sums, the
// grouped partitions and the last get's rows by position. A larger set
// replaces the current one without waiting for the device: the old set is
// retired behind an event recorded on `st` (the work queued before uses it)
// and freed by mlkv_sync, mlkv_reserve or mlkv_close. The new row cache is
// cleared on `st`, ahead of the kernels that read it.
int ensure_workspace(mlkv_table* t, int64_t n, hipStream_t st) {
  if (n <= t->ws_n) return MLKV_OK;
  int64_t want = std::max<int64_t>(n, std::max<int64_t>(65536, 2 * t->ws_n));
  want = (want + kPutTile - 1) / kPutTile * kPutTile;
  hipError_t e = hipSuccess;
  if (t->ws_n > 0) {
    ScratchSet old = current_set(t);
    if ((e = hipEventCreateWithFlags(&old.done, hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventRecord(old.done, st)) != hipSuccess) {
      if (old.done != nullptr) (void)hipEventDestroy(old.done);
      return hip_fail(e, "retiring scratch");
    }
    t->retired.push_back(old);
    clear_workspace_ptrs(t);
  }
  const int64_t get_tiles = (want + kGetTileMin - 1) / kGetTileMin + t->cus + 1;
  // put tiles are kPutTile keys, or fewer so that every CU gets one
  const int64_t put_tiles = std::max<int64_t>(want / kPutTile, t->cus + 1);
  const int64_t slots = std::max<int64_t>(want, put_tiles * kPutTile);
  const uint64_t spill_words = 4ull * (uint64_t)want + 4096;
  const uint64_t rl_entries = 2ull * (uint64_t)want + 64ull * kMaxRanges;
  if ((e = dev_alloc(&t->newlist, sizeof(NewKey) * ((size_t)slots + kGetTile))) != hipSuccess ||
      (e = dev_alloc(&t->tile_cnt, sizeof(uint32_t) * (size_t)get_tiles)) != hipSuccess ||
      (e = dev_alloc(&t->items, sizeof(uint64_t) * (size_t)slots)) != hipSuccess ||
      (e = dev_alloc(&t->meta, sizeof(uint32_t) * (size_t)kMaxParts * (size_t)put_tiles)) != hipSuccess ||
      (e = dev_alloc(&t->spill, sizeof(uint64_t) * (size_t)spill_words)) != hipSuccess ||
      // radix counts: 2^kRsMaxBits digit rows of (radix tiles rounded up to 4), then the item total
      (e = dev_alloc(&t->rs_cnt, sizeof(uint32_t) * (((size_t)(put_tiles + 3) / 4 + 4) * (1u << kRsMaxBits) + 64))) !=
          hipSuccess ||
      (e = dev_alloc(&t->partials, sizeof(double) * (size_t)want * (size_t)t->dim)) != hipSuccess ||
      (e = dev_alloc(&t->pc_key, sizeof(uint64_t) * (size_t)slots)) != hipSuccess ||
      (e = dev_alloc(&t->pc_row, sizeof(uint32_t) * (size_t)slots)) != hipSuccess ||
      (e = dev_alloc(&t->mid_xkey, sizeof(uint64_t) * (size_t)slots)) != hipSuccess ||
      (e = dev_alloc(&t->mid_xslot, sizeof(uint32_t) * (size_t)slots)) != hipSuccess ||
      // range lists: twice the keys in all, so that a range may hold twice its share
      (e = dev_alloc(&t->rl_list, sizeof(NewKey) * rl_entries)) != hipSuccess ||
      (e = dev_alloc(&t->rl_cnt, sizeof(uint32_t) * (2 * kMaxRanges + 1))) != hipSuccess ||
      (e = dev_alloc(&t->rl_cuts, sizeof(uint64_t) * kMaxRanges)) != hipSuccess ||
      (e = hipMemsetAsync(t->rl_cnt, 0, sizeof(uint32_t) * (2 * kMaxRanges + 1), st)) != hipSuccess ||
      (e = hipMemsetAsync(t->pc_key, 0xFF, sizeof(uint64_t) * (size_t)slots, st)) != hipSuccess) {  // no key cached
    free_workspace(t);
    return hip_fail(e, "scratch allocation");
  }
  if (t->cache_rows > 0 &&
      ((e = dev_alloc(&t->miss, sizeof(uint32_t) * (size_t)want)) != hipSuccess ||
       (e = dev_alloc(&t->plan_slot, sizeof(uint32_t) * (size_t)want)) != hipSuccess)) {
    free_workspace(t);
    return hip_fail(e, "lookahead scratch allocation");
  }
  t->ws_n = want;
  t->spill_words = spill_words;
  t->rl_entries = rl_entries;
  return MLKV_OK;
}

int check_table(mlkv_table* t) {
  if (t == nullptr) return fail(MLKV_EINVAL, "table is NULL");
  hipError_t e = hipSetDevice(t->device);
  if (e != hipSuccess) return hip_fail(e, "hipSetDevice");
  return MLKV_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

RowStore store_of(const mlkv_table* t) {
  RowStore s;
  s.rows = t->rows;
  s.host = t->host_rows;
  s.slot = t->slot_of_row;
  s.dirty = t->dirty;
  s.D = t->dim;
  return s;
}

hipEvent_t prof_event(mlkv_table* t) {
  if (!t->prof_pool.empty()) {
    hipEvent_t e = t->prof_pool.back();
    t->prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void prof_hook(void* ctx, int kernel, int phase, hipStream_t st) {
  mlkv_table* t = static_cast<mlkv_table*>(ctx);
  hipEvent_t e = prof_event(t);
  if (e == nullptr) return;
  (void)hipEventRecord(e, st);
  if (phase == 0) {
    t->prof_open[kernel] = e;
  } else if (t->prof_open[kernel] != nullptr) {
    t->prof_recs.push_back({kernel, t->prof_open[kernel], e});
    t->prof_open[kernel] = nullptr;
  } else {
    t->prof_pool.push_back(e);
  }
}

LaunchHook hook_of(mlkv_table* t) {
  LaunchHook h;
  if (t->prof_on) {
    h.fn = prof_hook;
    h.ctx = t;
  }
  return h;
}

void prof_release(mlkv_table* t) {
  for (auto& r : t->prof_recs) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  for (auto e : t->prof_pool) (void)hipEventDestroy(e);
  t->prof_recs.clear();
  t->prof_pool.clear();
}

}  // namespace

extern "C" {

const char* mlkv_last_error(void) { return g_err.c_str(); }

}  // extern "C"

namespace {

// Opens a table; cache_rows > 0 makes it tiered (rows at home in pinned host
// memory, cache_rows of them in an HBM cache).
mlkv_table* open_table(int32_t dim, int64_t capacity, uint64_t seed, float max_load, int64_t cache_rows) {
  if (dim < 1 || dim > 1024) {
    fail(MLKV_EINVAL, "dim must be in [1, 1024]");
    return nullptr;
  }
  if (capacity < 1 || capacity > 0xFFFFFFFEll) {
    fail(MLKV_EINVAL, "capacity must be in [1, 2^32 - 2]");
    return nullptr;
  }
  if (!(max_load > 0.0f) || !(max_load <= 0.9f)) {
    fail(MLKV_EINVAL, "max_load must be in (0, 0.9]");
    return nullptr;
  }
  // buckets: a power of two with 8 * nb * max_load >= capacity
  const double need = std::ceil((double)capacity / (8.0 * (double)max_load));
  uint32_t lg = 0;
  while ((double)(1ull << lg) < need) ++lg;
  if (lg > 28) {
    fail(MLKV_EINVAL, "hash index would exceed 2^31 slots; raise max_load or lower capacity");
    return nullptr;
  }
  mlkv_table* t = new mlkv_table();
  t->dim = dim;
  t->capacity = capacity;
  t->seed = seed;
  t->max_load = max_load;
  t->nb_log2 = lg;
  t->nb = 1ull << lg;
  hipError_t e = hipGetDevice(&t->device);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&t->cus, hipDeviceAttributeMultiprocessorCount, t->device);
  if (e != hipSuccess) {
    hip_fail(e, "hipGetDevice");
    delete t;
    return nullptr;
  }
  t->cus = std::max(1, t->cus);
  t->cache_rows = cache_rows;
  const int64_t hbm_rows = cache_rows > 0 ? cache_rows : capacity;
  if ((e = dev_alloc(&t->idx, sizeof(Bucket) * t->nb)) != hipSuccess ||
      (e = dev_alloc(&t->rows, sizeof(float) * (size_t)hbm_rows * (size_t)dim)) != hipSuccess ||
      (e = dev_alloc(&t->state, sizeof(float) * (size_t)capacity)) != hipSuccess ||
      (e = dev_alloc(&t->ctrl, sizeof(Ctrl))) != hipSuccess) {
    hip_fail(e, "table allocation");
    mlkv_close(t);
    return nullptr;
  }
  if (cache_rows > 0) {
    // the rows' home: pinned host memory the device reads and writes directly
    void* h = nullptr;
    e = hipHostMalloc(&h, sizeof(float) * (size_t)capacity * (size_t)dim, hipHostMallocMapped);
    if (e == hipSuccess) {
      t->host_alloc = h;
      void* d = nullptr;
      e = hipHostGetDevicePointer(&d, h, 0);
      t->host_rows = static_cast<float*>(d);
    }
    if (e == hipSuccess) e = dev_alloc(&t->slot_of_row, sizeof(uint32_t) * (size_t)capacity);
    if (e == hipSuccess) e = dev_alloc(&t->row_of_slot, sizeof(uint32_t) * (size_t)cache_rows);
    if (e == hipSuccess) e = dev_alloc(&t->dirty, (size_t)cache_rows);
    if (e == hipSuccess) e = dev_alloc(&t->keep, sizeof(uint32_t) * (size_t)cache_rows);
    if (e == hipSuccess) e = hipMemset(t->slot_of_row, 0xFF, sizeof(uint32_t) * (size_t)capacity);  // no row cached
    if (e == hipSuccess) e = hipMemset(t->row_of_slot, 0xFF, sizeof(uint32_t) * (size_t)cache_rows);
    if (e == hipSuccess) e = hipMemset(t->dirty, 0, (size_t)cache_rows);
    if (e == hipSuccess) e = hipMemset(t->keep, 0, sizeof(uint32_t) * (size_t)cache_rows);
    if (e != hipSuccess) {
      hip_fail(e, "tiered table allocation");
      mlkv_close(t);
      return nullptr;
    }
  }
  // empty index: all key tags EMPTY (all ones) and all row ids pending (all ones)
  Ctrl c;
  std::memset(&c, 0, sizeof(c));
  if ((e = hipMemset(t->idx, 0xFF, sizeof(Bucket) * t->nb)) != hipSuccess ||
      (e = hipMemcpy(t->ctrl, &c, sizeof(Ctrl), hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipDeviceSynchronize()) != hipSuccess) {
    hip_fail(e, "table initialisation");
    mlkv_close(t);
    return nullptr;
  }
  return t;
}

}  // namespace

extern "C" {

mlkv_table* mlkv_open_ex(int32_t dim, int64_t capacity, uint64_t seed, float max_load) {
  return open_table(dim, capacity, seed, max_load, 0);
}

mlkv_table* mlkv_open_tiered(int32_t dim, int64_t capacity, uint64_t seed, float max_load, int64_t cache_rows) {
  if (cache_rows < 1 || cache_rows > capacity) {
    fail(MLKV_EINVAL, "cache_rows must be in [1, capacity]");
    return nullptr;
  }
  return open_table(dim, capacity, seed, max_load, cache_rows);
}

mlkv_table* mlkv_open(int32_t dim, int64_t capacity) {
  return mlkv_open_ex(dim, capacity, MLKV_DEFAULT_SEED, 0.75f);
}

mlkv_table* mlkv_open_bounded(int32_t dim, int64_t capacity, uint64_t seed, float max_load,
                              int64_t staleness_bound) {
  if (staleness_bound < 0 || staleness_bound > (int64_t)kClockCount - 1) {
    fail(MLKV_EINVAL, "staleness_bound must be in [0, 2^24 - 2]");
    return nullptr;
  }
  mlkv_table* t = mlkv_open_ex(dim, capacity, seed, max_load);
  if (t == nullptr) return nullptr;
  hipError_t e = dev_alloc(&t->clock, sizeof(unsigned long long) * (size_t)capacity);
  if (e == hipSuccess) e = hipMemset(t->clock, 0, sizeof(unsigned long long) * (size_t)capacity);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    hip_fail(e, "staleness counts allocation");
    mlkv_close(t);
    return nullptr;
  }
  t->bound = staleness_bound;
  return t;
}

void mlkv_close(mlkv_table* t) {
  if (t == nullptr) return;
  (void)hipSetDevice(t->device);
  (void)hipDeviceSynchronize();
  (void)release_retired(t);
  free_workspace(t);
  prof_release(t);
  (void)hipFree(t->idx);
  (void)hipFree(t->rows);
  (void)hipFree(t->state);
  (void)hipFree(t->ctrl);
  (void)hipFree(t->clock);
  (void)hipFree(t->slot_of_row);
  (void)hipFree(t->row_of_slot);
  (void)hipFree(t->dirty);
  (void)hipFree(t->keep);
  if (t->host_alloc != nullptr) (void)hipHostFree(t->host_alloc);
  delete t;
}

}  // extern "C"

namespace {

// Per-call scratch of a get held outside the table (the allocation-free
// entry point): the new-key lists, the per-tile counts and the key-range
// overflow lists. Such a get leaves the table's record of found rows alone.
struct GetScratch {
  NewKey* newlist;
  uint32_t* tile_cnt;
  uint64_t* xkey;
  uint32_t* xslot;
};

// Host-side checks of a get call's arguments (nothing is queued).
int check_get(mlkv_table* t, const uint64_t* d_keys, int64_t n, uint8_t* d_blocked, bool count) {
  if (n < 0 || n > 0x7FFFFFFFll) return fail(MLKV_EINVAL, "n must be in [0, 2^31 - 1]");
  if (n == 0) return MLKV_OK;
  if (d_keys == nullptr) return fail(MLKV_EINVAL, "keys is NULL");
  const bool track = count && t->clock != nullptr;
  if (track && d_blocked == nullptr) return fail(MLKV_EINVAL, "blocked is NULL");
  if (track && t->cepoch >= (1ull << (64 - kClockBits)))
    return fail(MLKV_EINVAL, "the table has served 2^40 get calls, the most a bounded table counts");
  return MLKV_OK;
}

// The launch arguments of a get of n > 0 keys with the table's epoch; the
// row records and key-range lists are the table's (the put's items and
// metadata, idle during a get), or `fixed`'s.
GetArgs get_args(mlkv_table* t, const uint64_t* d_keys, int64_t n, float* d_out, uint8_t* d_blocked, bool count,
                 const GetScratch* fixed) {
  const bool track = count && t->clock != nullptr;
  GetArgs a;
  a.idx = t->idx;
  a.nb_log2 = t->nb_log2;
  a.keys = d_keys;
  a.n = n;
  a.out = d_out;
  a.store = store_of(t);
  a.state = t->state;
  a.D = t->dim;
  a.seed = t->seed;
  a.capacity = t->capacity;
  a.newlist = fixed ? fixed->newlist : t->newlist;
  a.tile_cnt = fixed ? fixed->tile_cnt : t->tile_cnt;
  a.ctrl = t->ctrl;
  a.epoch = t->epoch;
  a.xkey = fixed ? fixed->xkey : t->items;
  a.xslot = fixed ? fixed->xslot : t->meta;
  a.clock = track ? t->clock : nullptr;
  a.cepoch = t->cepoch;
  a.bound = (uint32_t)std::max<int64_t>(t->bound, 0);
  a.blocked = d_blocked;
  a.pc_key = fixed ? nullptr : t->pc_key;
  a.pc_row = fixed ? nullptr : t->pc_row;
  // after a lookahead, the positions of its keys skip the probe (tables
  // without a staleness bound)
  a.pc_in = (!fixed && t->pc_lookahead && a.clock == nullptr) ? 1 : 0;
  if (!fixed) {
    const uint32_t par = (uint32_t)(t->rl_calls & 1u);
    a.rl.list = t->rl_list;
    a.rl.entries = t->rl_entries;
    a.rl.cnt = t->rl_cnt + par * kMaxRanges;
    a.rl.cnt_next = t->rl_cnt + (par ^ 1u) * kMaxRanges;
    a.rl.cuts = t->rl_cuts;
    a.rl.cuts_g = t->rl_cnt + 2 * kMaxRanges;
  }
  a.cus = t->cus;
  return a;
}

bool get_vec4(const mlkv_table* t, const float* d_out) {
  return (t->dim % 4 == 0) && (d_out == nullptr || aligned16(d_out));
}

// The table's state after a get call was queued.
void get_done(mlkv_table* t, bool count, bool fixed) {
  if (!fixed) {
    t->pc_lookahead = !count;  // a lookahead is the one get call that counts nothing
    t->rl_calls++;             // the range counts it used are cleared for the call after next
  }
  t->epoch++;
  if (count && t->clock != nullptr) t->cepoch++;
}

// The get pipeline (probe + gather, then rows for new keys); d_blocked is
// written when the table has a staleness bound and the call counts (a
// lookahead does not). With `fixed`, the call uses that scratch, allocates
// nothing and records no launch timings.
int get_call(mlkv_table* t, const uint64_t* d_keys, int64_t n, float* d_out, uint8_t* d_blocked,
             bool count, void* hip_stream, const GetScratch* fixed = nullptr) {
  int rc = check_table(t);
  if (rc) return rc;
  if ((rc = check_get(t, d_keys, n, d_blocked, count)) != MLKV_OK || n == 0) return rc;
  if (fixed == nullptr && (rc = ensure_workspace(t, n, static_cast<hipStream_t>(hip_stream))) != MLKV_OK)
    return rc;
  const GetArgs a = get_args(t, d_keys, n, d_out, d_blocked, count, fixed);
  hipError_t e = launch_get(a, get_vec4(t, d_out), static_cast<hipStream_t>(hip_stream),
                            fixed ? LaunchHook{} : hook_of(t));
  if (e != hipSuccess) return hip_fail(e, "mlkv_get launch");
  get_done(t, count, fixed != nullptr);
  return MLKV_OK;
}

// ---- scratch of the allocation-free get ----
// A file-scope device array, one copy per GPU, sized for kNoAllocMaxKeys keys:
// new-key lists (16 B per key), per-tile counts, key-range lists (12 B per key).
constexpr int64_t kNoAllocMaxKeys = MLKV_NOALLOC_MAX_KEYS;
constexpr size_t kNaNewlist = 0;
// a tile's list starts at its first position; the last tile may reach past n
constexpr size_t kNaTileCnt = kNaNewlist + sizeof(NewKey) * ((size_t)kNoAllocMaxKeys + kGetTile);
constexpr size_t kNaXkey = kNaTileCnt + 4096;
constexpr size_t kNaXslot = kNaXkey + sizeof(uint64_t) * (size_t)kNoAllocMaxKeys;
constexpr size_t kNaBytes = kNaXslot + sizeof(uint32_t) * (size_t)kNoAllocMaxKeys;
static_assert(kNaTileCnt + sizeof(uint32_t) * ((kNoAllocMaxKeys + kGetTileMin - 1) / kGetTileMin) <= kNaXkey,
              "tile counts fit their region");

__device__ __align__(256) unsigned char scratch[kNaBytes];

// Device address of `scratch` on each device (the name itself is only a
// host-side stand-in), taken once per device with that device current.
std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
void* g_scratch_addr[kMaxDevices] = {};

int noalloc_scratch(int device, GetScratch* out) {
  if (device < 0 || device >= kMaxDevices) return fail(MLKV_EDEVICE, "device ordinal out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[device] == nullptr) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr) return fail(MLKV_EDEVICE, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_addr[device] = p;
  }
  unsigned char* base = static_cast<unsigned char*>(g_scratch_addr[device]);
  out->newlist = reinterpret_cast<NewKey*>(base + kNaNewlist);
  out->tile_cnt = reinterpret_cast<uint32_t*>(base + kNaTileCnt);
  out->xkey = reinterpret_cast<uint64_t*>(base + kNaXkey);
  out->xslot = reinterpret_cast<uint32_t*>(base + kNaXslot);
  return MLKV_OK;
}

}  // namespace

extern "C" {

int mlkv_get(mlkv_table* t, const uint64_t* d_keys, int64_t n, float* d_out, void* hip_stream) {
  if (t != nullptr && t->clock != nullptr)
    return fail(MLKV_EINVAL, "the table has a staleness bound: use mlkv_get_bounded");
  return get_call(t, d_keys, n, d_out, nullptr, true, hip_stream);
}

int mlkv_get_noalloc(mlkv_table* t, const uint64_t* d_keys, int64_t n, float* d_out, void* hip_stream) {
  int rc = check_table(t);  // makes the table's device current
  if (rc) return rc;
  if (t->clock != nullptr) return fail(MLKV_EINVAL, "the table has a staleness bound: use mlkv_get_bounded");
  if (n < 0 || n > kNoAllocMaxKeys)
    return fail(MLKV_EINVAL, "mlkv_get_noalloc takes at most MLKV_NOALLOC_MAX_KEYS (65536) keys");
  GetScratch s;
  if ((rc = noalloc_scratch(t->device, &s)) != MLKV_OK) return rc;
  return get_call(t, d_keys, n, d_out, nullptr, true, hip_stream, &s);
}

int mlkv_lookahead(mlkv_table* t, const uint64_t* d_keys, int64_t n, void* hip_stream) {
  int rc = get_call(t, d_keys, n, nullptr, nullptr, false, hip_stream);
  if (rc != MLKV_OK || t->cache_rows == 0 || n == 0) return rc;
  // tiered: the keys are resolved; now their rows come into the HBM cache
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  if (++t->tier_tag == 0) ++t->tier_tag;  // 0 is the tag of no call
  TierArgs a;
  a.idx = t->idx;
  a.nb_log2 = t->nb_log2;
  a.keys = d_keys;
  a.pc_key = t->pc_key;  // written by the get kernels of this lookahead
  a.pc_row = t->pc_row;
  a.n = n;
  a.slot_of_row = t->slot_of_row;
  a.row_of_slot = t->row_of_slot;
  a.dirty = t->dirty;
  a.keep = t->keep;
  a.tag = t->tier_tag;
  a.parity = (uint32_t)(t->tier_calls++ & 1u);  // alternates on every call, also when the tag wraps
  a.miss = t->miss;
  a.plan_slot = t->plan_slot;
  a.cache_rows = t->cache_rows;
  a.cache = t->rows;
  a.host = t->host_rows;
  a.D = t->dim;
  a.ctrl = t->ctrl;
  hipError_t e = launch_tier_lookahead(a, st, hook_of(t));
  if (e != hipSuccess) return hip_fail(e, "lookahead copy launch");
  return MLKV_OK;
}

int mlkv_cache_stats(mlkv_table* t, int64_t* out) {
  int rc = check_table(t);
  if (rc) return rc;
  if (out == nullptr) return fail(MLKV_EINVAL, "out is NULL");
  if (t->cache_rows == 0) return fail(MLKV_EINVAL, "the table is not tiered");
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  Ctrl c;
  e = hipMemcpy(&c, t->ctrl, sizeof(Ctrl), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "read cache counters");
  out[0] = (int64_t)c.tier_loaded;
  out[1] = (int64_t)c.tier_evicted;
  out[2] = (int64_t)c.tier_written;
  out[3] = (int64_t)c.tier_filled;
  out[4] = t->cache_rows;
  return MLKV_OK;
}

int mlkv_get_bounded(mlkv_table* t, const uint64_t* d_keys, int64_t n, float* d_out, uint8_t* d_blocked,
                     void* hip_stream) {
  if (t != nullptr && t->clock == nullptr)
    return fail(MLKV_EINVAL, "the table has no staleness bound: use mlkv_get");
  return get_call(t, d_keys, n, d_out, d_blocked, true, hip_stream);
}

int mlkv_read_staleness(mlkv_table* t, const int64_t* d_rows, int64_t n, uint32_t* d_out, void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  if (t->clock == nullptr) return fail(MLKV_EINVAL, "the table has no staleness bound");
  if (n < 0 || n > 0x7FFFFFFFll) return fail(MLKV_EINVAL, "n must be in [0, 2^31 - 1]");
  if (n == 0) return MLKV_OK;
  if (d_rows == nullptr || d_out == nullptr) return fail(MLKV_EINVAL, "rows or out is NULL");
  hipError_t e = launch_read_clock(t->clock, &t->ctrl->size[t->epoch & 1], d_rows, n, d_out, t->ctrl,
                                   static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "mlkv_read_staleness launch");
  return MLKV_OK;
}

}  // extern "C"

namespace {

// Host-side checks of a put call's arguments (nothing is queued).
int check_put(mlkv_table* t, const uint64_t* d_keys, const float* src, int64_t n, int op, float lr, float eps) {
  if (n < 0 || n > 0x3FFFFFFFll) return fail(MLKV_EINVAL, "n must be in [0, 2^30 - 1]");
  if (op != kOpAssign && !std::isfinite(lr)) return fail(MLKV_EINVAL, "lr must be finite");
  if (op == kOpAdagrad && (!std::isfinite(eps) || eps < 0.0f))
    return fail(MLKV_EINVAL, "eps must be finite and >= 0");
  if (n == 0) return MLKV_OK;
  if (d_keys == nullptr || src == nullptr) return fail(MLKV_EINVAL, "keys or rows is NULL");
  if (t->dedup == kDedupRadix && n > kRsMaxKeys) return fail(MLKV_EINVAL, "radix dedup takes at most 2^20 keys");
  return MLKV_OK;
}

// The launch arguments of a put of n > 0 keys with the table's epoch.
PutArgs put_args(mlkv_table* t, const uint64_t* d_keys, const float* src, int64_t n, int op, float lr, float eps) {
  const uint32_t pb = call_part_bits(n, t->cus);
  // keys per put_probe tile: a multiple of 64, at most kPutTile, so that the
  // tiles cover every CU when the batch is small
  const int64_t per_cu = (n + t->cus - 1) / t->cus;
  const int tlen = (int)std::min<int64_t>(kPutTile, std::max<int64_t>(64, (per_cu + 63) / 64 * 64));
  PutArgs a;
  a.idx = t->idx;
  a.nb_log2 = t->nb_log2;
  a.keys = d_keys;
  a.grads = src;
  a.n = n;
  a.store = store_of(t);
  a.state = t->state;
  a.D = t->dim;
  a.seed = t->seed;
  a.capacity = t->capacity;
  a.lr = lr;
  a.eps = eps;
  a.op = op;
  a.pb = (int)pb;
  a.tlen = tlen;
  a.items = t->items;
  a.partials = t->partials;
  a.meta = t->meta;
  a.newlist = t->newlist;
  a.tile_cnt = t->tile_cnt;
  a.spill = t->spill;
  a.spill_words = t->spill_words;
  a.ctrl = t->ctrl;
  a.epoch = t->epoch;
  a.clock = t->clock;
  a.pc_key = t->pc_key;
  a.pc_row = t->pc_row;
  a.dedup = t->dedup;
  a.cus = t->cus;
  a.rs_bits = t->rs_bits;
  a.rs_buf = t->spill;  // two n-item buffers (the spill area holds 4n words; radix puts never spill)
  a.rs_cnt = t->rs_cnt;
  return a;
}

// The put pipeline (probe, group, apply) with update `op` for every distinct
// key; `src` holds n rows of gradients (or values for kOpAssign).
int put_call(mlkv_table* t, const uint64_t* d_keys, const float* src, int64_t n, int op, float lr, float eps,
             void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  if ((rc = check_put(t, d_keys, src, n, op, lr, eps)) != MLKV_OK || n == 0) return rc;
  if ((rc = ensure_workspace(t, n, static_cast<hipStream_t>(hip_stream))) != MLKV_OK) return rc;
  const PutArgs a = put_args(t, d_keys, src, n, op, lr, eps);
  const bool vec4 = (t->dim % 4 == 0) && aligned16(src);
  hipError_t e = launch_put(a, vec4, static_cast<hipStream_t>(hip_stream), hook_of(t));
  if (e != hipSuccess) return hip_fail(e, "put launch");
  t->epoch++;
  return MLKV_OK;
}

}  // namespace

extern "C" {

int mlkv_put_grad(mlkv_table* t, const uint64_t* d_keys, const float* d_grads, int64_t n, float lr,
                  float eps, void* hip_stream) {
  return put_call(t, d_keys, d_grads, n, kOpAdagrad, lr, eps, hip_stream);
}

int mlkv_put_grad_sgd(mlkv_table* t, const uint64_t* d_keys, const float* d_grads, int64_t n, float lr,
                      void* hip_stream) {
  return put_call(t, d_keys, d_grads, n, kOpSgd, lr, 0.0f, hip_stream);
}

int mlkv_get_put_grad(mlkv_table* t, const uint64_t* d_get_keys, int64_t n_get, float* d_out, uint8_t* d_blocked,
                      const uint64_t* d_put_keys, const float* d_grads, int64_t n_put, float lr, float eps,
                      void* get_done_event, void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  if ((rc = check_get(t, d_get_keys, n_get, d_blocked, true)) != MLKV_OK) return rc;
  if ((rc = check_put(t, d_put_keys, d_grads, n_put, kOpAdagrad, lr, eps)) != MLKV_OK) return rc;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  hipEvent_t done = static_cast<hipEvent_t>(get_done_event);
  hipError_t e = hipSuccess;
  if (n_put == 0) {
    if ((rc = get_call(t, d_get_keys, n_get, d_out, d_blocked, true, hip_stream)) != MLKV_OK) return rc;
    if (done != nullptr && (e = hipEventRecord(done, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    return MLKV_OK;
  }
  if (n_get == 0) {
    if (done != nullptr && (e = hipEventRecord(done, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    return put_call(t, d_put_keys, d_grads, n_put, kOpAdagrad, lr, eps, hip_stream);
  }
  if ((rc = ensure_workspace(t, std::max(n_get, n_put), st)) != MLKV_OK) return rc;
  // the get takes this epoch, the put the next; the put's probe kernel runs
  // first (it reads the rows the last get recorded), then the get's kernels,
  // then the put's row updates
  PutArgs p = put_args(t, d_put_keys, d_grads, n_put, kOpAdagrad, lr, eps);
  p.epoch = t->epoch + 1;
  p.ahead = 1;
  GetArgs g = get_args(t, d_get_keys, n_get, d_out, d_blocked, true, nullptr);
  g.xkey = t->mid_xkey;
  g.xslot = t->mid_xslot;
  const bool pvec4 = (t->dim % 4 == 0) && aligned16(d_grads);
  const LaunchHook hook = hook_of(t);
  e = launch_put(p, pvec4, st, hook, kPutProbe);
  if (e == hipSuccess) e = launch_get(g, get_vec4(t, d_out), st, hook);
  if (e == hipSuccess && done != nullptr) e = hipEventRecord(done, st);
  if (e == hipSuccess) e = launch_put(p, pvec4, st, hook, kPutAfterProbe);
  if (e != hipSuccess) return hip_fail(e, "mlkv_get_put_grad launch");
  get_done(t, true, false);
  t->epoch++;  // the put
  return MLKV_OK;
}

int mlkv_set_dedup(mlkv_table* t, int mode) {
  int rc = check_table(t);
  if (rc) return rc;
  if (mode != kDedupHash && mode != kDedupRadix) return fail(MLKV_EINVAL, "unknown dedup mode");
  if (mode == kDedupRadix) {
    // sort keys: rows below capacity, a new key's index slot above it
    const uint64_t top = (uint64_t)t->capacity + ((uint64_t)kSlots << t->nb_log2);
    if (top > 0xFFFFFFFFull) return fail(MLKV_EINVAL, "radix dedup needs capacity + index slots < 2^32");
    int b = 0;
    while ((1ull << b) < top) ++b;
    t->rs_bits = b;
  }
  t->dedup = mode;
  return MLKV_OK;
}

int mlkv_put(mlkv_table* t, const uint64_t* d_keys, const float* d_values, int64_t n, void* hip_stream) {
  return put_call(t, d_keys, d_values, n, kOpAssign, 0.0f, 0.0f, hip_stream);
}

int mlkv_sync(mlkv_table* t, void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  if ((rc = release_retired(t)) != MLKV_OK) return rc;
  int latched = 0;
  e = hipMemcpy(&latched, &t->ctrl->latched, sizeof(int), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "read error latch");
  if (latched != 0) {
    const int zero = 0;
    e = hipMemcpy(&t->ctrl->latched, &zero, sizeof(int), hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail(e, "clear error latch");
    if (latched == kErrAbsent)
      return fail(MLKV_EINVAL, "the put of mlkv_get_put_grad held a key absent from the table before the call");
    return fail(latched, latched == MLKV_EFULL ? "a call exceeded the table capacity"
                                               : "a call contained the reserved key");
  }
  return MLKV_OK;
}

int64_t mlkv_size(mlkv_table* t) {
  if (check_table(t)) return -1;
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    hip_fail(e, "hipDeviceSynchronize");
    return -1;
  }
  unsigned long long s = 0;
  e = hipMemcpy(&s, &t->ctrl->size[t->epoch & 1], sizeof(s), hipMemcpyDeviceToHost);
  if (e != hipSuccess) {
    hip_fail(e, "read size");
    return -1;
  }
  return (int64_t)s;
}

int64_t mlkv_num_slots(mlkv_table* t) {
  if (t == nullptr) return -1;
  return (int64_t)(t->nb * kSlots);
}

int mlkv_reserve(mlkv_table* t, int64_t n) {
  int rc = check_table(t);
  if (rc) return rc;
  if (n < 0 || n > 0x7FFFFFFFll) return fail(MLKV_EINVAL, "n must be in [0, 2^31 - 1]");
  if ((rc = ensure_workspace(t, n, nullptr)) != MLKV_OK) return rc;
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
  return release_retired(t);
}

int mlkv_lookup_rows(mlkv_table* t, const uint64_t* d_keys, int64_t n, int64_t* d_rows_out,
                     void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  if (n < 0 || n > 0x7FFFFFFFll) return fail(MLKV_EINVAL, "n must be in [0, 2^31 - 1]");
  if (n == 0) return MLKV_OK;
  if (d_keys == nullptr || d_rows_out == nullptr) return fail(MLKV_EINVAL, "NULL pointer");
  hipError_t e = launch_lookup(t->idx, t->nb_log2, d_keys, n, d_rows_out,
                               static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "mlkv_lookup_rows launch");
  return MLKV_OK;
}

int mlkv_export(mlkv_table* t, int64_t nrows, float* d_rows_out, float* d_state_out,
                uint64_t* d_slot_keys_out, uint32_t* d_slot_rows_out, void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  const int64_t size = mlkv_size(t);
  if (size < 0) return MLKV_EDEVICE;
  if (nrows < 0 || nrows > size) return fail(MLKV_EINVAL, "nrows must be in [0, size]");
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  hipError_t e = hipSuccess;
  if (d_rows_out && nrows > 0) e = launch_export_rows(store_of(t), nrows, t->dim, d_rows_out, st);
  if (e == hipSuccess && d_state_out && nrows > 0)
    e = hipMemcpyAsync(d_state_out, t->state, sizeof(float) * (size_t)nrows, hipMemcpyDeviceToDevice, st);
  if (e == hipSuccess && (d_slot_keys_out || d_slot_rows_out))
    e = launch_export_slots(t->idx, t->nb * kSlots, d_slot_keys_out, d_slot_rows_out, st);
  if (e != hipSuccess) return hip_fail(e, "mlkv_export");
  return MLKV_OK;
}

int mlkv_read_rows(mlkv_table* t, const int64_t* d_rows, int64_t n, float* d_rows_out, float* d_state_out,
                   void* hip_stream) {
  int rc = check_table(t);
  if (rc) return rc;
  if (n < 0 || n > 0x7FFFFFFFll) return fail(MLKV_EINVAL, "n must be in [0, 2^31 - 1]");
  if (n == 0) return MLKV_OK;
  if (d_rows == nullptr) return fail(MLKV_EINVAL, "rows is NULL");
  hipError_t e = launch_read_rows(store_of(t), t->state, t->dim, &t->ctrl->size[t->epoch & 1], d_rows, n,
                                  d_rows_out, d_state_out, t->ctrl, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "mlkv_read_rows launch");
  return MLKV_OK;
}

int mlkv_profile_enable(mlkv_table* t, int enable) {
  if (t == nullptr) return fail(MLKV_EINVAL, "table is NULL");
  t->prof_on = enable != 0;
  return MLKV_OK;
}

int mlkv_profile_read(mlkv_table* t, double* total_ms, int64_t* launches) {
  int rc = check_table(t);
  if (rc) return rc;
  if (total_ms == nullptr || launches == nullptr) return fail(MLKV_EINVAL, "NULL output");
  for (int k = 0; k < K_COUNT; ++k) {
    total_ms[k] = 0.0;
    launches[k] = 0;
  }
  for (auto& r : t->prof_recs) {
    hipError_t e = hipEventSynchronize(r.stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.0f;
    e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    total_ms[r.kernel] += ms;
    launches[r.kernel] += 1;
    t->prof_pool.push_back(r.start);
    t->prof_pool.push_back(r.stop);
  }
  t->prof_recs.clear();
  return MLKV_OK;
}

const char* mlkv_kernel_name(int kernel) {
  static const char* names[K_COUNT] = {"get_probe_gather", "assign_new", "put_probe", "put_reduce",
                                       "tier_mark", "tier_plan", "tier_copy", "rsort_count",
                                       "rsort_scatter", "rsort_reduce"};
  return (kernel >= 0 && kernel < K_COUNT) ? names[kernel] : nullptr;
}

}  // extern "C"
