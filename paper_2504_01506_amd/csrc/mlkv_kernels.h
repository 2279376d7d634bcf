// Launch interface between the host table manager and the HIP kernels.
#pragma once

#include <algorithm>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mlkv_device.h"

namespace mlkv {

constexpr int kGetTile = 256;    // keys per probe_gather block at most (one per lane)
constexpr int kGetTileMin = 64;  // ... and at least, unless the batch is smaller

// Positions per get_probe_gather block for a batch of n keys on a device of
// `cus` compute units: the blocks come in whole rounds of one per CU, with
// equal tiles, so that no CU runs a block more than another.
inline int get_tile_len(int64_t n, int cus) {
  const int64_t per_round = (int64_t)kGetTile * cus;
  const int64_t rounds = (n + per_round - 1) / per_round;
  int64_t t = (n + rounds * cus - 1) / (rounds * cus);
  if (t < kGetTileMin) t = kGetTileMin;
  if (t > kGetTile) t = kGetTile;
  return (int)t;
}
constexpr int kPutTile = 1024;   // keys per put_probe block
constexpr int kPutThreads = 1024; // threads of a put_probe block
constexpr int kMaxParts = 4096;  // partitions (MSD digits) per put call
constexpr int kRedCap = 3072;    // partition items grouped in LDS by a put_reduce block
constexpr int kRedHash = 4096;   // LDS hash slots for that grouping (load <= 0.75)
constexpr int kPartTarget = 1024; // put keys per partition the partition count aims for
constexpr int kPresumMin = 2;    // a key repeated this often in a put_probe tile is summed there

// Error code a kernel latches when a put whose probe ran ahead of a get met a
// key that was not in the table before the two calls (reported as MLKV_EINVAL).
constexpr int kErrAbsent = -5;

// Kernels of the library, for per-launch timing.
enum KernelId : int {
  K_GET_PROBE_GATHER = 0,
  K_ASSIGN_NEW = 1,
  K_PUT_PROBE = 2,
  K_PUT_REDUCE = 3,
  K_TIER_MARK = 4,
  K_TIER_PLAN = 5,
  K_TIER_COPY = 6,
  K_RSORT_COUNT = 7,
  K_RSORT_SCATTER = 8,
  K_RSORT_REDUCE = 9,
  K_COUNT = 10
};

// How a put finds the equal keys of its batch.
enum Dedup : int {
  kDedupHash = 0,   // hash partition of the items, grouping in LDS per partition
  kDedupRadix = 1   // stable LSD radix sort of the items by row, run-length encoding
};
constexpr int kRsTile = 4096;    // items per radix-sort block (four put tiles)
constexpr int kRsMaxBits = 9;    // bits per radix pass at most
constexpr int kRsChunk = 2048;   // sorted items per radix reduce block at most, before the cut moves to a run start
constexpr int64_t kRsMaxKeys = 1 << 20;  // keys per put call with radix dedup

// Update a put call applies to each distinct key's row.
enum PutOp : int {
  kOpAdagrad = 0,  // sum the key's gradient rows, one row-wise Adagrad step
  kOpSgd = 1,      // sum the key's gradient rows, one SGD step
  kOpAssign = 2    // the value row at the key's last position replaces the row
};


// Optional callback around each launch (phase 0 before, 1 after), on the launch stream.
struct LaunchHook {
  void (*fn)(void* ctx, int kernel, int phase, hipStream_t st) = nullptr;
  void* ctx = nullptr;
  void operator()(int kernel, int phase, hipStream_t st) const {
    if (fn) fn(ctx, kernel, phase, st);
  }
};

// A get call's new keys filed by key range as the probe kernel inserts them,
// with the cut points the last ranking by key ranges left (the keys of
// global ranks floor(j M / G), j = 1 .. G - 1, of a call that inserted M keys
// with G ranges): range q holds the keys in [cut q-1, cut q). Row assignment
// then takes each range's keys from its list instead of searching every
// tile's list. The cut points serve a call with the same G; any sorted set of
// them is correct, the last call's keep the ranges about even.
constexpr int kMaxRanges = 512;  // ranges of a get call at most (its row-assignment blocks, two per CU)
struct RangeLists {
  NewKey* list = nullptr;      // [entries]: range q's keys from q * cap on; nullptr: no lists
  uint64_t entries = 0;
  uint32_t cap = 0;            // entries per range (set at launch: entries / ranges)
  uint32_t* cnt = nullptr;     // [kMaxRanges] this call's counts per range (zero before it)
  uint32_t* cnt_next = nullptr;  // [kMaxRanges] the next call's counts, cleared by this call
  uint64_t* cuts = nullptr;    // [kMaxRanges - 1] the cut points
  uint32_t* cuts_g = nullptr;  // the number of ranges the cut points are for (0: none)
};

struct GetArgs {
  Bucket* idx;
  uint32_t nb_log2;
  const uint64_t* keys;
  int64_t n;
  float* out;
  RowStore store;
  float* state;
  int D;
  uint64_t seed;
  int64_t capacity;
  NewKey* newlist;
  uint32_t* tile_cnt;
  Ctrl* ctrl;
  uint64_t epoch;
  uint64_t* xkey;   // [n] scratch: new keys of a key range too large for LDS
  uint32_t* xslot;  // [n] their index slots
  // staleness bound (nullptr clock: not tracked): per-row words of
  // (get-call epoch << kClockBits) | count, this call's epoch, the bound, and
  // the per-position blocked flags the call writes
  unsigned long long* clock;
  uint64_t cepoch;
  uint32_t bound;
  uint8_t* blocked;
  // per position: the key found present and its row (the key is the empty
  // key where the position held no present key); a later put reads them.
  // nullptr: not recorded
  uint64_t* pc_key;
  uint32_t* pc_row;
  // 1: a position whose key equals pc_key[i] takes pc_row[i] without probing
  // (a present key's row never changes, so any recorded pair stays true);
  // not with a staleness clock
  int pc_in;
  RangeLists rl;
  int cus;  // compute units of the device
};

struct PutArgs {
  Bucket* idx;
  uint32_t nb_log2;
  const uint64_t* keys;
  const float* grads;
  int64_t n;
  RowStore store;
  float* state;
  int D;
  uint64_t seed;
  int64_t capacity;
  float lr;
  float eps;
  int op;     // PutOp
  int pb;     // 2^pb partitions
  int tlen;   // keys per put_probe tile (<= kPutTile)
  uint64_t* items;
  double* partials;  // [n][D] fp64 sums of keys repeated within a tile
  uint32_t* meta;
  NewKey* newlist;
  uint32_t* tile_cnt;
  uint64_t* spill;
  uint64_t spill_words;
  Ctrl* ctrl;
  uint64_t epoch;
  unsigned long long* clock;  // per-row staleness words, or nullptr when not tracked
  const uint64_t* pc_key;     // the last get's present keys and rows by position
  const uint32_t* pc_row;
  int dedup;                  // Dedup
  int cus;                    // compute units (radix reduce blocks at least)
  int rs_bits;                // radix dedup: bits of the sort key (rows below capacity, new keys' slots above)
  uint64_t* rs_buf;           // radix dedup: two n-item ping-pong buffers
  uint32_t* rs_cnt;           // radix dedup: per-tile digit counts, then the item total
  // 1: the put's probe kernel runs ahead of the kernels of a get whose epoch
  // is this one's less one, its other kernels after them (the probe inserts
  // nothing: a key absent from the table before that get fails the put; it
  // writes no new-key list or tile counts, which are the get's, and marks its
  // errors in the control block's fields for such puts)
  int ahead = 0;
};

// Which kernels of a put launch_put queues: all of them, only the probe
// kernel, or the kernels after it.
enum PutPhase : int { kPutAll = 0, kPutProbe = 1, kPutAfterProbe = 2 };

// Lookahead of a tiered table, after the get kernels have resolved its n keys.
struct TierArgs {
  Bucket* idx;
  uint32_t nb_log2;
  const uint64_t* keys;
  const uint64_t* pc_key;  // the get's present keys and rows by position
  const uint32_t* pc_row;
  int64_t n;
  uint32_t* slot_of_row;  // [capacity]
  uint32_t* row_of_slot;  // [cache_rows]
  uint8_t* dirty;         // [cache_rows]
  uint32_t* keep;         // [cache_rows]
  uint32_t tag;           // this lookahead call (never 0)
  uint32_t parity;        // ping-pong index of the miss counter
  uint32_t* miss;         // [n] scratch
  uint32_t* plan_slot;    // [n] scratch
  int64_t cache_rows;
  float* cache;
  float* host;
  int D;
  Ctrl* ctrl;
};

hipError_t launch_get(const GetArgs& a, bool vec4, hipStream_t st, const LaunchHook& hook);
hipError_t launch_tier_lookahead(const TierArgs& a, hipStream_t st, const LaunchHook& hook);
hipError_t launch_put(const PutArgs& a, bool vec4, hipStream_t st, const LaunchHook& hook, int phase = kPutAll);
hipError_t launch_lookup(Bucket* idx, uint32_t nb_log2, const uint64_t* keys, int64_t n,
                         int64_t* rows_out, hipStream_t st);
hipError_t launch_export_slots(const Bucket* idx, uint64_t nslots, uint64_t* keys_out,
                               uint32_t* rows_out, hipStream_t st);
hipError_t launch_read_clock(const unsigned long long* clock, const unsigned long long* size_now,
                             const int64_t* ids, int64_t n, uint32_t* out, Ctrl* ctrl, hipStream_t st);
hipError_t launch_read_rows(const RowStore& store, const float* state, int D, const unsigned long long* size_now,
                            const int64_t* ids, int64_t n, float* w_out, float* st_out, Ctrl* ctrl,
                            hipStream_t st);
hipError_t launch_export_rows(const RowStore& store, int64_t nrows, int D, float* out, hipStream_t st);

}  // namespace mlkv
