// Device-side building blocks shared by the kernels of libmlkv (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mlkv {

constexpr uint64_t kEmptyKey = ~0ull;
constexpr uint32_t kPendingRow = 0xFFFFFFFFu;
constexpr int kSlots = 8;          // slots per bucket
constexpr int kMaxProbe = 4096;    // buckets visited before a call reports overflow

// One bucket = one 128-byte line: 8 key tags, the 8 row ids, 8 spare words.
struct __align__(128) Bucket {
  uint64_t key[kSlots];
  uint32_t row[kSlots];
  uint32_t aux[kSlots];
};
static_assert(sizeof(Bucket) == 128, "bucket must be one 128-byte line");

// Staleness word of a row (bounded staleness, Sec. III-C1): the low
// kClockBits bits count the gets served on the row that no put has completed
// yet, the high bits hold the epoch of the last get call that counted it (so
// that a key occurring several times in one call is counted once).
constexpr int kClockBits = 24;
constexpr unsigned long long kClockCount = (1ull << kClockBits) - 1;

// Where the values of row r live. An ordinary table keeps every row in one HBM
// array. A tiered table keeps every row in pinned host memory (its home) and
// a fixed number of rows in an HBM cache: slot[r] is r's cache slot, or
// kNoSlot when r is only at home. Writing a cached row marks its slot dirty
// (written back to the home when the slot is reused).
constexpr uint32_t kNoSlot = 0xFFFFFFFFu;
struct RowStore {
  float* rows;           // HBM: all rows [capacity][D], or the cache [cache rows][D]
  float* host;           // tiered: pinned host rows [capacity][D]; else nullptr
  const uint32_t* slot;  // tiered: [capacity] cache slot of each row; else nullptr
  uint8_t* dirty;        // tiered: [cache rows] slot written since it was loaded
  int D;
  __device__ __forceinline__ const float* ptr(uint32_t r) const { return row_read(rows, host, slot, D, r); }
  // the row about to be written (marks a cached row's slot dirty)
  __device__ __forceinline__ float* wptr(uint32_t r) const { return row_write(rows, host, slot, dirty, D, r); }

 private:
  static __device__ __forceinline__ const float* row_read(float* rows, float* host, const uint32_t* slot, int D,
                                                         uint32_t r) {
    if (slot == nullptr) return rows + (size_t)r * (size_t)D;
    const uint32_t s = slot[r];
    return s != kNoSlot ? rows + (size_t)s * (size_t)D : host + (size_t)r * (size_t)D;
  }
  static __device__ __forceinline__ float* row_write(float* rows, float* host, const uint32_t* slot, uint8_t* dirty,
                                                     int D, uint32_t r) {
    if (slot == nullptr) return rows + (size_t)r * (size_t)D;
    const uint32_t s = slot[r];
    if (s == kNoSlot) return host + (size_t)r * (size_t)D;
    dirty[s] = 1;
    return rows + (size_t)s * (size_t)D;
  }
};

// A key first inserted by the current call, owned by the lane that won its slot.
struct NewKey {
  uint64_t key;
  uint32_t slot;
  uint32_t pad;
};

// Per-table control block in device memory.
struct Ctrl {
  unsigned long long size[2];         // rows in use, ping-pong on the call epoch
  unsigned long long bad_epoch;       // epoch of a call that met the reserved key
  unsigned long long overflow_epoch;  // epoch of a call whose inserts overran the probe bound
  unsigned long long spill_next;      // bump allocator for partitions larger than LDS
  unsigned long long new_epoch;       // epoch of a call that inserted at least one key
  // a put whose probe kernel runs ahead of a get's kernels (and its other
  // kernels after them) marks its own errors here, so that the get does not
  // overwrite them: the epoch of such a put that met the reserved key, and of
  // one that met a key absent from the table before the pair of calls
  unsigned long long apput_bad_epoch;
  unsigned long long apput_absent_epoch;
  // a get whose probe kernel filed its new keys in range lists (see
  // RangeLists), and one whose lists overflowed
  unsigned long long rl_epoch;
  unsigned long long rl_overflow_epoch;
  int latched;                        // first device-side error since mlkv_sync
  unsigned int pad[7];
  // tiered tables: rows a lookahead call claimed as misses (ping-pong on the
  // call count), the FIFO cursor over cache slots, the entries of the last
  // copy plan, and running totals
  unsigned long long tier_nmiss[2];
  unsigned long long tier_cursor;
  unsigned long long tier_nplan;
  unsigned long long tier_loaded;   // rows copied from host memory into the cache
  unsigned long long tier_evicted;  // rows whose slot was given to another row
  unsigned long long tier_written;  // evicted rows written back (dirty)
  unsigned long long tier_filled;   // slots holding a row
};

// ---------------------------------------------------------------------------
// Hashing
// ---------------------------------------------------------------------------
// Bucket choice: a 64-bit finaliser (MurmurHash3 fmix64) then the top bits.
__device__ __forceinline__ uint64_t index_hash(uint64_t k) {
  k ^= k >> 33;
  k *= 0xff51afd7ed558ccdull;
  k ^= k >> 33;
  k *= 0xc4ceb9fe1a85ec53ull;
  k ^= k >> 33;
  return k;
}

// SplitMix64 output function (Steele, Lea & Flood 2014).
__device__ __forceinline__ uint64_t splitmix_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Initial value of column c of a new key, given s0 = mix64(key ^ seed): the
// top 24 bits of mix64(s0 + c * golden gamma), centred and scaled by
// 0.01f * 2^-23, i.e. uniform on [-0.01, 0.01).
__device__ __forceinline__ float init_elem(uint64_t s0, int c) {
  const uint64_t h = splitmix_mix(s0 + (uint64_t)(uint32_t)c * 0x9E3779B97F4A7C15ull);
  const int t = (int)(uint32_t)(h >> 40) - (1 << 23);
  constexpr float kScale = 0.01f * 0x1p-23f;
  return __fmul_rn((float)t, kScale);
}

// ---------------------------------------------------------------------------
// Probe / insert, one key per lane.
// ---------------------------------------------------------------------------
enum ProbeStatus : int {
  P_HIT = 0,        // key present from an earlier call; row valid
  P_NEW_MINE = 1,   // this lane inserted the key (row pending)
  P_NEW_OTHER = 2,  // another lane of this call inserted it (row pending)
  P_ABSENT = 3,     // not present (lookup only)
  P_OVERFLOW = 4,   // probe bound reached while inserting
  P_BAD = 5,        // reserved key
  P_NONE = 6        // lane has no key
};

struct Probe {
  uint32_t slot;
  uint32_t row;
  int status;
};

// First bucket of a key's probe chain (the bucket index), used to issue the
// loads of several keys before examining any of them.
__device__ __forceinline__ uint64_t home_bucket(uint64_t key, uint32_t nb_log2) {
  return nb_log2 ? (index_hash(key) >> (64 - nb_log2)) : 0;
}

struct BucketView {
  uint64_t k[8];
  uint32_t r[8];
};

__device__ __forceinline__ BucketView load_bucket(const Bucket* B) {
  BucketView v;
  const ulonglong2* kp = reinterpret_cast<const ulonglong2*>(B->key);
  const uint4* rp = reinterpret_cast<const uint4*>(B->row);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const ulonglong2 x = kp[q];
    v.k[2 * q] = x.x;
    v.k[2 * q + 1] = x.y;
  }
  const uint4 r0 = rp[0], r1 = rp[1];
  v.r[0] = r0.x; v.r[1] = r0.y; v.r[2] = r0.z; v.r[3] = r0.w;
  v.r[4] = r1.x; v.r[5] = r1.y; v.r[6] = r1.z; v.r[7] = r1.w;
  return v;
}

// Linear probing over buckets. A bucket holding an EMPTY tag ends the chain.
// Inserts claim the first EMPTY tag in chain order with a CAS; a failed CAS
// returns the tag that is really there, so a stale view of the line never
// produces a duplicate key (tags only ever go from EMPTY to a key in a call).
// `v` is the already loaded view of bucket `b`, the key's home bucket.
__device__ __forceinline__ Probe probe_with(Bucket* __restrict__ idx, uint32_t nb_log2, uint64_t key,
                                            bool insert, uint64_t b, BucketView v) {
  const uint64_t mask = (nb_log2 >= 64) ? ~0ull : ((1ull << nb_log2) - 1);
  const uint64_t limit = mask < (uint64_t)kMaxProbe ? mask + 1 : (uint64_t)kMaxProbe;
  for (uint64_t p = 0; p < limit; ++p) {
    if (p > 0) v = load_bucket(idx + b);
    int hit = -1;
    bool has_empty = false;
#pragma unroll
    for (int j = kSlots - 1; j >= 0; --j) {
      if (v.k[j] == key) hit = j;
      has_empty |= (v.k[j] == kEmptyKey);
    }
    if (hit >= 0) {
      uint32_t r = v.r[0];
#pragma unroll
      for (int j = 1; j < kSlots; ++j)
        if (hit == j) r = v.r[j];
      return {(uint32_t)(b * kSlots + hit), r, r == kPendingRow ? P_NEW_OTHER : P_HIT};
    }
    if (has_empty) {
      if (!insert) return {0, kPendingRow, P_ABSENT};
      Bucket* B = idx + b;
      for (int j = 0; j < kSlots; ++j) {
        if (v.k[j] != kEmptyKey) continue;
        const uint64_t old = atomicCAS(reinterpret_cast<unsigned long long*>(&B->key[j]),
                                       (unsigned long long)kEmptyKey, (unsigned long long)key);
        if (old == kEmptyKey) return {(uint32_t)(b * kSlots + j), kPendingRow, P_NEW_MINE};
        if (old == key) return {(uint32_t)(b * kSlots + j), kPendingRow, P_NEW_OTHER};
      }
      // every EMPTY tag seen was taken by other keys meanwhile: the chain goes on
    }
    b = (b + 1) & mask;
  }
  return {0, kPendingRow, insert ? P_OVERFLOW : P_ABSENT};
}

__device__ __forceinline__ Probe probe_key(Bucket* __restrict__ idx, uint32_t nb_log2, uint64_t key,
                                           bool insert) {
  const uint64_t b = home_bucket(key, nb_log2);
  return probe_with(idx, nb_log2, key, insert, b, load_bucket(idx + b));
}

// ---------------------------------------------------------------------------
// Block-wide helpers
// ---------------------------------------------------------------------------
// Barrier that orders LDS only: global loads and stores issued before it stay
// in flight (a full __syncthreads waits for them too).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Exclusive scan over the block; NT threads, s_w needs NT/64 words.
template <int NT>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* s_w, uint32_t* total) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_w[w] = x;
  lds_barrier();
  if (w == 0) {
    uint32_t s = lane < NT / 64 ? s_w[lane] : 0u;
#pragma unroll
    for (int o = 1; o < NT / 64; o <<= 1) {
      const uint32_t y = __shfl_up(s, o, 64);
      if (lane >= o) s += y;
    }
    if (lane < NT / 64) s_w[lane] = s;
  }
  lds_barrier();
  const uint32_t pre = (w > 0 ? s_w[w - 1] : 0u) + x - v;
  *total = s_w[NT / 64 - 1];
  lds_barrier();
  return pre;
}

// As block_exclusive_scan, on 64-bit values (two 32-bit fields can be
// scanned at once when the low field's total stays below 2^32).
template <int NT>
__device__ __forceinline__ uint64_t block_exclusive_scan_u64(uint64_t v, unsigned long long* s_w, uint64_t* total) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  unsigned long long x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const unsigned long long y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_w[w] = x;
  lds_barrier();
  if (w == 0) {
    unsigned long long s = lane < NT / 64 ? s_w[lane] : 0ull;
#pragma unroll
    for (int o = 1; o < NT / 64; o <<= 1) {
      const unsigned long long y = __shfl_up(s, o, 64);
      if (lane >= o) s += y;
    }
    if (lane < NT / 64) s_w[lane] = s;
  }
  lds_barrier();
  const uint64_t pre = (w > 0 ? s_w[w - 1] : 0ull) + x - v;
  *total = s_w[NT / 64 - 1];
  lds_barrier();
  return pre;
}

template <int NT>
__device__ __forceinline__ uint64_t block_sum_u64(uint64_t v, unsigned long long* s_w) {
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor((unsigned long long)v, o, 64);
  if (lane == 0) s_w[w] = v;
  lds_barrier();
  uint64_t t = 0;
#pragma unroll
  for (int j = 0; j < NT / 64; ++j) t += s_w[j];
  lds_barrier();
  return t;
}

// Bitonic sort of N (power of two) 64-bit words, ascending, by the whole block.
template <int NT, class P>
__device__ __forceinline__ void block_bitonic_sort(P a, uint32_t N) {
  for (uint32_t k = 2; k <= N; k <<= 1) {
    for (uint32_t j = k >> 1; j > 0; j >>= 1) {
      for (uint32_t i = threadIdx.x; i < N; i += NT) {
        const uint32_t ixj = i ^ j;
        if (ixj > i) {
          const uint64_t x = a[i];
          const uint64_t y = a[ixj];
          const bool up = (i & k) == 0;
          if ((x > y) == up) {
            a[i] = y;
            a[ixj] = x;
          }
        }
      }
      __syncthreads();
    }
  }
}

// ---------------------------------------------------------------------------
// Lane <-> row-element mapping. A wave is split into RPW = 64/LPR lane groups;
// a group of LPR lanes covers one row, VEC consecutive floats per lane per
// chunk, K chunks: column of (chunk k, element v) = (k*LPR + q)*VEC + v.
// ---------------------------------------------------------------------------
template <int VEC_, int LPR_, int K_>
struct RowMap {
  static constexpr int VEC = VEC_;
  static constexpr int LPR = LPR_;
  static constexpr int K = K_;
  static constexpr int RPW = 64 / LPR_;
};

template <int VEC>
struct VecT;
template <>
struct VecT<1> {
  using T = float;
  static __device__ __forceinline__ float get(const T& x, int) { return x; }
  static __device__ __forceinline__ void set(T& x, int, float v) { x = v; }
};
template <>
struct VecT<4> {
  using T = float4;
  static __device__ __forceinline__ float get(const T& x, int v) {
    return v == 0 ? x.x : v == 1 ? x.y : v == 2 ? x.z : x.w;
  }
  static __device__ __forceinline__ void set(T& x, int v, float f) {
    if (v == 0) x.x = f;
    else if (v == 1) x.y = f;
    else if (v == 2) x.z = f;
    else x.w = f;
  }
};

}  // namespace mlkv
