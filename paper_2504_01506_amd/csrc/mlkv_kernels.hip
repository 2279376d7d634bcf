// HIP kernels of libmlkv for gfx950 (MI355X): hash-index probe, row gather,
// in-batch dedup by MSD radix partition + LDS sort + run-length encoding, and
// the fp64 segment-reduce fused with the row-wise Adagrad scatter-update.
#include "mlkv_kernels.h"

#include <type_traits>

namespace mlkv {

// ===========================================================================
// Get: probe + gather (+ insert-on-miss), one key per lane.
// ===========================================================================
template <int VEC>
__device__ __forceinline__ typename VecT<VEC>::T load_vec(const float* p) {
  if constexpr (VEC == 4) {
    return *reinterpret_cast<const float4*>(p);
  } else {
    return *p;
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float* p, const typename VecT<VEC>::T& v) {
  if constexpr (VEC == 4) {
    *reinterpret_cast<float4*>(p) = v;
  } else {
    *p = v;
  }
}

// Loads W consecutive 32-bit words (W = 1, 2, 4 or 8; 16-byte aligned when W >= 4).
template <int W>
__device__ __forceinline__ void load_words(uint32_t* dst, const uint32_t* src) {
  if constexpr (W >= 4) {
#pragma unroll
    for (int h = 0; h < W / 4; ++h) {
      const uint4 v = reinterpret_cast<const uint4*>(src)[h];
      dst[4 * h] = v.x;
      dst[4 * h + 1] = v.y;
      dst[4 * h + 2] = v.z;
      dst[4 * h + 3] = v.w;
    }
  } else if constexpr (W == 2) {
    const uint2 v = *reinterpret_cast<const uint2*>(src);
    dst[0] = v.x;
    dst[1] = v.y;
  } else {
    dst[0] = *src;
  }
}

template <int VEC>
__device__ __forceinline__ typename VecT<VEC>::T init_vec(uint64_t s0, int col) {
  typename VecT<VEC>::T v;
#pragma unroll
  for (int e = 0; e < VEC; ++e) VecT<VEC>::set(v, e, init_elem(s0, col + e));
  return v;
}

// The wave copies the rows of its 64 positions into `out`: rows of keys that
// were present are read from the table (how = 1), rows of keys new in this
// call are generated from their seed (how = 0; they equal what the table will
// hold), and positions of blocked keys are not written (how = 2, only with
// kTrack: skipping stores costs registers, so tables without a staleness
// bound use a variant without it).
template <class M, bool kTrack>
__device__ __forceinline__ void wave_emit_rows(float* __restrict__ out, const RowStore& store,
                                               int D, int64_t wave_base, int64_t n, int how,
                                               uint32_t row, uint64_t s0, int lane) {
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  constexpr int ITERS = 64 / RPW;
  constexpr int UNITS = ITERS * K;
  constexpr int CH = UNITS < 16 ? UNITS : 16;
  const int g = lane / LPR;
  const int q = lane % LPR;
#pragma unroll 1
  for (int u0 = 0; u0 < UNITS; u0 += CH) {
    typename VecT<VEC>::T v[CH];
    uint32_t skip = 0;  // units whose position is blocked
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int uu = u0 + u;
      const int it = uu / K;
      const int k = uu % K;
      const int r = it * RPW + g;
      const uint32_t rr = __shfl(row, r, 64);
      const int hh = __shfl(how, r, 64);
      const uint64_t ss = __shfl((unsigned long long)s0, r, 64);
      const int col = (k * LPR + q) * VEC;
      const int64_t p = wave_base + r;
      if constexpr (kTrack) skip |= (hh == 2 ? 1u : 0u) << u;
      if (uu < UNITS && p < n && col < D) {
        if (hh == 1) v[u] = load_vec<VEC>(store.ptr(rr) + col);
        else if (hh == 0) v[u] = init_vec<VEC>(ss, col);
      }
    }
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int uu = u0 + u;
      const int it = uu / K;
      const int k = uu % K;
      const int r = it * RPW + g;
      const int col = (k * LPR + q) * VEC;
      const int64_t p = wave_base + r;
      if (uu < UNITS && p < n && col < D && (!kTrack || !((skip >> u) & 1u)))
        store_vec<VEC>(out + (size_t)p * (size_t)D + col, v[u]);
    }
  }
}

// kPcIn: a position whose key equals pc_key[i] takes pc_row[i] without
// probing (an instance of its own, so that other gets run unchanged)
template <class M, bool kTrack, bool kPcIn>
__global__ __launch_bounds__(kGetTile) void k_get_probe_gather(
    Bucket* __restrict__ idx, uint32_t nb_log2, const uint64_t* __restrict__ keys, int64_t n,
    float* __restrict__ out, const RowStore store, int D, uint64_t seed,
    NewKey* __restrict__ newlist, uint32_t* __restrict__ tile_cnt, Ctrl* ctrl, uint64_t epoch,
    unsigned long long* __restrict__ clock, uint64_t cepoch, uint32_t bound, uint8_t* __restrict__ blocked,
    uint64_t* __restrict__ pc_key, uint32_t* __restrict__ pc_row, int tlen, const RangeLists rl,
    uint32_t nranges) {
  __shared__ uint32_t s_cnt;
  __shared__ uint64_t s_nkey[kGetTile];  // the tile's new keys and their slots
  __shared__ uint32_t s_nslot[kGetTile];
  __shared__ uint64_t s_cuts[kMaxRanges - 1];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // the block's tile: tlen (<= kGetTile) positions, so that every CU gets the
  // same number of positions
  const int64_t base = (int64_t)blockIdx.x * tlen;
  const int64_t end = min(n, base + tlen);
  const int64_t i = base + tid;
  if (tid == 0) s_cnt = 0;
  __syncthreads();
  uint64_t key = 0;
  Probe pr = {0, kPendingRow, P_NONE};
  bool recorded = false;  // the key and its row came from the row cache
  if (i < end) {
    key = keys[i];
    if (key == kEmptyKey) {
      pr.status = P_BAD;
      ctrl->bad_epoch = epoch;
    } else {
      if constexpr (kPcIn) {
        const uint64_t ck = pc_key[i];
        const uint32_t cr = pc_row[i];
        if (ck == key) {
          pr = {0u, cr, P_HIT};
          recorded = true;
        }
      }
      if (!recorded) {
        pr = probe_key(idx, nb_log2, key, true);
        if (pr.status == P_OVERFLOW) ctrl->overflow_epoch = epoch;
      }
    }
  }
  if (pr.status == P_NEW_MINE) {
    const uint32_t j = atomicAdd(&s_cnt, 1u);
    s_nkey[j] = key;
    s_nslot[j] = pr.slot;
    ctrl->new_epoch = epoch;
  }
  // a key present before the call, with its row, for a put of the same
  // batch: a key's row never changes once assigned, so the pair stays valid
  if (i < end && pc_key != nullptr && !recorded) {
    pc_key[i] = pr.status == P_HIT ? key : kEmptyKey;
    pc_row[i] = pr.row;
  }
  int how = pr.status == P_HIT ? 1 : 0;
  if (kTrack && i < end) {
    // bounded staleness: a present key is served while its count before the
    // call is at most the bound. Serving it stamps the word with the call's
    // epoch and that count plus one. Nothing else writes the word during the
    // call, so a position reads either the word from before the call or the
    // stamp; every position that reads the former stores the same stamp, and
    // a plain store suffices (hot keys would serialise atomics). The count
    // thus rises once per call, however often the key occurs.
    bool blk = false;
    if (pr.status == P_HIT) {
      unsigned long long* cw = clock + pr.row;
      const unsigned long long w = *cw;
      if ((w >> kClockBits) != cepoch) {
        if ((w & kClockCount) > bound) blk = true;
        else *cw = (cepoch << kClockBits) | ((w & kClockCount) + 1);
      }
    }
    if (blk) how = 2;
    blocked[i] = blk ? 1 : 0;
  }
  if (out != nullptr) {
    const uint64_t s0 = splitmix_mix(key ^ seed);
    wave_emit_rows<M, kTrack>(out, store, D, base + wave * 64, end, how, pr.row, s0, lane);
  }
  __syncthreads();
  // the tile's list of new keys, in ascending key order (each at its rank)
  const uint32_t c = s_cnt;
  if ((uint32_t)tid < c) {
    const uint64_t k = s_nkey[tid];
    uint32_t r = 0;
    for (uint32_t e = 0; e < c; ++e) r += s_nkey[e] < k ? 1u : 0u;
    newlist[base + r] = NewKey{k, s_nslot[tid], 0u};
  }
  if (tid == 0) tile_cnt[blockIdx.x] = c;
  // the same keys filed by key range, when the cut points are for this
  // call's number of ranges (block-uniform: c and the cut count)
  if (rl.list != nullptr && c > 0 && *rl.cuts_g == nranges) {
    for (uint32_t e = tid; e + 1 < nranges; e += kGetTile) s_cuts[e] = rl.cuts[e];
    __syncthreads();
    if ((uint32_t)tid < c) {
      const uint64_t k = s_nkey[tid];
      uint32_t q = 0;  // range q holds [cut q-1, cut q): q = cut points <= k
      for (uint32_t step = kMaxRanges / 2; step >= 1; step >>= 1)
        if (q + step < nranges && s_cuts[q + step - 1] <= k) q += step;
      const uint32_t at = atomicAdd(&rl.cnt[q], 1u);
      if (at < rl.cap) rl.list[(size_t)q * rl.cap + at] = NewKey{k, s_nslot[tid], 0u};
      else ctrl->rl_overflow_epoch = epoch;
    }
    if (tid == 0) ctrl->rl_epoch = epoch;
  }
}

// ===========================================================================
// Streaming every new key of the call through LDS (used to rank new keys).
// ===========================================================================
constexpr int kChunk = 2048;

// Calls body(s_chunk, cnt) for consecutive chunks of this call's new keys;
// the block's NT threads must all call it. s_pref: NT+1 words.
template <int NT, class Body>
__device__ __forceinline__ void for_each_new_key_chunk(const NewKey* __restrict__ newlist,
                                       const uint32_t* __restrict__ tile_cnt, int ntiles,
                                       int tile_size, uint32_t* s_pref, uint32_t* s_w,
                                       uint64_t* s_chunk, Body body) {
  constexpr int PER = kChunk / NT;
  for (int t0 = 0; t0 < ntiles; t0 += NT) {
    const int nt = min(NT, ntiles - t0);
    const uint32_t c = (int)threadIdx.x < nt ? tile_cnt[t0 + threadIdx.x] : 0u;
    uint32_t total;
    const uint32_t pre = block_exclusive_scan<NT>(c, s_w, &total);
    s_pref[threadIdx.x] = pre;
    __syncthreads();
    for (uint32_t k0 = 0; k0 < total; k0 += kChunk) {
      const uint32_t cnt = min((uint32_t)kChunk, total - k0);
      uint64_t v[PER];
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const uint32_t k = threadIdx.x + e * NT;
        v[e] = 0;
        if (k < cnt) {
          const uint32_t gk = k0 + k;
          int lo = 0, hi = nt - 1;
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (s_pref[mid] <= gk) lo = mid;
            else hi = mid - 1;
          }
          v[e] = newlist[(size_t)(t0 + lo) * tile_size + (gk - s_pref[lo])].key;
        }
      }
#pragma unroll
      for (int e = 0; e < PER; ++e) {
        const uint32_t k = threadIdx.x + e * NT;
        if (k < cnt) s_chunk[k] = v[e];
      }
      __syncthreads();
      body(s_chunk, cnt);
      __syncthreads();
    }
    __syncthreads();
  }
}

// Sum of the per-tile new-key counts, i.e. the number M of distinct keys the
// call inserts.
template <int NT>
__device__ __forceinline__ uint64_t count_new_keys(const uint32_t* __restrict__ tile_cnt, int ntiles,
                                                   unsigned long long* s_w64) {
  uint64_t m = 0;
  for (int t = threadIdx.x; t < ntiles; t += NT) m += tile_cnt[t];
  return block_sum_u64<NT>(m, s_w64);
}

// Decides whether the call fails, and publishes the size for the next call.
__device__ __forceinline__ int call_verdict(Ctrl* ctrl, uint64_t epoch, uint64_t size0, uint64_t M,
                                            int64_t capacity, uint64_t bad_epoch, uint64_t overflow_epoch,
                                            uint64_t absent_epoch = 0) {
  int err = 0;
  if (bad_epoch == epoch) err = -1;                                           // MLKV_EINVAL
  else if (absent_epoch == epoch) err = kErrAbsent;                          // MLKV_EINVAL, its own message
  else if (overflow_epoch == epoch || size0 + M > (uint64_t)capacity) err = -2;  // MLKV_EFULL
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctrl->size[(epoch + 1) & 1] = err ? size0 : size0 + M;
    if (err) atomicCAS(&ctrl->latched, 0, err);
  }
  return err;
}

// ===========================================================================
// Get, second kernel: assign rows to the call's new keys (ascending key order),
// write their initial rows and zero accumulators; or roll the call back.
// ===========================================================================
constexpr int kAssignThreads = 256;
constexpr int kAssignBatch = 8;
constexpr int kAssignMine = kAssignBatch * kAssignThreads;
// With few new keys each block ranks its tiles' keys against all of them,
// streamed through LDS once per NT tiles of the call: about 13 us plus 44 ns
// per (new key x NT tiles) on MI355X (55 us at 256 new keys of a 213k-key,
// 832-tile batch; 1.4 ms at 8192), while key ranges take 44-50 us from a few
// hundred keys up when each block must search every tile's list for its
// range, and far less with range lists (those calls always take them). The
// direct ranking is otherwise used up to kAssignDirectWork new
// keys x tile chunks.
constexpr uint64_t kAssignDirectWork = 768;
constexpr int kRangeSamples = 2048;  // sample of the new keys that splits the key space among the blocks
constexpr int kRangeCap = 3072;      // keys of a block's key range ranked in LDS at once

// Each tile's list of new keys is sorted (ascending key). For the key range
// [lo, hi) this returns the thread's share of the number of new keys below lo
// and calls emit(offset, n) for each tile run of the range's keys (offset
// into the lists, n > 0 entries). Threads take kSearchTiles tiles at a time
// and search both bounds in all of them together (branch-free binary search,
// each step one load per bound and tile in flight).
constexpr int kSearchTiles = 16;
template <int NT, class Emit>
__device__ __forceinline__ uint64_t search_tile_lists(const NewKey* __restrict__ newlist,
                                                      const uint32_t* __restrict__ tile_cnt, int ntiles,
                                                      int tile_size, uint64_t lo, uint64_t hi, Emit emit) {
  uint64_t below = 0;
  for (int t0 = threadIdx.x; t0 < ntiles; t0 += NT * kSearchTiles) {
    uint32_t c[kSearchTiles], a[kSearchTiles], b[kSearchTiles];
#pragma unroll
    for (int u = 0; u < kSearchTiles; ++u) {
      const int t = t0 + u * NT;
      c[u] = t < ntiles ? tile_cnt[t] : 0u;
      a[u] = 0;  // keys below lo
      b[u] = 0;  // keys below hi
    }
    // a tile holds at most kGetTile (a power of two) keys
    for (uint32_t step = (uint32_t)kGetTile; step >= 1; step >>= 1) {
#pragma unroll
      for (int u = 0; u < kSearchTiles; ++u) {
        const NewKey* l = newlist + (size_t)(t0 + u * NT) * tile_size;
        if (a[u] + step <= c[u] && l[a[u] + step - 1].key < lo) a[u] += step;
        if (b[u] + step <= c[u] && l[b[u] + step - 1].key < hi) b[u] += step;
      }
    }
#pragma unroll
    for (int u = 0; u < kSearchTiles; ++u) {
      below += a[u];
      if (b[u] > a[u]) emit((uint32_t)(t0 + u * NT) * (uint32_t)tile_size + a[u], b[u] - a[u]);
    }
  }
  return below;
}

// Ascending bitonic sort of NT * kSortPT keys, thread t holding the
// elements kSortPT t .. kSortPT t + kSortPT - 1 in v. Compare-exchanges whose
// partner lies in the same thread run in registers; the others exchange
// through LDS, alternating between buf0 and buf1 (NT * kSortPT keys each), so
// one barrier per such stage suffices.
constexpr int kSortPT = 8;
template <int NT>
__device__ __forceinline__ void sort_keys_8pt(uint64_t (&v)[kSortPT], uint64_t* buf0, uint64_t* buf1) {
  constexpr uint32_t N = (uint32_t)NT * kSortPT;
  const uint32_t t = threadIdx.x;
  auto reg_stage = [&](auto J, uint32_t k) {
    constexpr uint32_t j = decltype(J)::value;
#pragma unroll
    for (uint32_t r = 0; r < kSortPT; ++r) {
      if ((r & j) == 0) {
        const bool asc = ((t * kSortPT + r) & k) == 0;
        const uint64_t a = v[r], b = v[r + j];
        if ((a > b) == asc) {
          v[r] = b;
          v[r + j] = a;
        }
      }
    }
  };
  bool second = false;
  for (uint32_t k = 2; k <= N; k <<= 1) {
    for (uint32_t j = k >> 1; j >= kSortPT; j >>= 1) {
      uint64_t* b = second ? buf1 : buf0;
      second = !second;
#pragma unroll
      for (uint32_t r = 0; r < kSortPT; ++r) b[r * NT + t] = v[r];
      lds_barrier();
      const uint32_t pt = t ^ (j / kSortPT);
#pragma unroll
      for (uint32_t r = 0; r < kSortPT; ++r) {
        const uint32_t i = t * kSortPT + r;
        const uint64_t p = b[r * NT + pt];
        const bool asc = (i & k) == 0, low = (i & j) == 0;
        v[r] = (asc == low) ? (v[r] < p ? v[r] : p) : (v[r] > p ? v[r] : p);
      }
    }
    if (k >= 8) reg_stage(std::integral_constant<uint32_t, 4>{}, k);
    if (k >= 4) reg_stage(std::integral_constant<uint32_t, 2>{}, k);
    reg_stage(std::integral_constant<uint32_t, 1>{}, k);
  }
}

// Staleness word of a row that a get inserts: served once by this call.
__device__ __forceinline__ unsigned long long new_row_clock(uint64_t cepoch) {
  return ((unsigned long long)cepoch << kClockBits) | 1ull;
}

// A failed get call gives back the counts it raised: every row stamped with
// its epoch loses one, and the stamp (needed only within the call) is cleared.
__device__ __forceinline__ void rollback_clocks(unsigned long long* __restrict__ clock, uint64_t nrows,
                                                uint64_t cepoch) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  for (uint64_t r = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; r < nrows; r += stride) {
    const unsigned long long w = clock[r];
    if ((w >> kClockBits) == cepoch) clock[r] = (w & kClockCount) - 1;
  }
}

// Initial rows of new keys ks[j] (j < m) at rows base + rk[j]: a wave per
// row, its lanes along the row, kInitRows rows of a wave at a time so that
// each lane has that many independent hash chains in flight (the 64-bit
// multiplies of one chain are serial).
constexpr int kInitRows = 4;
template <int NT, class KP, class RP>
__device__ __forceinline__ void write_init_rows(const KP ks, const RP rk, uint32_t m, uint64_t base,
                                                const RowStore& store, int D, uint64_t seed) {
  constexpr uint32_t NW = NT / 64;
  const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (uint32_t j0 = wave; j0 < m; j0 += NW * kInitRows) {
    float* w[kInitRows];
    uint64_t s0[kInitRows];
#pragma unroll
    for (int r = 0; r < kInitRows; ++r) {
      const uint32_t j = j0 + (uint32_t)r * NW;
      w[r] = nullptr;
      s0[r] = 0;
      if (j < m) {
        w[r] = store.wptr((uint32_t)(base + rk[j]));
        s0[r] = splitmix_mix(ks[j] ^ seed);
      }
    }
    for (int col = (int)lane; col < D; col += 64) {
#pragma unroll
      for (int r = 0; r < kInitRows; ++r)
        if (w[r] != nullptr) w[r][col] = init_elem(s0[r], col);
    }
  }
}

// Rows for the new keys ks[0, m) (index slots sl[...]) whose ranks among all
// new keys of the call are base + rk[...]: index row ids, zero accumulators,
// initial rows (written along rows).
template <int NT, class KP, class SP, class RP>
__device__ __forceinline__ void write_new_rows(const KP ks, const SP sl, const RP rk, uint32_t m, uint64_t base,
                                               Bucket* __restrict__ idx, const RowStore& store,
                                               float* __restrict__ state, int D, uint64_t seed,
                                               unsigned long long* __restrict__ clock, uint64_t cepoch) {
  for (uint32_t j = threadIdx.x; j < m; j += NT) {
    const uint32_t slot = sl[j];
    const uint32_t row = (uint32_t)(base + rk[j]);
    idx[slot / kSlots].row[slot % kSlots] = row;
    state[row] = 0.0f;
    if (clock != nullptr) clock[row] = new_row_clock(cepoch);
  }
  write_init_rows<NT>(ks, rk, m, base, store, D, seed);
}

__global__ __launch_bounds__(kAssignThreads) void k_assign_new(
    Bucket* __restrict__ idx, const NewKey* __restrict__ newlist, const uint32_t* __restrict__ tile_cnt,
    int ntiles, int tile_size, const RowStore store, float* __restrict__ state, int D,
    uint64_t seed, int64_t capacity, Ctrl* ctrl, uint64_t epoch, uint64_t* __restrict__ xkey,
    uint32_t* __restrict__ xslot, unsigned long long* __restrict__ clock, uint64_t cepoch, const RangeLists rl) {
  constexpr int NT = kAssignThreads;
  __shared__ unsigned long long s_w64[NT / 64];
  __shared__ uint32_t s_w[NT / 64];
  __shared__ __align__(16) uint32_t s_pref[NT + 1];
  __shared__ uint32_t s_nc;
  __shared__ uint64_t s_cut[2];
  // one LDS buffer of 48 KiB; the two ranking methods lay it out differently
  __shared__ uint64_t s_buf[kChunk + 2 * kAssignMine];
  static_assert(kRangeCap * 14 <= (int)sizeof(s_buf) && kRangeSamples * 12 <= (int)sizeof(s_buf), "LDS");
  static_assert(kRangeSamples == NT * kSortPT && kRangeCap <= 65536, "sample and range sizes");

  // the next call's range counts start at zero (this call's are read below)
  if (rl.list != nullptr && blockIdx.x == 0)
    for (int e = threadIdx.x; e < kMaxRanges; e += NT) rl.cnt_next[e] = 0u;
  const uint64_t size0 = ctrl->size[epoch & 1];
  const bool any_new = ctrl->new_epoch == epoch;
  const uint64_t M = any_new ? count_new_keys<NT>(tile_cnt, ntiles, s_w64) : 0ull;
  const int err = call_verdict(ctrl, epoch, size0, M, capacity, ctrl->bad_epoch, ctrl->overflow_epoch);
  if (err && clock != nullptr) rollback_clocks(clock, size0, cepoch);
  if (M == 0) return;

  if (err) {  // undo this call's insertions: the index returns to its state before the call
    for (int t = blockIdx.x; t < ntiles; t += gridDim.x) {
      const uint32_t c = tile_cnt[t];
      for (uint32_t j = threadIdx.x; j < c; j += NT) {
        const uint32_t slot = newlist[(size_t)t * tile_size + j].slot;
        idx[slot / kSlots].key[slot % kSlots] = kEmptyKey;
      }
    }
    return;
  }

  // the probe kernel filed the new keys by range (RangeLists): ranking them
  // by range then costs little for any number of them
  const bool listed = rl.list != nullptr && ctrl->rl_epoch == epoch && ctrl->rl_overflow_epoch != epoch;
  if (listed || M * (uint64_t)((ntiles + NT - 1) / NT) > kAssignDirectWork) {
    // ---- many new keys: key ranges. Block g ranks the new keys of the g-th
    // key range among themselves, after the count of new keys below the
    // range. The probe kernel has filed the keys by range when cut points for
    // this many ranges were left (RangeLists): the range's keys are its list,
    // the keys below it the lists before. Otherwise every block takes the
    // same sample of the new keys (sample k is the new key at position
    // floor(k M / S) of the tiles' lists laid end to end) and the same cut
    // points from it, which give block g the keys in [lo, hi); a binary
    // search of both bounds in every tile's sorted list of new keys counts
    // the keys below lo and finds the block's own. No block waits for another.
    const uint32_t g = blockIdx.x, G = gridDim.x;
    uint64_t* s_key = s_buf;                                                 // [kRangeCap]
    uint32_t* s_sr = reinterpret_cast<uint32_t*>(s_buf + kRangeCap);        // [kRangeCap]
    uint16_t* s_ord = reinterpret_cast<uint16_t*>(s_sr + kRangeCap);        // [kRangeCap]
    const NewKey* my_list = listed ? rl.list + (size_t)g * rl.cap : nullptr;
    uint64_t below = 0, lo = 0, hi = kEmptyKey;
    uint32_t c = 0;
    if (listed) {
      uint64_t mine = 0;
      for (uint32_t r = threadIdx.x; r < g; r += NT) mine += rl.cnt[r];
      below = block_sum_u64<NT>(mine, s_w64);
      c = rl.cnt[g];
      if (c <= (uint32_t)kRangeCap)
        for (uint32_t j = threadIdx.x; j < c; j += NT) {
          const NewKey nk = my_list[j];
          s_key[j] = nk.key;
          s_sr[j] = nk.slot;
        }
      __syncthreads();
    } else {
      constexpr uint32_t S = kRangeSamples;
      uint32_t* s_sat = reinterpret_cast<uint32_t*>(s_buf + S);     // [S] offsets of the samples in the lists
      {
        const int tpt = (ntiles + NT - 1) / NT;  // consecutive tiles per thread
        const int tb = min(ntiles, (int)threadIdx.x * tpt), te = min(ntiles, tb + tpt);
        uint32_t mine = 0;
        for (int t = tb; t < te; ++t) mine += tile_cnt[t];
        uint32_t tot;
        uint64_t pre = block_exclusive_scan<NT>(mine, s_w, &tot);
        uint64_t k = (pre * S + M - 1) / M;  // first sample at or after pre
        for (int t = tb; t < te && k < S; ++t) {
          const uint32_t c = tile_cnt[t];
          for (; k < S; ++k) {
            const uint64_t gk = k * M / S;
            if (gk >= pre + c) break;
            s_sat[k] = (uint32_t)t * (uint32_t)tile_size + (uint32_t)(gk - pre);
          }
          pre += c;
        }
      }
      __syncthreads();
      uint64_t v[kSortPT];
  #pragma unroll
      for (uint32_t u = 0; u < kSortPT; ++u) v[u] = newlist[s_sat[threadIdx.x + u * NT]].key;
      // the cut points: the samples of rank g S / G and (g + 1) S / G of the
      // sorted sample (with fewer new keys than samples a key is sampled more
      // than once, and equal cut points give an empty range); eight sample
      // gaps per range keep the largest range near twice the mean
      sort_keys_8pt<NT>(v, s_buf, s_buf + S);
      {
        const uint32_t r1 = (uint32_t)((uint64_t)g * S / G), r2 = (uint32_t)((uint64_t)(g + 1) * S / G);
  #pragma unroll
        for (uint32_t u = 0; u < kSortPT; ++u) {
          if (threadIdx.x * kSortPT + u == r1) s_cut[0] = v[u];
          if (threadIdx.x * kSortPT + u == r2) s_cut[1] = v[u];
        }
        if (threadIdx.x == 0) s_nc = 0;
      }
      __syncthreads();
      lo = g == 0 ? 0ull : s_cut[0];
      hi = g + 1 == G ? kEmptyKey : s_cut[1];
      // keys in [lo, hi) first go to LDS: key, slot (later the rank), and
      // their order by local sub-range
      below = search_tile_lists<NT>(newlist, tile_cnt, ntiles, tile_size, lo, hi, [&](uint32_t off, uint32_t cnt) {
        const uint32_t at = atomicAdd(&s_nc, cnt);
        for (uint32_t e = 0; e < cnt && at + e < (uint32_t)kRangeCap; ++e) {
          s_key[at + e] = newlist[off + e].key;
          s_sr[at + e] = off + e;  // slot and position are read later
        }
      });
      below = block_sum_u64<NT>(below, s_w64);  // its barriers also publish s_nc and the gathered keys
      c = s_nc;
      if (c <= (uint32_t)kRangeCap) {
        // the slot of each gathered key, from its list entry
        for (uint32_t j = threadIdx.x; j < c; j += NT) s_sr[j] = newlist[s_sr[j]].slot;
      }
      __syncthreads();
    }
    const uint64_t base = size0 + below;
    // cut points for the next call: cut j is the key of global rank
    // floor(j M / G), so the keys of rank R give cuts j in [ceil(R G / M),
    // ceil((R + 1) G / M))
    auto leave_cuts = [&](uint64_t key, uint64_t R) {
      if (rl.list == nullptr) return;
      const uint64_t jb = (R * G + M - 1) / M, je = ((R + 1) * G + M - 1) / M;
      for (uint64_t j = jb < 1 ? 1 : jb; j < je && j < G; ++j) rl.cuts[j - 1] = key;
    };
    if (c <= (uint32_t)kRangeCap) {
      // rank among the range's keys, through kSub local sub-ranges cut at a
      // sample of the gathered keys: sub-range counts and their prefix, the
      // keys listed by sub-range, then each key ranked inside its sub-range
      constexpr int kSub = 32;
      uint64_t* s_lc = reinterpret_cast<uint64_t*>(s_pref);  // [kSub - 1] local cut points (s_pref is free)
      uint32_t* s_sc = s_pref + 2 * kSub;                      // [kSub + 1] counts, then prefix, then cursors
      const uint32_t nl = c < (uint32_t)(kSub * 4) ? 0u : (uint32_t)kSub - 1;  // small ranges: one sub-range
      if (threadIdx.x < nl) {  // local cut l: the rank-l key of an evenly spaced sample of the gathered keys
        const uint64_t x = s_key[(uint64_t)(threadIdx.x + 1) * c / kSub];
        uint32_t rr = 0;
        for (uint32_t l = 0; l < nl; ++l) rr += s_key[(uint64_t)(l + 1) * c / kSub] < x ? 1u : 0u;
        s_lc[rr] = x;
      }
      if (threadIdx.x <= (uint32_t)kSub) s_sc[threadIdx.x] = 0;
      __syncthreads();
      uint32_t sub[kRangeCap / NT];
#pragma unroll
      for (int u = 0; u < kRangeCap / NT; ++u) {
        const uint32_t j = threadIdx.x + u * NT;
        sub[u] = 0;
        if (j < c) {
          const uint64_t key = s_key[j];
          uint32_t l = 0;  // sub-range l holds keys in [cut l-1, cut l): l = cuts <= key
          if (nl) {
#pragma unroll
            for (uint32_t step = kSub / 2; step >= 1; step >>= 1)
              if (l + step <= nl && s_lc[l + step - 1] <= key) l += step;
          }
          sub[u] = l;
          atomicAdd(&s_sc[l], 1u);
        }
      }
      __syncthreads();
      if (threadIdx.x == 0) {
        uint32_t acc = 0;
        for (int l = 0; l <= kSub; ++l) {
          const uint32_t x = s_sc[l];
          s_sc[l] = acc;
          acc += x;
        }
      }
      __syncthreads();
      uint32_t sbeg[kRangeCap / NT];
#pragma unroll
      for (int u = 0; u < kRangeCap / NT; ++u) {
        const uint32_t j = threadIdx.x + u * NT;
        sbeg[u] = 0;
        if (j < c) sbeg[u] = s_sc[sub[u]];
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kRangeCap / NT; ++u) {
        const uint32_t j = threadIdx.x + u * NT;
        if (j < c) s_ord[atomicAdd(&s_sc[sub[u]], 1u)] = (uint16_t)j;
      }
      __syncthreads();
      // after the cursors ran, s_sc[l] is the end of sub-range l
      uint32_t rk[kRangeCap / NT];
#pragma unroll
      for (int u = 0; u < kRangeCap / NT; ++u) {
        const uint32_t j = threadIdx.x + u * NT;
        rk[u] = 0;
        if (j < c) {
          const uint64_t key = s_key[j];
          const uint32_t b0 = sbeg[u], e0 = s_sc[sub[u]];
          uint32_t r = b0, i = b0;
          for (; i + 4 <= e0; i += 4) {
            const uint32_t o0 = s_ord[i], o1 = s_ord[i + 1], o2 = s_ord[i + 2], o3 = s_ord[i + 3];
            r += (s_key[o0] < key ? 1u : 0u) + (s_key[o1] < key ? 1u : 0u) + (s_key[o2] < key ? 1u : 0u) +
                 (s_key[o3] < key ? 1u : 0u);
          }
          for (; i < e0; ++i) r += s_key[s_ord[i]] < key ? 1u : 0u;
          rk[u] = r;
          const uint32_t slot = s_sr[j];
          idx[slot / kSlots].row[slot % kSlots] = (uint32_t)(base + r);
          state[base + r] = 0.0f;
          if (clock != nullptr) clock[base + r] = new_row_clock(cepoch);
          leave_cuts(key, below + r);
        }
      }
      __syncthreads();
#pragma unroll
      for (int u = 0; u < kRangeCap / NT; ++u) {
        const uint32_t j = threadIdx.x + u * NT;
        if (j < c) s_sr[j] = rk[u];
      }
      __syncthreads();
      write_init_rows<NT>(s_key, s_sr, c, base, store, D, seed);
    } else {
      // more keys in the range than LDS holds: gather them in global scratch
      // at [below, below + c), which no other block's range overlaps, then
      // rank them in chunks streamed through LDS
      __syncthreads();
      if (threadIdx.x == 0) s_nc = 0;
      __syncthreads();
      if (listed) {
        for (uint32_t j = threadIdx.x; j < c; j += NT) {
          const NewKey nk = my_list[j];
          xkey[below + j] = nk.key;
          xslot[below + j] = nk.slot;
        }
      } else {
        search_tile_lists<NT>(newlist, tile_cnt, ntiles, tile_size, lo, hi, [&](uint32_t off, uint32_t cnt) {
          const uint32_t at = atomicAdd(&s_nc, cnt);
          for (uint32_t e = 0; e < cnt; ++e) {
            const NewKey nk = newlist[off + e];
            xkey[below + at + e] = nk.key;
            xslot[below + at + e] = nk.slot;
          }
        });
      }
      __syncthreads();
      const uint64_t* rk_key = xkey + below;
      const uint32_t* rk_slot = xslot + below;
      uint64_t* s_cmp = s_buf;                                                    // [kChunk]
      uint64_t* s_mk = s_buf + kChunk;                                            // [kAssignMine]
      uint32_t* s_ms = reinterpret_cast<uint32_t*>(s_buf + kChunk + kAssignMine);  // [kAssignMine]
      uint32_t* s_mr = s_ms + kAssignMine;                                        // [kAssignMine]
      constexpr int PER = kAssignMine / NT;
      for (uint32_t j0 = 0; j0 < c; j0 += kAssignMine) {
        const uint32_t m = min((uint32_t)kAssignMine, c - j0);
        uint64_t mk[PER];
        uint32_t r[PER];
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const uint32_t j = threadIdx.x + u * NT;
          mk[u] = j < m ? rk_key[j0 + j] : 0ull;
          r[u] = 0;
        }
        for (uint32_t e0 = 0; e0 < c; e0 += kChunk) {
          const uint32_t cnt = min((uint32_t)kChunk, c - e0);
          for (uint32_t e = threadIdx.x; e < cnt; e += NT) s_cmp[e] = rk_key[e0 + e];
          __syncthreads();
          for (uint32_t e = 0; e < cnt; ++e) {
            const uint64_t v = s_cmp[e];
#pragma unroll
            for (int u = 0; u < PER; ++u) r[u] += v < mk[u] ? 1u : 0u;
          }
          __syncthreads();
        }
#pragma unroll
        for (int u = 0; u < PER; ++u) {
          const uint32_t j = threadIdx.x + u * NT;
          if (j < m) {
            s_mk[j] = mk[u];
            s_ms[j] = rk_slot[j0 + j];
            s_mr[j] = r[u];
            leave_cuts(mk[u], below + r[u]);
          }
        }
        __syncthreads();
        write_new_rows<NT>(s_mk, s_ms, s_mr, m, base, idx, store, state, D, seed, clock, cepoch);
        __syncthreads();
      }
    }
    if (rl.list != nullptr && g == 0 && threadIdx.x == 0) *rl.cuts_g = G;
    return;
  }

  // ---- few new keys: this block owns the tiles t = blockIdx.x (mod
  // gridDim.x); it takes them kAssignBatch at a time (thread j holds entry j
  // of each tile) and ranks their keys against all M new keys of the call.
  uint64_t* s_chunk = s_buf;                                              // [kChunk]
  uint64_t* s_key = s_buf + kChunk;                                       // [kAssignMine]
  uint32_t* s_slot = reinterpret_cast<uint32_t*>(s_key + kAssignMine);    // [kAssignMine]
  uint32_t* s_rank = s_slot + kAssignMine;                                // [kAssignMine]
  static_assert(kGetTile == NT, "one thread per entry of a probe tile");
  for (int tb = blockIdx.x; tb < ntiles; tb += gridDim.x * kAssignBatch) {
    uint32_t have = 0;
#pragma unroll
    for (int b = 0; b < kAssignBatch; ++b) {
      const int t = tb + b * (int)gridDim.x;
      const uint32_t c = t < ntiles ? tile_cnt[t] : 0u;
      const uint32_t j = threadIdx.x;
      const int m = b * NT + (int)j;
      if (j < c) {
        const NewKey nk = newlist[(size_t)t * tile_size + j];
        s_key[m] = nk.key;
        s_slot[m] = nk.slot;
        have = 1;
      } else {
        s_slot[m] = kPendingRow;  // marks an unused entry
      }
      s_rank[m] = 0;
    }
    if (block_sum_u64<NT>(have, s_w64) == 0) continue;
    for_each_new_key_chunk<NT>(newlist, tile_cnt, ntiles, tile_size, s_pref, s_w, s_chunk,
                               [&](const uint64_t* ck, uint32_t cnt) {
#pragma unroll
                                 for (int b = 0; b < kAssignBatch; ++b) {
                                   const int m = b * NT + (int)threadIdx.x;
                                   if (s_slot[m] == kPendingRow) continue;
                                   const uint64_t mk = s_key[m];
                                   uint32_t r = 0;
                                   for (uint32_t e = 0; e < cnt; ++e) r += ck[e] < mk ? 1u : 0u;
                                   s_rank[m] += r;
                                 }
                               });
#pragma unroll
    for (int b = 0; b < kAssignBatch; ++b) {
      const int m = b * NT + (int)threadIdx.x;
      const uint32_t slot = s_slot[m];
      if (slot == kPendingRow) continue;
      const uint32_t row = (uint32_t)(size0 + s_rank[m]);
      idx[slot / kSlots].row[slot % kSlots] = row;
      state[row] = 0.0f;
      if (clock != nullptr) clock[row] = new_row_clock(cepoch);
    }
    // initial rows, a wave per row
    for (int b = 0; b < kAssignBatch; ++b) {
      const int t = tb + b * (int)gridDim.x;
      const uint32_t c = t < ntiles ? tile_cnt[t] : 0u;
      write_init_rows<NT>(s_key + b * NT, s_rank + b * NT, c, size0, store, D, seed);
    }
    __syncthreads();
  }
}

// ===========================================================================
// Put. The (key, position) pairs of a call flow through "items":
//   bit 63     1 if the key is inserted by this call (row not yet known)
//   bits 31-62 the key's row, or its index slot when bit 63 is set
//   bit 30     1 if the item stands for several positions of one tile whose
//              gradient rows were already summed (fp64) into partials[pos]
//   bits 0-29  the position of the key in the batch (the first one for a
//              summed item)
// Sorting items groups the positions of each key (single positions first,
// then summed tiles, each in ascending order) and puts new keys last.
// ===========================================================================
constexpr uint64_t kItemSummed = 1ull << 30;

__device__ __forceinline__ uint64_t make_item(bool fresh, uint32_t tag, uint32_t low31) {
  return ((uint64_t)(fresh ? 1u : 0u) << 63) | ((uint64_t)tag << 31) | (uint64_t)(low31 & 0x7FFFFFFFu);
}
__device__ __forceinline__ uint32_t item_pos(uint64_t it) { return (uint32_t)(it & 0x3FFFFFFFull); }
__device__ __forceinline__ uint32_t item_low31(uint64_t it) { return (uint32_t)(it & 0x7FFFFFFFull); }
__device__ __forceinline__ bool item_summed(uint64_t it) { return (it & kItemSummed) != 0; }
__device__ __forceinline__ uint32_t item_tag(uint64_t it) { return (uint32_t)(it >> 31); }
__device__ __forceinline__ bool item_fresh(uint64_t it) { return (it >> 63) != 0; }
__device__ __forceinline__ uint64_t item_group(uint64_t it) { return it >> 31; }

// Partition of a key's group: top bits of a hash of (fresh, row or slot).
__device__ __forceinline__ uint32_t group_partition(uint64_t group, int pb) {
  return pb ? (uint32_t)(index_hash(group) >> (64 - pb)) : 0u;
}

// ---------------------------------------------------------------------------
// Put, first kernel (one block per tile of kPutTile keys, kPutThreads
// threads): probe (+ insert) each key; find the keys that occur more than once
// in the tile with an LDS hash table and sum each one's gradient rows
// (positions ascending, fp64) into one partial; partition the resulting items
// by a hash of the key (one MSD radix digit).
// ---------------------------------------------------------------------------
constexpr int kTileHash = 2 * kPutTile;  // LDS hash slots per tile

// kAhead: the put's probe runs ahead of the kernels of the get whose epoch is
// one less, its other kernels after them (PutArgs::ahead): it looks keys up
// without inserting, and a key absent from the table fails the put.
template <class M, bool kAhead>
__global__ __launch_bounds__(kPutThreads) void k_put_probe(
    Bucket* __restrict__ idx, uint32_t nb_log2, const uint64_t* __restrict__ keys,
    const float* __restrict__ grads, int64_t n, int tlen, int D, int op, int pb, int ntiles,
    uint64_t* __restrict__ items,
    uint32_t* __restrict__ meta, double* __restrict__ partials, NewKey* __restrict__ newlist,
    uint32_t* __restrict__ tile_cnt, Ctrl* ctrl, uint64_t epoch, const uint64_t* __restrict__ pc_key,
    const uint32_t* __restrict__ pc_row) {
  constexpr int NT = kPutThreads;
  constexpr int KPT = kPutTile / kPutThreads;  // keys per thread
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  constexpr int NG = (NT / 64) * RPW;
  using V = typename VecT<VEC>::T;
  __shared__ uint32_t s_hist[kMaxParts];
  __shared__ unsigned long long s_hkey[kTileHash];  // key of each hash slot
  __shared__ uint32_t s_hcnt[kTileHash];            // occurrences of the key in the tile
  __shared__ uint32_t s_hfirst[kTileHash];          // first entry holding the key
  __shared__ uint32_t s_hcur[kTileHash];            // fill cursor of the key's entry list
  __shared__ uint16_t s_hdup[kTileHash];            // index of a repeated key
  __shared__ uint16_t s_lanes[kPutTile];            // entries of repeated keys, grouped
  __shared__ uint16_t s_doff[kPutTile / 2 + 1];     // start of each repeated key's entries
  __shared__ uint32_t s_w[NT / 64];
  __shared__ uint32_t s_cnt;
  const int NP = 1 << pb;
  const int tid = threadIdx.x;
  const int tile = blockIdx.x;
  const int64_t base = (int64_t)tile * tlen;        // batch position of the tile's entry 0
  const int64_t sbase = (int64_t)tile * kPutTile;   // the tile's slots in items / newlist
  if (tile == 0 && tid == 0) ctrl->spill_next = 0;
  for (int d = tid; d < NP; d += NT) s_hist[d] = 0;
  for (int h = tid; h < kTileHash; h += NT) {
    s_hkey[h] = ~0ull;
    s_hcnt[h] = 0;
    s_hfirst[h] = 0xFFFFFFFFu;
    s_hcur[h] = 0;
  }
  if (tid == 0) s_cnt = 0;

  // entry e = kk * NT + tid of the tile is batch position base + e. The
  // index buckets of the tile's keys are loaded first; while they are in
  // flight the tile's keys are deduplicated in LDS (a key and its slot are
  // one to one), and the probe reads the buckets afterwards.
  // a key that the last get found present at the same position takes the
  // row it found there; the others load their home bucket
  uint64_t key[KPT];
  bool inb[KPT];
  uint64_t hb[KPT];
  BucketView bv[KPT];
  uint64_t ck[KPT];
  uint32_t crow[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    const int64_t i = base + kk * NT + tid;
    inb[kk] = kk * NT + tid < tlen && i < n;
    key[kk] = inb[kk] ? keys[i] : kEmptyKey;
    ck[kk] = inb[kk] ? pc_key[i] : kEmptyKey;
    crow[kk] = inb[kk] ? pc_row[i] : kPendingRow;
  }
  bool cached[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    cached[kk] = key[kk] != kEmptyKey && ck[kk] == key[kk];
    if (key[kk] != kEmptyKey && !cached[kk]) {
      hb[kk] = home_bucket(key[kk], nb_log2);
      bv[kk] = load_bucket(idx + hb[kk]);
    }
  }
  lds_barrier();  // the hash table is initialised

  uint32_t hs[KPT];
  bool valid[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    const int e = kk * NT + tid;
    valid[kk] = key[kk] != kEmptyKey;
    // count the tile's occurrences of every key
    hs[kk] = 0;
    if (valid[kk]) {
      uint32_t h = (uint32_t)index_hash(key[kk]) & (kTileHash - 1);
      while (true) {
        const unsigned long long old = atomicCAS(&s_hkey[h], ~0ull, (unsigned long long)key[kk]);
        if (old == ~0ull || old == key[kk]) break;
        h = (h + 1) & (kTileHash - 1);
      }
      hs[kk] = h;
      atomicAdd(&s_hcnt[h], 1u);
      atomicMin(&s_hfirst[h], (uint32_t)e);
    }
  }
  lds_barrier();
  // a key repeated in the tile ("dup") gets the sorted list of its entries;
  // one repeated at least dup_min times is merged into one item (an
  // assignment keeps the last position; a sum adds the key's gradient rows
  // here, in fp64), the entries of the others stay items of their own, which
  // the key's first entry emits together in position order
  const uint32_t dup_min = op == kOpAssign ? 2u : (uint32_t)kPresumMin;
  uint32_t cnt[KPT];
  bool dup[KPT], merged[KPT], owner[KPT];
  uint32_t n_own = 0, l_own = 0;
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    const int e = kk * NT + tid;
    cnt[kk] = valid[kk] ? s_hcnt[hs[kk]] : 0u;
    dup[kk] = cnt[kk] >= 2;
    merged[kk] = cnt[kk] >= dup_min;
    owner[kk] = dup[kk] && s_hfirst[hs[kk]] == (uint32_t)e;
    n_own += owner[kk] ? 1u : 0u;
    l_own += owner[kk] ? cnt[kk] : 0u;
  }

  // repeated groups: index them, then list their entries contiguously. The
  // in-tile sums below take one work item per repeated key, or, for a key
  // with more than kSumChunk entries, one per chunk of kSumChunk entries.
  constexpr int UNR = (K * VEC >= 16) ? 2 : (K * VEC >= 8) ? 4 : 8;  // rows loaded together
  constexpr uint32_t kSumChunk = 2 * UNR;
  auto n_items = [](uint32_t c) { return c <= kSumChunk ? 1u : (c + kSumChunk - 1) / kSumChunk; };
  uint32_t w_own = 0;
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) w_own += owner[kk] && merged[kk] ? n_items(cnt[kk]) : 0u;
  // one scan for the three prefixes, packed 10 | 11 | 11 bits (a tile holds
  // at most 512 repeated keys and 1024 entries, so no field overflows)
  static_assert(kPutTile <= 1024, "packed prefix fields");
  uint32_t ptot;
  const uint32_t ppre = block_exclusive_scan<NT>(n_own | (l_own << 10) | (w_own << 21), s_w, &ptot);
  const uint32_t ndup = ptot & 0x3FFu, nlanes = (ptot >> 10) & 0x7FFu, nwork = ptot >> 21;
  uint32_t dpre = ppre & 0x3FFu, lpre = (ppre >> 10) & 0x7FFu, wpre = ppre >> 21;
  uint32_t my_d[KPT], my_w[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    my_d[kk] = dpre;
    my_w[kk] = wpre;
    if (owner[kk]) {
      s_hdup[hs[kk]] = (uint16_t)dpre;
      s_doff[dpre] = (uint16_t)lpre;
      ++dpre;
      lpre += cnt[kk];
      wpre += merged[kk] ? n_items(cnt[kk]) : 0u;
    }
  }
  if (tid == 0) s_doff[ndup] = (uint16_t)nlanes;
  lds_barrier();
  uint32_t my_off[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    my_off[kk] = 0;
    if (dup[kk]) {
      my_off[kk] = s_doff[s_hdup[hs[kk]]];
      s_lanes[my_off[kk] + atomicAdd(&s_hcur[hs[kk]], 1u)] = (uint16_t)(kk * NT + tid);
    }
  }
  lds_barrier();
  // first work item of each repeated key (the fill cursors are no longer needed)
  uint16_t* s_wfirst = reinterpret_cast<uint16_t*>(s_hcur);
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk)
    if (owner[kk]) s_wfirst[my_d[kk]] = (uint16_t)my_w[kk];
  if (tid == 0) s_wfirst[ndup] = (uint16_t)nwork;
  // sort each repeated group's entry list: an entry's rank is the number of
  // smaller entries in its group's list
  uint32_t rank[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    rank[kk] = 0;
    if (dup[kk]) {
      const uint32_t e = kk * NT + tid;
      for (uint32_t m = 0; m < cnt[kk]; ++m) rank[kk] += s_lanes[my_off[kk] + m] < e ? 1u : 0u;
    }
  }
  lds_barrier();
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk)
    if (dup[kk]) s_lanes[my_off[kk] + rank[kk]] = (uint16_t)(kk * NT + tid);
  lds_barrier();

  // each lane group sums the rows of repeated keys, positions ascending (an
  // assignment needs no sum: its item is the key's last position instead).
  // Work items are dealt to the groups in turn. A key of at most kSumChunk
  // entries leaves its fp64 sum over the partials row of its first entry; a
  // longer key's chunks leave partial sums over the rows of their own first
  // entries (the first chunk over the key's second entry), which are added
  // in chunk order at the end of the kernel.
  const int lane = tid & 63;
  const int g = lane / LPR;
  const int q = lane % LPR;
  const int gid = (tid >> 6) * RPW + g;
  // some merged key has more than kSumChunk entries
  bool my_chunked = false;
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) my_chunked |= owner[kk] && cnt[kk] > kSumChunk;
  const bool chunked = __syncthreads_or(my_chunked ? 1 : 0) != 0;
  double acc[K][VEC];
  auto store_row = [&](uint32_t entry) {
    double* dst = partials + (size_t)(base + s_lanes[entry]) * (size_t)D;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
#pragma unroll
      for (int v = 0; v < VEC; ++v)
        if (col + v < D) dst[col + v] = acc[k][v];
    }
  };
  if (op != kOpAssign) {
    for (uint32_t w = gid; w < nwork; w += NG) {
      // the key of item w: the last d with s_wfirst[d] <= w (keys that are
      // not merged have no work item and share the next key's first one)
      uint32_t d = 0, dh = ndup;
      while (d + 1 < dh) {
        const uint32_t mid = (d + dh) >> 1;
        if (s_wfirst[mid] <= w) d = mid;
        else dh = mid;
      }
      const uint32_t c = w - s_wfirst[d];
      const uint32_t kb = s_doff[d], kend = s_doff[d + 1];
      const bool whole = kend - kb <= kSumChunk;
      const uint32_t b = kb + c * kSumChunk, e = whole ? kend : min(b + kSumChunk, kend);
#pragma unroll
      for (int k = 0; k < K; ++k)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[k][v] = 0.0;
      for (uint32_t j = b; j < e; j += UNR) {
        V gv[UNR][K];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          if (j + u < e) {
            const float* gr = grads + (size_t)(base + s_lanes[j + u]) * (size_t)D;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int col = (k * LPR + q) * VEC;
              if (col < D) gv[u][k] = load_vec<VEC>(gr + col);
            }
          }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
          if (j + u < e) {
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int col = (k * LPR + q) * VEC;
              if (col < D) {
#pragma unroll
                for (int v = 0; v < VEC; ++v) acc[k][v] += (double)VecT<VEC>::get(gv[u][k], v);
              }
            }
          }
        }
      }
      store_row(whole ? kb : (c == 0 ? kb + 1 : b));
    }
  }

  // probe (and insert) each key now that its bucket has arrived
  Probe pr[KPT];
  // ahead of a get: the size word that get starts from (it writes the other)
  const uint64_t size_before = kAhead ? ctrl->size[(epoch + 1) & 1] : 0ull;
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    pr[kk] = {0, kPendingRow, inb[kk] ? P_BAD : P_NONE};
    if (cached[kk]) {
      pr[kk] = {0, crow[kk], P_HIT};
    } else if (key[kk] != kEmptyKey) {
      pr[kk] = probe_with(idx, nb_log2, key[kk], !kAhead, hb[kk], bv[kk]);
      if constexpr (kAhead) {
        if (pr[kk].status != P_HIT || pr[kk].row >= size_before) {
          pr[kk].status = P_ABSENT;
          ctrl->apput_absent_epoch = epoch;
        }
      } else {
        if (pr[kk].status == P_OVERFLOW) ctrl->overflow_epoch = epoch;
      }
    } else if (pr[kk].status == P_BAD) {
      if constexpr (kAhead) ctrl->apput_bad_epoch = epoch;
      else ctrl->bad_epoch = epoch;
    }
  }
  uint64_t x[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    const int e = kk * NT + tid;
    valid[kk] = pr[kk].status == P_HIT || pr[kk].status == P_NEW_MINE || pr[kk].status == P_NEW_OTHER;
    if (pr[kk].status == P_NEW_MINE) {
      const uint32_t j = atomicAdd(&s_cnt, 1u);
      newlist[(size_t)sbase + j] = NewKey{key[kk], pr[kk].slot, 0u};
      ctrl->new_epoch = epoch;
    }
    const bool fresh = pr[kk].status != P_HIT;
    uint32_t pos = (uint32_t)(base + e);
    if (op == kOpAssign && owner[kk]) pos = (uint32_t)(base + s_lanes[s_doff[s_hdup[hs[kk]] + 1] - 1]);
    x[kk] = valid[kk] ? make_item(fresh, fresh ? pr[kk].slot : pr[kk].row, pos) : ~0ull;
  }

  // emit single positions, one item per merged key, and the entries of each
  // other repeated key together, in position order, from its first entry
  bool emit[KPT];
  uint32_t d[KPT], r[KPT], ne[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    emit[kk] = valid[kk] && (!dup[kk] || owner[kk]);
    ne[kk] = dup[kk] && !merged[kk] ? cnt[kk] : 1u;
    d[kk] = 0;
    r[kk] = 0;
    if (emit[kk]) {
      d[kk] = group_partition(item_group(x[kk]), pb);
      r[kk] = atomicAdd(&s_hist[d[kk]], ne[kk]);
    }
  }
  lds_barrier();
  constexpr int PER = kMaxParts / NT;
  uint32_t c[PER];
  uint32_t sum = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int dd = tid * PER + j;
    c[j] = dd < NP ? s_hist[dd] : 0u;
    sum += c[j];
  }
  uint32_t tot;
  uint32_t off = block_exclusive_scan<NT>(sum, s_w, &tot);
  uint32_t offs[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int dd = tid * PER + j;
    offs[j] = off;
    if (dd < NP) meta[(size_t)dd * ntiles + tile] = off | (c[j] << 16);
    off += c[j];
  }
  lds_barrier();
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int dd = tid * PER + j;
    if (dd < NP) s_hist[dd] = offs[j];
  }
  lds_barrier();
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    if (!emit[kk]) continue;
    uint64_t* dst = items + (size_t)sbase + s_hist[d[kk]] + r[kk];
    if (dup[kk] && !merged[kk]) {
      const uint32_t kb = s_doff[s_hdup[hs[kk]]];
      for (uint32_t i = 0; i < cnt[kk]; ++i)
        dst[i] = (x[kk] & ~0x7FFFFFFFull) | (uint64_t)(uint32_t)(base + s_lanes[kb + i]);
    } else {
      dst[0] = merged[kk] && op != kOpAssign ? (x[kk] | kItemSummed) : x[kk];
    }
  }
  if (!kAhead && tid == 0) tile_cnt[tile] = s_cnt;  // ahead of a get, the counts are the get's
  // keys summed in chunks: add the chunks' partial sums in order
  if (op != kOpAssign && chunked) {
    __syncthreads();
    for (uint32_t d = gid; d < ndup; d += NG) {
      const uint32_t kb = s_doff[d], kend = s_doff[d + 1];
      if (kend - kb <= kSumChunk) continue;
#pragma unroll
      for (int k = 0; k < K; ++k)
#pragma unroll
        for (int v = 0; v < VEC; ++v) acc[k][v] = 0.0;
      for (uint32_t b = kb; b < kend; b += kSumChunk) {
        const double* src = partials + (size_t)(base + s_lanes[b == kb ? kb + 1 : b]) * (size_t)D;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
#pragma unroll
          for (int v = 0; v < VEC; ++v)
            if (col + v < D) acc[k][v] += src[col + v];
        }
      }
      store_row(kb);
    }
  }
}

// ---------------------------------------------------------------------------
// Segment sums and row updates (shared by put_reduce and its spill path)
// ---------------------------------------------------------------------------

// Sum over the LPR lanes of a lane group (LPR a power of two, groups aligned);
// every lane of the group receives the same value. Steps within 16 lanes use
// DPP moves, wider steps lane shuffles.
template <int LPR>
__device__ __forceinline__ double group_sum(double x) {
  auto dpp = [](double v, auto ctrl_tag) {
    constexpr int ctrl = decltype(ctrl_tag)::value;
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), ctrl, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), ctrl, 0xF, 0xF, false);
    return __hiloint2double(hi, lo);
  };
  using Xor1 = std::integral_constant<int, 0xB1>;       // quad_perm [1,0,3,2]
  using Xor2 = std::integral_constant<int, 0x4E>;       // quad_perm [2,3,0,1]
  using HalfMirror = std::integral_constant<int, 0x141>;  // row_half_mirror
  using Mirror = std::integral_constant<int, 0x140>;      // row_mirror
  if constexpr (LPR >= 2) x += dpp(x, Xor1{});
  if constexpr (LPR >= 4) x += dpp(x, Xor2{});
  if constexpr (LPR >= 8) x += dpp(x, HalfMirror{});
  if constexpr (LPR >= 16) x += dpp(x, Mirror{});
  if constexpr (LPR >= 32) x += __shfl_xor(x, 16, 64);
  if constexpr (LPR >= 64) x += __shfl_xor(x, 32, 64);
  return x;
}

template <class M>
struct SegmentOps {
  static constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  using V = typename VecT<VEC>::T;

  // Row-wise Adagrad step of one row, given its summed gradient g (fp32):
  // m = fp32(sum g^2 / D) over the group's lanes; G' = G + m;
  // den = sqrt(G') + eps; w -= lr * (g / den); writes w and G'.
  static __device__ __forceinline__ void adagrad(const V (&g)[K], V (&w)[K], float G, float* __restrict__ wrow,
                                                 float* __restrict__ state, uint32_t row, int D, int q,
                                                 bool d_pow2, double inv_d, float lr, float eps) {
    double sq = 0.0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
#pragma unroll
      for (int x = 0; x < VEC; ++x) {
        const double gx = (double)VecT<VEC>::get(g[k], x);
        if (col + x < D) sq += gx * gx;
      }
    }
    sq = group_sum<LPR>(sq);
    // D a power of two: multiplying by 1/D is exact, hence equal to sq / D
    const float m = (float)(d_pow2 ? sq * inv_d : sq / (double)D);
    const float Gn = __fadd_rn(G, m);
    const float den = __fadd_rn(__builtin_sqrtf(Gn), eps);  // correctly rounded sqrt
    // g / den: a correctly rounded IEEE quotient per element, so that den = 0
    // (eps = 0 with an underflowing m), subnormal denominators and overflowing
    // quotients give the same infinities and NaNs as a plain fp32 division
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
      if (col < D) {
#pragma unroll
        for (int x = 0; x < VEC; ++x) {
          const float gx = VecT<VEC>::get(g[k], x);
          const float qv = __fdiv_rn(gx, den);
          const float p = __fmul_rn(lr, qv);
          VecT<VEC>::set(w[k], x, __fsub_rn(VecT<VEC>::get(w[k], x), p));
        }
        store_vec<VEC>(wrow + col, w[k]);
      }
    }
    if (q == 0) state[row] = Gn;
  }

  // One SGD step: w -= lr * g (separate fp32 operations).
  static __device__ __forceinline__ void sgd(const V (&g)[K], V (&w)[K], float* __restrict__ wrow, int D, int q,
                                             float lr) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
      if (col < D) {
#pragma unroll
        for (int x = 0; x < VEC; ++x)
          VecT<VEC>::set(w[k], x, __fsub_rn(VecT<VEC>::get(w[k], x), __fmul_rn(lr, VecT<VEC>::get(g[k], x))));
        store_vec<VEC>(wrow + col, w[k]);
      }
    }
  }

  // The row becomes g.
  static __device__ __forceinline__ void assign(const V (&g)[K], float* __restrict__ wrow, int D, int q) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
      if (col < D) store_vec<VEC>(wrow + col, g[k]);
    }
  }

  // The update of op for one row; w and G are the row's current values
  // (not read for kOpAssign, G only for kOpAdagrad).
  static __device__ __forceinline__ void update(int op, const V (&g)[K], V (&w)[K], float G,
                                                float* __restrict__ wrow, float* __restrict__ state,
                                                uint32_t row, int D, int q, bool d_pow2, double inv_d, float lr,
                                                float eps) {
    if (op == kOpAdagrad) adagrad(g, w, G, wrow, state, row, D, q, d_pow2, inv_d, lr, eps);
    else if (op == kOpSgd) sgd(g, w, wrow, D, q, lr);
    else assign(g, wrow, D, q);
  }

  static __device__ __forceinline__ void zero(double (&acc)[K][VEC]) {
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int x = 0; x < VEC; ++x) acc[k][x] = 0.0;
  }

  // g = fp32(acc) over the fp64 partials row at position pos (that row is no
  // longer read once its segment is summed).
  static __device__ __forceinline__ void store_g(const double (&acc)[K][VEC], const double* partials,
                                                 uint32_t pos, int D, int q) {
    float* gp = reinterpret_cast<float*>(const_cast<double*>(partials) + (size_t)pos * (size_t)D);
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
      if (col < D) {
        V v;
#pragma unroll
        for (int x = 0; x < VEC; ++x) VecT<VEC>::set(v, x, (float)acc[k][x]);
        store_vec<VEC>(gp + col, v);
      }
    }
  }
};

struct RedCtx {
  int op;
  Bucket* idx;
  const float* grads;
  const double* partials;
  RowStore store;
  float* state;
  int D;
  uint64_t seed;
  float lr;
  float eps;
  uint64_t size0;
  unsigned long long* clock;  // staleness words, or nullptr
};

// A put completes one served get on the row (bounded staleness, Sec.
// III-C1): its count drops by one, never below 0. One lane per row.
__device__ __forceinline__ void put_clock(unsigned long long* __restrict__ clock, uint32_t row) {
  const unsigned long long w = clock[row];
  if ((w & kClockCount) != 0) clock[row] = w - 1;
}

// The same from the low 32 bits of the word, loaded ahead with the row: they
// hold the count (a nonzero count drops without borrowing from the epoch
// bits above it, so only the low word is written).
static_assert(kClockBits < 32, "the count fits the low word of a staleness word");
__device__ __forceinline__ uint32_t clock_low(const unsigned long long* __restrict__ clock, uint32_t row) {
  return reinterpret_cast<const uint32_t*>(clock + row)[0];  // little-endian: the low word comes first
}
__device__ __forceinline__ void put_clock_low(unsigned long long* __restrict__ clock, uint32_t row, uint32_t lo) {
  if ((lo & (uint32_t)kClockCount) != 0u) reinterpret_cast<uint32_t*>(clock + row)[0] = lo - 1u;
}

// Run-length encodes items sorted by value: seg[s] = first item of segment s,
// seg[S] = mp, sid[j] = segment of item j. Returns S (block-uniform).
template <int NT, class IP, class SP, class DP>
__device__ __forceinline__ uint32_t encode_segments(IP it, uint32_t mp, SP seg, DP sid, uint32_t* s_w) {
  uint32_t S = 0;
  for (uint32_t b0 = 0; b0 < mp; b0 += NT) {
    const uint32_t j = b0 + threadIdx.x;
    const uint32_t head = (j < mp) && (j == 0 || item_group(it[j]) != item_group(it[j - 1])) ? 1u : 0u;
    uint32_t tot;
    const uint32_t pre = block_exclusive_scan<NT>(head, s_w, &tot);
    if (head) seg[S + pre] = j;
    if (j < mp) sid[j] = S + pre + head - 1;
    S += tot;
  }
  if (threadIdx.x == 0) seg[S] = mp;
  __syncthreads();
  return S;
}

// Keys new in this call (fresh items) get their rows: row = size + rank of
// the key among all new keys of the call. The block's new keys (up to NT at a
// time) are sorted in LDS; every new key of the call, streamed through LDS,
// adds one to the count of the first of them above it, and a key's rank is
// the sum of the counts up to its own position. Initial row and zero
// accumulator are written, and the row replaces the slot in the segment's
// first item, whose "fresh" bit stays set. s_chunk: at least (kChunk + NT)
// 64-bit words plus NT + 1 32-bit words of LDS.
template <int NT, class IP, class SP>
__device__ __forceinline__ void resolve_new_rows(IP it, SP seg, uint32_t S, const RedCtx& c,
                                                 const NewKey* __restrict__ newlist,
                                                 const uint32_t* __restrict__ tile_cnt, int ntiles,
                                                 uint32_t* s_pref, uint32_t* s_w,
                                                 unsigned long long* s_w64, uint64_t* s_chunk) {
  uint64_t* s_pk = s_chunk + kChunk;                          // [NT] the batch's new keys, sorted
  uint32_t* s_cnt = reinterpret_cast<uint32_t*>(s_pk + NT);  // [NT + 1] counts, then their prefix
  for (uint32_t s0 = 0; s0 < S; s0 += NT) {
    const uint32_t s = s0 + threadIdx.x;
    bool pend = false;
    uint32_t slot = 0;
    uint64_t x = 0;
    if (s < S) {
      x = it[seg[s]];
      pend = item_fresh(x);
      slot = item_tag(x);
    }
    uint32_t np;
    const uint32_t pi = block_exclusive_scan<NT>(pend ? 1u : 0u, s_w, &np);
    if (np == 0) continue;
    const uint64_t key = pend ? c.idx[slot / kSlots].key[slot % kSlots] : 0ull;
    uint32_t np2 = 1;
    while (np2 < np) np2 <<= 1;
    for (uint32_t j = threadIdx.x; j < np2; j += NT) s_pk[j] = kEmptyKey;  // no key equals it
    for (uint32_t j = threadIdx.x; j <= np; j += NT) s_cnt[j] = 0;
    __syncthreads();
    if (pend) s_pk[pi] = key;
    __syncthreads();
    block_bitonic_sort<NT>(s_pk, np2);
    for_each_new_key_chunk<NT>(newlist, tile_cnt, ntiles, kPutTile, s_pref, s_w, s_chunk,
                               [&](const uint64_t* ck, uint32_t cnt) {
                                 for (uint32_t e = threadIdx.x; e < cnt; e += NT) {
                                   const uint64_t xk = ck[e];
                                   uint32_t lo = 0, hi = np;  // first pending key above xk
                                   while (lo < hi) {
                                     const uint32_t mid = (lo + hi) >> 1;
                                     if (s_pk[mid] <= xk) lo = mid + 1;
                                     else hi = mid;
                                   }
                                   if (lo < np) atomicAdd(&s_cnt[lo], 1u);
                                 }
                               });
    {
      const uint32_t v = threadIdx.x < np ? s_cnt[threadIdx.x] : 0u;
      uint32_t tot;
      const uint32_t ex = block_exclusive_scan<NT>(v, s_w, &tot);
      if (threadIdx.x < np) s_cnt[threadIdx.x] = ex + v;  // new keys below the key at this position
      __syncthreads();
    }
    if (pend) {
      uint32_t lo = 0, hi = np - 1;  // the key's own position
      while (lo < hi) {
        const uint32_t mid = (lo + hi) >> 1;
        if (s_pk[mid] < key) lo = mid + 1;
        else hi = mid;
      }
      const uint32_t rank = s_cnt[lo];
      const uint32_t row = (uint32_t)(c.size0 + rank);
      c.idx[slot / kSlots].row[slot % kSlots] = row;
      it[seg[s]] = make_item(true, row, item_low31(x));
      const uint64_t s0k = splitmix_mix(key ^ c.seed);
      float* w = c.store.wptr(row);
      for (int col = 0; col < c.D; ++col) w[col] = init_elem(s0k, col);
      c.state[row] = 0.0f;
    }
    __syncthreads();
  }
  __syncthreads();
}

// Update, phase A: the fp64 sum of every segment that needs one (more than
// one item, or an in-tile sum as its only item) over items [0, mA), written
// as fp32 g over the partials row of the segment's first item. Each lane
// group takes an equal contiguous slice of the items and walks it in batches
// (all gradient rows of a batch are loaded together). The piece of a segment
// that began before the slice goes to s_part[group]; after a barrier, the
// group where a cut segment began adds the pieces of the following groups in
// slice order.
template <class M, int NT, class IP, class SP, class DP>
__device__ __forceinline__ void sum_segments(IP it, SP seg, DP sid, uint32_t mA, const RedCtx& c,
                                             double* s_part) {
  using Ops = SegmentOps<M>;
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  constexpr int NG = (NT / 64) * RPW;
  constexpr int B = (K * VEC >= 8) ? 2 : 4;
  using V = typename VecT<VEC>::T;
  const int lane = threadIdx.x & 63;
  const int g = lane / LPR;
  const int q = lane % LPR;
  const int gid = (threadIdx.x >> 6) * RPW + g;
  const int D = c.D;

  const uint32_t L = (mA + NG - 1) / NG;
  const uint32_t lo = min(mA, (uint32_t)gid * L);
  const uint32_t hi = min(mA, lo + L);

  double acc[K][VEC];
  Ops::zero(acc);
  for (uint32_t j0 = lo; j0 < hi; j0 += B) {
    V gv[B][K];
    double pv[B][K][VEC];
    uint32_t first[B];
    bool use[B], ends[B], owned[B], summ[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t j = j0 + u;
      use[u] = false;
      ends[u] = false;
      owned[u] = false;
      summ[u] = false;
      first[u] = 0;
      if (j < hi) {
        const uint64_t x = it[j];
        const uint32_t sj = sid[j];
        const uint32_t b = seg[sj], e = seg[sj + 1];
        summ[u] = item_summed(x);
        use[u] = (e - b > 1) || summ[u];
        ends[u] = e == j + 1;
        owned[u] = b >= lo;
        first[u] = b;
        if (use[u]) {
          if (summ[u]) {
            const double* pr = c.partials + (size_t)item_pos(x) * (size_t)D;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int col = (k * LPR + q) * VEC;
#pragma unroll
              for (int v = 0; v < VEC; ++v)
                if (col + v < D) pv[u][k][v] = pr[col + v];
            }
          } else {
            const float* gr = c.grads + (size_t)item_pos(x) * (size_t)D;
#pragma unroll
            for (int k = 0; k < K; ++k) {
              const int col = (k * LPR + q) * VEC;
              if (col < D) gv[u][k] = load_vec<VEC>(gr + col);
            }
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      if (!use[u]) continue;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int col = (k * LPR + q) * VEC;
        if (col < D) {
#pragma unroll
          for (int x = 0; x < VEC; ++x)
            acc[k][x] += summ[u] ? pv[u][k][x] : (double)VecT<VEC>::get(gv[u][k], x);
        }
      }
      if (ends[u]) {
        if (owned[u]) {
          Ops::store_g(acc, c.partials, item_pos(it[first[u]]), D, q);
        } else {
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int col = (k * LPR + q) * VEC;
#pragma unroll
            for (int x = 0; x < VEC; ++x)
              if (col + x < D) s_part[(size_t)gid * D + col + x] = acc[k][x];
          }
        }
        Ops::zero(acc);
      }
    }
  }
  // the slice ends inside a segment
  uint32_t tail = 0xFFFFFFFFu;
  if (lo < hi) {
    const uint32_t sl = sid[hi - 1];
    if (seg[sl + 1] > hi) {
      if (seg[sl] >= lo) {
        tail = sl;
      } else {
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
#pragma unroll
          for (int x = 0; x < VEC; ++x)
            if (col + x < D) s_part[(size_t)gid * D + col + x] = acc[k][x];
        }
      }
    }
  }
  __syncthreads();
  if (tail != 0xFFFFFFFFu) {
    const uint32_t end = seg[tail + 1];
    for (uint32_t h = gid + 1; h < (uint32_t)NG && h * L < end; ++h) {
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int col = (k * LPR + q) * VEC;
#pragma unroll
        for (int x = 0; x < VEC; ++x)
          if (col + x < D) acc[k][x] += s_part[(size_t)h * D + col + x];
      }
    }
    Ops::store_g(acc, c.partials, item_pos(it[seg[tail]]), D, q);
  }
  __syncthreads();
}

// Update, phase B: one Adagrad step per segment. Segments are dealt to lane
// groups in turn (group gid takes gid, gid + NG, ...), so the groups of a
// wave update rows together. g is read from the partials row phase A wrote,
// or from the segment's only gradient row.
template <class M, int NT, class IP, class SP>
__device__ __forceinline__ void update_segments(IP it, SP seg, uint32_t S, const RedCtx& c) {
  using Ops = SegmentOps<M>;
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  constexpr int NG = (NT / 64) * RPW;
  constexpr int BB = (K * VEC >= 8) ? 2 : 4;
  using V = typename VecT<VEC>::T;
  const int lane = threadIdx.x & 63;
  const int g = lane / LPR;
  const int q = lane % LPR;
  const int gid = (threadIdx.x >> 6) * RPW + g;
  const int D = c.D;
  const bool d_pow2 = (D & (D - 1)) == 0;
  const double inv_d = 1.0 / (double)D;

  for (uint32_t s0 = gid; s0 < S; s0 += (uint32_t)NG * BB) {
    V gf[BB][K], w[BB][K];
    float G[BB];
    uint32_t row[BB];
#pragma unroll
    for (int u = 0; u < BB; ++u) {
      const uint32_t s = s0 + u * NG;
      G[u] = 0.0f;
      row[u] = 0;
      if (s < S) {
        const uint32_t b = seg[s];
        const uint64_t x = it[b];
        row[u] = item_tag(x);
        const bool from_a = c.op != kOpAssign && ((seg[s + 1] - b > 1) || item_summed(x));
        // an assignment takes the value row at the key's last position
        const uint32_t pos = c.op == kOpAssign ? item_pos(it[seg[s + 1] - 1]) : item_pos(x);
        const float* src = from_a ? reinterpret_cast<const float*>(c.partials + (size_t)pos * (size_t)D)
                                  : c.grads + (size_t)pos * (size_t)D;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
          if (col < D) {
            gf[u][k] = load_vec<VEC>(src + col);
            w[u][k] = load_vec<VEC>(c.store.ptr(row[u]) + col);
          }
        }
        if (c.op == kOpAdagrad) G[u] = c.state[row[u]];
      }
    }
#pragma unroll
    for (int u = 0; u < BB; ++u) {
      if (s0 + u * NG < S) {
        Ops::update(c.op, gf[u], w[u], G[u], c.store.wptr(row[u]), c.state, row[u], D, q, d_pow2, inv_d, c.lr,
                    c.eps);
        if (c.clock != nullptr && q == 0) put_clock(c.clock, row[u]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Put, second kernel: one block per partition. The block gathers the
// partition's items, groups them by key in LDS with each key's items in
// ascending position, gives keys new in the call their rows, then sums every
// key's gradient rows in fp64 and applies the update to its row. A partition
// larger than the block's LDS share takes the global spill path.
// ---------------------------------------------------------------------------
template <class M>
struct ReduceCfg {
  static constexpr int DMAX = M::LPR * M::K * M::VEC;
  // the pieces of segments cut between lane groups (one fp64 row per group,
  // NT * K * VEC doubles) take 32 KiB at every row map
  static constexpr int NT = DMAX <= 256 ? 1024 : DMAX <= 512 ? 512 : 256;
  static constexpr int NG = (NT / 64) * M::RPW;
  // gradient rows a lane group has in flight in the sums, and rows it
  // updates at a time for keys seen once (at 1024 threads a lane has 128
  // registers: four rows in flight fit them without spilling)
  static constexpr int B = (M::K * M::VEC >= 16) ? 2 : (M::K * M::VEC >= 8 || NT >= 1024) ? 4 : 8;
  static constexpr int BS = B;
};

constexpr size_t align16(size_t x) { return (x + 15) & ~(size_t)15; }
constexpr int kMaxGroups = 256;  // lane groups of a reduce block at most
// Segments of more than kLongSeg items are put in order through a bitmask of
// their items' places in the gathered list (at most kMaskSegs of them per
// partition; others compare their items pairwise).
constexpr uint32_t kLongSeg = 32;
constexpr int kMaskSegs = 32;
constexpr int kMaskWords = kRedCap / 32;

// Dynamic LDS of a reduce block, in bytes. The first region (gathered items
// and grouping tables) is dead once the items are grouped; it then holds a
// chunk of new keys (rows for keys new in the call) and after that the
// pieces of cut segments.
template <int NT>
struct ReduceLds {
  static constexpr size_t it = 0;                                    // u64[kRedCap] gather order
  static constexpr size_t hidx = it + 8 * (size_t)kRedCap;            // u32[kRedHash]
  static constexpr size_t hcnt = hidx + 4 * (size_t)kRedHash;         // u32[kRedHash]
  static constexpr size_t inv = hcnt + 4 * (size_t)kRedHash;          // u16[kRedHash]
  static constexpr size_t slot = inv + 2 * (size_t)kRedHash;          // u16[kRedCap]
  static constexpr size_t ord = slot + 2 * (size_t)kRedCap;           // u16[kRedCap]
  static constexpr size_t reuse = align16(ord + 2 * (size_t)kRedCap);  // end of the reused region
  static constexpr size_t srt = reuse;                                // u64[kRedCap] grouped items
  static constexpr size_t seg = srt + 8 * (size_t)kRedCap;            // u32[kRedCap + 1]
  static constexpr size_t sid = align16(seg + 4 * ((size_t)kRedCap + 1));  // u16[kRedCap]
  static constexpr size_t lid = align16(sid + 2 * (size_t)kRedCap);   // u16[kRedCap] mask of each segment
  static constexpr size_t mask = align16(lid + 2 * (size_t)kRedCap);  // u32[kMaskSegs][kMaskWords]
  static constexpr size_t pref = align16(mask + 4 * (size_t)kMaskSegs * kMaskWords);  // u32[NT + 1]
  static constexpr size_t w = align16(pref + 4 * ((size_t)NT + 1));   // u32[NT / 64]
  static constexpr size_t w64 = align16(w + 4 * (size_t)(NT / 64));   // u64[NT / 64]
  static constexpr size_t misc = align16(w64 + 8 * (size_t)(NT / 64));  // u32[8]
  static constexpr size_t base = misc + 32;                           // u64
  static constexpr size_t slo = base + 16;                            // u32[kMaxGroups + 1]
  static constexpr size_t total = align16(slo + 4 * ((size_t)kMaxGroups + 1));
};

// Groups a partition's items by key in LDS.
// In:  it[0, mp), the partition's items in the order put_probe's tiles
//      listed them: tiles ascending, and within a tile a key's items
//      together in ascending position; so the items of each key appear in
//      position order (an in-tile sum is one item at the first position it
//      covers).
// Out: srt[0, mp) = the items grouped into segments, one per key, each
//      segment's items in ascending position; segments [0, SA) need a sum
//      (more than one item, or an in-tile sum as the only item) and hold the
//      items [0, MA); segments [SA, S) are single items that need none.
//      seg[s] = first item of segment s, seg[S] = mp; sid[i] = segment of
//      item i; info = {S, SA, MA, any key new in the call}.
// Segment order: keys go to an LDS hash table with linear probing. The set of
// occupied slots does not depend on the order of insertion, only which key
// sits where inside a run of occupied slots does; keys are therefore given
// the slots of their run in ascending order, and segments follow these
// places. Every order above thus depends only on the set of items.
template <int NT>
__device__ __forceinline__ void group_by_key(const uint64_t* it, uint32_t mp, uint64_t* srt, uint32_t* seg,
                                             uint16_t* sid, uint32_t* hidx, uint32_t* hcnt, uint16_t* inv,
                                             uint16_t* slot, uint16_t* ord, uint16_t* lid, uint32_t* mask,
                                             unsigned long long* s_w64, uint32_t* info) {
  constexpr int IPT = (kRedCap + NT - 1) / NT;
  constexpr int HPT = kRedHash / NT;
  static_assert(kRedHash % NT == 0 && kRedCap < kRedHash && kRedHash <= 65536, "grouping table sizes");
  constexpr uint32_t kNone = 0xFFFFFFFFu;
  constexpr uint32_t kMask = kRedHash - 1;
  const int tid = threadIdx.x;
  for (int h = tid; h < kRedHash; h += NT) {
    hidx[h] = kNone;
    hcnt[h] = 0u;
  }
  for (int w = tid; w < kMaskSegs * kMaskWords; w += NT) mask[w] = 0u;
  if (tid == 0) info[4] = 0u;  // masks handed out
  lds_barrier();

  // 1. one slot per key (the first item to take it), and its item count
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t j = tid + k * NT;
    if (j < mp) {
      const uint64_t gr = item_group(it[j]);
      uint32_t h = (uint32_t)index_hash(gr) & kMask;
      while (true) {
        const uint32_t old = atomicCAS(&hidx[h], kNone, j);
        if (old == kNone || item_group(it[old]) == gr) break;
        h = (h + 1) & kMask;
      }
      slot[j] = (uint16_t)h;
      atomicAdd(&hcnt[h], 1u);
    }
  }
  lds_barrier();

  // 2. the place of each key within its run of occupied slots (a run always
  // ends: fewer items than slots)
#pragma unroll
  for (int q = 0; q < HPT; ++q) {
    const uint32_t h = tid * HPT + q;
    const uint32_t j = hidx[h];
    if (j != kNone) {
      const uint64_t key = item_group(it[j]);
      uint32_t cs = h;
      while (hidx[(cs - 1) & kMask] != kNone) cs = (cs - 1) & kMask;
      uint32_t r = 0;
      for (uint32_t c = cs; hidx[c] != kNone; c = (c + 1) & kMask) r += item_group(it[hidx[c]]) < key ? 1u : 0u;
      inv[(cs + r) & kMask] = (uint16_t)h;
    }
  }
  lds_barrier();

  // 3. segment numbers and first items, places in order, segments that need
  // a sum first (one scan of three counts of 21 bits each)
  uint32_t cnt[HPT], hs[HPT];
  bool need[HPT], occ[HPT];
  uint64_t mine = 0;
  bool fresh = false;
#pragma unroll
  for (int q = 0; q < HPT; ++q) {
    const uint32_t pl = tid * HPT + q;
    occ[q] = hidx[pl] != kNone;  // occupied places are the occupied slots
    need[q] = false;
    cnt[q] = 0;
    hs[q] = 0;
    if (occ[q]) {
      hs[q] = inv[pl];
      const uint64_t x = it[hidx[hs[q]]];
      cnt[q] = hcnt[hs[q]];
      need[q] = cnt[q] > 1 || item_summed(x);
      fresh |= item_fresh(x);
      mine += need[q] ? (1ull | ((uint64_t)cnt[q] << 21)) : (1ull << 42);
    }
  }
  uint64_t tot;
  const uint64_t pre = block_exclusive_scan_u64<NT>(mine, s_w64, &tot);  // barriers: every read above is done
  constexpr uint64_t F = (1ull << 21) - 1;
  const uint32_t SA = (uint32_t)(tot & F), MA = (uint32_t)((tot >> 21) & F), S = SA + (uint32_t)(tot >> 42);
  uint32_t sa = (uint32_t)(pre & F), ia = (uint32_t)((pre >> 21) & F), sb = (uint32_t)(pre >> 42);
#pragma unroll
  for (int q = 0; q < HPT; ++q) {
    if (occ[q]) {
      uint32_t s, off;
      if (need[q]) {
        s = sa++;
        off = ia;
        ia += cnt[q];
      } else {
        s = SA + sb;
        off = MA + sb;
        ++sb;
      }
      seg[s] = off;
      hcnt[hs[q]] = off | (s << 16);
      hidx[hs[q]] = 0u;  // fill cursor
      uint32_t l = 0xFFFFu;
      if (cnt[q] > kLongSeg) {
        l = atomicAdd(&info[4], 1u);  // which mask a long segment gets does not matter
        if (l >= (uint32_t)kMaskSegs) l = 0xFFFFu;
      }
      lid[s] = (uint16_t)l;
    }
  }
  if (tid == 0) {
    seg[S] = mp;
    info[0] = S;
    info[1] = SA;
    info[2] = MA;
  }
  const bool any_fresh = __syncthreads_or(fresh ? 1 : 0) != 0;
  if (tid == 0) info[3] = any_fresh ? 1u : 0u;

  // 4. drop each item into its segment (any order within it); a long
  // segment also marks its items' places in its mask
  uint32_t sg[IPT];
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t j = tid + k * NT;
    sg[k] = 0;
    if (j < mp) {
      const uint32_t v = hcnt[slot[j]];
      sg[k] = v >> 16;
      ord[(v & 0xFFFFu) + atomicAdd(&hidx[slot[j]], 1u)] = (uint16_t)j;
      const uint32_t l = lid[sg[k]];
      if (l != 0xFFFFu) atomicOr(&mask[l * kMaskWords + (j >> 5)], 1u << (j & 31));
    }
  }
  lds_barrier();
  // 5. each item at its rank within its segment: the number of the segment's
  // items at earlier places (the items of a key come in position order)
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t j = tid + k * NT;
    if (j < mp) {
      const uint32_t b = seg[sg[k]], e = seg[sg[k] + 1];
      uint32_t r = 0;
      if (e - b > 1) {
        const uint32_t l = lid[sg[k]];
        if (l != 0xFFFFu) {
          const uint32_t* mw = mask + l * kMaskWords;
          const uint32_t wj = j >> 5;
          for (uint32_t w = 0; w < wj; ++w) r += __popc(mw[w]);
          r += __popc(mw[wj] & ((1u << (j & 31)) - 1u));
        } else {
          for (uint32_t i = b; i < e; ++i) r += ord[i] < j ? 1u : 0u;
        }
      }
      srt[b + r] = it[j];
      sid[b + r] = (uint16_t)sg[k];
    }
  }
  lds_barrier();
}

// One lane's VEC elements of a row, fp32 (a gradient row) or fp64 (an in-tile
// sum), as loaded.
template <int VEC>
struct RawRow;
template <>
struct RawRow<4> {
  uint4 lo, hi;
};
template <>
struct RawRow<1> {
  uint2 lo;
};

template <int VEC>
__device__ __forceinline__ void load_raw(RawRow<VEC>& r, const float* __restrict__ grads,
                                         const double* __restrict__ partials, size_t off, bool summed) {
  if constexpr (VEC == 4) {
    if (summed) {
      const uint4* p = reinterpret_cast<const uint4*>(partials + off);
      r.lo = p[0];
      r.hi = p[1];
    } else {
      r.lo = *reinterpret_cast<const uint4*>(grads + off);
    }
  } else {
    if (summed) r.lo = *reinterpret_cast<const uint2*>(partials + off);
    else r.lo.x = *reinterpret_cast<const uint32_t*>(grads + off);
  }
}

template <int VEC>
__device__ __forceinline__ void add_raw(double* acc, const RawRow<VEC>& r, bool summed) {
  if constexpr (VEC == 4) {
    if (summed) {
      acc[0] += __hiloint2double((int)r.lo.y, (int)r.lo.x);
      acc[1] += __hiloint2double((int)r.lo.w, (int)r.lo.z);
      acc[2] += __hiloint2double((int)r.hi.y, (int)r.hi.x);
      acc[3] += __hiloint2double((int)r.hi.w, (int)r.hi.z);
    } else {
      acc[0] += (double)__uint_as_float(r.lo.x);
      acc[1] += (double)__uint_as_float(r.lo.y);
      acc[2] += (double)__uint_as_float(r.lo.z);
      acc[3] += (double)__uint_as_float(r.lo.w);
    }
  } else {
    acc[0] += summed ? __hiloint2double((int)r.lo.y, (int)r.lo.x) : (double)__uint_as_float(r.lo.x);
  }
}

// One update step (op of c) for the rows rw[u] with on[u], given their summed
// gradients gq[u]: the rows (and accumulators) of the N keys are loaded
// together, updated and written back; a bounded table's counts drop (kClk:
// the table has staleness words).
template <class M, int N, bool kClk>
__device__ __forceinline__ void update_rows(const bool (&on)[N], const uint32_t (&rw)[N],
                                            const typename VecT<M::VEC>::T (&gq)[N][M::K], const RedCtx& c, int q,
                                            bool d_pow2, double inv_d) {
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K;
  using V = typename VecT<VEC>::T;
  const int D = c.D;
  V w[N][K];
  float G[N];
  float* wr[N];
  uint32_t cl[N];  // low words of the rows' staleness words (bounded tables)
  const bool clk = kClk && q == 0;
#pragma unroll
  for (int u = 0; u < N; ++u) {
    G[u] = 0.0f;
    wr[u] = nullptr;
    cl[u] = 0u;
    if (on[u]) {
      wr[u] = c.store.wptr(rw[u]);
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int col = (k * LPR + q) * VEC;
        if (col < D) w[u][k] = load_vec<VEC>(wr[u] + col);
      }
      if (c.op == kOpAdagrad) G[u] = c.state[rw[u]];
      if (clk) cl[u] = clock_low(c.clock, rw[u]);
    }
  }
#pragma unroll
  for (int u = 0; u < N; ++u)
    if (on[u]) {
      SegmentOps<M>::update(c.op, gq[u], w[u], G[u], wr[u], c.state, rw[u], D, q, d_pow2, inv_d, c.lr, c.eps);
      if (clk) put_clock_low(c.clock, rw[u], cl[u]);
    }
}

// Sums and updates of a grouped partition (update op != kOpAssign).
// Lane group gid takes an even share [lo, hi) of the items of segments that
// need a sum and walks it B items at a time (their gradient rows, and the row
// and accumulator of each segment starting among them, loaded together),
// accumulating in fp64; a segment that starts and ends in the share is updated
// as soon as it ends. The part of a segment begun in an earlier share goes to
// LDS (a group has at most one); after a barrier, the group where a segment
// cut between shares began adds the later parts in share order and updates
// it. Each group also updates an even share of the keys seen once (g is their
// gradient row).
template <class M, int NT, bool kClk>
__device__ __forceinline__ void sum_and_update(const uint64_t* srt, const uint32_t* seg, const uint16_t* sid,
                                               uint32_t S, uint32_t SA, uint32_t MA, const RedCtx& c,
                                               double* s_piece, uint32_t* s_slo) {
  using Ops = SegmentOps<M>;
  using Cfg = ReduceCfg<M>;
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K;
  constexpr int NG = Cfg::NG, B = Cfg::B, BS = Cfg::BS, DMAX = Cfg::DMAX;
  static_assert(NG <= kMaxGroups, "lane groups");
  using V = typename VecT<VEC>::T;
  const int lane = threadIdx.x & 63;
  const int q = lane % LPR;
  const int gid = (threadIdx.x >> 6) * M::RPW + lane / LPR;
  const int D = c.D;
  const bool d_pow2 = (D & (D - 1)) == 0;
  const double inv_d = 1.0 / (double)D;

  for (int h = threadIdx.x; h <= NG; h += NT) s_slo[h] = (uint32_t)((uint64_t)MA * h / NG);
  lds_barrier();
  const uint32_t lo = s_slo[gid], hi = s_slo[gid + 1];

  auto put_piece = [&](const double (&a)[K][VEC]) {
    double* dst = s_piece + (size_t)gid * DMAX;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
#pragma unroll
      for (int x = 0; x < VEC; ++x)
        if (col + x < D) dst[col + x] = a[k][x];
    }
  };
  auto to_f32 = [&](V (&g)[K], const double (&a)[K][VEC]) {
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int x = 0; x < VEC; ++x) VecT<VEC>::set(g[k], x, (float)a[k][x]);
  };
  // ---- segments that need a sum ----
  // The row and accumulator of a segment this group owns are loaded with the
  // batch that holds its first item; at most one segment is open at a time.
  double acc[K][VEC];
  Ops::zero(acc);
  V wc[K];
  float Gc = 0.0f;
  uint32_t Cc = 0u;  // low word of the open segment's staleness word (bounded tables)
  const bool clk = kClk && q == 0;
  uint32_t rowc = 0;
  float* wrc = nullptr;
  bool last_ends = true, last_owned = true;
  uint32_t last_end = 0;
  for (uint32_t j0 = lo; j0 < hi; j0 += B) {
    uint64_t x[B];
    uint32_t fst[B], end[B];
    RawRow<VEC> raw[B][K];
    V wl[B][K];
    float Gl[B];
    uint32_t Cl[B];
    float* wp[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t j = j0 + u;
      x[u] = 0;
      fst[u] = 0;
      end[u] = 0;
      Gl[u] = 0.0f;
      Cl[u] = 0u;
      wp[u] = nullptr;
      if (j < hi) {
        x[u] = srt[j];
        const uint32_t s = sid[j];
        fst[u] = seg[s];
        end[u] = seg[s + 1];
        const bool summ = item_summed(x[u]);
        const size_t base = (size_t)item_pos(x[u]) * (size_t)D;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
          if (col < D) load_raw<VEC>(raw[u][k], c.grads, c.partials, base + col, summ);
        }
        if (fst[u] == j && j >= lo) {  // an owned segment starts: its row (the first item carries it)
          const uint32_t r = item_tag(x[u]);
          wp[u] = c.store.wptr(r);
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int col = (k * LPR + q) * VEC;
            if (col < D) wl[u][k] = load_vec<VEC>(wp[u] + col);
          }
          if (c.op == kOpAdagrad) Gl[u] = c.state[r];
          if (clk) Cl[u] = clock_low(c.clock, r);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t j = j0 + u;
      if (j < hi) {
        if (fst[u] == j) {  // (j >= lo here)
          rowc = item_tag(x[u]);
          wrc = wp[u];
#pragma unroll
          for (int k = 0; k < K; ++k) wc[k] = wl[u][k];
          Gc = Gl[u];
          Cc = Cl[u];
        }
        const bool summ = item_summed(x[u]);
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
          if (col < D) add_raw<VEC>(acc[k], raw[u][k], summ);
        }
        last_ends = end[u] == j + 1;
        last_owned = fst[u] >= lo;
        last_end = end[u];
        if (last_ends) {
          if (last_owned) {
            V g[K];
            to_f32(g, acc);
            Ops::update(c.op, g, wc, Gc, wrc, c.state, rowc, D, q, d_pow2, inv_d, c.lr, c.eps);
            if (clk) put_clock_low(c.clock, rowc, Cc);
          } else {
            put_piece(acc);  // the end of a segment begun in an earlier share
          }
          Ops::zero(acc);
        }
      }
    }
  }
  const bool tail = lo < hi && !last_ends && last_owned;
  if (lo < hi && !last_ends && !last_owned) put_piece(acc);  // the share lies inside one segment

  // ---- keys seen once: g is the key's gradient row ----
  {
    const uint32_t S1 = S - SA;
    const uint32_t k0 = SA + (uint32_t)((uint64_t)S1 * gid / NG), k1 = SA + (uint32_t)((uint64_t)S1 * (gid + 1) / NG);
    for (uint32_t s0 = k0; s0 < k1; s0 += BS) {
      bool on[BS];
      uint32_t rw[BS];
      V gq[BS][K];
#pragma unroll
      for (int u = 0; u < BS; ++u) {
        const uint32_t s = s0 + u;
        on[u] = s < k1;
        rw[u] = 0;
        if (on[u]) {
          const uint64_t xs = srt[MA + (s - SA)];
          rw[u] = item_tag(xs);
          const float* gr = c.grads + (size_t)item_pos(xs) * (size_t)D;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int col = (k * LPR + q) * VEC;
            if (col < D) gq[u][k] = load_vec<VEC>(gr + col);
          }
        }
      }
      update_rows<M, BS, kClk>(on, rw, gq, c, q, d_pow2, inv_d);
    }
  }

  __syncthreads();  // the pieces of cut segments are in LDS
  if (tail) {
    // the segment ends in share hl: add the pieces of shares gid+1 .. hl in
    // order (an empty share holds none)
    uint32_t hl = gid + 1;
    while (hl + 1 < (uint32_t)NG && s_slo[hl + 1] < last_end) ++hl;
    for (uint32_t h = gid + 1; h <= hl; ++h) {
      if (s_slo[h] >= s_slo[h + 1]) continue;
      const double* src = s_piece + (size_t)h * DMAX;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int col = (k * LPR + q) * VEC;
#pragma unroll
        for (int xx = 0; xx < VEC; ++xx)
          if (col + xx < D) acc[k][xx] += src[col + xx];
      }
    }
    V g[K];
    to_f32(g, acc);  // the row, accumulator and staleness word came with the segment's first item
    Ops::update(c.op, g, wc, Gc, wrc, c.state, rowc, D, q, d_pow2, inv_d, c.lr, c.eps);
    if (clk) put_clock_low(c.clock, rowc, Cc);
  }
}

// Put with the assignment op: each key's row becomes the value row at its
// last position. Lane groups take even shares of the segments.
// An upsert whose keys were all present before the call: each key's row
// takes the value at the key's last position, so the partition needs no
// grouping, only the largest position per row (an LDS hash table from row to
// position + 1), then one write per row, lane groups taking equal shares of
// the rows in slot order.
constexpr uint32_t kNoRowKey = 0xFFFFFFFFu;  // an empty slot (no row has this id)
template <class M, int NT, bool kClk>
__device__ __forceinline__ void upsert_last(const uint64_t* __restrict__ it, uint32_t mp, const RedCtx& c,
                                            uint32_t* s_row, uint32_t* s_last, uint16_t* s_list, uint32_t* s_w) {
  static_assert(kRedHash == 4096 && kRedHash % NT == 0, "12-bit slot hash, whole slots per thread");
  for (uint32_t h = threadIdx.x; h < (uint32_t)kRedHash; h += NT) {
    s_row[h] = kNoRowKey;
    s_last[h] = 0u;
  }
  __syncthreads();
  for (uint32_t j = threadIdx.x; j < mp; j += NT) {
    const uint64_t x = it[j];
    const uint32_t row = item_tag(x);
    uint32_t h = (row * 0x9E3779B1u) >> 20;
    while (true) {
      const uint32_t old = atomicCAS(&s_row[h], kNoRowKey, row);
      if (old == kNoRowKey || old == row) break;
      h = (h + 1) & (kRedHash - 1);
    }
    atomicMax(&s_last[h], item_pos(x) + 1u);
  }
  __syncthreads();
  constexpr int PER = kRedHash / NT;
  uint32_t occ = 0;
#pragma unroll
  for (int e = 0; e < PER; ++e) occ += s_row[threadIdx.x * PER + e] != kNoRowKey ? 1u : 0u;
  uint32_t S;
  uint32_t at = block_exclusive_scan<NT>(occ, s_w, &S);
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const uint32_t h = threadIdx.x * PER + e;
    if (s_row[h] != kNoRowKey) s_list[at++] = (uint16_t)h;
  }
  __syncthreads();
  using Cfg = ReduceCfg<M>;
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, NG = Cfg::NG, BS = Cfg::BS;
  using V = typename VecT<VEC>::T;
  const int lane = threadIdx.x & 63;
  const int q = lane % LPR;
  const int gid = (threadIdx.x >> 6) * M::RPW + lane / LPR;
  const int D = c.D;
  const uint32_t k0 = (uint32_t)((uint64_t)S * gid / NG), k1 = (uint32_t)((uint64_t)S * (gid + 1) / NG);
  for (uint32_t s0 = k0; s0 < k1; s0 += BS) {
    V v[BS][K];
    uint32_t rw[BS], cl[BS];
    const bool clk = kClk && q == 0;
#pragma unroll
    for (int u = 0; u < BS; ++u) {
      const uint32_t sl = s0 + u;
      rw[u] = 0;
      cl[u] = 0u;
      if (sl < k1) {
        const uint32_t h = s_list[sl];
        rw[u] = s_row[h];
        const float* src = c.grads + (size_t)(s_last[h] - 1u) * (size_t)D;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
          if (col < D) v[u][k] = load_vec<VEC>(src + col);
        }
        if (clk) cl[u] = clock_low(c.clock, rw[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < BS; ++u) {
      if (s0 + u >= k1) continue;
      SegmentOps<M>::assign(v[u], c.store.wptr(rw[u]), D, q);
      if (clk) put_clock_low(c.clock, rw[u], cl[u]);
    }
  }
}

template <class M, int NT, bool kClk>
__device__ __forceinline__ void assign_segments(const uint64_t* srt, const uint32_t* seg, uint32_t S,
                                                const RedCtx& c) {
  using Cfg = ReduceCfg<M>;
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, NG = Cfg::NG, BS = Cfg::BS;
  using V = typename VecT<VEC>::T;
  const int lane = threadIdx.x & 63;
  const int q = lane % LPR;
  const int gid = (threadIdx.x >> 6) * M::RPW + lane / LPR;
  const int D = c.D;
  const uint32_t k0 = (uint32_t)((uint64_t)S * gid / NG), k1 = (uint32_t)((uint64_t)S * (gid + 1) / NG);
  for (uint32_t s0 = k0; s0 < k1; s0 += BS) {
    V v[BS][K];
    uint32_t rw[BS], cl[BS];
    const bool clk = kClk && q == 0;
#pragma unroll
    for (int u = 0; u < BS; ++u) {
      const uint32_t s = s0 + u;
      rw[u] = 0;
      cl[u] = 0u;
      if (s < k1) {
        rw[u] = item_tag(srt[seg[s]]);
        const float* src = c.grads + (size_t)item_pos(srt[seg[s + 1] - 1]) * (size_t)D;
#pragma unroll
        for (int k = 0; k < K; ++k) {
          const int col = (k * LPR + q) * VEC;
          if (col < D) v[u][k] = load_vec<VEC>(src + col);
        }
        if (clk) cl[u] = clock_low(c.clock, rw[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < BS; ++u) {
      if (s0 + u >= k1) continue;
      SegmentOps<M>::assign(v[u], c.store.wptr(rw[u]), D, q);
      if (clk) put_clock_low(c.clock, rw[u], cl[u]);
    }
  }
}

// Partition larger than the block's LDS share: the same steps on a global
// scratch area (bitonic sort in place).
template <class M, int NT>
__device__ __forceinline__ void reduce_partition_global(uint32_t p, uint32_t mp, const uint64_t* __restrict__ items,
                                                     const uint32_t* __restrict__ meta, int ntiles,
                                                     const RedCtx& c, const NewKey* __restrict__ newlist,
                                                     const uint32_t* __restrict__ tile_cnt, Ctrl* ctrl,
                                                     uint64_t* __restrict__ spill, uint64_t spill_words,
                                                     double* s_part, uint32_t* s_pref, uint32_t* s_w,
                                                     unsigned long long* s_w64, uint64_t* s_base) {
  uint32_t P2 = 1;
  while (P2 < mp) P2 <<= 1;
  if (threadIdx.x == 0) {
    const uint64_t need = 2ull * P2 + 2;
    const uint64_t b = atomicAdd(&ctrl->spill_next, (unsigned long long)need);
    *s_base = (b + need <= spill_words) ? b : ~0ull;
  }
  __syncthreads();
  const uint64_t base = *s_base;
  if (base == ~0ull) {  // cannot happen when the spill area holds 4n words
    if (threadIdx.x == 0) atomicCAS(&ctrl->latched, 0, -4);
    return;
  }
  uint64_t* it = spill + base;
  uint32_t* seg = reinterpret_cast<uint32_t*>(spill + base + P2);
  uint32_t* sid = seg + P2 + 1;
  uint32_t dst = 0;
  for (int t0 = 0; t0 < ntiles; t0 += NT) {
    const int t = t0 + (int)threadIdx.x;
    const uint32_t mt = t < ntiles ? meta[(size_t)p * ntiles + t] : 0u;
    const uint32_t off = mt & 0xFFFFu, cnt = mt >> 16;
    uint32_t tot;
    const uint32_t pre = block_exclusive_scan<NT>(cnt, s_w, &tot);
    for (uint32_t j = 0; j < cnt; ++j) it[dst + pre + j] = items[(size_t)t * kPutTile + off + j];
    dst += tot;
  }
  for (uint32_t j = mp + threadIdx.x; j < P2; j += NT) it[j] = ~0ull;
  __syncthreads();
  block_bitonic_sort<NT>(it, P2);
  const uint32_t S = encode_segments<NT>(it, mp, seg, sid, s_w);
  resolve_new_rows<NT>(it, seg, S, c, newlist, tile_cnt, ntiles, s_pref, s_w, s_w64,
                       reinterpret_cast<uint64_t*>(s_part));
  if (c.op != kOpAssign) sum_segments<M, NT>(it, seg, sid, mp, c, s_part);
  update_segments<M, NT>(it, seg, S, c);
}

// kUpsert: the instance for upserts (PutOp kOpAssign), whose partitions
// without keys new in the call take the value at each key's last position
// without grouping (upsert_last).
template <class M, int NT, bool kClk, bool kUpsert>
__global__ __launch_bounds__(NT) void k_put_reduce(
    Bucket* __restrict__ idx, const uint64_t* __restrict__ items, const uint32_t* __restrict__ meta,
    int ntiles, const NewKey* __restrict__ newlist, const uint32_t* __restrict__ tile_cnt,
    const float* __restrict__ grads, double* __restrict__ partials, const RowStore store,
    float* __restrict__ state, int D, uint64_t seed, float lr, float eps, int64_t capacity, Ctrl* ctrl,
    uint64_t epoch, uint64_t* __restrict__ spill, uint64_t spill_words, int op,
    unsigned long long* __restrict__ clock) {
  using L = ReduceLds<NT>;
  constexpr int IPT = (kRedCap + NT - 1) / NT;
  extern __shared__ __align__(16) unsigned char s_raw[];
  uint64_t* s_it = reinterpret_cast<uint64_t*>(s_raw + L::it);
  uint32_t* s_hidx = reinterpret_cast<uint32_t*>(s_raw + L::hidx);
  uint32_t* s_hcnt = reinterpret_cast<uint32_t*>(s_raw + L::hcnt);
  uint16_t* s_inv = reinterpret_cast<uint16_t*>(s_raw + L::inv);
  uint16_t* s_slot = reinterpret_cast<uint16_t*>(s_raw + L::slot);
  uint16_t* s_ord = reinterpret_cast<uint16_t*>(s_raw + L::ord);
  double* s_piece = reinterpret_cast<double*>(s_raw);       // reused region
  uint64_t* s_chunk = reinterpret_cast<uint64_t*>(s_raw);   // reused region
  uint64_t* s_srt = reinterpret_cast<uint64_t*>(s_raw + L::srt);
  uint32_t* s_seg = reinterpret_cast<uint32_t*>(s_raw + L::seg);
  uint16_t* s_sid = reinterpret_cast<uint16_t*>(s_raw + L::sid);
  uint16_t* s_lid = reinterpret_cast<uint16_t*>(s_raw + L::lid);
  uint32_t* s_mask = reinterpret_cast<uint32_t*>(s_raw + L::mask);
  uint32_t* s_pref = reinterpret_cast<uint32_t*>(s_raw + L::pref);
  uint32_t* s_w = reinterpret_cast<uint32_t*>(s_raw + L::w);
  unsigned long long* s_w64 = reinterpret_cast<unsigned long long*>(s_raw + L::w64);
  uint32_t* s_info = reinterpret_cast<uint32_t*>(s_raw + L::misc);
  uint64_t* s_base = reinterpret_cast<uint64_t*>(s_raw + L::base);
  uint32_t* s_slo = reinterpret_cast<uint32_t*>(s_raw + L::slo);

  const uint32_t p = blockIdx.x;
  const int tid = threadIdx.x;
  const uint64_t size0 = ctrl->size[epoch & 1];
  const uint64_t new_e = ctrl->new_epoch, ovf_e = ctrl->overflow_epoch;
  const uint64_t bad_e = ctrl->apput_bad_epoch == epoch ? epoch : ctrl->bad_epoch;
  const uint64_t abs_e = ctrl->apput_absent_epoch;
  const uint32_t* pm = meta + (size_t)p * ntiles;
  const bool one_chunk = ntiles <= NT;  // common case: one thread per tile
  const uint32_t mt0 = one_chunk && tid < ntiles ? pm[tid] : 0u;

  // entries of this partition in every tile
  uint32_t mp, pre0 = 0;
  if (one_chunk) {
    pre0 = block_exclusive_scan<NT>(mt0 >> 16, s_w, &mp);
  } else {
    uint64_t mp64 = 0;
    for (int t = tid; t < ntiles; t += NT) mp64 += pm[t] >> 16;
    mp = (uint32_t)block_sum_u64<NT>(mp64, s_w64);
  }

  const uint64_t Mnew = new_e == epoch ? count_new_keys<NT>(tile_cnt, ntiles, s_w64) : 0ull;
  const int err = call_verdict(ctrl, epoch, size0, Mnew, capacity, bad_e, ovf_e, abs_e);
  if (mp == 0) return;
  if (err) {
    if (Mnew == 0) return;
    // undo the insertions of this call whose slots fall in this partition
    for (int t = tid; t < ntiles; t += NT) {
      const uint32_t mt = pm[t];
      const uint32_t off = mt & 0xFFFFu, cnt = mt >> 16;
      for (uint32_t j = 0; j < cnt; ++j) {
        const uint64_t x = items[(size_t)t * kPutTile + off + j];
        if (item_fresh(x)) {
          const uint32_t slot = item_tag(x);
          idx[slot / kSlots].key[slot % kSlots] = kEmptyKey;
        }
      }
    }
    return;
  }

  const RedCtx c{op, idx, grads, partials, store, state, D, seed, lr, eps, size0, clock};
  if (mp > (uint32_t)kRedCap) {
    reduce_partition_global<M, NT>(p, mp, items, meta, ntiles, c, newlist, tile_cnt, ctrl, spill, spill_words,
                                   s_piece, s_pref, s_w, s_w64, s_base);
    return;
  }

  // ---- gather the partition's items into LDS, tile order ----
  {
    uint32_t dst = 0;
    for (int t0 = 0; t0 < ntiles; t0 += NT) {
      const int nt = min(NT, ntiles - t0);
      uint32_t mt = mt0, pre = pre0, tot = mp;
      if (!one_chunk) {
        mt = tid < nt ? pm[t0 + tid] : 0u;
        pre = block_exclusive_scan<NT>(mt >> 16, s_w, &tot);
      }
      s_pref[tid] = pre | (mt << 16);  // items before this tile | offset in the tile
      __syncthreads();
      uint64_t v[IPT];
#pragma unroll
      for (int e = 0; e < IPT; ++e) {
        const uint32_t k = tid + e * NT;
        v[e] = 0;
        if (k < tot) {
          int lo = 0, hi = nt - 1;
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((s_pref[mid] & 0xFFFFu) <= k) lo = mid;
            else hi = mid - 1;
          }
          const uint32_t pe = s_pref[lo];
          v[e] = items[(size_t)(t0 + lo) * kPutTile + (pe >> 16) + (k - (pe & 0xFFFFu))];
        }
      }
#pragma unroll
      for (int e = 0; e < IPT; ++e) {
        const uint32_t k = tid + e * NT;
        if (k < tot) s_it[dst + k] = v[e];
      }
      dst += tot;
      __syncthreads();
    }
  }

  if constexpr (kUpsert) {
    uint32_t fresh = 0;
    for (uint32_t j = tid; j < mp; j += NT) fresh |= item_fresh(s_it[j]) ? 1u : 0u;
    if (__syncthreads_or((int)fresh) == 0) {
      upsert_last<M, NT, kClk>(s_it, mp, c, s_hidx, s_hcnt, s_slot, s_w);
      return;
    }
  }
  group_by_key<NT>(s_it, mp, s_srt, s_seg, s_sid, s_hidx, s_hcnt, s_inv, s_slot, s_ord, s_lid, s_mask, s_w64, s_info);
  const uint32_t S = s_info[0], SA = s_info[1], MA = s_info[2];
  if (s_info[3] != 0u)
    resolve_new_rows<NT>(s_srt, s_seg, S, c, newlist, tile_cnt, ntiles, s_pref, s_w, s_w64, s_chunk);
  if (op == kOpAssign) assign_segments<M, NT, kClk>(s_srt, s_seg, S, c);
  else sum_and_update<M, NT, kClk>(s_srt, s_seg, s_sid, S, SA, MA, c, s_piece, s_slo);
}

// ===========================================================================
// Put with dedup by radix sort (Dedup kDedupRadix), the alternative to the
// hash partition: put_probe with a single partition (its in-tile sums leave
// each key at most one item per put tile), then a stable LSD radix sort of
// all items by the key's row (rows below capacity, keys new in the call by
// capacity + index slot), in passes of at most kRsMaxBits bits, each a count
// kernel and a scatter kernel; then blocks that take even shares of the
// sorted items, each cut moved forward to the start of a key's run,
// run-length encode them in LDS and apply the updates as put_reduce does.
// Stability keeps a key's items in put-tile order, which is position order.
// ===========================================================================
static_assert(kPresumMin == 2, "radix dedup: one item per key and put tile");
static_assert(kRsTile == 4 * kPutTile, "a radix tile is four put tiles");
constexpr int kRsThreads = 1024;
constexpr int kRsPer = kRsTile / kRsThreads;
constexpr int kRsDigits = 1 << kRsMaxBits;

__device__ __forceinline__ uint32_t rs_key(uint64_t x, uint32_t cap) {
  return item_fresh(x) ? cap + item_tag(x) : item_tag(x);
}

// The items a radix tile reads. First pass: put_probe's items, tile t being
// put tiles 4t .. 4t+3, kPutTile slots each, the first (meta >> 16) of them
// used. Later passes: the dense output of the previous pass.
struct RsSrc {
  const uint64_t* src;
  const uint32_t* meta;   // first pass only
  int ntiles;             // put tiles
  const uint32_t* total;  // later passes: items in all
};

// Loads the tile's items: v[k] = item of element k * kRsThreads + tid, ok[k]
// whether it exists.
__device__ __forceinline__ void rs_load(const RsSrc& s, uint64_t (&v)[kRsPer], bool (&ok)[kRsPer]) {
  const int64_t base = (int64_t)blockIdx.x * kRsTile;
  const uint32_t T = s.meta == nullptr ? *s.total : 0u;
#pragma unroll
  for (int k = 0; k < kRsPer; ++k) {
    const int64_t i = base + k * kRsThreads + threadIdx.x;
    if (s.meta != nullptr) {
      const int pt = (int)(i / kPutTile);
      ok[k] = pt < s.ntiles && (uint32_t)(i % kPutTile) < (s.meta[pt] >> 16);
    } else {
      ok[k] = i < (int64_t)T;
    }
    v[k] = ok[k] ? s.src[i] : 0ull;
  }
}

// Digit counts of one radix tile: cnt[d * stride + tile], digit-major, so that
// a digit's counts over the tiles are contiguous (stride >= tiles, a multiple of 4).
__global__ __launch_bounds__(kRsThreads) void k_rsort_count(RsSrc s, uint32_t cap, int shift, int bits,
                                                            uint32_t* __restrict__ cnt, int stride) {
  __shared__ uint32_t h[kRsDigits];
  const int R = 1 << bits;
  for (int d = threadIdx.x; d < R; d += kRsThreads) h[d] = 0;
  uint64_t v[kRsPer];
  bool ok[kRsPer];
  rs_load(s, v, ok);
  __syncthreads();
#pragma unroll
  for (int k = 0; k < kRsPer; ++k)
    if (ok[k]) atomicAdd(&h[(rs_key(v[k], cap) >> shift) & (uint32_t)(R - 1)], 1u);
  __syncthreads();
  for (int d = threadIdx.x; d < R; d += kRsThreads) cnt[(size_t)d * stride + blockIdx.x] = h[d];
}

// Stable scatter of one radix tile by digit. An item goes to: items of smaller
// digits in all tiles + items of its digit in earlier tiles + items of its
// digit before it in this tile. The last term comes from a multisplit per
// wave (lanes with the same digit found by one ballot per digit bit), waves
// and batches taken in element order.
__global__ __launch_bounds__(kRsThreads) void k_rsort_scatter(RsSrc s, uint32_t cap, int shift, int bits,
                                                              const uint32_t* __restrict__ cnt, int rtiles,
                                                              int stride, uint64_t* __restrict__ dst,
                                                              uint32_t* __restrict__ total_out) {
  constexpr int NT = kRsThreads, NW = NT / 64;
  __shared__ uint32_t s_wc[NW * kRsDigits];  // per wave and digit: items, then where they start
  __shared__ uint32_t s_run[kRsDigits];      // per digit: where the next batch's items start
  __shared__ uint32_t s_w[NW];
  const int R = 1 << bits;  // 16 .. kRsDigits
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t = blockIdx.x;
  uint64_t v[kRsPer];
  bool ok[kRsPer];
  rs_load(s, v, ok);
  // the TPD threads of a digit (adjacent lanes) share the digit's counts
  // over the tiles, four at a time (a digit's row is 16-byte aligned; the
  // entries past the last tile are not counts)
  {
    const int TPD = NT / R;
    const int d = tid / TPD, part = tid % TPD;
    uint32_t all = 0, before = 0;
    const uint4* row = reinterpret_cast<const uint4*>(cnt + (size_t)d * stride);
    for (int u4 = part; u4 * 4 < rtiles; u4 += TPD) {
      const uint4 c = row[u4];
      const int u = u4 * 4;
      const uint32_t c0 = c.x, c1 = u + 1 < rtiles ? c.y : 0u, c2 = u + 2 < rtiles ? c.z : 0u,
                     c3 = u + 3 < rtiles ? c.w : 0u;
      all += c0 + c1 + c2 + c3;
      before += (u < t ? c0 : 0u) + (u + 1 < t ? c1 : 0u) + (u + 2 < t ? c2 : 0u) + (u + 3 < t ? c3 : 0u);
    }
    for (int o = 1; o < TPD; o <<= 1) {
      all += __shfl_xor(all, o, 64);
      before += __shfl_xor(before, o, 64);
    }
    uint32_t T;
    const uint32_t ex = block_exclusive_scan<NT>(part == 0 ? all : 0u, s_w, &T);
    if (part == 0) s_run[d] = ex + before;
    if (total_out != nullptr && t == 0 && tid == 0) *total_out = T;
  }
  const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
  for (int k = 0; k < kRsPer; ++k) {
    for (int e = tid; e < NW * R; e += NT) s_wc[e] = 0u;
    const uint32_t dg = ok[k] ? (rs_key(v[k], cap) >> shift) & (uint32_t)(R - 1) : 0u;
    uint64_t m = __ballot(ok[k] ? 1 : 0);
    for (int b = 0; b < bits; ++b) {
      const bool on = (dg >> b) & 1u;
      const uint64_t bb = __ballot(on ? 1 : 0);
      m &= on ? bb : ~bb;
    }
    const uint32_t rank = (uint32_t)__popcll(m & lt);
    __syncthreads();  // the table is cleared (and s_run written)
    if (ok[k] && rank == 0) s_wc[wave * R + dg] = (uint32_t)__popcll(m);
    __syncthreads();
    if (tid < R) {
      uint32_t run = s_run[tid];
      for (int w = 0; w < NW; ++w) {
        const uint32_t c = s_wc[w * R + tid];
        s_wc[w * R + tid] = run;
        run += c;
      }
      s_run[tid] = run;
    }
    __syncthreads();
    if (ok[k]) dst[s_wc[wave * R + dg] + rank] = v[k];
    __syncthreads();  // before the table is cleared again
  }
}

// Cut point of the sorted items at or after p: the first position q >= p
// where a key's run starts (q = T if none).
template <int NT>
__device__ __forceinline__ uint32_t rs_cut(const uint64_t* __restrict__ it, uint32_t T, uint32_t p,
                                           uint32_t* s_min) {
  if (p == 0 || p >= T) return min(p, T);
  for (uint32_t q0 = p; q0 < T; q0 += NT) {
    const uint32_t q = q0 + threadIdx.x;
    if (threadIdx.x == 0) *s_min = T;
    __syncthreads();
    if (q < T && item_group(it[q]) != item_group(it[q - 1])) atomicMin(s_min, q);
    __syncthreads();
    const uint32_t f = *s_min;
    __syncthreads();
    if (f < T) return f;
  }
  return T;
}

// Run-length encoding of m sorted items it[0, m) (whole runs of equal keys)
// into group_by_key's output: srt, seg, sid, info = {S, SA, MA, any key new
// in the call}; segments that need a sum first (more than one item, or an
// in-tile sum as the only item), their items [0, MA).
template <int NT>
__device__ __forceinline__ void encode_runs(const uint64_t* it, uint32_t m, uint64_t* srt, uint32_t* seg,
                                            uint16_t* sid, uint32_t* r_start, uint32_t* r_dest, uint16_t* r_new,
                                            uint16_t* r_of, uint32_t* s_w, uint32_t* info) {
  constexpr int IPT = (kRedCap + NT - 1) / NT;
  const int tid = threadIdx.x;
  if (tid == 0) info[3] = 0u;
  // 1. runs: the thread's IPT consecutive items
  bool head[IPT];
  uint32_t nh = 0;
  bool fresh = false;
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t j = (uint32_t)tid * IPT + k;
    head[k] = j < m && (j == 0 || item_group(it[j]) != item_group(it[j - 1]));
    nh += head[k] ? 1u : 0u;
    fresh |= j < m && item_fresh(it[j]);
  }
  uint32_t S;
  uint32_t r = block_exclusive_scan<NT>(nh, s_w, &S);
  if (fresh) info[3] = 1u;
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t j = (uint32_t)tid * IPT + k;
    if (head[k]) r_start[r++] = j;
    if (j < m) r_of[j] = (uint16_t)(r - 1);
  }
  if (tid == 0) r_start[S] = m;
  __syncthreads();
  // 2. new places: runs that need a sum first, in order, then the others
  bool multi[IPT];
  uint32_t len[IPT];
  uint32_t packed = 0;  // runs that need a sum | their items << 16
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t q = (uint32_t)tid * IPT + k;
    multi[k] = false;
    len[k] = 0;
    if (q < S) {
      len[k] = r_start[q + 1] - r_start[q];
      multi[k] = len[k] > 1 || item_summed(it[r_start[q]]);
      packed += multi[k] ? (1u | (len[k] << 16)) : 0u;
    }
  }
  uint32_t tot;
  const uint32_t pre = block_exclusive_scan<NT>(packed, s_w, &tot);
  const uint32_t SA = tot & 0xFFFFu, MA = tot >> 16;
  uint32_t na = pre & 0xFFFFu, ia = pre >> 16;
#pragma unroll
  for (int k = 0; k < IPT; ++k) {
    const uint32_t q = (uint32_t)tid * IPT + k;
    if (q < S) {
      uint32_t ns, nd;
      if (multi[k]) {
        ns = na++;
        nd = ia;
        ia += len[k];
      } else {
        ns = SA + (q - na);  // the runs before q that need no sum, each one item
        nd = MA + (q - na);
      }
      r_new[q] = (uint16_t)ns;
      r_dest[q] = nd;
      seg[ns] = nd;
    }
  }
  if (tid == 0) {
    seg[S] = m;
    info[0] = S;
    info[1] = SA;
    info[2] = MA;
  }
  __syncthreads();
  // 3. every item to its place
  for (uint32_t j = tid; j < m; j += NT) {
    const uint32_t q = r_of[j];
    const uint32_t d = r_dest[q] + (j - r_start[q]);
    srt[d] = it[j];
    sid[d] = r_new[q];
  }
  __syncthreads();
}

template <class M, int NT, bool kClk>
__global__ __launch_bounds__(NT) void k_rsort_reduce(
    Bucket* __restrict__ idx, const uint64_t* __restrict__ sorted, const uint32_t* __restrict__ total,
    int ntiles, const NewKey* __restrict__ newlist, const uint32_t* __restrict__ tile_cnt,
    const float* __restrict__ grads, double* __restrict__ partials, const RowStore store,
    float* __restrict__ state, int D, uint64_t seed, float lr, float eps, int64_t capacity, Ctrl* ctrl,
    uint64_t epoch, int op, unsigned long long* __restrict__ clock) {
  using L = ReduceLds<NT>;
  extern __shared__ __align__(16) unsigned char s_raw[];
  uint64_t* s_it = reinterpret_cast<uint64_t*>(s_raw + L::it);
  uint32_t* s_rstart = reinterpret_cast<uint32_t*>(s_raw + L::hidx);  // [kRedCap + 1]
  uint32_t* s_rdest = reinterpret_cast<uint32_t*>(s_raw + L::hcnt);
  uint16_t* s_rnew = reinterpret_cast<uint16_t*>(s_raw + L::inv);
  uint16_t* s_rof = reinterpret_cast<uint16_t*>(s_raw + L::slot);
  double* s_piece = reinterpret_cast<double*>(s_raw);      // reused region
  uint64_t* s_chunk = reinterpret_cast<uint64_t*>(s_raw);  // reused region
  uint64_t* s_srt = reinterpret_cast<uint64_t*>(s_raw + L::srt);
  uint32_t* s_seg = reinterpret_cast<uint32_t*>(s_raw + L::seg);
  uint16_t* s_sid = reinterpret_cast<uint16_t*>(s_raw + L::sid);
  uint32_t* s_pref = reinterpret_cast<uint32_t*>(s_raw + L::pref);
  uint32_t* s_w = reinterpret_cast<uint32_t*>(s_raw + L::w);
  unsigned long long* s_w64 = reinterpret_cast<unsigned long long*>(s_raw + L::w64);
  uint32_t* s_info = reinterpret_cast<uint32_t*>(s_raw + L::misc);
  uint32_t* s_slo = reinterpret_cast<uint32_t*>(s_raw + L::slo);
  static_assert(kRedHash >= kRedCap + 1, "run starts fit the hash region");

  const uint64_t size0 = ctrl->size[epoch & 1];
  const uint64_t new_e = ctrl->new_epoch, ovf_e = ctrl->overflow_epoch;
  const uint64_t bad_e = ctrl->apput_bad_epoch == epoch ? epoch : ctrl->bad_epoch;
  const uint64_t Mnew = new_e == epoch ? count_new_keys<NT>(tile_cnt, ntiles, s_w64) : 0ull;
  const int err = call_verdict(ctrl, epoch, size0, Mnew, capacity, bad_e, ovf_e, ctrl->apput_absent_epoch);
  const uint32_t T = *total;
  const uint32_t nb = gridDim.x, b = blockIdx.x;
  const uint32_t lo = rs_cut<NT>(sorted, T, (uint32_t)((uint64_t)T * b / nb), s_info + 4);
  const uint32_t hi = rs_cut<NT>(sorted, T, (uint32_t)((uint64_t)T * (b + 1) / nb), s_info + 4);
  const uint32_t m = hi - lo;
  if (m == 0) return;
  if (err) {
    // undo the insertions of this call whose keys have their runs here
    for (uint32_t j = threadIdx.x; j < m; j += NT) {
      const uint64_t x = sorted[lo + j];
      if (item_fresh(x)) {
        const uint32_t slot = item_tag(x);
        idx[slot / kSlots].key[slot % kSlots] = kEmptyKey;
      }
    }
    return;
  }
  if (m > (uint32_t)kRedCap) {  // runs are at most one item per put tile; the host keeps this from happening
    if (threadIdx.x == 0) atomicCAS(&ctrl->latched, 0, -4);
    return;
  }
  for (uint32_t j = threadIdx.x; j < m; j += NT) s_it[j] = sorted[lo + j];
  __syncthreads();
  encode_runs<NT>(s_it, m, s_srt, s_seg, s_sid, s_rstart, s_rdest, s_rnew, s_rof, s_w, s_info);
  const uint32_t S = s_info[0], SA = s_info[1], MA = s_info[2];
  const RedCtx c{op, idx, grads, partials, store, state, D, seed, lr, eps, size0, clock};
  if (s_info[3] != 0u)
    resolve_new_rows<NT>(s_srt, s_seg, S, c, newlist, tile_cnt, ntiles, s_pref, s_w, s_w64, s_chunk);
  if (op == kOpAssign) assign_segments<M, NT, kClk>(s_srt, s_seg, S, c);
  else sum_and_update<M, NT, kClk>(s_srt, s_seg, s_sid, S, SA, MA, c, s_piece, s_slo);
}

// ===========================================================================
// Inspection kernels
// ===========================================================================
__global__ __launch_bounds__(256) void k_lookup(Bucket* __restrict__ idx, uint32_t nb_log2,
                                                const uint64_t* __restrict__ keys, int64_t n,
                                                int64_t* __restrict__ rows_out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  const uint64_t key = keys[i];
  int64_t r = -1;
  if (key != kEmptyKey) {
    const Probe pr = probe_key(idx, nb_log2, key, false);
    if (pr.status == P_HIT) r = pr.row;
  }
  rows_out[i] = r;
}

__global__ __launch_bounds__(256) void k_export_slots(const Bucket* __restrict__ idx, uint64_t nslots,
                                                      uint64_t* __restrict__ keys_out,
                                                      uint32_t* __restrict__ rows_out) {
  const uint64_t s = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  if (s >= nslots) return;
  const Bucket* B = idx + s / kSlots;
  if (keys_out) keys_out[s] = B->key[s % kSlots];
  if (rows_out) rows_out[s] = B->row[s % kSlots];
}

// Copies rows and accumulators by row id; ids outside [0, size) give NaN
// rows and latch MLKV_EINVAL (-1).
__global__ __launch_bounds__(256) void k_read_rows(const RowStore store, const float* __restrict__ state,
                                                   int D, const unsigned long long* size_now,
                                                   const int64_t* __restrict__ ids, int64_t n,
                                                   float* __restrict__ w_out, float* __restrict__ st_out,
                                                   Ctrl* ctrl) {
  const uint64_t size = *size_now;
  const uint64_t total = (uint64_t)n * (uint64_t)D;
  for (uint64_t e = (uint64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (uint64_t)gridDim.x * 256) {
    const uint64_t i = e / (uint64_t)D;
    const int c = (int)(e % (uint64_t)D);
    const int64_t r = ids[i];
    const bool ok = r >= 0 && (uint64_t)r < size;
    if (!ok && c == 0) atomicCAS(&ctrl->latched, 0, -1);
    if (w_out) w_out[e] = ok ? store.ptr((uint32_t)r)[c] : __builtin_nanf("");
    if (st_out && c == 0) st_out[i] = ok ? state[r] : __builtin_nanf("");
  }
}

// Staleness counts by row id; ids outside [0, size) give 0xFFFFFFFF and
// latch MLKV_EINVAL (-1).
__global__ __launch_bounds__(256) void k_read_clock(const unsigned long long* __restrict__ clock,
                                                    const unsigned long long* size_now,
                                                    const int64_t* __restrict__ ids, int64_t n,
                                                    uint32_t* __restrict__ out, Ctrl* ctrl) {
  const uint64_t size = *size_now;
  for (uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x; i < (uint64_t)n; i += (uint64_t)gridDim.x * 256) {
    const int64_t r = ids[i];
    const bool ok = r >= 0 && (uint64_t)r < size;
    if (!ok) atomicCAS(&ctrl->latched, 0, -1);
    out[i] = ok ? (uint32_t)(clock[r] & kClockCount) : 0xFFFFFFFFu;
  }
}

// ===========================================================================
// Launchers
// ===========================================================================
template <class M>
static hipError_t launch_get_t(const GetArgs& a, hipStream_t st, const LaunchHook& hook) {
  const int tlen = get_tile_len(a.n, a.cus);
  const int64_t ntiles = (a.n + tlen - 1) / tlen;
  const int grid = (int)std::min<int64_t>(ntiles, kMaxRanges);  // row assignment: one block per key range
  RangeLists rl = a.rl;
  if (rl.list != nullptr) rl.cap = (uint32_t)std::min<uint64_t>(rl.entries / (uint64_t)grid, 0xFFFFFFFFull);
  hook(K_GET_PROBE_GATHER, 0, st);
  auto kern = a.clock != nullptr ? k_get_probe_gather<M, true, false>
                                  : a.pc_in ? k_get_probe_gather<M, false, true> : k_get_probe_gather<M, false, false>;
  hipLaunchKernelGGL(kern, dim3((unsigned)ntiles), dim3(kGetTile), 0, st, a.idx, a.nb_log2, a.keys, a.n,
                     a.out, a.store, a.D, a.seed, a.newlist, a.tile_cnt, a.ctrl, a.epoch, a.clock, a.cepoch,
                     a.bound, a.blocked, a.pc_key, a.pc_row, tlen, rl, (uint32_t)grid);
  hook(K_GET_PROBE_GATHER, 1, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hook(K_ASSIGN_NEW, 0, st);
  hipLaunchKernelGGL(k_assign_new, dim3(grid), dim3(kAssignThreads), 0, st, a.idx, a.newlist,
                     a.tile_cnt, (int)ntiles, tlen, a.store, a.state, a.D, a.seed, a.capacity,
                     a.ctrl, a.epoch, a.xkey, a.xslot, a.clock, a.cepoch, rl);
  hook(K_ASSIGN_NEW, 1, st);
  return hipGetLastError();
}

// Lets kernel `f` (an instance of a reduce kernel) use `bytes` of dynamic
// LDS on the current device; `done` remembers the devices where that is set.
template <int kMaxDev>
static hipError_t lds_attr(const void* f, int bytes, bool (&done)[kMaxDev]) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kMaxDev && done[dev]) return hipSuccess;
  e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  if (e == hipSuccess && dev >= 0 && dev < kMaxDev) done[dev] = true;
  return e;
}

// Whether the put_reduce instance of row map M may use its dynamic LDS on
// each device (set once per device).
template <class M, bool kClk, bool kUpsert>
static hipError_t reduce_lds_attr() {
  static bool done[64] = {};
  constexpr int NT = ReduceCfg<M>::NT;
  return lds_attr(reinterpret_cast<const void*>(&k_put_reduce<M, NT, kClk, kUpsert>), (int)ReduceLds<NT>::total,
                  done);
}

// The same for the radix reduce instance of row map M.
template <class M, bool kClk>
static hipError_t rsort_lds_attr() {
  static bool done[64] = {};
  constexpr int NT = ReduceCfg<M>::NT;
  return lds_attr(reinterpret_cast<const void*>(&k_rsort_reduce<M, NT, kClk>), (int)ReduceLds<NT>::total, done);
}

// The probe kernel of a put, with 2^pb partitions.
template <class M>
static hipError_t launch_put_probe(const PutArgs& a, int pb, hipStream_t st, const LaunchHook& hook) {
  const int64_t ntiles = (a.n + a.tlen - 1) / a.tlen;
  auto kern = a.ahead ? k_put_probe<M, true> : k_put_probe<M, false>;
  hook(K_PUT_PROBE, 0, st);
  hipLaunchKernelGGL(kern, dim3((unsigned)ntiles), dim3(kPutThreads), 0, st, a.idx, a.nb_log2, a.keys, a.grads,
                     a.n, a.tlen, a.D, a.op, pb, (int)ntiles, a.items, a.meta, a.partials, a.newlist, a.tile_cnt,
                     a.ctrl, a.epoch, a.pc_key, a.pc_row);
  hook(K_PUT_PROBE, 1, st);
  return hipGetLastError();
}

// Put with radix dedup: put_probe (one partition), the radix passes, the
// reduce over the sorted items.
template <class M>
static hipError_t launch_put_radix(const PutArgs& a, hipStream_t st, const LaunchHook& hook, int phase) {
  constexpr int NT = ReduceCfg<M>::NT;
  using L = ReduceLds<NT>;
  const int64_t ntiles = (a.n + a.tlen - 1) / a.tlen;
  hipError_t e = hipSuccess;
  if (phase != kPutAfterProbe && (e = launch_put_probe<M>(a, 0, st, hook)) != hipSuccess) return e;
  if (phase == kPutProbe) return hipSuccess;
  // passes of at most kRsMaxBits bits (at least 4: a sort key spans at least 4 bits)
  const int passes = (a.rs_bits + kRsMaxBits - 1) / kRsMaxBits;
  const int bits = (a.rs_bits + passes - 1) / passes;
  const int rtiles = (int)((ntiles + 3) / 4);
  const int stride = (rtiles + 3) / 4 * 4;  // a digit's row of counts, padded to 16 bytes
  uint32_t* cnt = a.rs_cnt;
  uint32_t* total = a.rs_cnt + (size_t)stride * (1u << bits);
  uint64_t* buf[2] = {a.rs_buf, a.rs_buf + a.n};
  const uint32_t cap = (uint32_t)a.capacity;
  for (int p = 0; p < passes; ++p) {
    RsSrc src;
    src.src = p == 0 ? a.items : buf[(p - 1) & 1];
    src.meta = p == 0 ? a.meta : nullptr;
    src.ntiles = (int)ntiles;
    src.total = total;
    hook(K_RSORT_COUNT, 0, st);
    hipLaunchKernelGGL(k_rsort_count, dim3((unsigned)rtiles), dim3(kRsThreads), 0, st, src, cap, p * bits, bits,
                       cnt, stride);
    hook(K_RSORT_COUNT, 1, st);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hook(K_RSORT_SCATTER, 0, st);
    hipLaunchKernelGGL(k_rsort_scatter, dim3((unsigned)rtiles), dim3(kRsThreads), 0, st, src, cap, p * bits, bits,
                       (const uint32_t*)cnt, rtiles, stride, buf[p & 1], p == 0 ? total : (uint32_t*)nullptr);
    hook(K_RSORT_SCATTER, 1, st);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  const bool clk = a.clock != nullptr;
  if ((e = clk ? rsort_lds_attr<M, true>() : rsort_lds_attr<M, false>()) != hipSuccess) return e;
  // blocks: one per CU at least, at most kRsChunk sorted items each before the cuts move
  const int64_t nb = std::max<int64_t>(a.cus, (a.n + kRsChunk - 1) / kRsChunk);
  auto rkern = clk ? k_rsort_reduce<M, NT, true> : k_rsort_reduce<M, NT, false>;
  hook(K_RSORT_REDUCE, 0, st);
  hipLaunchKernelGGL(rkern, dim3((unsigned)nb), dim3(NT), L::total, st, a.idx, (const uint64_t*)buf[(passes - 1) & 1], (const uint32_t*)total,
                     (int)ntiles, a.newlist, a.tile_cnt, a.grads, a.partials, a.store, a.state, a.D, a.seed, a.lr,
                     a.eps, a.capacity, a.ctrl, a.epoch, a.op, a.clock);
  hook(K_RSORT_REDUCE, 1, st);
  return hipGetLastError();
}

template <class M>
static hipError_t launch_put_t(const PutArgs& a, hipStream_t st, const LaunchHook& hook, int phase) {
  constexpr int NT = ReduceCfg<M>::NT;
  using L = ReduceLds<NT>;
  static_assert((size_t)ReduceCfg<M>::NG * ReduceCfg<M>::DMAX * sizeof(double) <= L::reuse,
                "pieces of cut segments must fit the reused LDS region");
  static_assert((size_t)(kChunk + NT) * sizeof(uint64_t) + (size_t)(NT + 1) * sizeof(uint32_t) <= L::reuse,
                "new-key chunk, sorted new keys and their counts must fit the reused LDS region");
  static_assert(L::total <= 160 * 1024, "LDS budget of a gfx950 workgroup");
  if (a.dedup == kDedupRadix) return launch_put_radix<M>(a, st, hook, phase);
  const int64_t ntiles = (a.n + a.tlen - 1) / a.tlen;
  const int np = 1 << a.pb;
  hipError_t e = hipSuccess;
  if (phase != kPutAfterProbe && (e = launch_put_probe<M>(a, a.pb, st, hook)) != hipSuccess) return e;
  if (phase == kPutProbe) return hipSuccess;
  const bool clk = a.clock != nullptr;  // a bounded table: puts lower the staleness counts
  const bool ups = a.op == kOpAssign;
  if ((e = clk ? (ups ? reduce_lds_attr<M, true, true>() : reduce_lds_attr<M, true, false>())
               : (ups ? reduce_lds_attr<M, false, true>() : reduce_lds_attr<M, false, false>())) != hipSuccess)
    return e;
  auto kern = clk ? (ups ? k_put_reduce<M, NT, true, true> : k_put_reduce<M, NT, true, false>)
                  : (ups ? k_put_reduce<M, NT, false, true> : k_put_reduce<M, NT, false, false>);
  hook(K_PUT_REDUCE, 0, st);
  hipLaunchKernelGGL(kern, dim3((unsigned)np), dim3(NT),
                     L::total, st, a.idx, a.items, a.meta, (int)ntiles, a.newlist, a.tile_cnt, a.grads, a.partials,
                     a.store, a.state, a.D, a.seed, a.lr, a.eps, a.capacity, a.ctrl, a.epoch, a.spill, a.spill_words,
                     a.op, a.clock);
  hook(K_PUT_REDUCE, 1, st);
  return hipGetLastError();
}

// Row maps: float4 lanes when rows are 16-byte aligned multiples of 4 floats.
using MapD16 = RowMap<4, 4, 1>;     // dim <= 16
using MapD32 = RowMap<4, 8, 1>;     // dim <= 32
using MapD64 = RowMap<4, 16, 1>;    // dim <= 64
using MapD128 = RowMap<4, 32, 1>;   // dim <= 128
using MapD256 = RowMap<4, 64, 1>;   // dim <= 256
using MapD512 = RowMap<4, 64, 2>;   // dim <= 512
using MapD1024 = RowMap<4, 64, 4>;  // dim <= 1024
using MapAny = RowMap<1, 64, 16>;   // any dim <= 1024, one float per lane

template <class F>
static hipError_t dispatch_map(int D, bool vec4, F f) {
  if (!vec4) return f(MapAny{});
  if (D <= 16) return f(MapD16{});
  if (D <= 32) return f(MapD32{});
  if (D <= 64) return f(MapD64{});
  if (D <= 128) return f(MapD128{});
  if (D <= 256) return f(MapD256{});
  if (D <= 512) return f(MapD512{});
  return f(MapD1024{});
}

hipError_t launch_get(const GetArgs& a, bool vec4, hipStream_t st, const LaunchHook& hook) {
  return dispatch_map(a.D, vec4, [&](auto m) { return launch_get_t<decltype(m)>(a, st, hook); });
}

hipError_t launch_put(const PutArgs& a, bool vec4, hipStream_t st, const LaunchHook& hook, int phase) {
  return dispatch_map(a.D, vec4, [&](auto m) { return launch_put_t<decltype(m)>(a, st, hook, phase); });
}

hipError_t launch_lookup(Bucket* idx, uint32_t nb_log2, const uint64_t* keys, int64_t n, int64_t* rows_out,
                         hipStream_t st) {
  const int64_t grid = (n + 255) / 256;
  hipLaunchKernelGGL(k_lookup, dim3((unsigned)grid), dim3(256), 0, st, idx, nb_log2, keys, n, rows_out);
  return hipGetLastError();
}

hipError_t launch_export_slots(const Bucket* idx, uint64_t nslots, uint64_t* keys_out, uint32_t* rows_out,
                               hipStream_t st) {
  const uint64_t grid = (nslots + 255) / 256;
  hipLaunchKernelGGL(k_export_slots, dim3((unsigned)grid), dim3(256), 0, st, idx, nslots, keys_out, rows_out);
  return hipGetLastError();
}

hipError_t launch_read_rows(const RowStore& store, const float* state, int D, const unsigned long long* size_now,
                            const int64_t* ids, int64_t n, float* w_out, float* st_out, Ctrl* ctrl,
                            hipStream_t st) {
  const uint64_t total = (uint64_t)n * (uint64_t)D;
  const uint64_t grid = std::min<uint64_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_read_rows, dim3((unsigned)grid), dim3(256), 0, st, store, state, D, size_now, ids, n,
                     w_out, st_out, ctrl);
  return hipGetLastError();
}

// Rows 0 .. nrows-1 in order, from wherever each lives.
__global__ __launch_bounds__(256) void k_export_rows(const RowStore store, int64_t nrows, int D,
                                                     float* __restrict__ out) {
  const uint64_t total = (uint64_t)nrows * (uint64_t)D;
  for (uint64_t e = (uint64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (uint64_t)gridDim.x * 256) {
    const uint64_t r = e / (uint64_t)D;
    out[e] = store.ptr((uint32_t)r)[e % (uint64_t)D];
  }
}

hipError_t launch_export_rows(const RowStore& store, int64_t nrows, int D, float* out, hipStream_t st) {
  const uint64_t total = (uint64_t)nrows * (uint64_t)D;
  if (total == 0) return hipSuccess;
  const uint64_t grid = std::min<uint64_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_export_rows, dim3((unsigned)grid), dim3(256), 0, st, store, nrows, D, out);
  return hipGetLastError();
}

hipError_t launch_read_clock(const unsigned long long* clock, const unsigned long long* size_now,
                             const int64_t* ids, int64_t n, uint32_t* out, Ctrl* ctrl, hipStream_t st) {
  const uint64_t grid = std::min<uint64_t>(((uint64_t)n + 255) / 256, 65536);
  hipLaunchKernelGGL(k_read_clock, dim3((unsigned)grid), dim3(256), 0, st, clock, size_now, ids, n, out, ctrl);
  return hipGetLastError();
}

}  // namespace mlkv
