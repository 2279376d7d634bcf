// HIP kernels of libmlkv for gfx950 (MI355X): hash-index probe, row gather,
// in-batch dedup by MSD radix partition + LDS sort + run-length encoding, and
// the fp64 segment-reduce fused with the row-wise Adagrad scatter-update.
#include "mlkv_kernels.h"

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
// were present are read from the table, rows of keys new in this call are
// generated from their seed (they equal what the table will hold).
template <class M>
__device__ __forceinline__ void wave_emit_rows(float* __restrict__ out, const float* __restrict__ rows,
                                               int D, int64_t wave_base, int64_t n, bool hit,
                                               uint32_t row, uint64_t s0, int lane) {
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  constexpr int ITERS = 64 / RPW;
  constexpr int UNITS = ITERS * K;
  constexpr int CH = UNITS < 16 ? UNITS : 16;
  const int g = lane / LPR;
  const int q = lane % LPR;
  const int ihit = hit ? 1 : 0;
#pragma unroll 1
  for (int u0 = 0; u0 < UNITS; u0 += CH) {
    typename VecT<VEC>::T v[CH];
#pragma unroll
    for (int u = 0; u < CH; ++u) {
      const int uu = u0 + u;
      const int it = uu / K;
      const int k = uu % K;
      const int r = it * RPW + g;
      const uint32_t rr = __shfl(row, r, 64);
      const int hh = __shfl(ihit, r, 64);
      const uint64_t ss = __shfl((unsigned long long)s0, r, 64);
      const int col = (k * LPR + q) * VEC;
      const int64_t p = wave_base + r;
      if (uu < UNITS && p < n && col < D) {
        if (hh) v[u] = load_vec<VEC>(rows + (size_t)rr * (size_t)D + col);
        else v[u] = init_vec<VEC>(ss, col);
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
      if (uu < UNITS && p < n && col < D) store_vec<VEC>(out + (size_t)p * (size_t)D + col, v[u]);
    }
  }
}

template <class M>
__global__ __launch_bounds__(kGetTile) void k_get_probe_gather(
    Bucket* __restrict__ idx, uint32_t nb_log2, const uint64_t* __restrict__ keys, int64_t n,
    float* __restrict__ out, const float* __restrict__ rows, int D, uint64_t seed,
    NewKey* __restrict__ newlist, uint32_t* __restrict__ tile_cnt, Ctrl* ctrl, uint64_t epoch) {
  __shared__ uint32_t s_cnt;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t base = (int64_t)blockIdx.x * kGetTile;
  const int64_t i = base + tid;
  if (tid == 0) s_cnt = 0;
  __syncthreads();
  uint64_t key = 0;
  Probe pr = {0, kPendingRow, P_NONE};
  if (i < n) {
    key = keys[i];
    if (key == kEmptyKey) {
      pr.status = P_BAD;
      ctrl->bad_epoch = epoch;
    } else {
      pr = probe_key(idx, nb_log2, key, true);
      if (pr.status == P_OVERFLOW) ctrl->overflow_epoch = epoch;
    }
  }
  if (pr.status == P_NEW_MINE) {
    const uint32_t j = atomicAdd(&s_cnt, 1u);
    newlist[base + j] = NewKey{key, pr.slot, 0u};
    ctrl->new_epoch = epoch;
  }
  if (out != nullptr) {
    const uint64_t s0 = splitmix_mix(key ^ seed);
    wave_emit_rows<M>(out, rows, D, base + wave * 64, n, pr.status == P_HIT, pr.row, s0, lane);
  }
  __syncthreads();
  if (tid == 0) tile_cnt[blockIdx.x] = s_cnt;
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
                                            int64_t capacity) {
  int err = 0;
  if (ctrl->bad_epoch == epoch) err = -1;                          // MLKV_EINVAL
  else if (ctrl->overflow_epoch == epoch || size0 + M > (uint64_t)capacity) err = -2;  // MLKV_EFULL
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

__global__ __launch_bounds__(kAssignThreads) void k_assign_new(
    Bucket* __restrict__ idx, const NewKey* __restrict__ newlist, const uint32_t* __restrict__ tile_cnt,
    int ntiles, int tile_size, float* __restrict__ rows, float* __restrict__ state, int D,
    uint64_t seed, int64_t capacity, Ctrl* ctrl, uint64_t epoch) {
  constexpr int NT = kAssignThreads;
  __shared__ unsigned long long s_w64[NT / 64];
  __shared__ uint32_t s_w[NT / 64];
  __shared__ uint32_t s_pref[NT + 1];
  __shared__ uint64_t s_chunk[kChunk];
  __shared__ uint64_t s_key[kAssignMine];
  __shared__ uint32_t s_slot[kAssignMine];
  __shared__ uint32_t s_rank[kAssignMine];

  const uint64_t size0 = ctrl->size[epoch & 1];
  const bool any_new = ctrl->new_epoch == epoch;
  const uint64_t M = any_new ? count_new_keys<NT>(tile_cnt, ntiles, s_w64) : 0ull;
  const int err = call_verdict(ctrl, epoch, size0, M, capacity);
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

  // This block owns the tiles t = blockIdx.x (mod gridDim.x); it takes them
  // kAssignBatch at a time (thread j holds entry j of each tile) and ranks
  // their keys against all M new keys of the call.
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
    }
    // initial rows, written cooperatively (coalesced along each row)
    for (int b = 0; b < kAssignBatch; ++b) {
      const int t = tb + b * (int)gridDim.x;
      const uint32_t c = t < ntiles ? tile_cnt[t] : 0u;
      const uint64_t total = (uint64_t)c * (uint64_t)D;
      for (uint64_t e = threadIdx.x; e < total; e += NT) {
        const uint32_t j = (uint32_t)(e / (uint64_t)D);
        const int col = (int)(e - (uint64_t)j * D);
        const int m = b * NT + (int)j;
        const uint64_t row = size0 + s_rank[m];
        rows[row * (uint64_t)D + col] = init_elem(splitmix_mix(s_key[m] ^ seed), col);
      }
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

template <class M>
__global__ __launch_bounds__(kPutThreads) void k_put_probe(
    Bucket* __restrict__ idx, uint32_t nb_log2, const uint64_t* __restrict__ keys,
    const float* __restrict__ grads, int64_t n, int D, int pb, int ntiles, uint64_t* __restrict__ items,
    uint32_t* __restrict__ meta, double* __restrict__ partials, NewKey* __restrict__ newlist,
    uint32_t* __restrict__ tile_cnt, Ctrl* ctrl, uint64_t epoch) {
  constexpr int NT = kPutThreads;
  constexpr int KPT = kPutTile / kPutThreads;  // keys per thread
  constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  constexpr int NG = (NT / 64) * RPW;
  using V = typename VecT<VEC>::T;
  __shared__ uint32_t s_hist[kMaxParts];
  __shared__ unsigned long long s_hkey[kTileHash];  // group of each hash slot
  __shared__ uint32_t s_hcnt[kTileHash];            // occurrences of the group in the tile
  __shared__ uint32_t s_hfirst[kTileHash];          // first entry holding the group
  __shared__ uint32_t s_hcur[kTileHash];            // fill cursor of the group's entry list
  __shared__ uint16_t s_hdup[kTileHash];            // index of a repeated group
  __shared__ uint16_t s_lanes[kPutTile];            // entries of repeated groups, grouped
  __shared__ uint16_t s_doff[kPutTile / 2 + 1];     // start of each repeated group's entries
  __shared__ uint32_t s_w[NT / 64];
  __shared__ uint32_t s_cnt;
  const int NP = 1 << pb;
  const int tid = threadIdx.x;
  const int tile = blockIdx.x;
  const int64_t base = (int64_t)tile * kPutTile;
  if (tile == 0 && tid == 0) ctrl->spill_next = 0;
  for (int d = tid; d < NP; d += NT) s_hist[d] = 0;
  for (int h = tid; h < kTileHash; h += NT) {
    s_hkey[h] = ~0ull;
    s_hcnt[h] = 0;
    s_hfirst[h] = 0xFFFFFFFFu;
    s_hcur[h] = 0;
  }
  if (tid == 0) s_cnt = 0;

  // entry e = kk * NT + tid of the tile is batch position base + e
  uint64_t key[KPT];
  Probe pr[KPT];
  {
    uint64_t hb[KPT];
    BucketView bv[KPT];
#pragma unroll
    for (int kk = 0; kk < KPT; ++kk) {
      const int64_t i = base + kk * NT + tid;
      key[kk] = i < n ? keys[i] : kEmptyKey;
      pr[kk] = {0, kPendingRow, i < n ? P_BAD : P_NONE};
    }
#pragma unroll
    for (int kk = 0; kk < KPT; ++kk) {
      if (key[kk] != kEmptyKey) {
        hb[kk] = home_bucket(key[kk], nb_log2);
        bv[kk] = load_bucket(idx + hb[kk]);
      }
    }
#pragma unroll
    for (int kk = 0; kk < KPT; ++kk) {
      if (key[kk] != kEmptyKey) {
        pr[kk] = probe_with(idx, nb_log2, key[kk], true, hb[kk], bv[kk]);
        if (pr[kk].status == P_OVERFLOW) ctrl->overflow_epoch = epoch;
      } else if (pr[kk].status == P_BAD) {
        ctrl->bad_epoch = epoch;
      }
    }
  }
  __syncthreads();

  uint64_t x[KPT];
  uint32_t hs[KPT];
  bool valid[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    const int e = kk * NT + tid;
    valid[kk] = pr[kk].status == P_HIT || pr[kk].status == P_NEW_MINE || pr[kk].status == P_NEW_OTHER;
    if (pr[kk].status == P_NEW_MINE) {
      const uint32_t j = atomicAdd(&s_cnt, 1u);
      newlist[(size_t)base + j] = NewKey{key[kk], pr[kk].slot, 0u};
      ctrl->new_epoch = epoch;
    }
    const bool fresh = pr[kk].status != P_HIT;
    x[kk] = valid[kk] ? make_item(fresh, fresh ? pr[kk].slot : pr[kk].row, (uint32_t)(base + e)) : ~0ull;
    // count the tile's occurrences of every group
    hs[kk] = 0;
    if (valid[kk]) {
      const uint64_t grp = item_group(x[kk]);
      uint32_t h = (uint32_t)index_hash(grp) & (kTileHash - 1);
      while (true) {
        const unsigned long long old = atomicCAS(&s_hkey[h], ~0ull, (unsigned long long)grp);
        if (old == ~0ull || old == grp) break;
        h = (h + 1) & (kTileHash - 1);
      }
      hs[kk] = h;
      atomicAdd(&s_hcnt[h], 1u);
      atomicMin(&s_hfirst[h], (uint32_t)e);
    }
  }
  __syncthreads();
  uint32_t cnt[KPT];
  bool dup[KPT], owner[KPT];
  uint32_t n_own = 0, l_own = 0;
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    const int e = kk * NT + tid;
    cnt[kk] = valid[kk] ? s_hcnt[hs[kk]] : 0u;
    dup[kk] = cnt[kk] >= 2;
    owner[kk] = dup[kk] && s_hfirst[hs[kk]] == (uint32_t)e;
    n_own += owner[kk] ? 1u : 0u;
    l_own += owner[kk] ? cnt[kk] : 0u;
  }

  // repeated groups: index them, then list their entries contiguously
  uint32_t ndup, nlanes;
  uint32_t dpre = block_exclusive_scan<NT>(n_own, s_w, &ndup);
  uint32_t lpre = block_exclusive_scan<NT>(l_own, s_w, &nlanes);
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    if (owner[kk]) {
      s_hdup[hs[kk]] = (uint16_t)dpre;
      s_doff[dpre] = (uint16_t)lpre;
      ++dpre;
      lpre += cnt[kk];
    }
  }
  if (tid == 0) s_doff[ndup] = (uint16_t)nlanes;
  __syncthreads();
  uint32_t my_off[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    my_off[kk] = 0;
    if (dup[kk]) {
      my_off[kk] = s_doff[s_hdup[hs[kk]]];
      s_lanes[my_off[kk] + atomicAdd(&s_hcur[hs[kk]], 1u)] = (uint16_t)(kk * NT + tid);
    }
  }
  __syncthreads();
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
  __syncthreads();
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk)
    if (dup[kk]) s_lanes[my_off[kk] + rank[kk]] = (uint16_t)(kk * NT + tid);
  __syncthreads();

  // each lane group sums the rows of repeated groups, positions ascending
  {
    constexpr int UNR = (K * VEC >= 8) ? 4 : 8;
    const int lane = tid & 63;
    const int g = lane / LPR;
    const int q = lane % LPR;
    const int gid = (tid >> 6) * RPW + g;
    for (uint32_t dg = gid; dg < ndup; dg += NG) {
      const uint32_t b = s_doff[dg], e = s_doff[dg + 1];
      double acc[K][VEC];
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
      double* dst = partials + (size_t)(base + s_lanes[b]) * (size_t)D;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        const int col = (k * LPR + q) * VEC;
#pragma unroll
        for (int v = 0; v < VEC; ++v)
          if (col + v < D) dst[col + v] = acc[k][v];
      }
    }
  }

  // emit single positions, and one summed item per repeated key
  bool emit[KPT];
  uint32_t d[KPT], r[KPT];
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk) {
    emit[kk] = valid[kk] && (!dup[kk] || owner[kk]);
    d[kk] = 0;
    r[kk] = 0;
    if (emit[kk]) {
      d[kk] = group_partition(item_group(x[kk]), pb);
      r[kk] = atomicAdd(&s_hist[d[kk]], 1u);
    }
  }
  __syncthreads();
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
  __syncthreads();
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int dd = tid * PER + j;
    if (dd < NP) s_hist[dd] = offs[j];
  }
  __syncthreads();
#pragma unroll
  for (int kk = 0; kk < KPT; ++kk)
    if (emit[kk]) items[(size_t)base + s_hist[d[kk]] + r[kk]] = dup[kk] ? (x[kk] | kItemSummed) : x[kk];
  if (tid == 0) tile_cnt[tile] = s_cnt;
}

// ---------------------------------------------------------------------------
// Put, second kernel: one block per partition. Gathers the partition's items,
// sorts them, run-length encodes them into segments (one per distinct key,
// positions ascending), sums each segment's gradient rows in fp64 and applies
// one row-wise Adagrad step to the key's row.
// ---------------------------------------------------------------------------
template <class M>
struct SegmentOps {
  static constexpr int VEC = M::VEC, LPR = M::LPR, K = M::K, RPW = M::RPW;
  using V = typename VecT<VEC>::T;
  static constexpr int UNR = (K * VEC >= 8) ? 4 : 8;

  // acc += gradient rows of the sorted items [b, e)
  template <class IP>
  static __device__ __forceinline__ void accumulate(double (&acc)[K][VEC], IP it, uint32_t b, uint32_t e,
                                                    const float* __restrict__ grads, int D, int q) {
    for (uint32_t j = b; j < e; j += UNR) {
      V v[UNR][K];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        if (j + u < e) {
          const float* g = grads + (size_t)item_pos(it[j + u]) * (size_t)D;
#pragma unroll
          for (int k = 0; k < K; ++k) {
            const int col = (k * LPR + q) * VEC;
            if (col < D) v[u][k] = load_vec<VEC>(g + col);
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
              for (int x = 0; x < VEC; ++x) acc[k][x] += (double)VecT<VEC>::get(v[u][k], x);
            }
          }
        }
      }
    }
  }

  // Current row values (or the initial row of a key new in this call).
  static __device__ __forceinline__ void load_w(V (&w)[K], const float* __restrict__ rows, uint32_t row,
                                                bool isnew, uint64_t s0, int D, int q) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
      if (col < D) {
        if (isnew) w[k] = init_vec<VEC>(s0, col);
        else w[k] = load_vec<VEC>(rows + (size_t)row * (size_t)D + col);
      }
    }
  }

  // g = fp32(acc); m = fp32(sum g^2 / D) over the group's lanes; G' = G + m;
  // den = sqrt(G') + eps; w -= lr * (g / den); writes w and G'.
  static __device__ __forceinline__ void adagrad(const double (&acc)[K][VEC], V (&w)[K], float G0,
                                                 float* __restrict__ rows, float* __restrict__ state,
                                                 uint32_t row, int D, int q, int leader, float lr,
                                                 float eps) {
    float gf[K][VEC];
    double sq = 0.0;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
#pragma unroll
      for (int x = 0; x < VEC; ++x) {
        gf[k][x] = (float)acc[k][x];
        if (col + x < D) sq += (double)gf[k][x] * (double)gf[k][x];
      }
    }
#pragma unroll
    for (int o = LPR / 2; o > 0; o >>= 1) sq += __shfl_xor(sq, o, 64);
    const float m = (float)(sq / (double)D);
    const float G = __shfl(G0, leader, 64);
    const float Gn = __fadd_rn(G, m);
    const float den = __fadd_rn(__builtin_sqrtf(Gn), eps);  // correctly rounded sqrt
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int col = (k * LPR + q) * VEC;
      if (col < D) {
#pragma unroll
        for (int x = 0; x < VEC; ++x) {
          const float qv = __fdiv_rn(gf[k][x], den);
          const float p = __fmul_rn(lr, qv);
          VecT<VEC>::set(w[k], x, __fsub_rn(VecT<VEC>::get(w[k], x), p));
        }
        store_vec<VEC>(rows + (size_t)row * (size_t)D + col, w[k]);
      }
    }
    if (q == 0) state[row] = Gn;
  }

  static __device__ __forceinline__ void zero(double (&acc)[K][VEC]) {
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int x = 0; x < VEC; ++x) acc[k][x] = 0.0;
  }
};

struct RedCtx {
  Bucket* idx;
  const float* grads;
  const double* partials;
  float* rows;
  float* state;
  int D;
  uint64_t seed;
  float lr;
  float eps;
  uint64_t size0;
};

// Run-length encodes the sorted items: seg[s] = first item of segment s,
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

// Keys first inserted by this call (their items sort last) get rows
// size0 + rank among all new keys of the call; the row replaces the slot in
// the segment's first item, whose "fresh" bit stays set.
template <int NT, class IP, class SP>
__device__ __forceinline__ void resolve_new_rows(IP it, SP seg, uint32_t S, uint32_t mp, const RedCtx& c,
                                                 const NewKey* __restrict__ newlist,
                                                 const uint32_t* __restrict__ tile_cnt, int ntiles,
                                                 uint32_t* s_pref, uint32_t* s_w,
                                                 unsigned long long* s_w64, uint64_t* s_chunk) {
  if (!item_fresh(it[mp - 1])) return;  // block-uniform: no key of this partition is new
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
    const uint64_t npend = block_sum_u64<NT>(pend ? 1u : 0u, s_w64);
    if (npend == 0) continue;
    const uint64_t key = pend ? c.idx[slot / kSlots].key[slot % kSlots] : 0ull;
    uint32_t rank = 0;
    for_each_new_key_chunk<NT>(newlist, tile_cnt, ntiles, kPutTile, s_pref, s_w, s_chunk,
                               [&](const uint64_t* ck, uint32_t cnt) {
                                 if (pend)
                                   for (uint32_t e = 0; e < cnt; ++e) rank += ck[e] < key ? 1u : 0u;
                               });
    if (pend) {
      const uint32_t row = (uint32_t)(c.size0 + rank);
      c.idx[slot / kSlots].row[slot % kSlots] = row;
      it[seg[s]] = make_item(true, row, item_low31(x));
      // the new row starts from its initial value and a zero accumulator
      const uint64_t s0 = splitmix_mix(key ^ c.seed);
      float* w = c.rows + (size_t)row * (size_t)c.D;
      for (int col = 0; col < c.D; ++col) w[col] = init_elem(s0, col);
      c.state[row] = 0.0f;
    }
  }
  __syncthreads();
}

// Applies every segment. Each lane group takes an equal contiguous slice of
// the sorted items and walks it in batches: the gradient rows of a batch and
// the row / accumulator of every segment that ends in the batch are loaded
// together, then segments are summed (fp64) and the ones that start in the
// slice are updated. The piece of a segment that began before the slice goes
// to s_part[group]; after a barrier, the group where a cut segment began adds
// the pieces of the following groups in slice order and updates it.
template <class M, int NT, class IP, class SP, class DP>
__device__ __forceinline__ void apply_segments(IP it, SP seg, DP sid, uint32_t mp, const RedCtx& c,
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
  const int leader = g * LPR;
  const int D = c.D;

  const uint32_t L = (mp + NG - 1) / NG;
  const uint32_t lo = min(mp, (uint32_t)gid * L);
  const uint32_t hi = min(mp, lo + L);

  double acc[K][VEC];
  Ops::zero(acc);
  for (uint32_t j0 = lo; j0 < hi; j0 += B) {
    V gv[B][K];
    double pv[B][K][VEC];
    V wv[B][K];
    float G0[B];
    uint32_t sj[B];
    bool ends[B], owned[B], summ[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t j = j0 + u;
      ends[u] = false;
      owned[u] = false;
      summ[u] = false;
      G0[u] = 0.0f;
      if (j < hi) {
        const uint64_t x = it[j];
        sj[u] = sid[j];
        summ[u] = item_summed(x);
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
        ends[u] = seg[sj[u] + 1] == j + 1;
        owned[u] = seg[sj[u]] >= lo;
        if (ends[u] && owned[u]) {
          const uint32_t row = item_tag(it[seg[sj[u]]]);
          Ops::load_w(wv[u], c.rows, row, false, 0, D, q);
          G0[u] = c.state[row];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t j = j0 + u;
      if (j < hi) {
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
            Ops::adagrad(acc, wv[u], G0[u], c.rows, c.state, item_tag(it[seg[sj[u]]]), D, q, leader, c.lr,
                         c.eps);
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
    const uint32_t row = item_tag(it[seg[tail]]);
    V w[K];
    Ops::load_w(w, c.rows, row, false, 0, D, q);
    const float G = c.state[row];
    Ops::adagrad(acc, w, G, c.rows, c.state, row, D, q, leader, c.lr, c.eps);
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
  resolve_new_rows<NT>(it, seg, S, mp, c, newlist, tile_cnt, ntiles, s_pref, s_w, s_w64,
                       reinterpret_cast<uint64_t*>(s_part));
  apply_segments<M, NT>(it, seg, sid, mp, c, s_part);
}

template <class M>
__global__ __launch_bounds__(kRedThreads, (M::K * M::VEC >= 16) ? 2 : 4) void k_reduce_update(
    Bucket* __restrict__ idx, const uint64_t* __restrict__ items, const uint32_t* __restrict__ meta,
    int ntiles, const NewKey* __restrict__ newlist, const uint32_t* __restrict__ tile_cnt,
    const float* __restrict__ grads, const double* __restrict__ partials, float* __restrict__ rows, float* __restrict__ state, int D,
    uint64_t seed, float lr, float eps, int64_t capacity, Ctrl* ctrl, uint64_t epoch,
    uint64_t* __restrict__ spill, uint64_t spill_words) {
  constexpr int NT = kRedThreads;
  constexpr int NW = NT / 64;

  extern __shared__ double s_dyn[];  // pieces of cut segments [lane groups][D], or a chunk of new keys
  __shared__ uint64_t s_items[kRedCap];
  __shared__ uint16_t s_sid[kRedCap];
  __shared__ uint16_t s_seg[kRedCap + 1];
  __shared__ uint32_t s_pref[NT + 1];
  __shared__ uint32_t s_w[NW];
  __shared__ unsigned long long s_w64[NW];
  __shared__ uint64_t s_base;

  const uint32_t p = blockIdx.x;
  const int tid = threadIdx.x;
  const uint64_t size0 = ctrl->size[epoch & 1];
  const bool any_new = ctrl->new_epoch == epoch;
  const uint32_t* pm = meta + (size_t)p * ntiles;

  // entries of this partition in every tile
  uint64_t mp64 = 0;
  for (int t = tid; t < ntiles; t += NT) mp64 += pm[t] >> 16;
  const uint32_t mp = (uint32_t)block_sum_u64<NT>(mp64, s_w64);

  const uint64_t Mnew = any_new ? count_new_keys<NT>(tile_cnt, ntiles, s_w64) : 0ull;
  const int err = call_verdict(ctrl, epoch, size0, Mnew, capacity);
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

  const RedCtx c{idx, grads, partials, rows, state, D, seed, lr, eps, size0};
  if (mp > (uint32_t)kRedCap) {
    reduce_partition_global<M, NT>(p, mp, items, meta, ntiles, c, newlist, tile_cnt, ctrl, spill, spill_words,
                                   s_dyn, s_pref, s_w, s_w64, &s_base);
    return;
  }

  // ---- gather the partition's items into LDS ----
  {
    uint32_t dst = 0;
    for (int t0 = 0; t0 < ntiles; t0 += NT) {
      const int t = t0 + tid;
      const uint32_t mt = t < ntiles ? pm[t] : 0u;
      const uint32_t off = mt & 0xFFFFu, cnt = mt >> 16;
      uint32_t tot;
      const uint32_t pre = block_exclusive_scan<NT>(cnt, s_w, &tot);
      for (uint32_t j = 0; j < cnt; ++j) s_items[dst + pre + j] = items[(size_t)t * kPutTile + off + j];
      dst += tot;
    }
    __syncthreads();
  }

  // ---- sort: an item's rank is the number of smaller items (all items are
  // distinct, since positions are) ----
  {
    constexpr int IPT = kRedCap / NT;
    uint64_t v[IPT];
    uint32_t rk[IPT];
    int mine = 0;
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
      const uint32_t k = tid + j * NT;
      v[j] = k < mp ? s_items[k] : ~0ull;
      rk[j] = 0;
      mine += k < mp ? 1 : 0;
    }
    if (mine > 0) {
      for (uint32_t e = 0; e < mp; ++e) {
        const uint64_t a = s_items[e];
#pragma unroll
        for (int j = 0; j < IPT; ++j) rk[j] += a < v[j] ? 1u : 0u;
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < IPT; ++j)
      if (tid + j * NT < mp) s_items[rk[j]] = v[j];
    __syncthreads();
  }

  const uint32_t S = encode_segments<NT>(s_items, mp, s_seg, s_sid, s_w);
  resolve_new_rows<NT>(s_items, s_seg, S, mp, c, newlist, tile_cnt, ntiles, s_pref, s_w, s_w64,
                       reinterpret_cast<uint64_t*>(s_dyn));
  apply_segments<M, NT>(s_items, s_seg, s_sid, mp, c, s_dyn);
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
__global__ __launch_bounds__(256) void k_read_rows(const float* __restrict__ rows, const float* __restrict__ state,
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
    if (w_out) w_out[e] = ok ? rows[(uint64_t)r * (uint64_t)D + c] : __builtin_nanf("");
    if (st_out && c == 0) st_out[i] = ok ? state[r] : __builtin_nanf("");
  }
}

// ===========================================================================
// Launchers
// ===========================================================================
template <class M>
static hipError_t launch_get_t(const GetArgs& a, hipStream_t st, const LaunchHook& hook) {
  const int64_t ntiles = (a.n + kGetTile - 1) / kGetTile;
  hook(K_GET_PROBE_GATHER, 0, st);
  hipLaunchKernelGGL(k_get_probe_gather<M>, dim3((unsigned)ntiles), dim3(kGetTile), 0, st, a.idx,
                     a.nb_log2, a.keys, a.n, a.out, a.rows, a.D, a.seed, a.newlist, a.tile_cnt, a.ctrl,
                     a.epoch);
  hook(K_GET_PROBE_GATHER, 1, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int grid = (int)std::min<int64_t>(ntiles, 256);
  hook(K_ASSIGN_NEW, 0, st);
  hipLaunchKernelGGL(k_assign_new, dim3(grid), dim3(kAssignThreads), 0, st, a.idx, a.newlist,
                     a.tile_cnt, (int)ntiles, kGetTile, a.rows, a.state, a.D, a.seed, a.capacity,
                     a.ctrl, a.epoch);
  hook(K_ASSIGN_NEW, 1, st);
  return hipGetLastError();
}

template <class M>
static size_t reduce_dyn_bytes(int D) {
  const size_t part = (size_t)(kRedThreads / 64) * M::RPW * (size_t)D * sizeof(double);
  const size_t chunk = (size_t)kChunk * sizeof(uint64_t);
  return part > chunk ? part : chunk;
}

template <class M>
static hipError_t launch_put_t(const PutArgs& a, hipStream_t st, const LaunchHook& hook) {
  const int64_t ntiles = (a.n + kPutTile - 1) / kPutTile;
  hook(K_PUT_PROBE, 0, st);
  hipLaunchKernelGGL(k_put_probe<M>, dim3((unsigned)ntiles), dim3(kPutThreads), 0, st, a.idx, a.nb_log2,
                     a.keys, a.grads, a.n, a.D, a.pb, (int)ntiles, a.items, a.meta, a.partials,
                     a.newlist, a.tile_cnt, a.ctrl, a.epoch);
  hook(K_PUT_PROBE, 1, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const size_t dyn = reduce_dyn_bytes<M>(a.D);
  static bool attr_set = false;
  if (!attr_set) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_reduce_update<M>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hook(K_REDUCE_UPDATE, 0, st);
  hipLaunchKernelGGL(k_reduce_update<M>, dim3(1u << a.pb), dim3(kRedThreads), dyn, st, a.idx, a.items,
                     a.meta, (int)ntiles, a.newlist, a.tile_cnt, a.grads, a.partials, a.rows, a.state,
                     a.D, a.seed, a.lr, a.eps, a.capacity, a.ctrl, a.epoch, a.spill, a.spill_words);
  hook(K_REDUCE_UPDATE, 1, st);
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

hipError_t launch_put(const PutArgs& a, bool vec4, hipStream_t st, const LaunchHook& hook) {
  return dispatch_map(a.D, vec4, [&](auto m) { return launch_put_t<decltype(m)>(a, st, hook); });
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

hipError_t launch_read_rows(const float* rows, const float* state, int D, const unsigned long long* size_now,
                            const int64_t* ids, int64_t n, float* w_out, float* st_out, Ctrl* ctrl,
                            hipStream_t st) {
  const uint64_t total = (uint64_t)n * (uint64_t)D;
  const uint64_t grid = std::min<uint64_t>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_read_rows, dim3((unsigned)grid), dim3(256), 0, st, rows, state, D, size_now, ids, n,
                     w_out, st_out, ctrl);
  return hipGetLastError();
}

}  // namespace mlkv
