// Tiered tables: rows at home in pinned host memory, a fixed number of them
// cached in HBM. Lookahead (Sec. III-A, look-ahead prefetching of Sec. III-C2)
// makes the rows of a batch resident in the cache ahead of their gets:
//   mark    every position's row (the row the lookahead's get found there,
//           or, for a key it inserted, a lookup) is marked: a cached one is
//           kept for this call, an uncached one is claimed (once per row) as
//           a miss;
//   plan    one block walks the cache slots from a FIFO cursor and gives the
//           misses the first slots this call does not keep (row by row of
//           contiguous slots, places counted by wave ballots and a scan);
//   copy    a wave per four misses moves the directory entries (the slot's
//           old row goes home, the missing row comes in; misses beyond the
//           slots free to take stay at home), writes the evicted row back if
//           it is dirty, then copies the missing row in, over the host link.
// A taken slot is not kept by the call, so its old row is not one the call
// asked for, and every miss is claimed once: the entries each miss changes
// are its own, and the copy kernel changes them in parallel.
// Gets and puts read and write rows wherever they are (RowStore), so the
// cache never changes a result.
#include "mlkv_kernels.h"

namespace mlkv {

constexpr uint32_t kClaimed = 0xFFFFFFFEu;  // slot_of_row of a miss claimed by the current call
constexpr int kMarkThreads = 1024;  // one miss-counter addition per block, few blocks
constexpr int kPlanThreads = 1024;
constexpr int kCopyThreads = 256;
constexpr int kCopyRows = 4;  // rows a wave copies at a time
constexpr int kPlanPer = 16;  // rows of kPlanThreads consecutive cache slots a plan pass examines

__global__ __launch_bounds__(kMarkThreads) void k_tier_mark(Bucket* __restrict__ idx, uint32_t nb_log2,
                                                            const uint64_t* __restrict__ keys,
                                                            const uint64_t* __restrict__ pc_key,
                                                            const uint32_t* __restrict__ pc_row, int64_t n,
                                                            uint32_t* __restrict__ slot_of_row,
                                                            uint32_t* __restrict__ keep, uint32_t tag,
                                                            uint32_t* __restrict__ miss, Ctrl* ctrl,
                                                            uint32_t parity) {
  __shared__ uint32_t s_cnt, s_base;
  if (blockIdx.x == 0 && threadIdx.x == 0) ctrl->tier_nmiss[parity ^ 1u] = 0;  // for the next call
  if (threadIdx.x == 0) s_cnt = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * kMarkThreads + threadIdx.x;
  int64_t r = -1;
  uint32_t mine = 0xFFFFFFFFu;
  if (i < n) {
    const uint64_t key = keys[i];
    if (key != kEmptyKey && pc_key[i] == key) {
      r = pc_row[i];  // present before the call: the get recorded its row here
    } else if (key != kEmptyKey) {
      const Probe pr = probe_key(idx, nb_log2, key, false);
      if (pr.status == P_HIT) r = pr.row;  // else absent (the call's insert failed)
    }
    if (r >= 0) {
      const uint32_t s = slot_of_row[r];
      if (s < kClaimed) {
        keep[s] = tag;
      } else if (s == kNoSlot && atomicCAS(&slot_of_row[r], kNoSlot, kClaimed) == kNoSlot) {
        mine = atomicAdd(&s_cnt, 1u);
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0 && s_cnt > 0)
    s_base = (uint32_t)atomicAdd(&ctrl->tier_nmiss[parity], (unsigned long long)s_cnt);
  __syncthreads();
  if (mine != 0xFFFFFFFFu) miss[s_base + mine] = (uint32_t)r;
}

__global__ __launch_bounds__(kPlanThreads) void k_tier_plan(const uint32_t* __restrict__ keep, uint32_t tag,
                                                            uint32_t* __restrict__ plan_slot, uint64_t C, Ctrl* ctrl,
                                                            uint32_t parity) {
  constexpr int NT = kPlanThreads, NW = NT / 64;
  static_assert(kPlanPer * NW <= NT, "one scan entry per (row, wave)");
  __shared__ uint32_t s_row[kPlanPer * NW];  // free slots per (row, wave), then the slots before them
  __shared__ uint32_t s_w[NW];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const uint64_t below = lane ? (~0ull >> (64 - lane)) : 0ull;
  const uint64_t M = ctrl->tier_nmiss[parity];
  const uint64_t cur = ctrl->tier_cursor;
  // the first M slots from the cursor on that this call does not keep. A pass
  // examines kPlanPer rows of NT consecutive slots, thread t the t-th slot of
  // each row, so that the loads of a row are contiguous; a slot's place among
  // the free ones counts the free slots of earlier rows, of earlier waves in
  // its row and of earlier lanes in its wave (a ballot)
  uint64_t found = 0;
  for (uint64_t i0 = 0; i0 < C && found < M; i0 += (uint64_t)NT * kPlanPer) {
    // slot of position i from the cursor: cur + i < 2C, so one subtraction wraps it
    auto slot_at = [&](uint64_t i) { const uint64_t x = cur + i; return x >= C ? x - C : x; };
    uint32_t mine = 0;  // bit j: this thread's slot of row j is free to take
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j) {
      const uint64_t i = i0 + (uint64_t)j * NT + threadIdx.x;
      if (i < C && keep[slot_at(i)] != tag) mine |= 1u << j;
    }
    uint64_t bal[kPlanPer];
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j) {
      bal[j] = __ballot((mine >> j) & 1u);
      if (lane == 0) s_row[j * NW + w] = (uint32_t)__popcll(bal[j]);
    }
    __syncthreads();
    const uint32_t c = threadIdx.x < kPlanPer * NW ? s_row[threadIdx.x] : 0u;
    uint32_t tot;
    const uint32_t pre = block_exclusive_scan<NT>(c, s_w, &tot);  // its barriers: every count above is read
    if (threadIdx.x < kPlanPer * NW) s_row[threadIdx.x] = pre;
    __syncthreads();
#pragma unroll
    for (int j = 0; j < kPlanPer; ++j) {
      if ((mine >> j) & 1u) {
        const uint64_t v = found + s_row[j * NW + w] + (uint64_t)__popcll(bal[j] & below);
        if (v < M) plan_slot[v] = (uint32_t)slot_at(i0 + (uint64_t)j * NT + threadIdx.x);
      }
    }
    __syncthreads();  // s_row is rewritten by the next pass
    found += tot;
  }
  const uint64_t A = found < M ? found : M;
  __syncthreads();  // the plan's slots are written
  if (threadIdx.x == 0) {
    ctrl->tier_cursor = A > 0 ? (plan_slot[A - 1] + 1 == C ? 0 : plan_slot[A - 1] + 1) : cur;  // past the last slot taken
    ctrl->tier_nplan = A;
  }
}

// A wave per kCopyRows misses: a miss given a slot moves in (its slot's old
// row goes home, written back first if dirty), a miss beyond the slots free
// to take stays at home. Counters are added once per block.
__global__ __launch_bounds__(kCopyThreads) void k_tier_copy(const uint32_t* __restrict__ miss,
                                                            const uint32_t* __restrict__ plan_slot,
                                                            uint32_t* __restrict__ slot_of_row,
                                                            uint32_t* __restrict__ row_of_slot,
                                                            uint8_t* __restrict__ dirty, Ctrl* ctrl, uint32_t parity,
                                                            float* __restrict__ cache, float* __restrict__ host,
                                                            int D) {
  __shared__ unsigned long long s_ev, s_wb, s_in;
  if (threadIdx.x == 0) s_ev = s_wb = s_in = 0;
  __syncthreads();
  const uint64_t M = ctrl->tier_nmiss[parity];
  const uint64_t A = ctrl->tier_nplan;
  const int lane = threadIdx.x & 63;
  const uint64_t waves = (uint64_t)gridDim.x * (kCopyThreads / 64);
  const uint64_t w0 = (uint64_t)blockIdx.x * (kCopyThreads / 64) + (threadIdx.x >> 6);
  uint32_t ev = 0, wbn = 0, inn = 0;
  for (uint64_t e0 = w0 * kCopyRows; e0 < M; e0 += waves * kCopyRows) {
    uint32_t s[kCopyRows], old[kCopyRows], nw[kCopyRows];
    bool back[kCopyRows];
#pragma unroll
    for (int u = 0; u < kCopyRows; ++u) {
      const uint64_t e = e0 + u;
      s[u] = kNoSlot;
      old[u] = kNoSlot;
      nw[u] = kNoSlot;
      back[u] = false;
      if (e < M) {
        const uint32_t r = miss[e];
        if (e < A) {
          s[u] = plan_slot[e];
          old[u] = row_of_slot[s[u]];
          back[u] = old[u] != kNoSlot && dirty[s[u]] != 0;
          nw[u] = r;
        } else if (lane == 0) {
          slot_of_row[r] = kNoSlot;  // no slot for it: it stays at home
        }
      }
    }
    // the directory (one lane per entry; the copies below read no entry)
    if (lane == 0) {
#pragma unroll
      for (int u = 0; u < kCopyRows; ++u) {
        if (nw[u] == kNoSlot) continue;
        if (old[u] != kNoSlot) slot_of_row[old[u]] = kNoSlot;
        row_of_slot[s[u]] = nw[u];
        slot_of_row[nw[u]] = s[u];
        dirty[s[u]] = 0;
        ev += old[u] != kNoSlot ? 1u : 0u;
        wbn += back[u] ? 1u : 0u;
        inn += 1u;
      }
    }
    for (int col = lane; col < D; col += 64) {
      float wv[kCopyRows], nv[kCopyRows];
#pragma unroll
      for (int u = 0; u < kCopyRows; ++u) {
        if (back[u]) wv[u] = cache[(size_t)s[u] * D + col];
        if (nw[u] != kNoSlot) nv[u] = host[(size_t)nw[u] * D + col];
      }
#pragma unroll
      for (int u = 0; u < kCopyRows; ++u) {
        if (back[u]) host[(size_t)old[u] * D + col] = wv[u];
        if (nw[u] != kNoSlot) cache[(size_t)s[u] * D + col] = nv[u];
      }
    }
  }
  if (lane == 0 && inn > 0) {
    atomicAdd(&s_ev, (unsigned long long)ev);
    atomicAdd(&s_wb, (unsigned long long)wbn);
    atomicAdd(&s_in, (unsigned long long)inn);
  }
  __syncthreads();
  if (threadIdx.x == 0 && s_in > 0) {
    atomicAdd(&ctrl->tier_loaded, s_in);
    atomicAdd(&ctrl->tier_evicted, s_ev);
    atomicAdd(&ctrl->tier_written, s_wb);
    atomicAdd(&ctrl->tier_filled, s_in - s_ev);
  }
}

hipError_t launch_tier_lookahead(const TierArgs& a, hipStream_t st, const LaunchHook& hook) {
  if (a.n == 0) return hipSuccess;
  hook(K_TIER_MARK, 0, st);
  const int64_t mb = (a.n + kMarkThreads - 1) / kMarkThreads;
  hipLaunchKernelGGL(k_tier_mark, dim3((unsigned)mb), dim3(kMarkThreads), 0, st, a.idx, a.nb_log2, a.keys,
                     a.pc_key, a.pc_row, a.n, a.slot_of_row,
                     a.keep, a.tag, a.miss, a.ctrl, a.parity);
  hook(K_TIER_MARK, 1, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hook(K_TIER_PLAN, 0, st);
  hipLaunchKernelGGL(k_tier_plan, dim3(1), dim3(kPlanThreads), 0, st, a.keep, a.tag, a.plan_slot,
                     (uint64_t)a.cache_rows, a.ctrl, a.parity);
  hook(K_TIER_PLAN, 1, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // every miss (at most n) gets a wave's turn; at most 256 blocks, which
  // keep enough rows in flight for the host link and add the counters once each
  const int64_t per_block = (kCopyThreads / 64) * kCopyRows;
  const int64_t cb = std::max<int64_t>(1, std::min<int64_t>((a.n + per_block - 1) / per_block, 256));
  hook(K_TIER_COPY, 0, st);
  hipLaunchKernelGGL(k_tier_copy, dim3((unsigned)cb), dim3(kCopyThreads), 0, st, a.miss, a.plan_slot, a.slot_of_row,
                     a.row_of_slot, a.dirty, a.ctrl, a.parity, a.cache, a.host, a.D);
  hook(K_TIER_COPY, 1, st);
  return hipGetLastError();
}

}  // namespace mlkv
