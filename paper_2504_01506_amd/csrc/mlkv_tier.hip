// Tiered tables: rows at home in pinned host memory, a fixed number of them
// cached in HBM. Lookahead (Sec. III-A, look-ahead prefetching of Sec. III-C2)
// makes the rows of a batch resident in the cache ahead of their gets:
//   mark    every position's row: a cached one is kept for this call, an
//           uncached one is claimed (once per row) as a miss;
//   plan    one block walks the cache slots from a FIFO cursor and gives the
//           misses the first slots this call does not keep, evicting their
//           rows (dirty ones are written back); misses beyond the slots that
//           are free to take stay at home;
//   copy    a wave per planned slot writes back the evicted row, then copies
//           the missing row in, over the host link.
// Gets and puts read and write rows wherever they are (RowStore), so the
// cache never changes a result.
#include "mlkv_kernels.h"

namespace mlkv {

constexpr uint32_t kClaimed = 0xFFFFFFFEu;  // slot_of_row of a miss claimed by the current call
constexpr int kMarkThreads = 256;
constexpr int kPlanThreads = 1024;
constexpr int kCopyThreads = 256;
constexpr int kCopyRows = 4;  // rows a wave copies at a time

__global__ __launch_bounds__(kMarkThreads) void k_tier_mark(const int64_t* __restrict__ rows_of_pos, int64_t n,
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
    r = rows_of_pos[i];  // -1: key absent (a failed insert)
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

__global__ __launch_bounds__(kPlanThreads) void k_tier_plan(uint32_t* __restrict__ slot_of_row,
                                                            uint32_t* __restrict__ row_of_slot,
                                                            uint8_t* __restrict__ dirty,
                                                            const uint32_t* __restrict__ keep, uint32_t tag,
                                                            const uint32_t* __restrict__ miss,
                                                            uint32_t* __restrict__ plan_slot,
                                                            uint32_t* __restrict__ plan_old,
                                                            uint32_t* __restrict__ plan_new, uint64_t C, Ctrl* ctrl,
                                                            uint32_t parity) {
  constexpr int NT = kPlanThreads;
  __shared__ uint32_t s_w[NT / 64];
  __shared__ unsigned long long s_w64[NT / 64];
  const uint64_t M = ctrl->tier_nmiss[parity];
  const uint64_t cur = ctrl->tier_cursor;
  // the first M slots from the cursor on that this call does not keep
  uint64_t found = 0;
  for (uint64_t i0 = 0; i0 < C && found < M; i0 += NT) {
    const uint64_t i = i0 + threadIdx.x;
    const uint64_t s = (cur + i) % C;
    const uint32_t cand = (i < C && keep[s] != tag) ? 1u : 0u;
    uint32_t tot;
    const uint32_t pre = block_exclusive_scan<NT>(cand, s_w, &tot);
    const uint64_t v = found + pre;
    if (cand && v < M) plan_slot[v] = (uint32_t)s;
    found += tot;
  }
  const uint64_t A = found < M ? found : M;
  __syncthreads();  // the plan's slots are written
  // the taken slots change hands; misses without a slot stay at home
  uint64_t ev = 0, wb = 0;
  for (uint64_t v = threadIdx.x; v < M; v += NT) {
    const uint32_t r = miss[v];
    if (v >= A) {
      slot_of_row[r] = kNoSlot;
      continue;
    }
    const uint32_t s = plan_slot[v];
    const uint32_t old = row_of_slot[s];
    const bool write_back = old != kNoSlot && dirty[s] != 0;
    if (old != kNoSlot) {
      slot_of_row[old] = kNoSlot;
      ++ev;
    }
    wb += write_back ? 1 : 0;
    plan_old[v] = write_back ? old : kNoSlot;
    plan_new[v] = r;
    row_of_slot[s] = r;
    slot_of_row[r] = s;
    dirty[s] = 0;
  }
  ev = block_sum_u64<NT>(ev, s_w64);
  wb = block_sum_u64<NT>(wb, s_w64);
  // the cursor moves past the last slot taken
  __shared__ unsigned long long s_last;
  if (threadIdx.x == 0) s_last = cur;
  __syncthreads();
  if (A > 0 && threadIdx.x == 0) s_last = (plan_slot[A - 1] + 1) % C;
  __syncthreads();
  if (threadIdx.x == 0) {
    ctrl->tier_cursor = s_last;
    ctrl->tier_nplan = A;
    ctrl->tier_loaded += A;
    ctrl->tier_evicted += ev;
    ctrl->tier_written += wb;
    ctrl->tier_filled += A - ev;
  }
}

// A wave per planned slot (kCopyRows slots at a time): the evicted dirty row
// goes back to its home, then the missing row comes in.
__global__ __launch_bounds__(kCopyThreads) void k_tier_copy(const uint32_t* __restrict__ plan_slot,
                                                            const uint32_t* __restrict__ plan_old,
                                                            const uint32_t* __restrict__ plan_new,
                                                            const Ctrl* ctrl, float* __restrict__ cache,
                                                            float* __restrict__ host, int D) {
  const uint64_t A = ctrl->tier_nplan;
  const int lane = threadIdx.x & 63;
  const uint64_t waves = (uint64_t)gridDim.x * (kCopyThreads / 64);
  const uint64_t w0 = (uint64_t)blockIdx.x * (kCopyThreads / 64) + (threadIdx.x >> 6);
  for (uint64_t e0 = w0 * kCopyRows; e0 < A; e0 += waves * kCopyRows) {
    uint32_t s[kCopyRows], old[kCopyRows], nw[kCopyRows];
#pragma unroll
    for (int u = 0; u < kCopyRows; ++u) {
      const uint64_t e = e0 + u;
      s[u] = e < A ? plan_slot[e] : kNoSlot;
      old[u] = e < A ? plan_old[e] : kNoSlot;
      nw[u] = e < A ? plan_new[e] : kNoSlot;
    }
    for (int col = lane; col < D; col += 64) {
      float wv[kCopyRows], nv[kCopyRows];
#pragma unroll
      for (int u = 0; u < kCopyRows; ++u) {
        if (old[u] != kNoSlot) wv[u] = cache[(size_t)s[u] * D + col];
        if (nw[u] != kNoSlot) nv[u] = host[(size_t)nw[u] * D + col];
      }
#pragma unroll
      for (int u = 0; u < kCopyRows; ++u) {
        if (old[u] != kNoSlot) host[(size_t)old[u] * D + col] = wv[u];
        if (nw[u] != kNoSlot) cache[(size_t)s[u] * D + col] = nv[u];
      }
    }
  }
}

hipError_t launch_tier_lookahead(const TierArgs& a, hipStream_t st, const LaunchHook& hook) {
  if (a.n == 0) return hipSuccess;
  hook(K_TIER_MARK, 0, st);
  const int64_t mb = (a.n + kMarkThreads - 1) / kMarkThreads;
  hipLaunchKernelGGL(k_tier_mark, dim3((unsigned)mb), dim3(kMarkThreads), 0, st, a.rows_of_pos, a.n, a.slot_of_row,
                     a.keep, a.tag, a.miss, a.ctrl, a.parity);
  hook(K_TIER_MARK, 1, st);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hook(K_TIER_PLAN, 0, st);
  hipLaunchKernelGGL(k_tier_plan, dim3(1), dim3(kPlanThreads), 0, st, a.slot_of_row, a.row_of_slot, a.dirty, a.keep,
                     a.tag, a.miss, a.plan_slot, a.plan_old, a.plan_new, (uint64_t)a.cache_rows, a.ctrl, a.parity);
  hook(K_TIER_PLAN, 1, st);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t most = std::min<int64_t>(a.n, a.cache_rows);
  const int64_t per_block = (kCopyThreads / 64) * kCopyRows;
  const int64_t cb = std::max<int64_t>(1, std::min<int64_t>((most + per_block - 1) / per_block, 2048));
  hook(K_TIER_COPY, 0, st);
  hipLaunchKernelGGL(k_tier_copy, dim3((unsigned)cb), dim3(kCopyThreads), 0, st, a.plan_slot, a.plan_old,
                     a.plan_new, a.ctrl, a.cache, a.host, a.D);
  hook(K_TIER_COPY, 1, st);
  return hipGetLastError();
}

}  // namespace mlkv
