// The distinct element set U(z) of one request (Section 4.1), shared by the index kernels and the
// item-set attention kernel that builds it in its own prologue.  A bitmap of M bits in LDS marks
// the elements that occur; an exclusive scan of per-word popcounts gives every element its rank,
// so the distinct ids come out in ascending order and slot = rank(element) is exact and
// deterministic.
#pragma once

#include "fe_common.h"

namespace fe_dedup {

// Exclusive prefix sum of one value per thread over a workgroup of NT threads (wave scans on
// lane shuffles, then the wave totals through LDS s_wave[NT / 64]); *total receives the sum.
template <int NT>
FE_DEV uint32_t block_exclusive_scan(uint32_t x, uint32_t* s_wave, uint32_t* total) {
  constexpr int NW = NT / 64;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t inc = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(inc, o, 64);
    if (lane >= o) inc += t;
  }
  if (lane == 63) s_wave[wave] = inc;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    before += w < wave ? s_wave[w] : 0u;
    all += s_wave[w];
  }
  *total = all;
  return before + inc - x;
}

// Distinct set of the KL list entries lb[] over elements 0..M-1, for a workgroup of NT threads.
// Writes, when the pointers are set: ub[0 .. U_cap) = the distinct ids ascending, padded with -1;
// sb[i] = rank of lb[i] among them (-1 for an entry outside [0, M)); s_uniq[0 .. U) = the distinct
// ids in LDS (U <= U_cap is guaranteed by U_cap = min(M, KL)).  *bad = 1 if some entry lies
// outside [0, M).  bits and pre are LDS arrays of (M + 31) / 32 words.  Returns U; s_uniq and the
// return value are valid for the whole workgroup on return.
template <int NT>
FE_DEV int distinct_set(const int32_t* __restrict__ lb, int KL, int M, int U_cap, int32_t* __restrict__ ub,
                        int32_t* __restrict__ sb, int* bad_out, uint32_t* bits, uint32_t* pre, int32_t* s_uniq) {
  __shared__ uint32_t s_wave[NT / 64];
  const int W = (M + 31) >> 5;
  const int tid = threadIdx.x;
  for (int i = tid; i < W; i += NT) bits[i] = 0u;
  __syncthreads();
  int bad = 0;
  for (int i = tid; i < KL; i += NT) {
    const int v = lb[i];
    if (v >= 0 && v < M) atomicOr(&bits[v >> 5], 1u << (v & 31));
    else bad = 1;
  }
  bad = __syncthreads_or(bad);

  // per-thread contiguous chunk of words, then a block-wide exclusive scan of the chunk sums
  const int chunk = (W + NT - 1) / NT;
  const int w0 = min(W, tid * chunk), w1 = min(W, w0 + chunk);
  uint32_t local = 0;
  for (int w = w0; w < w1; ++w) local += __popc(bits[w]);
  uint32_t total;
  uint32_t run = block_exclusive_scan<NT>(local, s_wave, &total);
  for (int w = w0; w < w1; ++w) {
    pre[w] = run;
    uint32_t m = bits[w];
    while (m) {
      const int t = __ffs(m) - 1;
      const int id = (w << 5) + t;
      if (ub) ub[run] = id;
      if (s_uniq) s_uniq[run] = id;
      ++run;
      m &= m - 1;
    }
  }
  if (ub)
    for (int i = (int)total + tid; i < U_cap; i += NT) ub[i] = -1;
  __syncthreads();
  if (sb)
    for (int i = tid; i < KL; i += NT) {
      const int v = lb[i];
      int s = -1;
      if (v >= 0 && v < M) s = (int)(pre[v >> 5] + __popc(bits[v >> 5] & ((1u << (v & 31)) - 1u)));
      sb[i] = s;
    }
  *bad_out = bad;
  return (int)total;
}

}  // namespace fe_dedup
