// Index work of the joint pass: the distinct element set U(z) with occurrence ranks
// (Section 4.1), row gathers of element embeddings (Section 4.2), index-based sequence
// assembly with positions added after the gather (Section 4.3), and the score head with the
// argmax of eq. (1).
#include "fe_common.h"
#include "fe_dedup.h"
#include "flasheval.h"

#include <climits>

namespace {

// ------------------------------------------------------------------------------------------
// U(z): one workgroup per request (fe_dedup.h).
// ------------------------------------------------------------------------------------------

// The distinct set of request b = xcd_tile(blockIdx.x, B) (XCD-contiguous requests, so the
// kernels after it, mapped the same way, read slot and the element rows from their own L2):
// writes uniq (ascending, padded with -1 up to U_cap), n_uniq, slot and the status word, and,
// when s_uniq != nullptr, the distinct ids into LDS s_uniq[0 .. U).  bits and pre are LDS arrays
// of (M + 31) / 32 words.  Returns U; the ids in s_uniq are visible to the whole workgroup when
// it returns.
FE_DEV int dedup_request(const int32_t* __restrict__ lists, int KL, int M, int U_cap, int32_t* __restrict__ uniq,
                         int32_t* __restrict__ n_uniq, int32_t* __restrict__ slot, int32_t* __restrict__ status,
                         uint32_t* bits, uint32_t* pre, int32_t* s_uniq) {
  const int b = xcd_tile(blockIdx.x, gridDim.x);
  int bad = 0;
  const int U = fe_dedup::distinct_set<256>(lists + (long long)b * KL, KL, M, U_cap, uniq + (long long)b * U_cap,
                                            slot + (long long)b * KL, &bad, bits, pre, s_uniq);
  if (threadIdx.x == 0) {
    n_uniq[b] = (int32_t)U;
    status[b] = bad ? FE_DEV_BAD_INDEX : 0;
  }
  return U;
}

__global__ __launch_bounds__(256) void k_dedup(const int32_t* __restrict__ lists, int KL, int M, int U_cap,
                                               int32_t* __restrict__ uniq, int32_t* __restrict__ n_uniq,
                                               int32_t* __restrict__ slot, int32_t* __restrict__ status) {
  extern __shared__ uint32_t sm[];
  const int W = (M + 31) >> 5;
  dedup_request(lists, KL, M, U_cap, uniq, n_uniq, slot, status, sm, sm + W, nullptr);
}

// The distinct set and its element rows in one launch, for requests whose rows are few:
// out[b][r] = table[b][uniq[b][r]] (VPR 16-byte vectors per row) for r < U, zero rows up to
// U_cap.  Each thread keeps NI row loads in flight.
template <int VPR>
__global__ __launch_bounds__(256) void k_dedup_gather(const int32_t* __restrict__ lists, int KL, int M, int U_cap,
                                                      int32_t* __restrict__ uniq, int32_t* __restrict__ n_uniq,
                                                      int32_t* __restrict__ slot, int32_t* __restrict__ status,
                                                      const uint4* __restrict__ table, long long table_bs_v,
                                                      uint4* __restrict__ out) {
  extern __shared__ uint32_t sm[];
  const int W = (M + 31) >> 5;
  int32_t* s_uniq = reinterpret_cast<int32_t*>(sm + 2 * W);
  const int U = dedup_request(lists, KL, M, U_cap, uniq, n_uniq, slot, status, sm, sm + W, s_uniq);
  constexpr int RPI = 256 / VPR, NI = 8;
  const int b = xcd_tile(blockIdx.x, gridDim.x);
  const int v = threadIdx.x % VPR, rr = threadIdx.x / VPR;
  const uint4* tb = table + b * table_bs_v;
  uint4* ob = out + (long long)b * U_cap * VPR;
  for (int r0 = rr; r0 < U_cap; r0 += NI * RPI) {
    uint4 val[NI];
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = r0 + i * RPI;
      val[i] = make_uint4(0u, 0u, 0u, 0u);
      if (r < U) val[i] = tb[(long long)s_uniq[r] * VPR + v];
    }
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int r = r0 + i * RPI;
      if (r < U_cap) ob[(long long)r * VPR + v] = val[i];
    }
  }
}

// ------------------------------------------------------------------------------------------
// Row gather: out[b][r] = table[b][idx[b][r]] for r < nvalid[b], zero rows otherwise.  One
// 16-byte vector per thread; an id outside the table gives a zero row and a status bit.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gather_rows(const uint4* __restrict__ table, long long table_bs_v,
                                                     int n_rows_table, const int32_t* __restrict__ idx, int idx_bs,
                                                     const int32_t* __restrict__ nvalid, int B, int rows, int vpr,
                                                     uint4* __restrict__ out, int32_t* __restrict__ status,
                                                     int status_bit) {
  const long long total = (long long)B * rows * vpr;
  for (long long e = blockIdx.x * 256ll + threadIdx.x; e < total; e += (long long)gridDim.x * 256) {
    const long long row = e / vpr;
    const int v = (int)(e - row * vpr);
    const int b = (int)(row / rows), r = (int)(row - (long long)b * rows);
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (!nvalid || r < nvalid[b]) {
      const int id = idx[(long long)b * idx_bs + r];
      if (id >= 0 && id < n_rows_table) val = table[b * table_bs_v + (long long)id * vpr + v];
      else if (v == 0 && status) atomicOr(&status[b], status_bit);
    }
    out[e] = val;
  }
}

// ------------------------------------------------------------------------------------------
// Sequence assembly: seq[b][k][0] = cls + pos[0], seq[b][k][j+1] = H[b][slot] + pos[j+1].
// Pure data movement, bound by the HBM write of seq and by the latency of its two dependent
// loads (slot, then the element row).  A row is VPR 16-byte vectors; a workgroup owns
// NI * (256 / VPR) consecutive output rows and each thread NI of them (one vector each), so a
// thread's NI slot loads, then its NI row loads, are in flight together.
// Workgroups take XCD-contiguous row ranges (xcd_tile): XCD x assembles the lists of the x-th
// eighth of the requests, whose element rows H the item kernels wrote through that XCD's L2,
// and whose sequences the sequence encoder reads there next.  The sum is taken in fp32 and
// rounded once; an occurrence whose slot lies outside [0, U_cap) gives a zero row.
// ------------------------------------------------------------------------------------------
template <typename T, int VPR, int NI>
__global__ __launch_bounds__(256) void k_assemble(const int32_t* __restrict__ slot, const T* __restrict__ H,
                                                  int K, int L, int U_cap, int rows, const T* __restrict__ cls,
                                                  const T* __restrict__ pos, T* __restrict__ seq) {
  constexpr int VEC = 16 / sizeof(T), RPI = 256 / VPR;
  const int S = L + 1;
  const int v = threadIdx.x % VPR, rr = threadIdx.x / VPR;
  const int row0 = xcd_tile(blockIdx.x, gridDim.x) * (RPI * NI) + rr;
  const uint4* H4 = reinterpret_cast<const uint4*>(H);
  int src[NI], jpos[NI];   // src: H vector index, -1 for [CLS], -2 for a zero row
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int r = row0 + i * RPI;
    const int bk = r / S, j = r - bk * S;
    jpos[i] = j;
    src[i] = -2;
    if (r < rows) {
      if (j == 0) {
        src[i] = -1;
      } else {
        const int s = slot[bk * L + j - 1];
        if (s >= 0 && s < U_cap) src[i] = ((bk / K) * U_cap + s) * VPR + v;
      }
    }
  }
  uint4 a[NI], p[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    a[i] = src[i] >= 0 ? H4[src[i]] : reinterpret_cast<const uint4*>(cls)[v];
    p[i] = reinterpret_cast<const uint4*>(pos)[jpos[i] * VPR + v];
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int r = row0 + i * RPI;
    if (r >= rows) continue;
    const T* x = reinterpret_cast<const T*>(&a[i]);
    const T* q = reinterpret_cast<const T*>(&p[i]);
    T res[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) res[e] = src[i] == -2 ? from_f32<T>(0.f) : from_f32<T>(to_f32(x[e]) + to_f32(q[e]));
    reinterpret_cast<uint4*>(seq)[r * VPR + v] = *reinterpret_cast<const uint4*>(res);
  }
}

// Smallest index of the largest non-NaN value of s_score[0..K), -1 if every value is NaN; every
// thread of the 256-thread block calls it and gets the result.  Candidates are merged by the
// total order (larger value first, then smaller index) -- within each wave by a shuffle
// butterfly, then across the four waves through s_val / s_idx -- so the result does not depend
// on the merge order.
FE_DEV void select_merge(float& bv, int& bi, float ov, int oi) {
  if (oi >= 0 && (bi < 0 || ov > bv || (ov == bv && oi < bi))) {
    bv = ov;
    bi = oi;
  }
}

FE_DEV int block_select(const float* s_score, int K, float* s_val, int* s_idx) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  float bv = 0.f;
  int bi = -1;
  for (int k = tid; k < K; k += 256) {
    const float v = s_score[k];
    if (v != v) continue;
    select_merge(bv, bi, v, k);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o, 64);
    const int oi = __shfl_xor(bi, o, 64);
    select_merge(bv, bi, ov, oi);
  }
  if (lane == 0) {
    s_val[wave] = bv;
    s_idx[wave] = bi;
  }
  __syncthreads();
  float rv = s_val[0];
  int ri = s_idx[0];
#pragma unroll
  for (int w = 1; w < 4; ++w) select_merge(rv, ri, s_val[w], s_idx[w]);
  return ri;
}

// ------------------------------------------------------------------------------------------
// Score head and selection: one workgroup per request (XCD-contiguous, like the cross-sequence
// module that wrote Cp).  A group of LPR = min(16, D/4) lanes forms one dot product (lane l sums
// columns 4(l + LPR*i) .. +3 in a fixed order, then a fixed butterfly over the group), so
// identical rows give identical scores wherever they sit; each thread keeps RPT rows in flight.  A
// block reduction then keeps the largest non-NaN score with the smallest index.
// ------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void k_score_select(const float* __restrict__ Cp, int K, const float* __restrict__ w,
                                                      const float* __restrict__ bias, float* __restrict__ scores,
                                                      int32_t* __restrict__ best) {
  constexpr int LPR = D / 4 < 16 ? D / 4 : 16, NV = D / (4 * LPR), NG = 256 / LPR, RPT = 4;
  __shared__ float s_val[256];
  __shared__ int s_idx[256];
  __shared__ float s_score[4096];
  const int b = xcd_tile(blockIdx.x, gridDim.x), tid = threadIdx.x, l16 = tid % LPR, grp = tid / LPR;
  const float* cb = Cp + (long long)b * K * D;
  float4 wv[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) wv[i] = *reinterpret_cast<const float4*>(&w[4 * (l16 + LPR * i)]);
  const float b0 = bias[0];
  for (int k0 = grp; k0 < K; k0 += NG * RPT) {
    float4 xv[RPT][NV];
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      const int k = min(k0 + NG * r, K - 1);
#pragma unroll
      for (int i = 0; i < NV; ++i) xv[r][i] = *reinterpret_cast<const float4*>(&cb[(long long)k * D + 4 * (l16 + LPR * i)]);
    }
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < NV; ++i)
        acc += xv[r][i].x * wv[i].x + xv[r][i].y * wv[i].y + xv[r][i].z * wv[i].z + xv[r][i].w * wv[i].w;
#pragma unroll
      for (int o = 1; o < LPR; o <<= 1) acc += __shfl_xor(acc, o, LPR);
      const int k = k0 + NG * r;
      if (l16 == 0 && k < K) {
        scores[(long long)b * K + k] = acc + b0;
        s_score[k] = acc + b0;
      }
    }
  }
  __syncthreads();
  const int bi = block_select(s_score, K, s_val, s_idx);
  if (tid == 0) best[b] = bi;
}

// Section 4.4, multi-objective form: NOBJ task heads on the shared C'_k, fused by a weighted sum.
// One workgroup per request; head weights staged in LDS; each LPR-lane group takes one list at a
// time, reads C'_k once and forms every head's dot product from it.
//   obj[b][k][t] = C'_k . W[t] + bias[t];   fused[b][k] = sum_t alpha[t] obj[b][k][t] (t ascending)
//   best[b] = smallest k with the largest fused score, NaN skipped, -1 if all NaN.
template <int D>
__global__ __launch_bounds__(256) void k_score_objectives(const float* __restrict__ Cp, int K, int nobj,
                                                          const float* __restrict__ W, const float* __restrict__ bias,
                                                          const float* __restrict__ alpha, float* __restrict__ obj,
                                                          float* __restrict__ fused, int32_t* __restrict__ best) {
  constexpr int LPR = D / 4 < 16 ? D / 4 : 16, NV = D / (4 * LPR), NG = 256 / LPR;
  __shared__ __attribute__((aligned(16))) float s_w[FE_MAX_OBJECTIVES * D];
  __shared__ float s_val[256];
  __shared__ int s_idx[256];
  __shared__ float s_score[4096];
  const int b = xcd_tile(blockIdx.x, gridDim.x), tid = threadIdx.x, l16 = tid % LPR, grp = tid / LPR;
  for (int e = tid; e < nobj * D; e += 256) s_w[e] = W[e];
  __syncthreads();
  const float* cb = Cp + (long long)b * K * D;
  for (int k = grp; k < K; k += NG) {
    float4 xv[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) xv[i] = *reinterpret_cast<const float4*>(&cb[(long long)k * D + 4 * (l16 + LPR * i)]);
    float f = 0.f;
    for (int t = 0; t < nobj; ++t) {
      const float4* wt = reinterpret_cast<const float4*>(s_w + t * D);
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const float4 wv = wt[l16 + LPR * i];
        acc += xv[i].x * wv.x + xv[i].y * wv.y + xv[i].z * wv.z + xv[i].w * wv.w;
      }
#pragma unroll
      for (int o = 1; o < LPR; o <<= 1) acc += __shfl_xor(acc, o, LPR);
      const float st = acc + bias[t];
      if (l16 == 0) obj[((long long)b * K + k) * nobj + t] = st;
      f = t == 0 ? alpha[0] * st : fmaf(alpha[t], st, f);
    }
    if (l16 == 0) {
      fused[(long long)b * K + k] = f;
      s_score[k] = f;
    }
  }
  __syncthreads();
  const int bi = block_select(s_score, K, s_val, s_idx);
  if (tid == 0) best[b] = bi;
}

__global__ void k_fill_i32(int32_t* p, int n, int32_t v) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) p[i] = v;
}

// dst block (b * reps + r) = src block b, blocks of `words` 32-bit words (grid-stride; r < reps)
__global__ void k_repeat_blocks(const uint32_t* src, uint32_t* dst, long long words, int nblk, int reps) {
  const long long total = (long long)nblk * reps * words;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < total; e += (long long)gridDim.x * 256) {
    const long long blk = e / words, w = e - blk * words;
    dst[e] = src[(blk / reps) * words + w];
  }
}

// slot_k[q][j] = slot_all[q][q % K][j] for q < BK: list (q % K)'s ranks out of the slot map of all K
// lists that request q saw
__global__ void k_take_list_slots(const int32_t* slot_all, int32_t* slot_k, int BK, int K, int L) {
  const long long n = (long long)BK * L;
  for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n; e += (long long)gridDim.x * 256) {
    const long long q = e / L, j = e - q * L;
    slot_k[e] = slot_all[(q * K + q % K) * L + j];
  }
}

int grid_for(long long work) {
  long long g = (work + 255) / 256;
  if (g > 65536) g = 65536;
  return (int)(g < 1 ? 1 : g);
}

}  // namespace

hipError_t launch_fill_i32(int32_t* p, int n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

hipError_t launch_repeat_blocks(const void* src, void* dst, long long block_bytes, int nblk, int reps, hipStream_t s) {
  if (block_bytes % 4 != 0) return hipErrorInvalidValue;
  const long long words = block_bytes / 4;
  if (words == 0 || nblk <= 0 || reps <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_repeat_blocks, dim3(grid_for((long long)nblk * reps * words)), dim3(256), 0, s,
                     static_cast<const uint32_t*>(src), static_cast<uint32_t*>(dst), words, nblk, reps);
  return hipGetLastError();
}

hipError_t launch_take_list_slots(const int32_t* slot_all, int32_t* slot_k, int BK, int K, int L, hipStream_t s) {
  if (BK <= 0 || L <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_take_list_slots, dim3(grid_for((long long)BK * L)), dim3(256), 0, s, slot_all, slot_k, BK, K, L);
  return hipGetLastError();
}

hipError_t launch_dedup(const int32_t* lists, int B, int KL, int M, int U_cap, int32_t* uniq, int32_t* n_uniq,
                        int32_t* slot, int32_t* status, hipStream_t s) {
  const size_t lds = 2 * (size_t)((M + 31) / 32) * sizeof(uint32_t);
  hipLaunchKernelGGL(k_dedup, dim3(B), dim3(256), lds, s, lists, KL, M, U_cap, uniq, n_uniq, slot, status);
  return hipGetLastError();
}

bool dedup_gather_fits(int U_cap, int d, bool bf16_model) {
  const long long bytes = (long long)U_cap * d * (bf16_model ? 2 : 4);
  return bytes <= (128 << 10);
}

hipError_t launch_dedup_gather(const int32_t* lists, int B, int KL, int M, int U_cap, int32_t* uniq, int32_t* n_uniq,
                               int32_t* slot, int32_t* status, const void* table, long long table_bs, int d,
                               void* out, bool bf16_model, hipStream_t s) {
  if (!dedup_gather_fits(U_cap, d, bf16_model)) return hipErrorInvalidValue;
  const int esz = bf16_model ? 2 : 4;
  const int vpr = d * esz / 16;
  const size_t lds = (2 * (size_t)((M + 31) / 32) + U_cap) * sizeof(uint32_t);
  const uint4* t = static_cast<const uint4*>(table);
  uint4* o = static_cast<uint4*>(out);
  const long long tbs = table_bs * esz / 16;
#define FE_DG(V) hipLaunchKernelGGL(k_dedup_gather<V>, dim3(B), dim3(256), lds, s, lists, KL, M, U_cap, uniq, n_uniq, \
                                    slot, status, t, tbs, o)
  switch (vpr) {
    case 8: FE_DG(8); break;
    case 16: FE_DG(16); break;
    case 32: FE_DG(32); break;
    case 64: FE_DG(64); break;
    case 128: FE_DG(128); break;
    default: return hipErrorInvalidValue;
  }
#undef FE_DG
  return hipGetLastError();
}

hipError_t launch_gather_rows(const void* table, long long table_bs, int n_rows_table, const int32_t* idx, int idx_bs,
                              const int32_t* nvalid, int B, int rows, int d, void* out, int32_t* status,
                              int status_bit, bool bf16_model, hipStream_t s) {
  const int esz = bf16_model ? 2 : 4;
  const int vpr = d * esz / 16;
  const long long work = (long long)B * rows * vpr;
  hipLaunchKernelGGL(k_gather_rows, dim3(grid_for(work)), dim3(256), 0, s, static_cast<const uint4*>(table),
                     table_bs * esz / 16, n_rows_table, idx, idx_bs, nvalid, B, rows, vpr,
                     static_cast<uint4*>(out), status, status_bit);
  return hipGetLastError();
}

template <typename T, int VPR>
void assemble_as(const int32_t* slot, const void* H, int K, int L, int U_cap, int rows, const void* cls,
                 const void* pos, void* seq, hipStream_t s) {
  constexpr int NI = 1, RPB = NI * (256 / VPR);   // one row per thread: more workgroups beat more rows in flight per thread
  const int grid = (rows + RPB - 1) / RPB;
  hipLaunchKernelGGL((k_assemble<T, VPR, NI>), dim3(grid), dim3(256), 0, s, slot, static_cast<const T*>(H), K, L,
                     U_cap, rows, static_cast<const T*>(cls), static_cast<const T*>(pos), static_cast<T*>(seq));
}

hipError_t launch_assemble(const int32_t* slot, const void* H, int B, int K, int L, int U_cap, int d, const void* cls,
                           const void* pos, void* seq, bool bf16_model, hipStream_t s) {
  const long long rows = (long long)B * K * (L + 1);
  const long long vpr = (long long)d * (bf16_model ? 2 : 4) / 16;
  // every vector index of seq and H must fit the kernel's 32-bit arithmetic
  if (rows * vpr > INT_MAX || (long long)B * U_cap * vpr > INT_MAX) return hipErrorInvalidValue;
  if (rows == 0) return hipSuccess;
  const int R = (int)rows;
#define FE_ASM(TT, V) assemble_as<TT, V>(slot, H, K, L, U_cap, R, cls, pos, seq, s)
  if (bf16_model) {
    switch (vpr) {
      case 16: FE_ASM(bf16, 16); break;
      case 32: FE_ASM(bf16, 32); break;
      case 64: FE_ASM(bf16, 64); break;
      default: return hipErrorInvalidValue;
    }
  } else {
    switch (vpr) {
      case 8: FE_ASM(float, 8); break;
      case 16: FE_ASM(float, 16); break;
      case 32: FE_ASM(float, 32); break;
      case 64: FE_ASM(float, 64); break;
      case 128: FE_ASM(float, 128); break;
      default: return hipErrorInvalidValue;
    }
  }
#undef FE_ASM
  return hipGetLastError();
}

hipError_t launch_score_objectives(const float* Cp, int B, int K, int d, int nobj, const float* W, const float* bias,
                                   const float* alpha, float* obj, float* fused, int32_t* best, hipStream_t s) {
  if (nobj < 1 || nobj > FE_MAX_OBJECTIVES || K > 4096) return hipErrorInvalidValue;
#define FE_OBJ(DD) hipLaunchKernelGGL(k_score_objectives<DD>, dim3(B), dim3(256), 0, s, Cp, K, nobj, W, bias, alpha, obj, fused, best)
  switch (d) {
    case 32: FE_OBJ(32); break;
    case 64: FE_OBJ(64); break;
    case 128: FE_OBJ(128); break;
    case 256: FE_OBJ(256); break;
    case 512: FE_OBJ(512); break;
    default: return hipErrorInvalidValue;
  }
#undef FE_OBJ
  return hipGetLastError();
}

hipError_t launch_score_select(const float* Cp, int B, int K, int d, const float* w, const float* bias, float* scores,
                               int32_t* best, hipStream_t s) {
  switch (d) {
    case 32: hipLaunchKernelGGL(k_score_select<32>, dim3(B), dim3(256), 0, s, Cp, K, w, bias, scores, best); break;
    case 64: hipLaunchKernelGGL(k_score_select<64>, dim3(B), dim3(256), 0, s, Cp, K, w, bias, scores, best); break;
    case 128: hipLaunchKernelGGL(k_score_select<128>, dim3(B), dim3(256), 0, s, Cp, K, w, bias, scores, best); break;
    case 256: hipLaunchKernelGGL(k_score_select<256>, dim3(B), dim3(256), 0, s, Cp, K, w, bias, scores, best); break;
    case 512: hipLaunchKernelGGL(k_score_select<512>, dim3(B), dim3(256), 0, s, Cp, K, w, bias, scores, best); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
