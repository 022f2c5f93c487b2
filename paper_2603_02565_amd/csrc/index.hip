// Index work of the joint pass: the distinct element set U(z) with occurrence ranks
// (Section 4.1), row gathers of element embeddings (Section 4.2), index-based sequence
// assembly with positions added after the gather (Section 4.3), and the score head with the
// argmax of eq. (1).
#include "fe_common.h"
#include "flasheval.h"

namespace {

// ------------------------------------------------------------------------------------------
// U(z): one workgroup per request.  A bitmap of M bits in LDS marks the elements that occur;
// an exclusive scan of per-word popcounts gives every element its rank, so uniq comes out in
// ascending order and slot = rank(element) is exact and deterministic.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_dedup(const int32_t* __restrict__ lists, int KL, int M, int U_cap,
                                               int32_t* __restrict__ uniq, int32_t* __restrict__ n_uniq,
                                               int32_t* __restrict__ slot, int32_t* __restrict__ status) {
  extern __shared__ uint32_t sm[];
  __shared__ uint32_t s_part[256];
  const int W = (M + 31) >> 5;
  uint32_t* bits = sm;
  uint32_t* pre = sm + W;
  const int b = blockIdx.x, tid = threadIdx.x;
  const int32_t* lb = lists + (long long)b * KL;

  for (int i = tid; i < W; i += 256) bits[i] = 0u;
  __syncthreads();
  int bad = 0;
  for (int i = tid; i < KL; i += 256) {
    const int v = lb[i];
    if (v >= 0 && v < M) atomicOr(&bits[v >> 5], 1u << (v & 31));
    else bad = 1;
  }
  bad = __syncthreads_or(bad);

  // per-thread contiguous chunk of words, then a block-wide exclusive scan of the chunk sums
  const int chunk = (W + 255) / 256;
  const int w0 = min(W, tid * chunk), w1 = min(W, w0 + chunk);
  uint32_t local = 0;
  for (int w = w0; w < w1; ++w) local += __popc(bits[w]);
  s_part[tid] = local;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const uint32_t add = tid >= off ? s_part[tid - off] : 0u;
    __syncthreads();
    s_part[tid] += add;
    __syncthreads();
  }
  const uint32_t total = s_part[255];
  uint32_t run = s_part[tid] - local;
  int32_t* ub = uniq + (long long)b * U_cap;
  for (int w = w0; w < w1; ++w) {
    pre[w] = run;
    uint32_t m = bits[w];
    while (m) {
      const int t = __ffs(m) - 1;
      ub[run++] = (w << 5) + t;
      m &= m - 1;
    }
  }
  for (int i = (int)total + tid; i < U_cap; i += 256) ub[i] = -1;
  __syncthreads();
  int32_t* sb = slot + (long long)b * KL;
  for (int i = tid; i < KL; i += 256) {
    const int v = lb[i];
    int s = -1;
    if (v >= 0 && v < M) s = (int)(pre[v >> 5] + __popc(bits[v >> 5] & ((1u << (v & 31)) - 1u)));
    sb[i] = s;
  }
  if (tid == 0) {
    n_uniq[b] = (int32_t)total;
    status[b] = bad ? FE_DEV_BAD_INDEX : 0;
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
// Each thread produces one 16-byte vector of one output row; the sum is taken in fp32 and
// rounded once.  Pure data movement: bound by the HBM write of seq.
// ------------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void k_assemble(const int32_t* __restrict__ slot, const T* __restrict__ H,
                                                  int B, int K, int L, int U_cap, int d, const T* __restrict__ cls,
                                                  const T* __restrict__ pos, T* __restrict__ seq) {
  constexpr int VEC = 16 / sizeof(T);
  const int vpr = d / VEC;
  const int S = L + 1;
  const long long total = (long long)B * K * S * vpr;
  for (long long e = blockIdx.x * 256ll + threadIdx.x; e < total; e += (long long)gridDim.x * 256) {
    const long long orow = e / vpr;
    const int v = (int)(e - orow * vpr);
    const long long bk = orow / S;
    const int j = (int)(orow - bk * S);
    const int b = (int)(bk / K);
    T src[VEC], pv[VEC], res[VEC];
    *reinterpret_cast<uint4*>(pv) = reinterpret_cast<const uint4*>(pos + (long long)j * d)[v];
    bool zero = false;
    if (j == 0) {
      *reinterpret_cast<uint4*>(src) = reinterpret_cast<const uint4*>(cls)[v];
    } else {
      const int s = slot[bk * L + (j - 1)];
      if (s >= 0 && s < U_cap) *reinterpret_cast<uint4*>(src) = reinterpret_cast<const uint4*>(H + ((long long)b * U_cap + s) * d)[v];
      else zero = true;
    }
#pragma unroll
    for (int i = 0; i < VEC; ++i) res[i] = zero ? from_f32<T>(0.f) : from_f32<T>(to_f32(src[i]) + to_f32(pv[i]));
    reinterpret_cast<uint4*>(seq)[e] = *reinterpret_cast<uint4*>(res);
  }
}

// Smallest index of the largest non-NaN value of s_score[0..K), -1 if every value is NaN; every
// thread of the 256-thread block calls it and gets the result.
FE_DEV int block_select(const float* s_score, int K, float* s_val, int* s_idx) {
  const int tid = threadIdx.x;
  float bv = 0.f;
  int bi = -1;
  for (int k = tid; k < K; k += 256) {
    const float v = s_score[k];
    if (v != v) continue;
    if (bi < 0 || v > bv) { bv = v; bi = k; }
  }
  s_val[tid] = bv;
  s_idx[tid] = bi;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (tid < off) {
      const float ov = s_val[tid + off];
      const int oi = s_idx[tid + off];
      const int mi = s_idx[tid];
      if (oi >= 0 && (mi < 0 || ov > s_val[tid] || (ov == s_val[tid] && oi < mi))) {
        s_val[tid] = ov;
        s_idx[tid] = oi;
      }
    }
    __syncthreads();
  }
  return s_idx[0];
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

hipError_t launch_assemble(const int32_t* slot, const void* H, int B, int K, int L, int U_cap, int d, const void* cls,
                           const void* pos, void* seq, bool bf16_model, hipStream_t s) {
  const int esz = bf16_model ? 2 : 4;
  const long long work = (long long)B * K * (L + 1) * (d * esz / 16);
  if (bf16_model)
    hipLaunchKernelGGL(k_assemble<bf16>, dim3(grid_for(work)), dim3(256), 0, s, slot, static_cast<const bf16*>(H), B, K,
                       L, U_cap, d, static_cast<const bf16*>(cls), static_cast<const bf16*>(pos), static_cast<bf16*>(seq));
  else
    hipLaunchKernelGGL(k_assemble<float>, dim3(grid_for(work)), dim3(256), 0, s, slot, static_cast<const float*>(H), B,
                       K, L, U_cap, d, static_cast<const float*>(cls), static_cast<const float*>(pos),
                       static_cast<float*>(seq));
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
