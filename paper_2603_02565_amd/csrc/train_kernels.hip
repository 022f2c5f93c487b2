// fp32 kernels of the training step (Section 4.5): the forward with saved activations and its
// backward.  Plain, general kernels: a batched strided product, row-wise LayerNorm and softmax
// with their backward passes, elementwise steps, row gathers and their scatter-add backward, and
// the losses with the label construction of Appendix B.1.
#include "fe_common.h"
#include "train_kernels.h"

#include <algorithm>
#include <initializer_list>

namespace {

// ------------------------------------------------------------------------------------------
// C[z] = alpha * op(A[z]) op(B[z]) + beta * C[z] (+ bias[j]); element (i, k) of A[z] at
// A + z1*a_b1 + z2*a_b2 + i*a_rs + k*a_cs (likewise B with (k, j), C with (i, j) and unit column
// stride), z = z1*nb2 + z2.
//
// fp32 matrix cores: a workgroup of four waves owns a (32 WM) x (32 WN) output tile, each wave one
// 32 x 32 block accumulated by v_mfma_f32_32x32x2_f32 (lane l feeds A[l%32][l/32] and
// B[l/32][l%32] of a 32x32x2 step and holds D[8q + 4(l/32) + e][l%32] in accumulator 4q + e).
// k advances in steps of 32 through LDS, the next step's operands loaded into registers while
// the current step's products run.  AK / BK: the operand's k index is its contiguous one,
// so consecutive lanes load along k (else along i or j), which keeps the global loads coalesced
// for both orientations.
// ------------------------------------------------------------------------------------------
constexpr int GK = 32;
typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int WM, int WN, bool AK, bool BK, bool VA, bool VB>
__global__ __launch_bounds__(256) void k_gemm(TGemm g, int z0, int nz) {
  static_assert(WM * WN == 4, "four waves");
  constexpr int TM = 32 * WM, TN = 32 * WN, PA = TM + 4, PB = TN + 4;
  constexpr int NA = GK * TM / 256, NB = GK * TN / 256;   // elements per thread per k-step
  __shared__ __align__(16) float As[GK][PA];
  __shared__ __align__(16) float Bs[GK][PB];
  const int zz = z0 + blockIdx.z, z = zz % nz, kc = zz / nz;
  const int z1 = z / g.nb2, z2 = z % g.nb2;
  const int kbeg = g.ksplit > 0 ? kc * g.ksplit : 0;
  const int kend = g.ksplit > 0 ? min(g.K, kbeg + g.ksplit) : g.K;
  const float* A = g.A + z1 * g.a_b1 + z2 * g.a_b2;
  const float* B = g.B + z1 * g.b_b1 + z2 * g.b_b2;
  float* C = g.C + z1 * g.c_b1 + z2 * g.c_b2;
  const float* Rz = g.R + z1 * g.c_b1 + z2 * g.c_b2;
  const float* Mz = g.mask + z1 * g.c_b1 + z2 * g.c_b2;
  const int i0 = blockIdx.y * TM, j0 = blockIdx.x * TN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wi = (wave / WN) * 32, wj = (wave % WN) * 32;
  const int lr = lane & 31, lk = lane >> 5;
  float ra[NA], rb[NB];
  // the operands of k-step k0 into registers (zero outside the matrices and past kend).  VA / VB:
  // four consecutive elements of the contiguous index per load (the launcher has checked that
  // they are 16-byte aligned); NA / NB stay the number of scalars per thread.
  auto load = [&](int k0) {
    if constexpr (VA) {
#pragma unroll
      for (int q = 0; q < NA / 4; ++q) {
        const int e = threadIdx.x + 256 * q;
        const int i = AK ? i0 + e / (GK / 4) : i0 + 4 * (e % (TM / 4));
        const int k = AK ? k0 + 4 * (e % (GK / 4)) : k0 + e / (TM / 4);
        const float* src = A + i * g.a_rs + k * g.a_cs;
        if (AK ? (i < g.M && k + 3 < kend) : (i + 3 < g.M && k < kend)) {
          const float4 v = *reinterpret_cast<const float4*>(src);
          ra[4 * q] = v.x; ra[4 * q + 1] = v.y; ra[4 * q + 2] = v.z; ra[4 * q + 3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            ra[4 * q + c] = (AK ? (i < g.M && k + c < kend) : (i + c < g.M && k < kend))
                                ? src[AK ? c : c * g.a_rs] : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < NA; ++t) {
        const int e = threadIdx.x + 256 * t;
        const int kk = AK ? e % GK : e / TM, mm = AK ? e / GK : e % TM;
        const int i = i0 + mm, k = k0 + kk;
        ra[t] = (i < g.M && k < kend) ? A[i * g.a_rs + k * g.a_cs] : 0.f;
      }
    }
    if constexpr (VB) {
#pragma unroll
      for (int q = 0; q < NB / 4; ++q) {
        const int e = threadIdx.x + 256 * q;
        const int j = BK ? j0 + e / (GK / 4) : j0 + 4 * (e % (TN / 4));
        const int k = BK ? k0 + 4 * (e % (GK / 4)) : k0 + e / (TN / 4);
        const float* src = B + k * g.b_rs + j * g.b_cs;
        if (BK ? (j < g.N && k + 3 < kend) : (j + 3 < g.N && k < kend)) {
          const float4 v = *reinterpret_cast<const float4*>(src);
          rb[4 * q] = v.x; rb[4 * q + 1] = v.y; rb[4 * q + 2] = v.z; rb[4 * q + 3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            rb[4 * q + c] = (BK ? (j < g.N && k + c < kend) : (j + c < g.N && k < kend))
                                ? src[BK ? c : c * g.b_cs] : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        const int e = threadIdx.x + 256 * t;
        const int kk = BK ? e % GK : e / TN, nn = BK ? e / GK : e % TN;
        const int j = j0 + nn, k = k0 + kk;
        rb[t] = (j < g.N && k < kend) ? B[k * g.b_rs + j * g.b_cs] : 0.f;
      }
    }
  };
  auto store = [&]() {
    if constexpr (VA) {
#pragma unroll
      for (int q = 0; q < NA / 4; ++q) {
        const int e = threadIdx.x + 256 * q;
        if constexpr (AK) {
          const int mm = e / (GK / 4), kq = 4 * (e % (GK / 4));
#pragma unroll
          for (int c = 0; c < 4; ++c) As[kq + c][mm] = ra[4 * q + c];
        } else {
          *reinterpret_cast<float4*>(&As[e / (TM / 4)][4 * (e % (TM / 4))]) =
              make_float4(ra[4 * q], ra[4 * q + 1], ra[4 * q + 2], ra[4 * q + 3]);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < NA; ++t) {
        const int e = threadIdx.x + 256 * t;
        As[AK ? e % GK : e / TM][AK ? e / GK : e % TM] = ra[t];
      }
    }
    if constexpr (VB) {
#pragma unroll
      for (int q = 0; q < NB / 4; ++q) {
        const int e = threadIdx.x + 256 * q;
        if constexpr (BK) {
          const int nn = e / (GK / 4), kq = 4 * (e % (GK / 4));
#pragma unroll
          for (int c = 0; c < 4; ++c) Bs[kq + c][nn] = rb[4 * q + c];
        } else {
          *reinterpret_cast<float4*>(&Bs[e / (TN / 4)][4 * (e % (TN / 4))]) =
              make_float4(rb[4 * q], rb[4 * q + 1], rb[4 * q + 2], rb[4 * q + 3]);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        const int e = threadIdx.x + 256 * t;
        Bs[BK ? e % GK : e / TN][BK ? e / GK : e % TN] = rb[t];
      }
    }
  };
  f32x16 acc = {};
  const bool csum = g.colsum && blockIdx.y == 0 && threadIdx.x < TN;   // first row tile: column sums of B
  float cs = 0.f;
  load(kbeg);
  for (int k0 = kbeg; k0 < kend; k0 += GK) {
    store();
    __syncthreads();
    if (k0 + GK < kend) load(k0 + GK);   // the next step's loads are in flight during this step's products
#pragma unroll
    for (int t = 0; t < GK / 2; ++t)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[2 * t + lk][wi + lr], Bs[2 * t + lk][wj + lr], acc, 0, 0, 0);
    if (csum)
#pragma unroll
      for (int kk = 0; kk < GK; ++kk) cs += Bs[kk][threadIdx.x];
    __syncthreads();
  }
  if (csum && j0 + (int)threadIdx.x < g.N) atomicAdd(&g.colsum[j0 + threadIdx.x], g.alpha * cs);
  const int j = j0 + wj + lr;
  if (j >= g.N) return;
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = i0 + wi + 8 * q + 4 * lk + e;
      if (i >= g.M) continue;
      float r = g.alpha * acc[4 * q + e];
      const long long o = i * g.c_rs + j;
      float* c = C + o;
      if (g.ksplit > 0) {
        atomicAdd(c, r);
        continue;
      }
      if (g.bias) r += g.bias[j];
      if (g.R) r += Rz[o];
      if (g.relu) r = fmaxf(r, 0.f);
      if (g.mask && !(Mz[o] > 0.f)) r = 0.f;
      *c = g.beta != 0.f ? r + g.beta * *c : r;
    }
}

// Batched products with M, N <= 32 (attention inside short sequences): each wave owns one batch
// item's 32 x 32 tile, four items per workgroup, same k-steps and prefetch as k_gemm.
template <bool AK, bool BK, bool VA, bool VB>
__global__ __launch_bounds__(256) void k_gemm_small(TGemm g, int z0) {
  constexpr int P = 36, N1 = GK * 32 / 64;   // elements per lane per operand per k-step
  __shared__ __align__(16) float As[4][GK][P];
  __shared__ __align__(16) float Bs[4][GK][P];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int z = z0 + blockIdx.x * 4 + wave;
  const bool live = z < g.nbatch;
  const int z1 = live ? z / g.nb2 : 0, z2 = live ? z % g.nb2 : 0;
  const float* A = g.A + z1 * g.a_b1 + z2 * g.a_b2;
  const float* B = g.B + z1 * g.b_b1 + z2 * g.b_b2;
  float* C = g.C + z1 * g.c_b1 + z2 * g.c_b2;
  const float* Rz = g.R + z1 * g.c_b1 + z2 * g.c_b2;
  const float* Mz = g.mask + z1 * g.c_b1 + z2 * g.c_b2;
  const int lr = lane & 31, lk = lane >> 5;
  float ra[N1], rb[N1];
  // VA / VB: four consecutive elements of the contiguous index per load (aligned, checked by the
  // launcher); the registers hold the same N1 scalars either way
  auto load = [&](int k0) {
    if constexpr (VA) {
#pragma unroll
      for (int q = 0; q < N1 / 4; ++q) {
        const int e = lane + 64 * q;
        const int i = AK ? e / (GK / 4) : 4 * (e % 8), k = AK ? k0 + 4 * (e % (GK / 4)) : k0 + e / 8;
        const float* src = A + i * g.a_rs + k * g.a_cs;
        if (live && (AK ? (i < g.M && k + 3 < g.K) : (i + 3 < g.M && k < g.K))) {
          const float4 v = *reinterpret_cast<const float4*>(src);
          ra[4 * q] = v.x; ra[4 * q + 1] = v.y; ra[4 * q + 2] = v.z; ra[4 * q + 3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            ra[4 * q + c] = (live && (AK ? (i < g.M && k + c < g.K) : (i + c < g.M && k < g.K))) ? src[AK ? c : c * g.a_rs] : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < N1; ++t) {
        const int e = lane + 64 * t;
        const int kk = AK ? e % GK : e / 32, mm = AK ? e / GK : e % 32;
        const int k = k0 + kk;
        ra[t] = (live && mm < g.M && k < g.K) ? A[mm * g.a_rs + k * g.a_cs] : 0.f;
      }
    }
    if constexpr (VB) {
#pragma unroll
      for (int q = 0; q < N1 / 4; ++q) {
        const int e = lane + 64 * q;
        const int j = BK ? e / (GK / 4) : 4 * (e % 8), k = BK ? k0 + 4 * (e % (GK / 4)) : k0 + e / 8;
        const float* src = B + k * g.b_rs + j * g.b_cs;
        if (live && (BK ? (j < g.N && k + 3 < g.K) : (j + 3 < g.N && k < g.K))) {
          const float4 v = *reinterpret_cast<const float4*>(src);
          rb[4 * q] = v.x; rb[4 * q + 1] = v.y; rb[4 * q + 2] = v.z; rb[4 * q + 3] = v.w;
        } else {
#pragma unroll
          for (int c = 0; c < 4; ++c)
            rb[4 * q + c] = (live && (BK ? (j < g.N && k + c < g.K) : (j + c < g.N && k < g.K))) ? src[BK ? c : c * g.b_cs] : 0.f;
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < N1; ++t) {
        const int e = lane + 64 * t;
        const int kb = BK ? e % GK : e / 32, nn = BK ? e / GK : e % 32;
        const int kq = k0 + kb;
        rb[t] = (live && nn < g.N && kq < g.K) ? B[kq * g.b_rs + nn * g.b_cs] : 0.f;
      }
    }
  };
  f32x16 acc = {};
  load(0);
  for (int k0 = 0; k0 < g.K; k0 += GK) {
    if constexpr (VA) {
#pragma unroll
      for (int q = 0; q < N1 / 4; ++q) {
        const int e = lane + 64 * q;
        if constexpr (AK) {
#pragma unroll
          for (int c = 0; c < 4; ++c) As[wave][4 * (e % (GK / 4)) + c][e / (GK / 4)] = ra[4 * q + c];
        } else {
          *reinterpret_cast<float4*>(&As[wave][e / 8][4 * (e % 8)]) =
              make_float4(ra[4 * q], ra[4 * q + 1], ra[4 * q + 2], ra[4 * q + 3]);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < N1; ++t) {
        const int e = lane + 64 * t;
        As[wave][AK ? e % GK : e / 32][AK ? e / GK : e % 32] = ra[t];
      }
    }
    if constexpr (VB) {
#pragma unroll
      for (int q = 0; q < N1 / 4; ++q) {
        const int e = lane + 64 * q;
        if constexpr (BK) {
#pragma unroll
          for (int c = 0; c < 4; ++c) Bs[wave][4 * (e % (GK / 4)) + c][e / (GK / 4)] = rb[4 * q + c];
        } else {
          *reinterpret_cast<float4*>(&Bs[wave][e / 8][4 * (e % 8)]) =
              make_float4(rb[4 * q], rb[4 * q + 1], rb[4 * q + 2], rb[4 * q + 3]);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < N1; ++t) {
        const int e = lane + 64 * t;
        Bs[wave][BK ? e % GK : e / 32][BK ? e / GK : e % 32] = rb[t];
      }
    }
    __syncthreads();
    if (k0 + GK < g.K) load(k0 + GK);
#pragma unroll
    for (int t = 0; t < GK / 2; ++t)
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(As[wave][2 * t + lk][lr], Bs[wave][2 * t + lk][lr], acc, 0, 0, 0);
    __syncthreads();
  }
  if (!live || lr >= g.N) return;
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = 8 * q + 4 * lk + e;
      if (i >= g.M) continue;
      float r = g.alpha * acc[4 * q + e];
      const long long o = i * g.c_rs + lr;
      if (g.bias) r += g.bias[lr];
      if (g.R) r += Rz[o];
      if (g.relu) r = fmaxf(r, 0.f);
      if (g.mask && !(Mz[o] > 0.f)) r = 0.f;
      float* c = C + o;
      *c = g.beta != 0.f ? r + g.beta * *c : r;
    }
}

// ------------------------------------------------------------------------------------------
// LayerNorm over rows of d values (biased variance, eps 1e-5): one wave per row.
// ------------------------------------------------------------------------------------------
template <int V>
FE_DEV void ldv(const float* p, float* v) {
  if constexpr (V == 4) {
    const float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (V == 2) {
    const float2 t = *reinterpret_cast<const float2*>(p);
    v[0] = t.x; v[1] = t.y;
  } else {
    v[0] = *p;
  }
}
template <int V>
FE_DEV void stv(float* p, const float* v) {
  if constexpr (V == 4) *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  else if constexpr (V == 2) *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  else *p = v[0];
}

// V consecutive values per lane and load (d a multiple of 64 V, rows and vectors aligned to V floats)
template <int V>
__global__ __launch_bounds__(256) void k_ln_fwd(const float* X, long long x_rs, int rows, int d, const float* g,
                                                const float* b, float* Y, long long y_rs, float* mean, float* rstd) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* x = X + row * x_rs;
  float v[V];
  float s = 0.f;
  for (int j = lane * V; j < d; j += 64 * V) {
    ldv<V>(x + j, v);
#pragma unroll
    for (int c = 0; c < V; ++c) s += v[c];
  }
  const float mu = wave_sum(s) / d;
  float q = 0.f;
  for (int j = lane * V; j < d; j += 64 * V) {
    ldv<V>(x + j, v);
#pragma unroll
    for (int c = 0; c < V; ++c) q += (v[c] - mu) * (v[c] - mu);
  }
  const float rs = rsqrtf(wave_sum(q) / d + 1e-5f);
  float* y = Y + row * y_rs;
  for (int j = lane * V; j < d; j += 64 * V) {
    float gv[V], bv[V];
    ldv<V>(x + j, v);
    ldv<V>(g + j, gv);
    ldv<V>(b + j, bv);
#pragma unroll
    for (int c = 0; c < V; ++c) v[c] = (v[c] - mu) * rs * gv[c] + bv[c];
    stv<V>(y + j, v);
  }
  if (lane == 0) { mean[row] = mu; rstd[row] = rs; }
}

// dX += rstd (dxh - mean(dxh) - xh mean(dxh xh)) with dxh = dY g and xh the normalised input:
// one wave per row, V values per lane and load.
template <int V>
__global__ __launch_bounds__(256) void k_ln_bwd_rows(const float* X, long long x_rs, int rows, int d, const float* g,
                                                     const float* mean, const float* rstd, const float* dY,
                                                     long long dy_rs, float* dX, long long dx_rs) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* x = X + row * x_rs;
  const float* dy = dY + row * dy_rs;
  const float mu = mean[row], rs = rstd[row];
  float xv[V], dv[V], gv[V];
  float s1 = 0.f, s2 = 0.f;
  for (int j = lane * V; j < d; j += 64 * V) {
    ldv<V>(x + j, xv);
    ldv<V>(dy + j, dv);
    ldv<V>(g + j, gv);
#pragma unroll
    for (int c = 0; c < V; ++c) {
      const float xh = (xv[c] - mu) * rs, dxh = dv[c] * gv[c];
      s1 += dxh;
      s2 += dxh * xh;
    }
  }
  s1 = wave_sum(s1) / d;
  s2 = wave_sum(s2) / d;
  float* dx = dX + row * dx_rs;
  for (int j = lane * V; j < d; j += 64 * V) {
    float ov[V];
    ldv<V>(x + j, xv);
    ldv<V>(dy + j, dv);
    ldv<V>(g + j, gv);
    ldv<V>(dx + j, ov);
#pragma unroll
    for (int c = 0; c < V; ++c) ov[c] += rs * (dv[c] * gv[c] - s1 - (xv[c] - mu) * rs * s2);
    stv<V>(dx + j, ov);
  }
}

// dg[j] += sum_rows dY xh, db[j] += sum_rows dY: 64 columns x TRAIN_COL_ROWS rows per workgroup,
// its four waves every fourth row, one atomic per column and workgroup.
__global__ __launch_bounds__(256) void k_ln_bwd_params(const float* X, long long x_rs, int rows, int d,
                                                       const float* mean, const float* rstd, const float* dY,
                                                       long long dy_rs, float* dg, float* db) {
  __shared__ float part[2][4][64];
  const int c = threadIdx.x & 63, w = threadIdx.x >> 6, j = blockIdx.x * 64 + c;
  const int r0 = blockIdx.y * TRAIN_COL_ROWS, r1 = min(rows, r0 + TRAIN_COL_ROWS);
  float sg = 0.f, sb = 0.f;
  if (j < d)
    for (int r = r0 + w; r < r1; r += 4) {
      const float dy = dY[r * dy_rs + j];
      sg += dy * (X[r * x_rs + j] - mean[r]) * rstd[r];
      sb += dy;
    }
  part[0][w][c] = sg;
  part[1][w][c] = sb;
  __syncthreads();
  if (w == 0 && j < d) {
    atomicAdd(&dg[j], part[0][0][c] + part[0][1][c] + part[0][2][c] + part[0][3][c]);
    atomicAdd(&db[j], part[1][0][c] + part[1][1][c] + part[1][2][c] + part[1][3][c]);
  }
}

// ------------------------------------------------------------------------------------------
// Softmax over the keys of every score row: P = softmax(scale S) on keys j < klen(z1), 0 beyond;
// query rows i >= qlen(z1) are all zero.  Row r of batch z = z1*nb2 + z2 is S + z*nq*nk + r*nk.
// ------------------------------------------------------------------------------------------
// One wave per row; NV > 0: the row (nk <= 64 NV) stays in registers between the passes, NV = 0: it
// is re-read from memory (longer rows).
template <int NV>
__global__ __launch_bounds__(256) void k_softmax_fwd(const float* S, float* P, int nbatch, int nb2, int nq, int nk,
                                                     float scale, const int32_t* qlen, const int32_t* klen) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= (long long)nbatch * nq) return;
  const int z = (int)(row / nq), i = (int)(row % nq), z1 = z / nb2;
  const int kl = klen ? min(nk, klen[z1]) : nk;
  const bool live = (qlen ? i < qlen[z1] : true) && kl > 0;
  const float* s = S + row * nk;
  float* p = P + row * nk;
  if constexpr (NV > 0) {
    float v[NV];
    float mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int j = lane + 64 * u;
      v[u] = j < kl ? s[j] * scale : -INFINITY;
      mx = fmaxf(mx, v[u]);
    }
    mx = wave_max(mx);
    float sum = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int j = lane + 64 * u;
      v[u] = j < kl ? expf(v[u] - mx) : 0.f;
      sum += v[u];
    }
    sum = wave_sum(sum);
    const float inv = live ? 1.f / sum : 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int j = lane + 64 * u;
      if (j < nk) p[j] = v[u] * inv;
    }
  } else {
    float mx = -INFINITY;
    for (int j = lane; j < kl; j += 64) mx = fmaxf(mx, s[j] * scale);
    mx = wave_max(mx);
    float sum = 0.f;
    for (int j = lane; j < kl; j += 64) sum += expf(s[j] * scale - mx);
    sum = wave_sum(sum);
    const float inv = live ? 1.f / sum : 0.f;
    for (int j = lane; j < nk; j += 64) p[j] = (live && j < kl) ? expf(s[j] * scale - mx) * inv : 0.f;
  }
}

// dS = scale P (dP - sum_j P_j dP_j), in place over dP.
template <int NV>
__global__ __launch_bounds__(256) void k_softmax_bwd(const float* P, float* dP, long long rows, int nk, float scale) {
  const long long row = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* p = P + row * nk;
  float* dp = dP + row * nk;
  if constexpr (NV > 0) {
    float pv[NV], gv[NV];
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int j = lane + 64 * u;
      pv[u] = j < nk ? p[j] : 0.f;
      gv[u] = j < nk ? dp[j] : 0.f;
      s += pv[u] * gv[u];
    }
    s = wave_sum(s);
#pragma unroll
    for (int u = 0; u < NV; ++u) {
      const int j = lane + 64 * u;
      if (j < nk) dp[j] = scale * pv[u] * (gv[u] - s);
    }
  } else {
    float s = 0.f;
    for (int j = lane; j < nk; j += 64) s += p[j] * dp[j];
    s = wave_sum(s);
    for (int j = lane; j < nk; j += 64) dp[j] = scale * p[j] * (dp[j] - s);
  }
}

// ------------------------------------------------------------------------------------------
// Elementwise steps over n values.
// ------------------------------------------------------------------------------------------
__global__ void k_copy(const float* x, float* y, long long n) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = x[i];
}
__global__ void k_fill(float* y, long long n, float v) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = v;
}
// Y[b][r] = row idx[b][r] of table T + b*t_bs for r < n (n = nvalid ? nvalid[b] : rows); rows past
// n and ids outside [0, n_table) give zero rows.
__global__ void k_gather(const float* T, long long t_bs, int n_table, const int32_t* idx, int idx_bs,
                         const int32_t* nvalid, int rows, int d, float* Y) {
  const int b = blockIdx.y, r = blockIdx.x;
  const int n = nvalid ? nvalid[b] : rows;
  float* y = Y + ((long long)b * rows + r) * d;
  const int id = r < n ? idx[(long long)b * idx_bs + r] : -1;
  if (id < 0 || id >= n_table) {
    for (int j = threadIdx.x; j < d; j += blockDim.x) y[j] = 0.f;
    return;
  }
  const float* t = T + b * t_bs + (long long)id * d;
  for (int j = threadIdx.x; j < d; j += blockDim.x) y[j] = t[j];
}
// the gather's backward: dT row idx[b][r] += dY[b][r] for the rows the gather read
__global__ void k_scatter_add(const float* dY, const int32_t* idx, int idx_bs, const int32_t* nvalid, int rows,
                              int d, float* dT, long long t_bs, int n_table) {
  const int b = blockIdx.y, r = blockIdx.x;
  const int n = nvalid ? nvalid[b] : rows;
  if (r >= n) return;
  const int id = idx[(long long)b * idx_bs + r];
  if (id < 0 || id >= n_table) return;
  const float* dy = dY + ((long long)b * rows + r) * d;
  float* t = dT + b * t_bs + (long long)id * d;
  for (int j = threadIdx.x; j < d; j += blockDim.x) atomicAdd(&t[j], dy[j]);
}

// seq[b][k][0] = cls + pos[0]; seq[b][k][j+1] = H[b][slot[b][k][j]] + pos[j+1] (Section 4.3)
__global__ void k_assemble_f32(const float* H, int U_cap, const int32_t* slot, int K, int L, int d, const float* cls,
                               const float* pos, float* seq) {
  const int b = blockIdx.z, k = blockIdx.y, j = blockIdx.x;   // j = 0..L
  float* o = seq + (((long long)b * K + k) * (L + 1) + j) * d;
  const int sl = j == 0 ? 0 : slot[((long long)b * K + k) * L + j - 1];
  const float* src = j == 0 ? cls : H + ((long long)b * U_cap + sl) * d;
  // an entry outside the pool (slot -1) gives a zero row, as in the inference assembly
  for (int e = threadIdx.x; e < d; e += blockDim.x) o[e] = sl >= 0 ? src[e] + pos[(long long)j * d + e] : 0.f;
}
// the assembly's backward, element rows: dH[b][slot] += dseq rows (a distinct element's row receives
// the sum over its occurrences)
__global__ void k_assemble_bwd(const float* dseq, int U_cap, const int32_t* slot, int K, int L, int d, float* dH) {
  const int b = blockIdx.z, k = blockIdx.y, j = blockIdx.x + 1;
  const float* g = dseq + (((long long)b * K + k) * (L + 1) + j) * d;
  const int sl = slot[((long long)b * K + k) * L + j - 1];
  if (sl < 0) return;
  float* dst = dH + ((long long)b * U_cap + sl) * d;
  for (int e = threadIdx.x; e < d; e += blockDim.x) atomicAdd(&dst[e], g[e]);
}

// ... and positions and [CLS]: dpos[c] += sum over the B K sequences of dseq[.][c] for the (L+1) d
// entries c of a sequence, dcls[e] += the same sums of row 0; the zero rows of entries outside the
// pool (slot -1) carry no position and add nothing.  64 entries x TRAIN_COL_ROWS sequences per
// workgroup, one atomic per entry and workgroup.
__global__ __launch_bounds__(256) void k_assemble_bwd_pos(const float* dseq, const int32_t* slot, int L, int nseq,
                                                          int cols, int d, float* dpos, float* dcls) {
  __shared__ float part[4][64];
  const int c = blockIdx.x * 64 + (threadIdx.x & 63), w = threadIdx.x >> 6;
  const int r0 = blockIdx.y * TRAIN_COL_ROWS, r1 = min(nseq, r0 + TRAIN_COL_ROWS);
  const int j = c / d;                                   // row of the sequence: 0 [CLS], 1..L entries
  float sum = 0.f;
  if (c < cols)
    for (int r = r0 + w; r < r1; r += 4)
      if (j == 0 || slot[(long long)r * L + j - 1] >= 0) sum += dseq[(long long)r * cols + c];
  part[w][threadIdx.x & 63] = sum;
  __syncthreads();
  if (w == 0 && c < cols) {
    const float t = part[0][threadIdx.x] + part[1][threadIdx.x] + part[2][threadIdx.x] + part[3][threadIdx.x];
    atomicAdd(&dpos[c], t);
    if (c < d) atomicAdd(&dcls[c], t);
  }
}

// Loss of request b (Section 4.5) with its labels (Appendix B.1): r_k = sum_j relevant[b][l_kj],
// y = min argmax r_k; MSE target r_k, BCE target r_k / L.  Adds loss_b / B to *loss and writes
// dscores[b][k] = (1/B) dloss_b / ds_k.  One workgroup per request, K <= 1024.
__global__ __launch_bounds__(256) void k_loss(const float* s, const int32_t* lists, const int32_t* relevant, int M,
                                              int B, int K, int L, int kind, float* loss, float* ds) {
  __shared__ int sr[1024];
  __shared__ float red[256];
  __shared__ int sy;
  const int b = blockIdx.x;
  const float* sb = s + (long long)b * K;
  for (int k = threadIdx.x; k < K; k += 256) {
    int r = 0;
    for (int j = 0; j < L; ++j) {
      const int e = lists[((long long)b * K + k) * L + j];
      r += (e >= 0 && e < M) ? relevant[(long long)b * M + e] : 0;
    }
    sr[k] = r;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int y = 0;
    for (int k = 1; k < K; ++k) if (sr[k] > sr[y]) y = k;
    sy = y;
  }
  __syncthreads();
  // CE needs max and sum of exp over the K scores
  float mx = -INFINITY;
  for (int k = threadIdx.x; k < K; k += 256) mx = fmaxf(mx, sb[k]);
  red[threadIdx.x] = mx;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + o]);
    __syncthreads();
  }
  mx = red[0];
  __syncthreads();
  float part = 0.f;
  for (int k = threadIdx.x; k < K; k += 256) part += expf(sb[k] - mx);
  red[threadIdx.x] = part;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  const float sumexp = red[0];
  __syncthreads();
  float lpart = 0.f;
  for (int k = threadIdx.x; k < K; k += 256) {
    const float sk = sb[k];
    float l = 0.f, g = 0.f;
    if (kind == TRAIN_MSE) {
      const float t = (float)sr[k];
      l = (sk - t) * (sk - t) / K;
      g = 2.f * (sk - t) / K;
    } else if (kind == TRAIN_BCE) {
      const float t = (float)sr[k] / L;
      // t softplus(-s) + (1 - t) softplus(s), softplus(v) = max(v, 0) + log1p(exp(-|v|))
      const float sp_pos = fmaxf(sk, 0.f) + log1pf(expf(-fabsf(sk)));
      const float sp_neg = fmaxf(-sk, 0.f) + log1pf(expf(-fabsf(sk)));
      l = (t * sp_neg + (1.f - t) * sp_pos) / K;
      g = (1.f / (1.f + expf(-sk)) - t) / K;
    } else {
      const float p = expf(sk - mx) / sumexp;
      g = p - (k == sy ? 1.f : 0.f);
      if (k == sy) l = -(sk - mx - logf(sumexp));
    }
    lpart += l;
    ds[(long long)b * K + k] = g / B;
  }
  red[threadIdx.x] = lpart;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) atomicAdd(loss, red[0] / B);
}

inline unsigned blocks(long long n) { return (unsigned)((n + 255) / 256); }

}  // namespace

template <int WM, int WN, bool AK, bool BK, bool VA, bool VB>
void gemm_launch(const TGemm& g, long long total, hipStream_t s) {
  constexpr int TM = 32 * WM, TN = 32 * WN;
  const dim3 grid((unsigned)((g.N + TN - 1) / TN), (unsigned)((g.M + TM - 1) / TM), 1);
  for (long long z0 = 0; z0 < total; z0 += 65535) {
    dim3 gz = grid;
    gz.z = (unsigned)std::min<long long>(65535, total - z0);
    hipLaunchKernelGGL((k_gemm<WM, WN, AK, BK, VA, VB>), gz, dim3(256), 0, s, g, (int)z0, g.nbatch);
  }
}

// float4 loads of an operand are possible when its base and every stride but the contiguous one
// are multiples of four floats (so every group of four along the contiguous index is aligned)
inline bool vec4(const float* p, long long other_stride, long long b1, long long b2) {
  return reinterpret_cast<uintptr_t>(p) % 16 == 0 && other_stride % 4 == 0 && b1 % 4 == 0 && b2 % 4 == 0;
}

template <int WM, int WN, bool AK, bool BK>
void gemm_vec(const TGemm& g, long long total, hipStream_t s) {
  const bool va = vec4(g.A, AK ? g.a_rs : g.a_cs, g.a_b1, g.a_b2) && (AK ? g.a_cs == 1 : g.a_rs == 1);
  const bool vb = vec4(g.B, BK ? g.b_cs : g.b_rs, g.b_b1, g.b_b2) && (BK ? g.b_rs == 1 : g.b_cs == 1);
  if (va && vb) gemm_launch<WM, WN, AK, BK, true, true>(g, total, s);
  else if (va) gemm_launch<WM, WN, AK, BK, true, false>(g, total, s);
  else if (vb) gemm_launch<WM, WN, AK, BK, false, true>(g, total, s);
  else gemm_launch<WM, WN, AK, BK, false, false>(g, total, s);
}

template <int WM, int WN>
void gemm_orient(const TGemm& g, long long total, hipStream_t s) {
  const bool ak = g.a_cs == 1 && g.a_rs != 1, bk = g.b_rs == 1 && g.b_cs != 1;
  if (ak && bk) gemm_vec<WM, WN, true, true>(g, total, s);
  else if (ak) gemm_vec<WM, WN, true, false>(g, total, s);
  else if (bk) gemm_vec<WM, WN, false, true>(g, total, s);
  else gemm_vec<WM, WN, false, false>(g, total, s);
}

template <bool AK, bool BK>
void small_launch_vec(bool va, bool vb, const TGemm& g, unsigned nblk, int z0, hipStream_t s) {
  if (va && vb) hipLaunchKernelGGL((k_gemm_small<AK, BK, true, true>), dim3(nblk), dim3(256), 0, s, g, z0);
  else if (va) hipLaunchKernelGGL((k_gemm_small<AK, BK, true, false>), dim3(nblk), dim3(256), 0, s, g, z0);
  else if (vb) hipLaunchKernelGGL((k_gemm_small<AK, BK, false, true>), dim3(nblk), dim3(256), 0, s, g, z0);
  else hipLaunchKernelGGL((k_gemm_small<AK, BK, false, false>), dim3(nblk), dim3(256), 0, s, g, z0);
}

void small_launch(bool ak, bool bk, bool va, bool vb, const TGemm& g, unsigned nblk, int z0, hipStream_t s) {
  if (ak && bk) small_launch_vec<true, true>(va, vb, g, nblk, z0, s);
  else if (ak) small_launch_vec<true, false>(va, vb, g, nblk, z0, s);
  else if (bk) small_launch_vec<false, true>(va, vb, g, nblk, z0, s);
  else small_launch_vec<false, false>(va, vb, g, nblk, z0, s);
}

hipError_t t_gemm(const TGemm& g, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.nbatch <= 0) return hipSuccess;
  if (g.ksplit > 0 && (g.beta != 1.f || g.bias || g.R || g.relu || g.mask || g.ksplit % GK)) return hipErrorInvalidValue;
  if (g.colsum && g.nbatch != 1) return hipErrorInvalidValue;
  const int nk = g.ksplit > 0 ? (g.K + g.ksplit - 1) / g.ksplit : 1;
  const long long total = (long long)g.nbatch * nk;
  if (g.M <= 32 && g.N <= 32 && g.ksplit == 0 && !g.colsum) {
    const bool ak = g.a_cs == 1 && g.a_rs != 1, bk = g.b_rs == 1 && g.b_cs != 1;
    const bool va = vec4(g.A, ak ? g.a_rs : g.a_cs, g.a_b1, g.a_b2) && (ak ? g.a_cs == 1 : g.a_rs == 1);
    const bool vb = vec4(g.B, bk ? g.b_cs : g.b_rs, g.b_b1, g.b_b2) && (bk ? g.b_rs == 1 : g.b_cs == 1);
    for (long long z0 = 0; z0 < total; z0 += 4LL * 65535) {
      const unsigned nblk = (unsigned)std::min<long long>(65535, (total - z0 + 3) / 4);
      small_launch(ak, bk, va, vb, g, nblk, (int)z0, s);
    }
  } else if (g.N <= 32) {
    gemm_orient<4, 1>(g, total, s);                 // 128 x 32 tiles (one head's width)
  } else {
    gemm_orient<2, 2>(g, total, s);                 // 64 x 64 tiles
  }
  return hipGetLastError();
}

// widest V in {4, 2, 1} with d a multiple of 64 V and every pointer and row stride aligned to V floats
inline int ln_width(int d, std::initializer_list<const void*> ptrs, std::initializer_list<long long> strides) {
  for (int V : {4, 2}) {
    bool ok = d % (64 * V) == 0;
    for (const void* p : ptrs) ok = ok && reinterpret_cast<uintptr_t>(p) % (4 * V) == 0;
    for (long long st : strides) ok = ok && st % V == 0;
    if (ok) return V;
  }
  return 1;
}

hipError_t t_ln_fwd(const float* X, long long x_rs, int rows, int d, const float* g, const float* b, float* Y,
                    long long y_rs, float* mean, float* rstd, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  switch (ln_width(d, {X, g, b, Y}, {x_rs, y_rs})) {
    case 4: hipLaunchKernelGGL(k_ln_fwd<4>, grid, dim3(256), 0, s, X, x_rs, rows, d, g, b, Y, y_rs, mean, rstd); break;
    case 2: hipLaunchKernelGGL(k_ln_fwd<2>, grid, dim3(256), 0, s, X, x_rs, rows, d, g, b, Y, y_rs, mean, rstd); break;
    default: hipLaunchKernelGGL(k_ln_fwd<1>, grid, dim3(256), 0, s, X, x_rs, rows, d, g, b, Y, y_rs, mean, rstd);
  }
  return hipGetLastError();
}

hipError_t t_ln_bwd(const float* X, long long x_rs, int rows, int d, const float* g, const float* mean,
                    const float* rstd, const float* dY, long long dy_rs, float* dX, long long dx_rs, float* dg,
                    float* db, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  switch (ln_width(d, {X, g, dY, dX}, {x_rs, dy_rs, dx_rs})) {
    case 4: hipLaunchKernelGGL(k_ln_bwd_rows<4>, grid, dim3(256), 0, s, X, x_rs, rows, d, g, mean, rstd, dY, dy_rs, dX, dx_rs); break;
    case 2: hipLaunchKernelGGL(k_ln_bwd_rows<2>, grid, dim3(256), 0, s, X, x_rs, rows, d, g, mean, rstd, dY, dy_rs, dX, dx_rs); break;
    default: hipLaunchKernelGGL(k_ln_bwd_rows<1>, grid, dim3(256), 0, s, X, x_rs, rows, d, g, mean, rstd, dY, dy_rs, dX, dx_rs);
  }
  hipLaunchKernelGGL(k_ln_bwd_params, dim3((unsigned)((d + 63) / 64), (unsigned)((rows + TRAIN_COL_ROWS - 1) / TRAIN_COL_ROWS)),
                     dim3(256), 0, s, X, x_rs, rows, d, mean, rstd, dY, dy_rs, dg, db);
  return hipGetLastError();
}

template <class F>
void by_row_length(int nk, F&& launch) {
  if (nk <= 64) launch(std::integral_constant<int, 1>());
  else if (nk <= 128) launch(std::integral_constant<int, 2>());
  else if (nk <= 256) launch(std::integral_constant<int, 4>());
  else if (nk <= 512) launch(std::integral_constant<int, 8>());
  else launch(std::integral_constant<int, 0>());
}

hipError_t t_softmax_fwd(const float* S, float* P, int nbatch, int nb2, int nq, int nk, float scale,
                         const int32_t* qlen, const int32_t* klen, hipStream_t s) {
  const long long rows = (long long)nbatch * nq;
  if (rows <= 0) return hipSuccess;
  by_row_length(nk, [&](auto nv) {
    hipLaunchKernelGGL((k_softmax_fwd<decltype(nv)::value>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, S, P,
                       nbatch, nb2, nq, nk, scale, qlen, klen);
  });
  return hipGetLastError();
}

hipError_t t_softmax_bwd(const float* P, float* dP, long long rows, int nk, float scale, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  by_row_length(nk, [&](auto nv) {
    hipLaunchKernelGGL((k_softmax_bwd<decltype(nv)::value>), dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, P, dP,
                       rows, nk, scale);
  });
  return hipGetLastError();
}
hipError_t t_copy(const float* x, float* y, long long n, hipStream_t s) {
  if (n > 0) hipLaunchKernelGGL(k_copy, dim3(blocks(n)), dim3(256), 0, s, x, y, n);
  return hipGetLastError();
}
hipError_t t_fill(float* y, long long n, float v, hipStream_t s) {
  if (n > 0) hipLaunchKernelGGL(k_fill, dim3(blocks(n)), dim3(256), 0, s, y, n, v);
  return hipGetLastError();
}
hipError_t t_gather(const float* T, long long t_bs, int n_table, const int32_t* idx, int idx_bs, const int32_t* nvalid,
                    int B, int rows, int d, float* Y, hipStream_t s) {
  if (B <= 0 || rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_gather, dim3((unsigned)rows, (unsigned)B), dim3(128), 0, s, T, t_bs, n_table, idx, idx_bs, nvalid,
                     rows, d, Y);
  return hipGetLastError();
}
hipError_t t_scatter_add(const float* dY, const int32_t* idx, int idx_bs, const int32_t* nvalid, int B, int rows, int d,
                         float* dT, long long t_bs, int n_table, hipStream_t s) {
  if (B <= 0 || rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_scatter_add, dim3((unsigned)rows, (unsigned)B), dim3(128), 0, s, dY, idx, idx_bs, nvalid, rows, d,
                     dT, t_bs, n_table);
  return hipGetLastError();
}
hipError_t t_assemble(const float* H, int B, int U_cap, const int32_t* slot, int K, int L, int d, const float* cls,
                      const float* pos, float* seq, hipStream_t s) {
  hipLaunchKernelGGL(k_assemble_f32, dim3((unsigned)(L + 1), (unsigned)K, (unsigned)B), dim3(128), 0, s, H, U_cap, slot, K,
                     L, d, cls, pos, seq);
  return hipGetLastError();
}
hipError_t t_assemble_bwd(const float* dseq, int B, int U_cap, const int32_t* slot, int K, int L, int d, float* dH,
                          float* dcls, float* dpos, hipStream_t s) {
  if (L > 0)
    hipLaunchKernelGGL(k_assemble_bwd, dim3((unsigned)L, (unsigned)K, (unsigned)B), dim3(128), 0, s, dseq, U_cap, slot, K,
                       L, d, dH);
  const int nseq = B * K, cols = (L + 1) * d;
  hipLaunchKernelGGL(k_assemble_bwd_pos, dim3((unsigned)((cols + 63) / 64), (unsigned)((nseq + TRAIN_COL_ROWS - 1) / TRAIN_COL_ROWS)),
                     dim3(256), 0, s, dseq, slot, L, nseq, cols, d, dpos, dcls);
  return hipGetLastError();
}
hipError_t t_loss(const float* scores, const int32_t* lists, const int32_t* relevant, int M, int B, int K, int L, int kind,
                  float* loss, float* dscores, hipStream_t s) {
  if (K > 1024) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_loss, dim3((unsigned)B), dim3(256), 0, s, scores, lists, relevant, M, B, K, L, kind, loss, dscores);
  return hipGetLastError();
}
