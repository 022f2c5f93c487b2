// fp32 row-tile matrix product with a LayerNorm prologue and bias / ReLU / residual epilogues,
// plus the standalone row LayerNorm used by both model types.
//
// On fp32 models every projection of the joint pass (q|k|v, attention output, FFN up and down,
// the context-side key/value cache) is one call of k_gemm: C = epi(LN(A) x W + b), on the
// v_mfma_f32_16x16x4_f32 matrix cores.  (bf16 models use the fused kernels of fused.hip.)  Operand tiles are staged through LDS; the LayerNorm
// statistics of a row tile are computed once in fp32 before the k loop and applied while the
// A tile is copied into LDS, so the normalised activations never round-trip through HBM.
#include "fe_common.h"

namespace {

template <typename T> struct Tile;
// bf16: 64x64 output tile, 4 waves in a 2x2 grid of 32x32 MFMA blocks, k staged 64 at a time.
template <> struct Tile<bf16> { static constexpr int TM = 64, TN = 64, KC = 64, PAD = 8; };
// fp32: 64x32 output tile, each wave 16 rows x two 16x16 MFMA blocks, k staged 32 at a time.
template <> struct Tile<float> { static constexpr int TM = 64, TN = 32, KC = 32, PAD = 4; };

FE_DEV void load4(const void* p, bool f32, float* v) {
  if (f32) {
    float4 t = *reinterpret_cast<const float4*>(p);
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else {
    bf16x4 t = *reinterpret_cast<const bf16x4*>(p);
    v[0] = (float)t[0]; v[1] = (float)t[1]; v[2] = (float)t[2]; v[3] = (float)t[3];
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  constexpr int TM = Tile<T>::TM, TN = Tile<T>::TN, KC = Tile<T>::KC, LDS_LD = KC + Tile<T>::PAD;
  __shared__ __attribute__((aligned(16))) T As[TM * LDS_LD];
  __shared__ __attribute__((aligned(16))) T Bs[TN * LDS_LD];
  __shared__ float s_mean[TM], s_rstd[TM];
  __shared__ int s_valid[TM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int row0 = blockIdx.x * TM, col0 = blockIdx.y * TN;
  const bool a_f32 = a.a_f32 || sizeof(T) == 4;   // act-typed input of an fp32 model is fp32 too
  const size_t asz = a_f32 ? 4 : sizeof(T);
  const char* A = static_cast<const char*>(a.A);

  int my_valid = 0;
  if (tid < TM) {
    const int r = row0 + tid;
    my_valid = r < a.R;
    if (my_valid && a.nvalid) my_valid = (r % a.rows_per_batch) < a.nvalid[r / a.rows_per_batch];
    s_valid[tid] = my_valid;
  }
  if (!__syncthreads_or(my_valid)) return;   // tile made only of padding rows

  const bool ln = a.ln_g != nullptr;
  if (ln) {
    // wave w owns tile rows 16w..16w+15; two-pass mean / biased variance in fp32
    for (int i = 0; i < TM / 4; ++i) {
      const int rr = wave * (TM / 4) + i;
      const int r = row0 + rr;
      float mean = 0.f, rstd = 0.f;
      if (s_valid[rr]) {
        const char* rowp = A + (size_t)r * a.lda * asz;
        float vals[8];
        int nv = 0;
        float sum = 0.f;
        for (int k = lane * 4; k < a.K; k += 256) {
          float v4[4];
          load4(rowp + (size_t)k * asz, a_f32, v4);
          for (int j = 0; j < 4; ++j) { vals[nv * 4 + j] = v4[j]; sum += v4[j]; }
          ++nv;
        }
        mean = wave_sum(sum) / (float)a.K;
        float sq = 0.f;
        for (int t = 0; t < nv * 4; ++t) { const float dlt = vals[t] - mean; sq += dlt * dlt; }
        rstd = rsqrtf(wave_sum(sq) / (float)a.K + 1e-5f);
      }
      if (lane == 0) { s_mean[rr] = mean; s_rstd[rr] = rstd; }
    }
    __syncthreads();
  }

  f32x16 acc16 = {};
  f32x4 acc4a = {}, acc4b = {};

  const T* Wt = static_cast<const T*>(a.Wt);
  for (int k0 = 0; k0 < a.K; k0 += KC) {
    // ---- stage A (LayerNorm applied, rounded to the operand type) in groups of 4 along k
    for (int gi = tid; gi < TM * KC / 4; gi += 256) {
      const int rr = gi / (KC / 4), kk = (gi % (KC / 4)) * 4;
      // padding rows load row0 (inside the tile's allocation) and are stored as zeros
      const bool ok = s_valid[rr];
      float v[4];
      load4(A + ((size_t)(ok ? row0 + rr : row0) * a.lda + k0 + kk) * asz, a_f32, v);
      if (ln) {
        const float4 gg = *reinterpret_cast<const float4*>(a.ln_g + k0 + kk);
        const float4 bb = *reinterpret_cast<const float4*>(a.ln_b + k0 + kk);
        const float mu = s_mean[rr], rs = s_rstd[rr];
        v[0] = (v[0] - mu) * rs * gg.x + bb.x; v[1] = (v[1] - mu) * rs * gg.y + bb.y;
        v[2] = (v[2] - mu) * rs * gg.z + bb.z; v[3] = (v[3] - mu) * rs * gg.w + bb.w;
      }
      T* dst = &As[rr * LDS_LD + kk];
      for (int j = 0; j < 4; ++j) dst[j] = from_f32<T>(ok ? v[j] : 0.f);
    }
    // ---- stage W^T rows col0..col0+TN, 16 bytes per load
    constexpr int VB = 16 / sizeof(T);
    for (int gi = tid; gi < TN * KC / VB; gi += 256) {
      const int cc = gi / (KC / VB), kk = (gi % (KC / VB)) * VB;
      const uint4 w = *reinterpret_cast<const uint4*>(Wt + (size_t)(col0 + cc) * a.K + k0 + kk);
      *reinterpret_cast<uint4*>(&Bs[cc * LDS_LD + kk]) = w;
    }
    __syncthreads();
    if constexpr (sizeof(T) == 2) {
      const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
      for (int ks = 0; ks < KC; ks += 16) {
        const bf16x8 af = *reinterpret_cast<const bf16x8*>(&As[(wm * 32 + (lane & 31)) * LDS_LD + ks + (lane >> 5) * 8]);
        const bf16x8 bf = *reinterpret_cast<const bf16x8*>(&Bs[(wn * 32 + (lane & 31)) * LDS_LD + ks + (lane >> 5) * 8]);
        acc16 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf, acc16, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int ks = 0; ks < KC; ks += 4) {
        const float af = As[(wave * 16 + (lane & 15)) * LDS_LD + ks + (lane >> 4)];
        const float b0 = Bs[(lane & 15) * LDS_LD + ks + (lane >> 4)];
        const float b1 = Bs[(16 + (lane & 15)) * LDS_LD + ks + (lane >> 4)];
        acc4a = __builtin_amdgcn_mfma_f32_16x16x4f32(af, b0, acc4a, 0, 0, 0);
        acc4b = __builtin_amdgcn_mfma_f32_16x16x4f32(af, b1, acc4b, 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // ---- epilogue
  auto emit = [&](int rr, int cc, float v) {
    if (!s_valid[rr]) return;
    const int r = row0 + rr, n = col0 + cc;
    if (a.bias) v += a.bias[n];
    const long long off = (long long)(n / a.col_block) * a.col_block_stride + (long long)r * a.ldc + (n % a.col_block);
    if (a.epi == EPI_RESID) {
      const long long roff = (long long)r * a.ldr + n;
      const float res = a.res_f32 ? static_cast<const float*>(a.res)[roff] : to_f32(static_cast<const T*>(a.res)[roff]);
      static_cast<float*>(a.C)[off] = res + v;
      return;
    }
    if (a.epi == EPI_RELU) v = fmaxf(v, 0.f);
    if (a.c_f32) static_cast<float*>(a.C)[off] = v;
    else static_cast<T*>(a.C)[off] = from_f32<T>(v);
  };
  if constexpr (sizeof(T) == 2) {
    const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      emit(wm * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3), wn * 32 + (lane & 31), acc16[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      emit(wave * 16 + (lane >> 4) * 4 + i, lane & 15, acc4a[i]);
      emit(wave * 16 + (lane >> 4) * 4 + i, 16 + (lane & 15), acc4b[i]);
    }
  }
}

// Row r of a wide model (d = 512 NC): each lane holds 8 consecutive values of every 512-column
// chunk (16- or 32-byte loads and stores), all indices compile-time.
template <typename T, int NC>
FE_DEV void ln_row_wide(const void* X, int x_f32, long long x_rs, int r, const float* g, const float* b, void* Y,
                        int y_f32, long long y_rs, bool valid, int lane) {
  constexpr int D = 512 * NC;
  // gains and offsets are requested with the row, so their latency overlaps the row's
  float4 gv[NC][2], bv[NC][2];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = c * 512 + lane * 8;
    gv[c][0] = *reinterpret_cast<const float4*>(g + k);
    gv[c][1] = *reinterpret_cast<const float4*>(g + k + 4);
    bv[c][0] = *reinterpret_cast<const float4*>(b + k);
    bv[c][1] = *reinterpret_cast<const float4*>(b + k + 4);
  }
  float v[8 * NC];
  float sum = 0.f;
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = c * 512 + lane * 8;
    if (x_f32 || sizeof(T) == 4) {
      const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(X) + (size_t)r * x_rs + k);
      const float4 t0 = src[0], t1 = src[1];
      v[8 * c] = t0.x; v[8 * c + 1] = t0.y; v[8 * c + 2] = t0.z; v[8 * c + 3] = t0.w;
      v[8 * c + 4] = t1.x; v[8 * c + 5] = t1.y; v[8 * c + 6] = t1.z; v[8 * c + 7] = t1.w;
    } else {
      const bf16x8 t = *reinterpret_cast<const bf16x8*>(static_cast<const bf16*>(X) + (size_t)r * x_rs + k);
#pragma unroll
      for (int j = 0; j < 8; ++j) v[8 * c + j] = (float)t[j];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) sum += v[8 * c + j];
  }
  const float mean = wave_sum(sum) * (1.f / D);
  float sq = 0.f;
#pragma unroll
  for (int t = 0; t < 8 * NC; ++t) { const float dl = v[t] - mean; sq += dl * dl; }
  const float rstd = rsqrtf(wave_sum(sq) * (1.f / D) + 1e-5f);
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int k = c * 512 + lane * 8;
    const float4 g0 = gv[c][0], g1 = gv[c][1], b0 = bv[c][0], b1 = bv[c][1];
    const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
    const float bb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
    float y[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) y[j] = valid ? (v[8 * c + j] - mean) * rstd * gg[j] + bb[j] : 0.f;
    if (y_f32) {
      float4* dst = reinterpret_cast<float4*>(static_cast<float*>(Y) + (size_t)r * y_rs + k);
      dst[0] = make_float4(y[0], y[1], y[2], y[3]);
      dst[1] = make_float4(y[4], y[5], y[6], y[7]);
    } else if constexpr (sizeof(T) == 2) {
      bf16x8 o;
#pragma unroll
      for (int j = 0; j < 8; ++j) o[j] = (bf16)y[j];
      *reinterpret_cast<bf16x8*>(static_cast<bf16*>(Y) + (size_t)r * y_rs + k) = o;
    } else {
      float4* dst = reinterpret_cast<float4*>(static_cast<float*>(Y) + (size_t)r * y_rs + k);
      dst[0] = make_float4(y[0], y[1], y[2], y[3]);
      dst[1] = make_float4(y[4], y[5], y[6], y[7]);
    }
  }
}

// One wave per row: Y = LN(X), padding rows (per nvalid) written as zeros.  NC > 0: d = 512 NC
// (ln_row_wide); NC = 0: any d <= 1024.  Separate instances, so that the general form's registers
// do not lower the occupancy of the wide one.
template <typename T, int NC>
__global__ __launch_bounds__(256) void k_layernorm(const void* X, int x_f32, long long x_rs, int R, int d,
                                                   const float* g, const float* b, void* Y, int y_f32,
                                                   long long y_rs, const int32_t* nvalid, int rpb) {
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= R) return;
  const bool valid = !nvalid || (r % rpb) < nvalid[r / rpb];
  if constexpr (NC > 0) {
    ln_row_wide<T, NC>(X, x_f32, x_rs, r, g, b, Y, y_f32, y_rs, valid, lane);
    return;
  }
  // up to four 4-column groups per lane (d <= 1024), all loads -- the row, the gains and the
  // offsets -- requested before the first use; compile-time indices keep everything in registers
  float vals[16];
  float4 gv[4], bv[4];
  float sum = 0.f;
  x_f32 = x_f32 || sizeof(T) == 4;
  const size_t xs = x_f32 ? 4 : sizeof(T);
  const char* xr = static_cast<const char*>(X) + (size_t)r * x_rs * xs;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int k = lane * 4 + c * 256;
    if (k >= d) continue;
    float v4[4];
    load4(xr + (size_t)k * xs, x_f32, v4);
    gv[c] = *reinterpret_cast<const float4*>(g + k);
    bv[c] = *reinterpret_cast<const float4*>(b + k);
#pragma unroll
    for (int j = 0; j < 4; ++j) { vals[c * 4 + j] = v4[j]; sum += v4[j]; }
  }
  const float mean = wave_sum(sum) / (float)d;
  float sq = 0.f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    if (lane * 4 + c * 256 >= d) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) { const float dl = vals[c * 4 + j] - mean; sq += dl * dl; }
  }
  const float rstd = rsqrtf(wave_sum(sq) / (float)d + 1e-5f);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int k = lane * 4 + c * 256;
    if (k >= d) continue;
    const float gg[4] = {gv[c].x, gv[c].y, gv[c].z, gv[c].w}, bb[4] = {bv[c].x, bv[c].y, bv[c].z, bv[c].w};
    float y[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) y[j] = valid ? (vals[c * 4 + j] - mean) * rstd * gg[j] + bb[j] : 0.f;
    if (y_f32) {
      *reinterpret_cast<float4*>(static_cast<float*>(Y) + (size_t)r * y_rs + k) = make_float4(y[0], y[1], y[2], y[3]);
    } else {
      T o[4];
      for (int j = 0; j < 4; ++j) o[j] = from_f32<T>(y[j]);
      if constexpr (sizeof(T) == 2) *reinterpret_cast<bf16x4*>(static_cast<T*>(Y) + (size_t)r * y_rs + k) = *reinterpret_cast<const bf16x4*>(o);
      else *reinterpret_cast<float4*>(static_cast<T*>(Y) + (size_t)r * y_rs + k) = *reinterpret_cast<const float4*>(o);
    }
  }
}

}  // namespace

hipError_t launch_gemm(const GemmArgs& a, bool bf16_model, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  if (bf16_model) return hipErrorInvalidValue;   // bf16 weights are packed for k_proj / k_ffn
  dim3 grid((a.R + Tile<float>::TM - 1) / Tile<float>::TM, a.N / Tile<float>::TN);
  hipLaunchKernelGGL(k_gemm<float>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_layernorm_masked(const void* X, int x_f32, long long x_rs, int R, int d, const float* g,
                                   const float* b, void* Y, int y_f32, long long y_rs, const int32_t* nvalid,
                                   int rpb, bool bf16_model, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (d > 1024 || d % 4) return hipErrorInvalidValue;
  const dim3 grid((R + 3) / 4);
  auto go = [&](auto kern) { hipLaunchKernelGGL(kern, grid, dim3(256), 0, s, X, x_f32, x_rs, R, d, g, b, Y, y_f32, y_rs, nvalid, rpb); };
  if (bf16_model) {
    if (d == 512) go(k_layernorm<bf16, 1>);
    else if (d == 1024) go(k_layernorm<bf16, 2>);
    else go(k_layernorm<bf16, 0>);
  } else {
    if (d == 512) go(k_layernorm<float, 1>);
    else if (d == 1024) go(k_layernorm<float, 2>);
    else go(k_layernorm<float, 0>);
  }
  return hipGetLastError();
}

hipError_t launch_layernorm(const void* X, int x_f32, long long x_rs, int R, int d, const float* g, const float* b,
                            void* Y, int y_f32, long long y_rs, bool bf16_model, hipStream_t s) {
  return launch_layernorm_masked(X, x_f32, x_rs, R, d, g, b, Y, y_f32, y_rs, nullptr, 1, bf16_model, s);
}
