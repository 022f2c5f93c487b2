// bf16 row-tile kernels of the joint pass: projections with a LayerNorm prologue, and the whole
// pre-LN feed-forward sub-block (LN -> W1 -> ReLU -> W2 -> residual) in one kernel.
//
// Layout choices for CDNA4:
//  * A workgroup owns TM consecutive rows and ALL output columns, so every input row is read
//    from HBM once and normalised once (LayerNorm statistics in fp32, two passes over values
//    held in registers).  The normalised tile lives in LDS as bf16 for the whole k loop.
//  * Weights are pre-packed in the B-operand order of v_mfma_f32_32x32x16_bf16 (see
//    fe_model_create): the operand of one instruction is 64 lanes x 16 contiguous bytes, read
//    straight from global memory (L2-resident) with one coalesced load per lane.
//  * The FFN hidden activations (TM x F) never leave the chip: they are produced 128 columns
//    at a time into LDS and immediately contracted with the matching rows of W2.
#include "fe_common.h"

namespace {

constexpr int WG = 256;
constexpr int APAD = 8;  // bf16 elements of padding per LDS row

// Stage rows row0..row0+TM-1 of A (fp32 or bf16, row stride lda) into LDS as bf16, as
// LayerNorm(A) when g != nullptr.  Rows whose s_valid flag is 0 are written as zeros.
template <int TM, int D>
FE_DEV void stage_rows(const void* A, bool a_f32, long long lda, int row0, const int* s_valid, const float* g,
                       const float* b, bf16* As) {
  constexpr int TPR = WG / TM;             // threads per row
  constexpr int LD = D + APAD;
  const int tid = threadIdx.x;
  const int rr = tid / TPR, part = tid % TPR;
  const bool valid = s_valid[rr];
  const long long r = row0 + rr;
  if (a_f32) {
    constexpr int NV = D / (4 * TPR);      // float4 vectors per thread
    float v[NV * 4];
    const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(A) + r * lda);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      float4 t = valid ? src[i * TPR + part] : make_float4(0.f, 0.f, 0.f, 0.f);
      v[4 * i] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
    }
    float mean = 0.f, rstd = 1.f;
    if (g) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < NV * 4; ++i) s += v[i];
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o, 64);
      mean = s / (float)D;
      float q = 0.f;
#pragma unroll
      for (int i = 0; i < NV * 4; ++i) { const float t = v[i] - mean; q += t * t; }
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) q += __shfl_xor(q, o, 64);
      rstd = rsqrtf(q / (float)D + 1e-5f);
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = (i * TPR + part) * 4;
      bf16x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float y = g ? (v[4 * i + j] - mean) * rstd * g[k + j] + b[k + j] : v[4 * i + j];
        o[j] = valid ? (bf16)y : (bf16)0.f;
      }
      *reinterpret_cast<bf16x4*>(&As[rr * LD + k]) = o;
    }
  } else {
    constexpr int NV = D / (8 * TPR);      // 8 x bf16 vectors per thread
    static_assert(NV >= 1, "row too short for this tile");
    float v[NV * 8];
    const bf16x8* src = reinterpret_cast<const bf16x8*>(static_cast<const bf16*>(A) + r * lda);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      bf16x8 t = valid ? src[i * TPR + part] : bf16x8{};
#pragma unroll
      for (int j = 0; j < 8; ++j) v[8 * i + j] = (float)t[j];
    }
    float mean = 0.f, rstd = 1.f;
    if (g) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < NV * 8; ++i) s += v[i];
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o, 64);
      mean = s / (float)D;
      float q = 0.f;
#pragma unroll
      for (int i = 0; i < NV * 8; ++i) { const float t = v[i] - mean; q += t * t; }
#pragma unroll
      for (int o = 1; o < TPR; o <<= 1) q += __shfl_xor(q, o, 64);
      rstd = rsqrtf(q / (float)D + 1e-5f);
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int k = (i * TPR + part) * 8;
      bf16x8 o;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float y = g ? (v[8 * i + j] - mean) * rstd * g[k + j] + b[k + j] : v[8 * i + j];
        o[j] = valid ? (bf16)y : (bf16)0.f;
      }
      *reinterpret_cast<bf16x8*>(&As[rr * LD + k]) = o;
    }
  }
}

FE_DEV bf16x8 a_frag(const bf16* As, int ld, int row_base, int k0, int lane) {
  return *reinterpret_cast<const bf16x8*>(&As[(row_base + (lane & 31)) * ld + k0 + (lane >> 5) * 8]);
}

FE_DEV bf16x8 b_frag(const bf16* Wp, int ksteps, int cb, int ks, int lane) {
  return reinterpret_cast<const bf16x8*>(Wp)[((long long)cb * ksteps + ks) * 64 + lane];
}

// row (within the 32-row block) of accumulator element i for this lane
FE_DEV int acc_row(int i, int lane) { return (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3); }

template <int TM>
FE_DEV bool mark_rows(int row0, int R, const int32_t* nvalid, int rpb, int* s_valid) {
  int v = 0;
  if ((int)threadIdx.x < TM) {
    const int r = row0 + threadIdx.x;
    v = r < R;
    if (v && nvalid) v = (r % rpb) < nvalid[r / rpb];
    s_valid[threadIdx.x] = v;
  }
  return __syncthreads_or(v);
}

// ------------------------------------------------------------------------------------------
// C = epi(LN(A) W + bias) for K = D, any N that is a multiple of 32.
// ------------------------------------------------------------------------------------------
template <int TM, int D>
__global__ __launch_bounds__(WG) void k_proj(GemmArgs a) {
  constexpr int RB = TM / 32, KS = D / 16, LD = D + APAD, NBW = 4 / RB;   // 4 accumulator blocks per wave
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LD];
  __shared__ int s_valid[TM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = blockIdx.x * TM;
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  stage_rows<TM, D>(a.A, a.a_f32, a.lda, row0, s_valid, a.ln_g, a.ln_b, As);
  __syncthreads();

  const bf16* Wp = static_cast<const bf16*>(a.Wt);
  const int ncb = a.N / 32;
  for (int cb0 = wave; cb0 < ncb; cb0 += 4 * NBW) {
    f32x16 acc[RB][NBW];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int j = 0; j < NBW; ++j) acc[rb][j] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 af[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) af[rb] = a_frag(As, LD, rb * 32, ks * 16, lane);
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        const int cb = cb0 + 4 * j;
        if (cb < ncb) {
          const bf16x8 bfr = b_frag(Wp, KS, cb, ks, lane);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) acc[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[rb], bfr, acc[rb][j], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      const int cb = cb0 + 4 * j;
      if (cb >= ncb) continue;
      const int n = cb * 32 + (lane & 31);
      const float bias = a.bias ? a.bias[n] : 0.f;
      const long long cofs = (long long)(n / a.col_block) * a.col_block_stride + (n % a.col_block);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int rr = rb * 32 + acc_row(i, lane);
          if (!s_valid[rr]) continue;
          const long long r = row0 + rr;
          float v = acc[rb][j][i] + bias;
          if (a.epi == EPI_RESID) {
            const long long ro = r * a.ldr + n;
            const float res = a.res_f32 ? static_cast<const float*>(a.res)[ro] : (float)static_cast<const bf16*>(a.res)[ro];
            static_cast<float*>(a.C)[r * a.ldc + n] = res + v;
          } else {
            if (a.epi == EPI_RELU) v = fmaxf(v, 0.f);
            if (a.c_f32) static_cast<float*>(a.C)[cofs + r * a.ldc] = v;
            else static_cast<bf16*>(a.C)[cofs + r * a.ldc] = (bf16)v;
          }
        }
    }
  }
}

// ------------------------------------------------------------------------------------------
// X += W2 ReLU(LN(X) W1 + b1) + b2 over TM = 64 rows, hidden produced 128 columns at a time.
// ------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(WG) void k_ffn(FfnArgs a) {
  constexpr int TM = 64, RB = 2, KS = D / 16, LD = D + APAD, HC = 128, HLD = HC + APAD;
  constexpr int OCB = D / 128;             // output column blocks per wave
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LD];
  __shared__ __attribute__((aligned(16))) bf16 Hs[TM * HLD];
  __shared__ int s_valid[TM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = blockIdx.x * TM;
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  stage_rows<TM, D>(a.X, true, D, row0, s_valid, a.ln_g, a.ln_b, As);
  __syncthreads();

  const bf16* W1 = static_cast<const bf16*>(a.W1p);
  const bf16* W2 = static_cast<const bf16*>(a.W2p);
  const int KS2 = a.F / 16;
  f32x16 acc_o[RB][OCB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int j = 0; j < OCB; ++j) acc_o[rb][j] = f32x16{};

  for (int h0 = 0; h0 < a.F; h0 += HC) {
    // hidden columns h0 + 32*wave .. +31 for all 64 rows
    const int cbh = h0 / 32 + wave;
    f32x16 acc_h[RB] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const bf16x8 bfr = b_frag(W1, KS, cbh, ks, lane);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        acc_h[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_frag(As, LD, rb * 32, ks * 16, lane), bfr, acc_h[rb], 0, 0, 0);
    }
    const float bias1 = a.b1[cbh * 32 + (lane & 31)];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        Hs[(rb * 32 + acc_row(i, lane)) * HLD + wave * 32 + (lane & 31)] = (bf16)fmaxf(acc_h[rb][i] + bias1, 0.f);
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < HC / 16; ++ks) {
      bf16x8 af[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) af[rb] = a_frag(Hs, HLD, rb * 32, ks * 16, lane);
#pragma unroll
      for (int j = 0; j < OCB; ++j) {
        const bf16x8 bfr = b_frag(W2, KS2, wave + 4 * j, h0 / 16 + ks, lane);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc_o[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[rb], bfr, acc_o[rb][j], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  float* X = a.X;
#pragma unroll
  for (int j = 0; j < OCB; ++j) {
    const int n = (wave + 4 * j) * 32 + (lane & 31);
    const float bias2 = a.b2[n];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int rr = rb * 32 + acc_row(i, lane);
        if (!s_valid[rr]) continue;
        float* p = X + (long long)(row0 + rr) * D + n;
        *p = *p + acc_o[rb][j][i] + bias2;
      }
  }
}

template <int TM>
hipError_t launch_proj_tm(const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.R + TM - 1) / TM);
  switch (a.K) {
    case 128: hipLaunchKernelGGL((k_proj<TM, 128>), grid, dim3(WG), 0, s, a); break;
    case 256: hipLaunchKernelGGL((k_proj<TM, 256>), grid, dim3(WG), 0, s, a); break;
    case 512: hipLaunchKernelGGL((k_proj<TM, 512>), grid, dim3(WG), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_proj(const GemmArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  // small row counts: 32-row tiles to put more workgroups on the 256 compute units
  if ((a.R + 63) / 64 < 512) return launch_proj_tm<32>(a, s);
  return launch_proj_tm<64>(a, s);
}

hipError_t launch_ffn(const FfnArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  dim3 grid((a.R + 63) / 64);
  switch (a.D) {
    case 128: hipLaunchKernelGGL(k_ffn<128>, grid, dim3(WG), 0, s, a); break;
    case 256: hipLaunchKernelGGL(k_ffn<256>, grid, dim3(WG), 0, s, a); break;
    case 512: hipLaunchKernelGGL(k_ffn<512>, grid, dim3(WG), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
