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
#include "fe_tile.h"

namespace {

using namespace fe_tile;

// ------------------------------------------------------------------------------------------
// C = epi(LN(A) W + bias) for K = D, any N that is a multiple of 32.
//
// Wave w owns the 32-column blocks w, w+4, w+8, ...; they are processed NBW at a time.  The
// weight fragments are streamed through registers in stages of 16 fragments (NBW column
// blocks x KB k-steps), double-buffered: the loads of stage t+1 are issued before the matrix
// instructions of stage t, and stage 0 is requested before the A tile is staged, so its
// latency hides behind the row loads and the LayerNorm.
// ------------------------------------------------------------------------------------------
template <int TM, int D, int EPI>
__global__ __launch_bounds__(WG) void k_proj(GemmArgs a) {
  constexpr int RB = TM / 32, KS = D / 16, LD = D + APAD, NBW = 4 / RB;
  constexpr int KB = 16 / NBW < KS ? 16 / NBW : KS;   // k-steps per stage
  constexpr int NSK = KS / KB;                         // stages per column group
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LD];
  __shared__ __attribute__((aligned(16))) float s_g[D], s_b[D];
  __shared__ __attribute__((aligned(16))) float Cs[4 * TM * 33];   // per-wave output staging
  __shared__ int s_valid[TM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = xcd_tile(blockIdx.x, gridDim.x) * TM;
  const bf16* Wp = static_cast<const bf16*>(a.Wt);
  const int ncb = a.N / 32;
  const int ngroups = wave < ncb ? (ncb - wave + 4 * NBW - 1) / (4 * NBW) : 0;
  const int nstages = ngroups * NSK;

  bf16x8 cur[NBW][KB], nxt[NBW][KB];
  auto load_stage = [&](int t, bf16x8 (&buf)[NBW][KB]) {
    const int gi = t / NSK, sk = t % NSK;
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      const int cb = min(wave + 4 * (gi * NBW + j), ncb - 1);   // clamped: always a real block
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) buf[j][kk] = b_frag(Wp, KS, cb, sk * KB + kk, lane);
    }
  };
  if (nstages > 0) load_stage(0, cur);

  copy_ln_params<D>(a.ln_g, a.ln_b, s_g, s_b);
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  stage_rows<TM, D>(a.A, a.a_f32, a.lda, row0, s_valid, a.ln_g ? s_g : nullptr, s_b, As);
  __syncthreads();

  f32x16 acc[RB][NBW];
  for (int t = 0; t < nstages; ++t) {
    const int gi = t / NSK, sk = t % NSK;
    if (t + 1 < nstages) load_stage(t + 1, nxt);
    if (sk == 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int j = 0; j < NBW; ++j) acc[rb][j] = f32x16{};
    }
#pragma unroll
    for (int kk = 0; kk < KB; ++kk) {
      bf16x8 af[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) af[rb] = a_frag(As, LD, rb * 32, (sk * KB + kk) * 16, lane);
#pragma unroll
      for (int j = 0; j < NBW; ++j)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[rb], cur[j][kk], acc[rb][j], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < NBW; ++j)
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) cur[j][kk] = nxt[j][kk];
    if (sk != NSK - 1) continue;

    // ---- epilogue of column group gi: each 32-column block goes through the wave's LDS
    // staging area and leaves as row-contiguous 16-byte vectors
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      const int cb = wave + 4 * (gi * NBW + j);
      if (cb >= ncb) continue;
      const float bias = a.bias ? a.bias[cb * 32 + (lane & 31)] : 0.f;
      float* st = &Cs[wave * TM * 33];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[(rb * 32 + acc_row(i, lane)) * 33 + (lane & 31)] = acc[rb][j][i] + bias;
      __builtin_amdgcn_wave_barrier();
      if constexpr (EPI == EPI_RESID) {
        // fp32 out = residual + value: 8 lanes x float4 per 32-column row segment
#pragma unroll
        for (int it = 0; it < TM * 8 / 64; ++it) {
          const int e = it * 64 + lane, rr = e >> 3, c4 = (e & 7) * 4;
          if (!s_valid[rr]) continue;
          const long long r = row0 + rr;
          const int n = cb * 32 + c4;
          float4 res;
          if (a.res_f32) {
            res = *reinterpret_cast<const float4*>(static_cast<const float*>(a.res) + r * a.ldr + n);
          } else {
            const bf16x4 rb4 = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(a.res) + r * a.ldr + n);
            res = make_float4((float)rb4[0], (float)rb4[1], (float)rb4[2], (float)rb4[3]);
          }
          const float* sv = &st[rr * 33 + c4];
          *reinterpret_cast<float4*>(static_cast<float*>(a.C) + r * a.ldc + n) =
              make_float4(res.x + sv[0], res.y + sv[1], res.z + sv[2], res.w + sv[3]);
        }
      } else {
        // bf16 out: 4 lanes x 8 values per 32-column row segment
#pragma unroll
        for (int it = 0; it < TM * 4 / 64; ++it) {
          const int e = it * 64 + lane, rr = e >> 2, c8 = (e & 3) * 8;
          if (!s_valid[rr]) continue;
          const int n = cb * 32 + c8;
          const float* sv = &st[rr * 33 + c8];
          bf16x8 o;
#pragma unroll
          for (int q = 0; q < 8; ++q) o[q] = (bf16)(EPI == EPI_RELU ? fmaxf(sv[q], 0.f) : sv[q]);
          const long long cofs = (long long)(n / a.col_block) * a.col_block_stride + (n % a.col_block);
          *reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.C) + cofs + (long long)(row0 + rr) * a.ldc) = o;
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

// ------------------------------------------------------------------------------------------
// X += W2 ReLU(LN(X) W1 + b1) + b2 over TM = 64 rows, hidden produced 128 columns at a time.
//
// Per 128-column hidden chunk: phase H (wave w: hidden columns 32w..32w+31 of the chunk for
// all 64 rows, written to LDS after bias and ReLU) and phase O (wave w: its D/4 output columns
// accumulated over the chunk).  Every phase's weight fragments are requested one phase ahead
// (W2 of chunk c during phase H of c, W1 of chunk c+1 during phase O of c), each into the
// register set the previous phase has just released.
// ------------------------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(WG) void k_ffn(FfnArgs a) {
  constexpr int TM = 64, RB = 2, KS = D / 16, LD = D + APAD, HC = 128, HLD = HC + APAD;
  constexpr int OCB = D / 128;             // output column blocks per wave
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LD];
  __shared__ __attribute__((aligned(16))) bf16 Hs[TM * HLD];
  __shared__ __attribute__((aligned(16))) float s_g[D], s_b[D];
  __shared__ __attribute__((aligned(16))) float Cs[4 * TM * 33];   // per-wave output staging
  __shared__ int s_valid[TM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = xcd_tile(blockIdx.x, gridDim.x) * TM;
  const bf16* W1 = static_cast<const bf16*>(a.W1p);
  const bf16* W2 = static_cast<const bf16*>(a.W2p);
  const int KS2 = a.F / 16;
  const int nchunks = a.F / HC;

  bf16x8 w1[KS], w2[OCB][HC / 16];
  auto load_w1 = [&](int c) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) w1[ks] = b_frag(W1, KS, c * 4 + wave, ks, lane);
  };
  auto load_w2 = [&](int c) {
#pragma unroll
    for (int j = 0; j < OCB; ++j)
#pragma unroll
      for (int ks = 0; ks < HC / 16; ++ks) w2[j][ks] = b_frag(W2, KS2, wave + 4 * j, c * (HC / 16) + ks, lane);
  };
  load_w1(0);

  copy_ln_params<D>(a.ln_g, a.ln_b, s_g, s_b);
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  stage_rows<TM, D>(a.X, true, D, row0, s_valid, s_g, s_b, As);
  load_w2(0);
  __syncthreads();

  f32x16 acc_o[RB][OCB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int j = 0; j < OCB; ++j) acc_o[rb][j] = f32x16{};

  for (int c = 0; c < nchunks; ++c) {
    const int cbh = c * 4 + wave;
    const float bias1 = a.b1[cbh * 32 + (lane & 31)];
    f32x16 acc_h[RB] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        acc_h[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_frag(As, LD, rb * 32, ks * 16, lane), w1[ks], acc_h[rb], 0, 0, 0);
    }
    if (c + 1 < nchunks) load_w1(c + 1);
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
      for (int j = 0; j < OCB; ++j)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc_o[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[rb], w2[j][ks], acc_o[rb][j], 0, 0, 0);
    }
    if (c + 1 < nchunks) load_w2(c + 1);
    __syncthreads();
  }
  float* X = a.X;
  float* st = &Cs[wave * TM * 33];
#pragma unroll
  for (int j = 0; j < OCB; ++j) {
    const int cb = wave + 4 * j;
    const float bias2 = a.b2[cb * 32 + (lane & 31)];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) st[(rb * 32 + acc_row(i, lane)) * 33 + (lane & 31)] = acc_o[rb][j][i] + bias2;
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int it = 0; it < TM * 8 / 64; ++it) {
      const int e = it * 64 + lane, rr = e >> 3, c4 = (e & 7) * 4;
      if (!s_valid[rr]) continue;
      float4* p = reinterpret_cast<float4*>(X + (long long)(row0 + rr) * D + cb * 32 + c4);
      const float4 x = *p;
      const float* sv = &st[rr * 33 + c4];
      *p = make_float4(x.x + sv[0], x.y + sv[1], x.z + sv[2], x.w + sv[3]);
    }
    __builtin_amdgcn_wave_barrier();
  }
}

template <int TM, int D>
hipError_t launch_proj_d(const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.R + TM - 1) / TM);
  switch (a.epi) {
    case EPI_STORE: hipLaunchKernelGGL((k_proj<TM, D, EPI_STORE>), grid, dim3(WG), 0, s, a); break;
    case EPI_RELU: hipLaunchKernelGGL((k_proj<TM, D, EPI_RELU>), grid, dim3(WG), 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((k_proj<TM, D, EPI_RESID>), grid, dim3(WG), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int TM>
hipError_t launch_proj_tm(const GemmArgs& a, hipStream_t s) {
  if (a.c_f32 && a.epi != EPI_RESID) return hipErrorInvalidValue;   // fp32 output only through the residual
  switch (a.K) {
    case 128: return launch_proj_d<TM, 128>(a, s);
    case 256: return launch_proj_d<TM, 256>(a, s);
    case 512:
      if constexpr (TM == 32) return launch_proj_d<TM, 512>(a, s);
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_proj(const GemmArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  // 32-row tiles: two workgroups fit per compute unit (a 64-row tile needs all 512 registers
  // of a lane and runs one wave per SIMD) and small batches still spread over 256 units
  return launch_proj_tm<32>(a, s);
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
