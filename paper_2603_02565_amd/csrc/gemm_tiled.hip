// Tiled bf16 matrix product for wide models (d >= 256), where a row tile can no longer afford to
// stream a whole weight matrix through its compute unit:
//   C = epi(A W + bias),  A [R][K] bf16 (row stride lda), W packed in the fragment order of
//   v_mfma_f32_32x32x16_bf16 (block (nb, ks) = output columns 32nb.., inputs 16ks..; 1 KiB, lane l
//   holding W[16ks + 8(l/32) + j][32nb + l%32]).
//
// A workgroup of four waves (2 x 2) owns a BM x BN output tile; each wave accumulates a quarter
// as blocks of 32 x 32.  The k loop runs in stages of BK: per stage the A tile (BM x BK) and the
// W tile (BK x BN) are copied global -> LDS by the direct LDS load (global_load_lds, 16 bytes per
// lane, no registers), both already in fragment order, so every MFMA operand is one
// conflict-free ds_read_b128 at lane * 16.  The stage buffers form a ring with all but one
// stage in flight while the oldest is multiplied.  Products are formed
// transposed (C^T = W^T A^T) as in the other kernels, so a lane holds four consecutive output
// columns of one row.  Epilogues: bf16 store (+ bias, optional ReLU), or fp32 residual add (the
// residual fp32 or bf16; it may alias the output).
// Rows >= R and padding rows (r % rows_per_batch >= nvalid[r / rows_per_batch]) are not stored;
// their A rows are read from the tile's first row instead.
#include "fe_common.h"

namespace {

constexpr int FRAG = 64 * 8;                             // bf16 elements of one 1 KiB fragment

FE_DEV void lds_dma16(const void* src, bf16* dst_wave_base) {
  __builtin_amdgcn_global_load_lds(src, dst_wave_base, 16, 0, 0);
}

template <int N>
FE_DEV void vmem_wait_le() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// BM x BN output tile per workgroup of WM x WN waves (each wave RBW x CBW blocks of 32 x 32), k
// in stages of BK through a ring of NST LDS buffers (NST - 1 stages in flight).
template <int BM, int BN, int BK, int NST, int WM, int WN, int EPI>
__global__ __launch_bounds__(64 * WM * WN, 2) void k_gemm_tiled(GemmArgs a) {
  constexpr int NW = WM * WN, KSS = BK / 16, RBW = BM / WM / 32, CBW = BN / WN / 32;
  constexpr int SA = (BM / 32) * KSS * FRAG, ST = SA + (BN / 32) * KSS * FRAG;
  constexpr int NCOPY = (BM / 32 + BN / 32) * KSS, DPW = NCOPY / NW;
  static_assert(NCOPY % NW == 0 && RBW >= 1 && CBW >= 1, "unsupported tile");
  __shared__ __attribute__((aligned(16))) bf16 smem[NST * ST];
  __shared__ int s_valid[BM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wm = wave / WN, wn = wave % WN;
  const int n_mt = (a.R + BM - 1) / BM;
  const int id = xcd_tile(blockIdx.x, gridDim.x);
  const int mt = id % n_mt, nt = id / n_mt;             // row tiles vary fastest: a weight tile stays hot in L2
  const int row0 = mt * BM, cb0 = nt * (BN / 32);
  const int KS = a.K / 16, nst = a.K / BK;

  int v = 0;
  for (int t = threadIdx.x; t < BM; t += 64 * NW) {
    const int r = row0 + t;
    int ok = r < a.R;
    if (ok && a.nvalid) ok = (r % a.rows_per_batch) < a.nvalid[r / a.rows_per_batch];
    s_valid[t] = ok;
    v |= ok;
  }
  if (!__syncthreads_or(v)) return;                    // a tile made only of padding rows

  if (a.zero && blockIdx.x == 0)
    for (int i = threadIdx.x; i < a.zero_n; i += 64 * NW) a.zero[i] = 0;
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* W = static_cast<const bf16*>(a.Wt);
  // the copies of stage s: wave w issues copies w, w + NW, ... of the (BM + BN) / 32 * KSS
  // fragments (A first); copy c lands at buffer (s % NST), offset c KiB.  Each copy's source for
  // stage 0 is formed once; stage s adds s * BK elements (A) or s * KSS fragments (W).
  const bf16* src0[DPW];
  bool is_a[DPW];
#pragma unroll
  for (int i = 0; i < DPW; ++i) {
    const int c = wave + NW * i;
    is_a[i] = c < (BM / 32) * KSS;
    if (is_a[i]) {
      const int rb = c / KSS, kk = c % KSS;
      const int rr = rb * 32 + (lane & 31);
      const int r = s_valid[rr] ? row0 + rr : row0;
      src0[i] = A + (long long)r * a.lda + kk * 16 + 8 * (lane >> 5);
    } else {
      const int cw = c - (BM / 32) * KSS, nb = cw / KSS, kk = cw % KSS;
      src0[i] = W + ((long long)(cb0 + nb) * KS + kk) * FRAG + lane * 8;
    }
  }
  auto issue = [&](int s) {
    bf16* buf = smem + (s % NST) * ST;
#pragma unroll
    for (int i = 0; i < DPW; ++i) {
      const int c = wave + NW * i;
      lds_dma16(src0[i] + (is_a[i] ? (long long)s * BK : (long long)s * KSS * FRAG), buf + c * FRAG);
    }
  };
  f32x16 acc[RBW][CBW];
#pragma unroll
  for (int i = 0; i < RBW; ++i)
#pragma unroll
    for (int j = 0; j < CBW; ++j) acc[i][j] = f32x16{};

#pragma unroll
  for (int p = 0; p < NST - 1; ++p)
    if (p < nst) issue(p);
  for (int s = 0; s < nst; ++s) {
    // this wave's copies of stage s have landed (later stages may still be in flight); the
    // barrier publishes every wave's copies and retires the reads of the buffer refilled next
    const int ahead = min(NST - 2, nst - 1 - s);
    if (ahead <= 0) vmem_wait_le<0>();
    else if (ahead == 1) vmem_wait_le<DPW>();
    else vmem_wait_le<2 * DPW>();
    lds_barrier();
    if (s + NST - 1 < nst) issue(s + NST - 1);         // into the buffer read in iteration s - 1
    const bf16* buf = smem + (s % NST) * ST;
#pragma unroll
    for (int kk = 0; kk < KSS; ++kk) {
      bf16x8 af[RBW], wf[CBW];
#pragma unroll
      for (int i = 0; i < RBW; ++i) af[i] = *reinterpret_cast<const bf16x8*>(buf + ((wm * RBW + i) * KSS + kk) * FRAG + lane * 8);
#pragma unroll
      for (int j = 0; j < CBW; ++j)
        wf[j] = *reinterpret_cast<const bf16x8*>(buf + SA + ((wn * CBW + j) * KSS + kk) * FRAG + lane * 8);
#pragma unroll
      for (int i = 0; i < RBW; ++i)
#pragma unroll
        for (int j = 0; j < CBW; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[j], af[i], acc[i][j], 0, 0, 0);
    }
  }

  // epilogue: lane holds row (wm*RBW + i)*32 + lane%32, columns (cb0 + wn*CBW + j)*32 + 8q + 4(lane/32) + e
#pragma unroll
  for (int i = 0; i < RBW; ++i) {
    const int rr = (wm * RBW + i) * 32 + (lane & 31);
    if (!s_valid[rr]) continue;
    const long long r = row0 + rr;
#pragma unroll
    for (int j = 0; j < CBW; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = (cb0 + wn * CBW + j) * 32 + 8 * q + 4 * (lane >> 5);
        const float4 bb = a.bias ? *reinterpret_cast<const float4*>(a.bias + n) : make_float4(0.f, 0.f, 0.f, 0.f);
        float o0 = acc[i][j][4 * q] + bb.x, o1 = acc[i][j][4 * q + 1] + bb.y;
        float o2 = acc[i][j][4 * q + 2] + bb.z, o3 = acc[i][j][4 * q + 3] + bb.w;
        if constexpr (EPI == EPI_RESID) {
          float4 rv;
          if (a.res_f32) {
            rv = *reinterpret_cast<const float4*>(static_cast<const float*>(a.res) + r * a.ldr + n);
          } else {
            const bf16x4 t = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(a.res) + r * a.ldr + n);
            rv = make_float4((float)t[0], (float)t[1], (float)t[2], (float)t[3]);
          }
          float* y = static_cast<float*>(a.C) + r * a.ldc + n;
          *reinterpret_cast<float4*>(y) = make_float4(rv.x + o0, rv.y + o1, rv.z + o2, rv.w + o3);
        } else {
          if constexpr (EPI == EPI_RELU) {
            o0 = fmaxf(o0, 0.f); o1 = fmaxf(o1, 0.f); o2 = fmaxf(o2, 0.f); o3 = fmaxf(o3, 0.f);
          }
          bf16x4 o;
          o[0] = (bf16)o0; o[1] = (bf16)o1; o[2] = (bf16)o2; o[3] = (bf16)o3;
          bf16* y = static_cast<bf16*>(a.C) + (long long)(n / a.col_block) * a.col_block_stride + r * a.ldc +
                    (n % a.col_block);
          *reinterpret_cast<bf16x4*>(y) = o;
        }
      }
    }
  }
}

template <int BM, int BN, int BK, int NST>
hipError_t launch_cfg(const GemmArgs& a, hipStream_t s) {
  const unsigned grid = (unsigned)(((a.R + BM - 1) / BM) * (a.N / BN));
  switch (a.epi) {
    case EPI_STORE: hipLaunchKernelGGL((k_gemm_tiled<BM, BN, BK, NST, 2, 2, EPI_STORE>), dim3(grid), dim3(256), 0, s, a); break;
    case EPI_RELU: hipLaunchKernelGGL((k_gemm_tiled<BM, BN, BK, NST, 2, 2, EPI_RELU>), dim3(grid), dim3(256), 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((k_gemm_tiled<BM, BN, BK, NST, 2, 2, EPI_RESID>), dim3(grid), dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

bool gemm_tiled_fits(int K, int N) { return K % 64 == 0 && N % 128 == 0 && K >= 64; }

// Two shapes, both two workgroups per compute unit: 64 x 128 tiles (k stages of 32, four
// buffers) when the product has at least two such tiles per workgroup slot, else 64 x 64 tiles
// (k stages of 64, three buffers) for products with few rows, where latency, not throughput,
// sets the time and more workgroups share it.
hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  if (!gemm_tiled_fits(a.K, a.N) || a.ln_g || a.a_f32 || (a.lda % 8)) return hipErrorInvalidValue;
  if (a.epi == EPI_RESID) {
    if (!a.c_f32 || !a.res || (a.ldc % 4) || (a.ldr % 4)) return hipErrorInvalidValue;
  } else if (a.c_f32 || (a.col_block % 32) || (a.ldc % 4)) {
    return hipErrorInvalidValue;
  }
  const long long tiles = (long long)((a.R + 63) / 64) * (a.N / 128);
  if (tiles >= 512) return launch_cfg<64, 128, 32, 4>(a, s);
  return launch_cfg<64, 64, 64, 3>(a, s);
}
