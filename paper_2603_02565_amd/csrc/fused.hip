// bf16 projections with a LayerNorm prologue: C = LN(A) W + bias, K = D.
//
// Layout choices for CDNA4:
//  * A workgroup owns TM consecutive rows and one slab of NCB 32-column blocks (grid.y walks
//    the slabs): the q|k|v projection is one slab of 3D columns (two, three or six narrower
//    slabs when the launch has few row tiles), the key/value cache of all item layers n slabs
//    of 2D columns.  Every input row is read once per slab and normalised
//    once (LayerNorm statistics in fp32, two passes over values held in registers); the
//    normalised tile lives in LDS as bf16 for the whole k loop.
//  * Weights are pre-packed in the fragment order of v_mfma_f32_32x32x16_bf16 (see
//    fe_model_create) and streamed from L2 through registers by ColGemm, all stages
//    compile-time; products are formed transposed so a lane holds 4 consecutive columns of
//    one row, and each finished 32x32 block leaves through a per-wave LDS staging area as
//    16-byte row segments.
#include "fe_common.h"
#include "fe_tile.h"

namespace {

using namespace fe_tile;

template <int TM, int D, int NCB>
__global__ __launch_bounds__(WG, 2) void k_proj(GemmArgs a) {
  constexpr int LD = D + APAD, KS = D / 16;
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LD];
  __shared__ __attribute__((aligned(16))) float s_g[D], s_b[D];
  __shared__ __attribute__((aligned(16))) bf16 Cs[4 * 32 * 40];   // per-wave 32 x 32 staging
  __shared__ int s_valid[TM];
  const int wave = threadIdx.x >> 6;
  const int row0 = xcd_tile(blockIdx.x, gridDim.x) * TM;
  const int cb0 = blockIdx.y * NCB;                 // first column block of the slab
  if (a.zero && blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < a.zero_n; i += WG) a.zero[i] = 0;

  copy_ln_params<D>(a.ln_g, a.ln_b, s_g, s_b);
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  ColGemm<TM, D, NCB> gq;
  gq.start(static_cast<const bf16x8*>(a.Wt) + (long long)cb0 * KS * 64);
  stage_rows<TM, D>(a.A, a.a_f32, a.lda, row0, s_valid, a.ln_g ? s_g : nullptr, s_b, As);
  lds_barrier();
  bf16* C = static_cast<bf16*>(a.C);
  bf16* st = Cs + wave * 32 * 40;
  gq.run(As, LD, [&](int, int cb, int rb, const f32x16& acc) {
    const int n = (cb0 + cb) * 32;                  // a 32-column block never straddles col_block
    bf16* out = C + (long long)(n / a.col_block) * a.col_block_stride + (n % a.col_block) + (long long)row0 * a.ldc;
    store_block_bf16(acc, a.bias + n, st, out, a.ldc, rb, s_valid);
  });
}

// q|k|v columns per workgroup: all 3D, or, for launches with few row tiles, a slab of 3D/S (S of 6,
// 3 or 2, at most 512 workgroups in all) so that more compute units share the weight stream.
// Every output element is formed the same way whatever the slab width.
template <int TM, int D, int NB>
void launch_qkv(const GemmArgs& a, unsigned tiles, hipStream_t s) {
  if constexpr (NB % 6 == 0 && (NB / 6) % 4 == 0) {
    if (tiles * 6 <= 512) {
      hipLaunchKernelGGL((k_proj<TM, D, NB / 6>), dim3(tiles, 6), dim3(WG), 0, s, a);
      return;
    }
  }
  if constexpr (NB % 3 == 0 && (NB / 3) % 4 == 0) {
    if (tiles * 3 <= 512) {
      hipLaunchKernelGGL((k_proj<TM, D, NB / 3>), dim3(tiles, 3), dim3(WG), 0, s, a);
      return;
    }
  }
  if constexpr (NB % 2 == 0 && (NB / 2) % 4 == 0) {
    if (tiles * 2 <= 512) {
      hipLaunchKernelGGL((k_proj<TM, D, NB / 2>), dim3(tiles, 2), dim3(WG), 0, s, a);
      return;
    }
  }
  hipLaunchKernelGGL((k_proj<TM, D, NB>), dim3(tiles, 1), dim3(WG), 0, s, a);
}

template <int TM, int D>
hipError_t launch_proj_d(const GemmArgs& a, hipStream_t s) {
  const unsigned tiles = (a.R + TM - 1) / TM;
  if (a.N == 3 * D) {
    launch_qkv<TM, D, 3 * D / 32>(a, tiles, s);
  } else if (a.N % (2 * D) == 0) {
    hipLaunchKernelGGL((k_proj<TM, D, 2 * D / 32>), dim3(tiles, a.N / (2 * D)), dim3(WG), 0, s, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_proj(const GemmArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  // bf16 output only; 32-column blocks must not straddle an output column block
  if (a.epi != EPI_STORE || a.c_f32 || !a.bias || a.col_block % 32) return hipErrorInvalidValue;
  switch (a.K) {
    case 128: return launch_proj_d<32, 128>(a, s);
    // 64-row tiles once they fill every workgroup slot: each weight fragment then feeds two row
    // blocks, halving the weight stream per row
    case 256: return a.R >= 512 * 64 ? launch_proj_d<64, 256>(a, s) : launch_proj_d<32, 256>(a, s);
    case 512: return launch_proj_d<32, 512>(a, s);
    default: return hipErrorInvalidValue;
  }
}
