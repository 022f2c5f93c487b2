// Device-side tile helpers shared by the bf16 row-tile kernels (fused.hip, layer.hip).
#pragma once

#include "fe_common.h"

namespace fe_tile {

constexpr int WG = 256;
constexpr int APAD = 8;  // bf16 elements of padding per LDS row

// Copy LayerNorm gains and offsets (D floats each) into LDS; visible after the next barrier.
template <int D>
FE_DEV void copy_ln_params(const float* g, const float* b, float* s_g, float* s_b) {
  if (!g) return;
  for (int i = threadIdx.x; i < D / 4; i += WG) {
    reinterpret_cast<float4*>(s_g)[i] = reinterpret_cast<const float4*>(g)[i];
    reinterpret_cast<float4*>(s_b)[i] = reinterpret_cast<const float4*>(b)[i];
  }
}

// Stage rows row0..row0+TM-1 of A (fp32 or bf16, row stride lda) into LDS as bf16, as
// LayerNorm(A) when g != nullptr (g, b point at the LDS copies of the gains and offsets).
// Rows whose s_valid flag is 0 are written as zeros.  The global loads of a thread (its row
// slice) are unconditional vector loads, so they are in flight together.
template <int TM, int D, typename TA>
FE_DEV void stage_rows_t(const TA* A, long long lda, int row0, const int* s_valid, const float* g, const float* b,
                         bf16* As) {
  constexpr int TPR = WG / TM;                   // threads per row
  constexpr int VE = 16 / sizeof(TA);            // elements per 16-byte vector
  constexpr int NV = D / (VE * TPR);             // vectors per thread
  static_assert(NV >= 1, "row too short for this tile");
  constexpr int LD = D + APAD;
  const int tid = threadIdx.x;
  const int rr = tid / TPR, part = tid % TPR;
  const bool valid = s_valid[rr];
  // padding rows read row0 (always a valid row of the tile) and are zeroed below
  const long long r = valid ? row0 + rr : row0;
  float v[NV * VE];
  const uint4* src = reinterpret_cast<const uint4*>(A + r * lda);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const uint4 t = src[i * TPR + part];
    const TA* e = reinterpret_cast<const TA*>(&t);
#pragma unroll
    for (int j = 0; j < VE; ++j) v[i * VE + j] = (float)e[j];
  }
  if (g) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NV * VE; ++i) s += v[i];
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) s += __shfl_xor(s, o, 64);
    const float mean = s / (float)D;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NV * VE; ++i) { const float t = v[i] - mean; q += t * t; }
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) q += __shfl_xor(q, o, 64);
    const float rstd = rsqrtf(q / (float)D + 1e-5f), nm = -mean * rstd;
    const float4* g4 = reinterpret_cast<const float4*>(g);   // LDS copies (copy_ln_params)
    const float4* b4 = reinterpret_cast<const float4*>(b);
#pragma unroll
    for (int i = 0; i < NV; ++i)
#pragma unroll
      for (int h = 0; h < VE / 4; ++h) {
        const int idx = (i * TPR + part) * (VE / 4) + h;
        const float4 gg = g4[idx], bb = b4[idx];
        float* x = &v[i * VE + 4 * h];
        x[0] = fmaf(fmaf(x[0], rstd, nm), gg.x, bb.x);
        x[1] = fmaf(fmaf(x[1], rstd, nm), gg.y, bb.y);
        x[2] = fmaf(fmaf(x[2], rstd, nm), gg.z, bb.z);
        x[3] = fmaf(fmaf(x[3], rstd, nm), gg.w, bb.w);
      }
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int k = (i * TPR + part) * VE;
#pragma unroll
    for (int h = 0; h < VE / 4; ++h) {
      bf16x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) o[j] = valid ? (bf16)v[i * VE + 4 * h + j] : (bf16)0.f;
      *reinterpret_cast<bf16x4*>(&As[rr * LD + k + 4 * h]) = o;
    }
  }
}

template <int TM, int D>
FE_DEV void stage_rows(const void* A, bool a_f32, long long lda, int row0, const int* s_valid, const float* g,
                       const float* b, bf16* As) {
  if (a_f32) stage_rows_t<TM, D>(static_cast<const float*>(A), lda, row0, s_valid, g, b, As);
  else stage_rows_t<TM, D>(static_cast<const bf16*>(A), lda, row0, s_valid, g, b, As);
}

FE_DEV bf16x8 a_frag(const bf16* As, int ld, int row_base, int k0, int lane) {
  return *reinterpret_cast<const bf16x8*>(&As[(row_base + (lane & 31)) * ld + k0 + (lane >> 5) * 8]);
}

template <int TM>
FE_DEV bool mark_rows(int row0, int R, const int32_t* nvalid, int rpb, int* s_valid) {
  int v = 0;
  if ((int)threadIdx.x < TM) {
    const int r = row0 + threadIdx.x;
    v = r < R;
    if (v && nvalid) v = (r % rpb) < nvalid[r / rpb];
    s_valid[threadIdx.x] = v;
  }
  return block_any<WG / 64>(v);
}


// Column-split product over an LDS tile: wave w computes the 32-column output blocks
// w + 4j (j < NCB/4) of As[TM][K] x W, NBW blocks at a time, with the weight fragments
// streamed through registers in stages of 8 fragments, PF stages ahead of the one being consumed
// (PF >= the stage count: every fragment is requested by start()).  All shapes are compile-time,
// so the stage loop unrolls completely and fragment addresses are immediate offsets.  start()
// issues the first PF stages (so their latency can hide behind other work); run() calls
// epi(jj, cb, rb, acc) for every finished 32x32 block, with jj the wave-local block index
// (compile-time after unrolling), cb = wave + 4*jj the column block and rb the row block.
//
// The product is formed transposed, C^T = W^T A^T: the packed weight fragments are the A
// operand and the activation fragments the B operand.  Each lane then holds one output ROW
// (rb*32 + lane%32) and, in acc[4q..4q+3], the four consecutive output columns
// 8q + 4*(lane/32) .. +3 of the block (q = 0..3), so epilogues write 8- or 16-byte vectors.
template <int TM, int K, int NCB, int PF = 1>
struct ColGemm {
  static constexpr int RB = TM / 32, KS = K / 16, NBW = 4 / RB;
  static constexpr int BPW = NCB / 4;                            // column blocks per wave
  static constexpr int KB = (8 / NBW < KS) ? 8 / NBW : KS;      // k-steps per stage (8 fragments)
  static constexpr int NSK = KS / KB;                            // stages per column group
  static constexpr int NG = (BPW + NBW - 1) / NBW;               // column groups per wave
  static constexpr int NST = NG * NSK;                           // stages per wave
  static constexpr int AHEAD = PF < NST ? PF : NST;              // stages in flight ahead
  static constexpr int NBUF = AHEAD < NST ? AHEAD + 1 : NST;     // register ring slots
  static_assert(NCB % 4 == 0 && KS % KB == 0 && PF >= 1, "unsupported shape");
  bf16x8 buf[NBUF][NBW][KB];
  const bf16x8* Wl;   // this wave's first column block, this lane's fragment slot

  static constexpr int blocks_in(int g) { return (g + 1) * NBW <= BPW ? NBW : BPW - g * NBW; }
  FE_DEV void load(int t) {
    const int g = t / NSK, sk = t % NSK;
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      if (j >= blocks_in(g)) continue;
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) buf[t % NBUF][j][kk] = Wl[((4 * (g * NBW + j)) * KS + sk * KB + kk) * 64];
    }
  }
  FE_DEV void start(const void* W) {
    const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 3);   // wave within its group of four
    Wl = reinterpret_cast<const bf16x8*>(W) + (long long)wave * KS * 64 + (threadIdx.x & 63);
#pragma unroll
    for (int t = 0; t < AHEAD; ++t) load(t);
  }
  template <class Epi>
  FE_DEV void run(const bf16* As, int lda, Epi&& epi) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 3);   // wave within its group of four
    f32x16 acc[RB][NBW];
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int g = t / NSK, sk = t % NSK;
      if (t + AHEAD < NST) load(t + AHEAD);
      if (sk == 0) {
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int j = 0; j < NBW; ++j) acc[rb][j] = f32x16{};
      }
      bf16x8 af[KB][RB];
#pragma unroll
      for (int kk = 0; kk < KB; ++kk)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) af[kk][rb] = a_frag(As, lda, rb * 32, (sk * KB + kk) * 16, lane);
      // every LDS read of the stage is issued before its first product, so the reads overlap
      // each other and the products wait only for the ones they consume
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < KB; ++kk)
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
          if (j >= blocks_in(g)) continue;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(buf[t % NBUF][j][kk], af[kk][rb], acc[rb][j], 0, 0, 0);
        }
      if (sk != NSK - 1) continue;
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        if (j >= blocks_in(g)) continue;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) epi(g * NBW + j, wave + 4 * (g * NBW + j), rb, acc[rb][j]);
      }
    }
  }
};

// Epilogues of a transposed 32x32 block (see ColGemm): row rb*32 + lane%32, columns
// cb*32 + 8q + 4*(lane/32) + e hold acc[4q + e].
FE_DEV void block_to_lds_bf16(const f32x16& acc, int cb, int rb, const float* bias, bf16* dst, int ld) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int qq = 0; qq < 4; ++qq) {
    const int n = cb * 32 + qq * 8 + (lane >> 5) * 4;
    const float4 bb = *reinterpret_cast<const float4*>(&bias[n]);
    bf16x4 o;
    o[0] = (bf16)(acc[4 * qq] + bb.x);
    o[1] = (bf16)(acc[4 * qq + 1] + bb.y);
    o[2] = (bf16)(acc[4 * qq + 2] + bb.z);
    o[3] = (bf16)(acc[4 * qq + 3] + bb.w);
    *reinterpret_cast<bf16x4*>(&dst[(rb * 32 + (lane & 31)) * ld + n]) = o;
  }
}

// Write a transposed 32x32 block plus bias as bf16 through the wave's LDS staging area st
// (32 x 40 bf16): the block's rows leave as 16-byte row segments.  out points at the block's
// first column in row 0 of the tile (row stride ld); rows rb*32 + r with s_valid set are written.
FE_DEV void store_block_bf16(const f32x16& acc, const float* bias, bf16* st, bf16* out, long long ld, int rb,
                             const int* s_valid) {
  const int lane = threadIdx.x & 63;
  block_to_lds_bf16(acc, 0, 0, bias, st, 40);
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int e = it * 64 + lane, r = e >> 2, c8 = (e & 3) * 8;
    const int rr = rb * 32 + r;
    if (s_valid[rr]) *reinterpret_cast<bf16x8*>(out + (long long)rr * ld + c8) = *reinterpret_cast<const bf16x8*>(&st[r * 40 + c8]);
  }
  __builtin_amdgcn_wave_barrier();
}

}  // namespace fe_tile
