// Fused pre-LN transformer layers for bf16 models.
//
// k_layer_small: a whole encoder block in one kernel for modules whose attention groups are
//   short (the intra-sequence encoder over [CLS; items] of each list, and the cross-sequence
//   module when K <= 64).  A workgroup owns a tile of whole groups (at most TM rows); every
//   intermediate stays on chip:
//     A  LN1(x) -> LDS; q|k|v = LN1(x) Wqkv + b -> LDS
//     B  attention inside each group, per (group, head, 16-query tile) on one wave, keys in
//        blocks of 16 (S^T = K Q^T on 16x16x32 MFMA, P V on 16x16x16 MFMA, online softmax)
//     C  x1 = x + O Wo + bo -> LDS (fp32); LN2(x1) -> LDS; FFN in 128-wide hidden chunks;
//        x2 = x1 + FFN -> global fp32.
// k_post: the same tail (C) for modules with long groups (context, distinct items, wide
//   cross-sequence sets) whose attention ran in the chunked attention kernel; it reads the
//   attention output O from global memory.  Its PROJ variant replaces the FFN by the item
//   layers' cross-attention query projection q = LN2(x1) Wq + bq.
#include "fe_common.h"
#include "fe_tile.h"

namespace {

using namespace fe_tile;

constexpr float kLog2e = 1.4426950408889634f;
constexpr int HC = 128;              // FFN hidden chunk
constexpr int HLD = HC + APAD;

// Column-split product over an LDS tile: wave w computes the 32-column output blocks
// w + 4j (j < NCB/4) of As[TM][K] x W, NBW blocks at a time, with the weight fragments
// streamed through registers one 8-fragment stage ahead (all shapes compile-time, so the
// stage loop unrolls completely and fragment addresses are immediate offsets).  start() issues the first
// stage (so its latency can hide behind other work); run() calls epi(cb, rb, acc) for every
// finished 32x32 block (row block rb).
//
// The product is formed transposed, C^T = W^T A^T: the packed weight fragments are the A
// operand and the activation fragments the B operand.  Each lane then holds one output ROW
// (rb*32 + lane%32) and, in acc[4q..4q+3], the four consecutive output columns
// 8q + 4*(lane/32) .. +3 of the block (q = 0..3), so epilogues write 8- or 16-byte vectors.
template <int TM, int K, int NCB>
struct ColGemm {
  static constexpr int RB = TM / 32, KS = K / 16, NBW = 4 / RB;
  static constexpr int BPW = NCB / 4;                            // column blocks per wave
  static constexpr int KB = (8 / NBW < KS) ? 8 / NBW : KS;      // k-steps per stage (8 fragments)
  static constexpr int NSK = KS / KB;                            // stages per column group
  static constexpr int NG = (BPW + NBW - 1) / NBW;               // column groups per wave
  static constexpr int NST = NG * NSK;                           // stages per wave
  static_assert(NCB % 4 == 0 && KS % KB == 0, "unsupported shape");
  bf16x8 buf[2][NBW][KB];
  const bf16x8* Wl;   // this wave's first column block, this lane's fragment slot

  static constexpr int blocks_in(int g) { return (g + 1) * NBW <= BPW ? NBW : BPW - g * NBW; }
  FE_DEV void load(int t) {
    const int g = t / NSK, sk = t % NSK;
#pragma unroll
    for (int j = 0; j < NBW; ++j) {
      if (j >= blocks_in(g)) continue;
#pragma unroll
      for (int kk = 0; kk < KB; ++kk) buf[t & 1][j][kk] = Wl[((4 * (g * NBW + j)) * KS + sk * KB + kk) * 64];
    }
  }
  FE_DEV void start(const void* W) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    Wl = reinterpret_cast<const bf16x8*>(W) + (long long)wave * KS * 64 + (threadIdx.x & 63);
    load(0);
  }
  template <class Epi>
  FE_DEV void run(const bf16* As, int lda, Epi&& epi) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    f32x16 acc[RB][NBW];
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int g = t / NSK, sk = t % NSK;
      if (t + 1 < NST) load(t + 1);
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
#pragma unroll
      for (int kk = 0; kk < KB; ++kk)
#pragma unroll
        for (int j = 0; j < NBW; ++j) {
          if (j >= blocks_in(g)) continue;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(buf[t & 1][j][kk], af[kk][rb], acc[rb][j], 0, 0, 0);
        }
      if (sk != NSK - 1) continue;
#pragma unroll
      for (int j = 0; j < NBW; ++j) {
        if (j >= blocks_in(g)) continue;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) epi(wave + 4 * (g * NBW + j), rb, acc[rb][j]);
      }
    }
  }
};

// FFN of a TM-row tile: acc_o += ReLU(As W1 + b1) W2 over 128-wide hidden chunks through Hs.
// Wave w produces hidden columns 32w..32w+31 of each chunk and accumulates output column
// blocks w + 4j.  Each phase's weight fragments are requested one phase ahead; the caller
// issues ffn_preload() for chunk 0 earlier.
template <int TM, int D>
struct Ffn {
  static constexpr int RB = TM / 32, KS = D / 16, OCB = D / 128;
  bf16x8 w1[KS], w2[OCB][HC / 16];
  const bf16x8 *W1l, *W2l;   // this wave's first column block, this lane's fragment slot
  int F;
  FE_DEV void load_w1(int c) {
    // W1 [D][F]: column block 4c + wave, k-steps 0..KS-1
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) w1[ks] = W1l[((long long)c * 4 * KS + ks) * 64];
  }
  FE_DEV void load_w2(int c) {
    // W2 [F][D]: column blocks wave + 4j, k-steps 8c..8c+7 of F/16
    const int ks2 = F / 16;
#pragma unroll
    for (int j = 0; j < OCB; ++j)
#pragma unroll
      for (int ks = 0; ks < HC / 16; ++ks) w2[j][ks] = W2l[((long long)4 * j * ks2 + c * (HC / 16) + ks) * 64];
  }
  FE_DEV void preload(const void* w1p, const void* w2p, int f) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    F = f;
    W1l = reinterpret_cast<const bf16x8*>(w1p) + (long long)wave * KS * 64 + lane;
    W2l = reinterpret_cast<const bf16x8*>(w2p) + (long long)wave * (f / 16) * 64 + lane;
    load_w1(0);
    load_w2(0);
  }
  FE_DEV void run(const bf16* As, bf16* Hs, const float* b1, f32x16 (&acc_o)[RB][OCB]) {
    constexpr int LD = D + APAD;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int j = 0; j < OCB; ++j) acc_o[rb][j] = f32x16{};
    const int nchunks = F / HC;
    for (int c = 0; c < nchunks; ++c) {
      // this lane's hidden columns of the chunk: 32*wave + 8q + 4*(lane/32) + e
      float4 bias1[4];
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        bias1[qq] = *reinterpret_cast<const float4*>(&b1[(c * 4 + wave) * 32 + qq * 8 + (lane >> 5) * 4]);
      f32x16 acc_h[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc_h[rb] = f32x16{};
      {
        // all A fragments of the phase first, so the matrix instructions run back to back
        bf16x8 af[KS][RB];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) af[ks][rb] = a_frag(As, LD, rb * 32, ks * 16, lane);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc_h[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w1[ks], af[ks][rb], acc_h[rb], 0, 0, 0);
      }
      if (c + 1 < nchunks) load_w1(c + 1);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          const float* bb = reinterpret_cast<const float*>(&bias1[qq]);
          bf16x4 h;
#pragma unroll
          for (int e = 0; e < 4; ++e) h[e] = (bf16)fmaxf(acc_h[rb][4 * qq + e] + bb[e], 0.f);
          *reinterpret_cast<bf16x4*>(&Hs[(rb * 32 + (lane & 31)) * HLD + wave * 32 + qq * 8 + (lane >> 5) * 4]) = h;
        }
      __syncthreads();
      {
        bf16x8 af[HC / 16][RB];
#pragma unroll
        for (int ks = 0; ks < HC / 16; ++ks)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) af[ks][rb] = a_frag(Hs, HLD, rb * 32, ks * 16, lane);
#pragma unroll
        for (int ks = 0; ks < HC / 16; ++ks)
#pragma unroll
          for (int j = 0; j < OCB; ++j)
#pragma unroll
            for (int rb = 0; rb < RB; ++rb)
              acc_o[rb][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w2[j][ks], af[ks][rb], acc_o[rb][j], 0, 0, 0);
      }
      if (c + 1 < nchunks) load_w2(c + 1);
      __syncthreads();
    }
  }
};

// Attention inside groups of S consecutive tile rows (S <= 16*NKB), reading q|k|v from the
// LDS tile QKVs (row stride ldq; query columns 0..D-1, keys D..2D-1, values 2D..3D-1) and
// writing the per-head outputs into Os (row stride lds).  One wave per (group, head, 16-query
// tile), two such units in flight per wave: the NKB score blocks are formed first as
// independent MFMA chains, then one softmax over the whole group, then P V.
template <int D, int DH, int NKB>
FE_DEV void group_attention(const bf16* QKVs, int ldq, bf16* Os, int lds, int ng, int S, float sl2) {
  constexpr int H = D / DH, NU = 2, UPG = H * NKB;   // units per group: heads x query tiles
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g4 = lane >> 4, c16 = lane & 15;
  const int units = ng * UPG;
  for (int u0 = wave * NU; u0 < units; u0 += 4 * NU) {
    int base[NU], hcol[NU], q[NU];
    bool live[NU];
    bf16x8 qf[NU][DH / 32];
    f32x4 sc[NU][NKB];
#pragma unroll
    for (int x = 0; x < NU; ++x) {
      const int u = min(u0 + x, units - 1);
      live[x] = u0 + x < units;
      const int grp = u / UPG, rem = u % UPG;
      hcol[x] = (rem / NKB) * DH;
      base[x] = grp * S;
      q[x] = (rem % NKB) * 16 + c16;
      const int qrow = base[x] + (q[x] < S ? q[x] : 0);
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
        qf[x][c] = *reinterpret_cast<const bf16x8*>(&QKVs[qrow * ldq + hcol[x] + c * 32 + g4 * 8]);
    }
    // scores: lane holds, for query c16, keys 16*kb + 4*g4 + j
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
      for (int x = 0; x < NU; ++x) {
        const int key = kb * 16 + c16;
        const int krow = base[x] + (key < S ? key : 0);
        sc[x][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < DH / 32; ++c) {
          const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&QKVs[krow * ldq + D + hcol[x] + c * 32 + g4 * 8]);
          sc[x][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[x][c], sc[x][kb], 0, 0, 0);
        }
      }
    bf16x4 pb[NU][NKB];
    float inv[NU];
#pragma unroll
    for (int x = 0; x < NU; ++x) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sc[x][kb][j] = (kb * 16 + g4 * 4 + j < S) ? sc[x][kb][j] * sl2 : -INFINITY;
          mx = fmaxf(mx, sc[x][kb][j]);
        }
      mx = rows_max(mx);
      float l = 0.f;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float e = __builtin_amdgcn_exp2f(sc[x][kb][j] - mx);   // v_exp_f32; exp2(-inf) = 0
          l += e;
          pb[x][kb][j] = (bf16)e;
        }
      inv[x] = 1.f / rows_sum(l);
    }
    // LDS element offsets of the value rows this lane feeds into P V (keys past S: row 0, weight 0)
    int vrow[NU][NKB][4];
#pragma unroll
    for (int x = 0; x < NU; ++x)
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int vk = kb * 16 + g4 * 4 + j;
          vrow[x][kb][j] = (base[x] + (vk < S ? vk : 0)) * ldq + 2 * D + hcol[x] + c16;
        }
#pragma unroll
    for (int i = 0; i < DH / 16; ++i) {
      f32x4 o[NU];
#pragma unroll
      for (int x = 0; x < NU; ++x) {
        o[x] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) {
          bf16x4 vf;
#pragma unroll
          for (int j = 0; j < 4; ++j) vf[j] = QKVs[vrow[x][kb][j] + i * 16];
          o[x] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vf, pb[x][kb], o[x], 0, 0, 0);
        }
      }
#pragma unroll
      for (int x = 0; x < NU; ++x) {
        if (!live[x] || q[x] >= S) continue;
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (bf16)(o[x][j] * inv[x]);
        *reinterpret_cast<bf16x4*>(&Os[(base[x] + q[x]) * lds + hcol[x] + i * 16 + g4 * 4]) = w;
      }
    }
  }
}

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
FE_DEV void block_to_lds_f32(const f32x16& acc, int cb, int rb, const float* bias, float* dst, int ld) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int qq = 0; qq < 4; ++qq) {
    const int n = cb * 32 + qq * 8 + (lane >> 5) * 4;
    const float4 bb = *reinterpret_cast<const float4*>(&bias[n]);
    *reinterpret_cast<float4*>(&dst[(rb * 32 + (lane & 31)) * ld + n]) =
        make_float4(acc[4 * qq] + bb.x, acc[4 * qq + 1] + bb.y, acc[4 * qq + 2] + bb.z, acc[4 * qq + 3] + bb.w);
  }
}

// Xs[r][:] += x_in[row0 + r][:] for valid tile rows (fp32 or bf16 input, 16-byte vectors).
template <int TM, int D>
FE_DEV void add_rows(float* Xs, int ldx, const void* Xin, bool xin_f32, long long row0, const int* s_valid) {
  for (int e = threadIdx.x; e < TM * D / 4; e += WG) {
    const int rr = e / (D / 4), c = (e % (D / 4)) * 4;
    if (!s_valid[rr]) continue;
    float4 x;
    if (xin_f32) {
      x = *reinterpret_cast<const float4*>(static_cast<const float*>(Xin) + (row0 + rr) * D + c);
    } else {
      const bf16x4 t = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(Xin) + (row0 + rr) * D + c);
      x = make_float4((float)t[0], (float)t[1], (float)t[2], (float)t[3]);
    }
    float* d = &Xs[rr * ldx + c];
    d[0] += x.x; d[1] += x.y; d[2] += x.z; d[3] += x.w;
  }
}

// Xout[row0 + r][:] = Xs[r][:] for valid rows.
template <int TM, int D>
FE_DEV void store_rows(const float* Xs, int ldx, float* Xout, long long row0, const int* s_valid) {
  for (int e = threadIdx.x; e < TM * D / 4; e += WG) {
    const int rr = e / (D / 4), c = (e % (D / 4)) * 4;
    if (!s_valid[rr]) continue;
    *reinterpret_cast<float4*>(Xout + (row0 + rr) * D + c) = *reinterpret_cast<const float4*>(&Xs[rr * ldx + c]);
  }
}

// tail shared by both kernels: x1 = Xs (already holds O Wo + bo + x), LN2 -> As, FFN, store
template <int TM, int D>
FE_DEV void ffn_tail(Ffn<TM, D>& ffn, float* Xs, int ldx, bf16* As, bf16* Hs, const float* s_g2, const float* s_b2,
                     const float* b1, const float* b2, float* Xout, long long row0, const int* s_valid) {
  constexpr int RB = TM / 32, OCB = D / 128;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  stage_rows_lds<TM, D>(Xs, ldx, s_valid, s_g2, s_b2, As);
  __syncthreads();
  f32x16 acc_o[RB][OCB];
  ffn.run(As, Hs, b1, acc_o);
#pragma unroll
  for (int j = 0; j < OCB; ++j)
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int n = (wave + 4 * j) * 32 + qq * 8 + (lane >> 5) * 4;
      const float4 bb = *reinterpret_cast<const float4*>(&b2[n]);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float4* x = reinterpret_cast<float4*>(&Xs[(rb * 32 + (lane & 31)) * ldx + n]);
        float4 v = *x;
        v.x += acc_o[rb][j][4 * qq] + bb.x;
        v.y += acc_o[rb][j][4 * qq + 1] + bb.y;
        v.z += acc_o[rb][j][4 * qq + 2] + bb.z;
        v.w += acc_o[rb][j][4 * qq + 3] + bb.w;
        *x = v;
      }
    }
  __syncthreads();
  store_rows<TM, D>(Xs, ldx, Xout, row0, s_valid);
}

template <int TM, int D>
struct SmallSmem {
  static constexpr int LDA = D + APAD, LDQ = 3 * D + APAD, LDX = D + 4;
  static constexpr int QKV_BYTES = TM * LDQ * 2;
  static constexpr int TAIL_BYTES = TM * LDX * 4 + TM * HLD * 2;
  static constexpr int BIG = QKV_BYTES > TAIL_BYTES ? QKV_BYTES : TAIL_BYTES;
};

template <int TM, int D, int DH, int NKB>
__global__ __launch_bounds__(WG, 2) void k_layer_small(LayerArgs a) {
  using L = SmallSmem<TM, D>;
  __shared__ __attribute__((aligned(16))) bf16 As[TM * L::LDA];
  __shared__ __attribute__((aligned(16))) char big[L::BIG];
  __shared__ __attribute__((aligned(16))) float s_g1[D], s_b1[D], s_g2[D], s_b2[D];
  __shared__ int s_valid[TM];
  bf16* QKVs = reinterpret_cast<bf16*>(big);
  float* Xs = reinterpret_cast<float*>(big);
  bf16* Hs = reinterpret_cast<bf16*>(big + TM * L::LDX * 4);
  const int lane = threadIdx.x & 63;

  const int g0 = blockIdx.x * a.gpt;
  const int ng = min(a.gpt, a.n_groups - g0);
  const long long row0 = (long long)g0 * a.S;
  const int nrows = ng * a.S;

  ColGemm<TM, D, 3 * D / 32> gq;
  gq.start(a.wqkv);
  copy_ln_params<D>(a.ln1g, a.ln1b, s_g1, s_b1);
  copy_ln_params<D>(a.ln2g, a.ln2b, s_g2, s_b2);
  if (!mark_rows<TM>(0, nrows, nullptr, 1, s_valid)) return;
  stage_rows<TM, D>(a.Xin, a.xin_f32, D, (int)row0, s_valid, s_g1, s_b1, As);
  __syncthreads();

  // A: q|k|v of the tile into LDS
  gq.run(As, L::LDA, [&](int cb, int rb, const f32x16& acc) { block_to_lds_bf16(acc, cb, rb, a.bqkv, QKVs, L::LDQ); });
  ColGemm<TM, D, D / 32> go;
  go.start(a.wo);
  __syncthreads();

  // B: attention inside each group -> As (the LN1 tile is no longer needed)
  group_attention<D, DH, NKB>(QKVs, L::LDQ, As, L::LDA, ng, a.S, a.scale * kLog2e);
  Ffn<TM, D> ffn;
  ffn.preload(a.w1, a.w2, a.F);
  __syncthreads();

  // C: x1 = x + O Wo + bo -> Xs (fp32); then LN2, FFN, x2 = x1 + FFN
  go.run(As, L::LDA, [&](int cb, int rb, const f32x16& acc) { block_to_lds_f32(acc, cb, rb, a.bo, Xs, L::LDX); });
  __syncthreads();
  add_rows<TM, D>(Xs, L::LDX, a.Xin, a.xin_f32, row0, s_valid);
  __syncthreads();
  ffn_tail<TM, D>(ffn, Xs, L::LDX, As, Hs, s_g2, s_b2, a.b1, a.b2, a.Xout, row0, s_valid);
}

template <int TM, int D, int TAIL>
__global__ __launch_bounds__(WG, 2) void k_post(PostArgs a) {
  constexpr int LDA = D + APAD, LDX = D + 4;
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LDA];
  __shared__ __attribute__((aligned(16))) float Xs[TM * LDX];
  __shared__ __attribute__((aligned(16))) bf16 Hs[TM * HLD];
  __shared__ __attribute__((aligned(16))) float s_g2[D], s_b2[D];
  __shared__ int s_valid[TM];
  const int lane = threadIdx.x & 63;
  const int row0 = blockIdx.x * TM;

  ColGemm<TM, D, D / 32> go;
  go.start(a.wo);
  copy_ln_params<D>(a.ln2g, a.ln2b, s_g2, s_b2);
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  stage_rows<TM, D>(a.O, false, D, row0, s_valid, nullptr, nullptr, As);
  Ffn<TM, D> ffn;
  ColGemm<TM, D, D / 32> gq;
  if constexpr (TAIL == 0) ffn.preload(a.w1, a.w2, a.F);
  __syncthreads();

  go.run(As, LDA, [&](int cb, int rb, const f32x16& acc) { block_to_lds_f32(acc, cb, rb, a.bo, Xs, LDX); });
  if constexpr (TAIL == 1) gq.start(a.wq);
  __syncthreads();
  add_rows<TM, D>(Xs, LDX, a.Xin, a.xin_f32, row0, s_valid);
  __syncthreads();
  if constexpr (TAIL == 0) {
    ffn_tail<TM, D>(ffn, Xs, LDX, As, Hs, s_g2, s_b2, a.b1, a.b2, a.Xout, row0, s_valid);
  } else {
    // x1 leaves as the new residual stream; q = LN2(x1) Wq + bq for the cross-attention
    store_rows<TM, D>(Xs, LDX, a.Xout, row0, s_valid);
    stage_rows_lds<TM, D>(Xs, LDX, s_valid, s_g2, s_b2, As);
    __syncthreads();
    bf16* Qs = reinterpret_cast<bf16*>(Xs);   // Xs is dead now: per-wave 32 x 32 bf16 staging
    const int wave = threadIdx.x >> 6;
    gq.run(As, LDA, [&](int cb, int rb, const f32x16& acc) {
      bf16* st = Qs + wave * 32 * 40;
      // the block's rows land in the wave's 32 x 32 staging area (columns relative to cb*32)
      block_to_lds_bf16(acc, 0, 0, a.bq + cb * 32, st, 40);
      __builtin_amdgcn_wave_barrier();
      // 32 rows x 64 bytes: 4 lanes per row, 16 bytes each, two passes
#pragma unroll
      for (int it = 0; it < 2; ++it) {
        const int e = it * 64 + lane, r = e >> 2, c8 = (e & 3) * 8;
        const int rr = rb * 32 + r;
        if (s_valid[rr])
          *reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.Qout) + (long long)(row0 + rr) * D + cb * 32 + c8) =
              *reinterpret_cast<const bf16x8*>(&st[r * 40 + c8]);
      }
      __builtin_amdgcn_wave_barrier();
    });
  }
}

template <int TM, int D, int DH>
hipError_t launch_small_t(const LayerArgs& a, hipStream_t s) {
  const int tiles = (a.n_groups + a.gpt - 1) / a.gpt;
  switch ((a.S + 15) / 16) {
    case 1: hipLaunchKernelGGL((k_layer_small<TM, D, DH, 1>), dim3(tiles), dim3(WG), 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_layer_small<TM, D, DH, 2>), dim3(tiles), dim3(WG), 0, s, a); break;
    case 3: hipLaunchKernelGGL((k_layer_small<TM, D, DH, 3>), dim3(tiles), dim3(WG), 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_layer_small<TM, D, DH, 4>), dim3(tiles), dim3(WG), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int TM, int D>
hipError_t launch_post_t(const PostArgs& a, hipStream_t s) {
  dim3 grid((a.R + TM - 1) / TM);
  if (a.tail == 0) hipLaunchKernelGGL((k_post<TM, D, 0>), grid, dim3(WG), 0, s, a);
  else hipLaunchKernelGGL((k_post<TM, D, 1>), grid, dim3(WG), 0, s, a);
  return hipGetLastError();
}

}  // namespace

// groups of up to 64 rows (the score blocks of a group are held in registers at once)
int layer_small_tile_rows(int d) { return d >= 512 ? 32 : 64; }

hipError_t launch_layer_small(LayerArgs a, hipStream_t s) {
  if (a.n_groups <= 0) return hipSuccess;
  const int tm = layer_small_tile_rows(a.D);
  if (a.S > tm) return hipErrorInvalidValue;
  a.gpt = tm / a.S;
  const int dh = a.D / a.H;
  switch (a.D) {
    case 128: return dh == 64 ? launch_small_t<64, 128, 64>(a, s) : launch_small_t<64, 128, 32>(a, s);
    case 256: return dh == 64 ? launch_small_t<64, 256, 64>(a, s) : launch_small_t<64, 256, 32>(a, s);
    case 512: return dh == 64 ? launch_small_t<32, 512, 64>(a, s) : launch_small_t<32, 512, 32>(a, s);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_post(const PostArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  switch (a.D) {
    case 128: return launch_post_t<64, 128>(a, s);
    case 256: return launch_post_t<64, 256>(a, s);
    case 512: return launch_post_t<32, 512>(a, s);
    default: return hipErrorInvalidValue;
  }
}
