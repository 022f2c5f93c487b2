// Fused pre-LN transformer layers for bf16 models.
//
// k_module_small: a whole encoder module -- every block and the final LayerNorm -- in one
//   kernel for modules whose attention groups are short (the intra-sequence encoder over
//   [CLS; items] of each list, the cross-sequence module when K <= 64, the context module when
//   T <= 64).  A workgroup owns a tile of whole groups (at most TM rows); the fp32 residual
//   stream stays in registers for all blocks and every intermediate stays on chip.  Per block:
//     A  LN1(x) -> LDS; q|k|v = LN1(x) Wqkv + b -> LDS
//     B  attention inside each group, per (group, head, 16-query tile) on one wave
//        (S^T = K Q^T on 16x16x32 MFMA, one softmax over the group, P V on 16x16x16 MFMA)
//     C  x += O Wo + bo; LN2(x) -> LDS; x += FFN in 128-wide hidden chunks.
// k_post: the tail (C) for modules with long groups (context, distinct items, wide
//   cross-sequence sets) whose attention ran in the chunked attention kernel; it reads the
//   attention output O and the residual stream from global memory.  Its second variant replaces
//   the FFN by the item layers' cross-attention query projection q = LN2(x1) Wq + bq.
#include <type_traits>

#include "fe_common.h"
#include "fe_tile.h"

namespace {

using namespace fe_tile;

constexpr float kLog2e = 1.4426950408889634f;
constexpr int HC = 128;              // FFN hidden chunk
constexpr int HLD = HC + APAD;

// Attention inside groups of S consecutive tile rows (S <= 16*NKB), reading q|k|v from the
// LDS tile QKVs (row stride ldq; query columns 0..D-1, keys D..2D-1, values 2D..3D-1) and
// writing the per-head outputs into Os (row stride lds); with FIRST_TILE only the first 16
// queries of each group are computed and only the first query's output is written, to row g of
// Os for group g (the compact [CLS] rows).  One wave per (group, head, 16-query
// tile), two such units in flight per wave: the NKB score blocks are formed first as
// independent MFMA chains, then one softmax over the whole group, then P V.
template <int D, int DH, int NKB, bool FIRST_TILE = false, int WAVES = 4>
FE_DEV void group_attention(const bf16* QKVs, int ldq, bf16* Os, int lds, int ng, int S, float sl2) {
  constexpr int H = D / DH, NU = 2, QT = FIRST_TILE ? 1 : NKB, UPG = H * QT;   // units per group
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g4 = lane >> 4, c16 = lane & 15;
  const int units = ng * UPG;
  for (int u0 = wave * NU; u0 < units; u0 += WAVES * NU) {
    int base[NU], hcol[NU], q[NU], grpx[NU];
    bool live[NU];
    bf16x8 qf[NU][DH / 32];
    f32x4 sc[NU][NKB];
#pragma unroll
    for (int x = 0; x < NU; ++x) {
      const int u = min(u0 + x, units - 1);
      live[x] = u0 + x < units;
      const int grp = u / UPG, rem = u % UPG;
      grpx[x] = grp;
      hcol[x] = (rem / QT) * DH;
      base[x] = grp * S;
      q[x] = (rem % QT) * 16 + c16;
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
      inv[x] = __builtin_amdgcn_rcpf(rows_sum(l));   // v_rcp_f32
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
        if (!live[x] || q[x] >= S || (FIRST_TILE && q[x] != 0)) continue;
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = (bf16)(o[x][j] * inv[x]);
        const int orow = FIRST_TILE ? grpx[x] : base[x] + q[x];
        *reinterpret_cast<bf16x4*>(&Os[orow * lds + hcol[x] + i * 16 + g4 * 4]) = w;
      }
    }
  }
}

// ------------------------------------------------------------------------------------------
// Whole modules over short groups, residual stream in registers.
//
// Wave w keeps the fp32 residual rows of its output column blocks cb = w + 4j (j < D/128) --
// the blocks its column-split products (Wo, the FFN down-projection) produce -- in the
// transposed accumulator layout: x.v[j][rb][4q + e] is row rb*32 + lane%32, column
// cb*32 + 8q + 4*(lane/32) + e.  Output-projection and FFN epilogues add into it directly;
// only the LayerNorm statistics cross waves (through a small LDS array).
// ------------------------------------------------------------------------------------------
template <int TM, int D>
struct Resid {
  static constexpr int RB = TM / 32, BPW = D / 128;
  f32x16 v[BPW][RB];
};

FE_DEV int resid_col(int j, int q) {
  return (__builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 3) + 4 * j) * 32 + 8 * q + 4 * ((threadIdx.x & 63) >> 5);
}

// x = rows row0.. of X (fp32 or bf16, row stride D); rows whose s_valid flag is 0 are zero.
// All loads of a lane are unconditional and independent, so they are in flight together.
template <int TM, int D, typename TX>
FE_DEV void resid_load_t(Resid<TM, D>& x, const TX* X, long long row0, const int* s_valid) {
  const int lane = threadIdx.x & 63;
  typedef TX vec4 __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int rb = 0; rb < TM / 32; ++rb) {
    const int r = rb * 32 + (lane & 31);
    const bool ok = s_valid[r];
    const TX* src = X + (ok ? row0 + r : row0) * D;
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const vec4 t = *reinterpret_cast<const vec4*>(src + resid_col(j, q));
#pragma unroll
        for (int e = 0; e < 4; ++e) x.v[j][rb][4 * q + e] = ok ? (float)t[e] : 0.f;
      }
  }
}

template <int TM, int D>
FE_DEV void resid_load(Resid<TM, D>& x, const void* X, bool x_f32, long long row0, const int* s_valid) {
  if (x_f32) resid_load_t<TM, D>(x, static_cast<const float*>(X), row0, s_valid);
  else resid_load_t<TM, D>(x, static_cast<const bf16*>(X), row0, s_valid);
}

// x[block jj, row block rb] += acc + bias (acc in the same transposed layout; bias [D]).
template <int TM, int D>
FE_DEV void resid_add(Resid<TM, D>& x, int jj, int rb, const f32x16& acc, const float* bias) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 bb = *reinterpret_cast<const float4*>(&bias[resid_col(jj, q)]);
    x.v[jj][rb][4 * q] += acc[4 * q] + bb.x;
    x.v[jj][rb][4 * q + 1] += acc[4 * q + 1] + bb.y;
    x.v[jj][rb][4 * q + 2] += acc[4 * q + 2] + bb.z;
    x.v[jj][rb][4 * q + 3] += acc[4 * q + 3] + bb.w;
  }
}

// Per row of x (this lane's rows rb*32 + lane%32): rstd = 1/sqrt(var + eps) and nm = -mean*rstd,
// so the normalised value is x*rstd + nm.  Each lane
// reduces its 16*D/128 values to a mean and a sum of squared deviations; partial results are
// merged pairwise with the update of Chan, Golub and LeVeque (equal counts: mean of the means,
// M2 = M2a + M2b + (ma - mb)^2 n/2), first across the two lanes that share a row
// (v_permlane32_swap), then across the four waves through s_stat [4][TM].  Contains one barrier;
// s_stat must not be read by an earlier call any more when a wave arrives here.
template <int TM, int D>
FE_DEV void resid_stats(const Resid<TM, D>& x, float2* s_stat, float (&nm)[TM / 32], float (&rstd)[TM / 32]) {
  constexpr int RB = TM / 32, BPW = D / 128, NL = 16 * BPW;
  const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) & 3;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < BPW; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i) sum += x.v[j][rb][i];
    const float m = sum * (1.f / NL);
    float m2 = 0.f;
#pragma unroll
    for (int j = 0; j < BPW; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float t = x.v[j][rb][i] - m;
        m2 += t * t;
      }
    const auto pm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    const auto pq = __builtin_amdgcn_permlane32_swap(__float_as_uint(m2), __float_as_uint(m2), false, false);
    const float ma = __uint_as_float(pm[0]), mb = __uint_as_float(pm[1]);
    const float dm = mb - ma;
    const float mw = 0.5f * (ma + mb);
    const float qw = __uint_as_float(pq[0]) + __uint_as_float(pq[1]) + dm * dm * (0.5f * NL);
    if (lane < 32) s_stat[wave * TM + rb * 32 + lane] = make_float2(mw, qw);
  }
  lds_barrier();
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = rb * 32 + (lane & 31);
    const float2 p0 = s_stat[r], p1 = s_stat[TM + r], p2 = s_stat[2 * TM + r], p3 = s_stat[3 * TM + r];
    const float mu = 0.25f * ((p0.x + p1.x) + (p2.x + p3.x));
    const float d0 = p0.x - mu, d1 = p1.x - mu, d2 = p2.x - mu, d3 = p3.x - mu;
    const float m2 = (p0.y + p1.y) + (p2.y + p3.y) + (d0 * d0 + d1 * d1 + d2 * d2 + d3 * d3) * (float)(2 * NL);
    rstd[rb] = rsqrtf(m2 * (1.f / D) + 1e-5f);
    nm[rb] = -mu * rstd[rb];
  }
}

// As (bf16, row stride D + APAD) = (x*rstd + nm) * g + b per row (g, b: [D], LDS or global).
template <int TM, int D>
FE_DEV void resid_norm_to_lds(const Resid<TM, D>& x, const float (&nm)[TM / 32], const float (&rstd)[TM / 32],
                              const float* g, const float* b, bf16* As) {
  constexpr int RB = TM / 32, LDA = D + APAD;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = rb * 32 + (lane & 31);
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = resid_col(j, q);
        const float4 gg = *reinterpret_cast<const float4*>(&g[c]);
        const float4 bb = *reinterpret_cast<const float4*>(&b[c]);
        const f32x16& v = x.v[j][rb];
        bf16x4 o;
        o[0] = (bf16)(fmaf(fmaf(v[4 * q], rstd[rb], nm[rb]), gg.x, bb.x));
        o[1] = (bf16)(fmaf(fmaf(v[4 * q + 1], rstd[rb], nm[rb]), gg.y, bb.y));
        o[2] = (bf16)(fmaf(fmaf(v[4 * q + 2], rstd[rb], nm[rb]), gg.z, bb.z));
        o[3] = (bf16)(fmaf(fmaf(v[4 * q + 3], rstd[rb], nm[rb]), gg.w, bb.w));
        *reinterpret_cast<bf16x4*>(&As[r * LDA + c]) = o;
      }
  }
}

// As = LayerNorm(x) with gains g and offsets b; contains the statistics barrier.
template <int TM, int D>
FE_DEV void resid_ln_to_lds(const Resid<TM, D>& x, const float* g, const float* b, float2* s_stat, bf16* As) {
  float nm[TM / 32], rstd[TM / 32];
  resid_stats<TM, D>(x, s_stat, nm, rstd);
  resid_norm_to_lds<TM, D>(x, nm, rstd, g, b, As);
}

// The vectors of one encoder block as the module kernel keeps them in LDS (fp32):
// [ln1g | ln1b | ln2g | ln2b | bqkv (3D) | bo | b2], 9D floats.
template <int D>
struct Vecs {
  static constexpr int G1 = 0, B1 = D, G2 = 2 * D, B2 = 3 * D, QKV = 4 * D, O = 7 * D, F2 = 8 * D, SIZE = 9 * D;
};

// Copy one block's vectors from global memory straight into the LDS block dst with
// global_load_lds (16 bytes per lane, no registers): wave w of W moves the 1 KiB chunks w, w + W, ....
// The data is visible to other waves once each issuing wave has passed vmem_wait() and then a
// barrier; until then dst must not be read, and it must not be written while still being read.
template <int D>
FE_DEV void vecs_dma(const EncW& w, float* dst) {
  using V = Vecs<D>;
  constexpr int NCHK = (V::SIZE * 4 + 1023) / 1024;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nwaves = blockDim.x >> 6;
  for (int ch = wave; ch < NCHK; ch += nwaves) {
    const int o = ch * 256 + lane * 4;              // this lane's first float
    if (o >= V::SIZE) continue;
    const float* src = o < V::B1    ? w.ln1g + o
                     : o < V::G2    ? w.ln1b + (o - V::B1)
                     : o < V::B2    ? w.ln2g + (o - V::G2)
                     : o < V::QKV   ? w.ln2b + (o - V::B2)
                     : o < V::O     ? w.bqkv + (o - V::QKV)
                     : o < V::F2    ? w.bo + (o - V::O)
                                    : w.b2 + (o - V::F2);
    __builtin_amdgcn_global_load_lds(src, dst + ch * 256, 16, 0, 0);
  }
}

// x += W2 ReLU(As W1 + b1) + b2 for the tile in As (LN2 output), hidden width F (a runtime
// multiple of HC = 128) in chunks of HC, accumulating straight into the register-resident residual
// (its blocks are the down-projection's output blocks).  Wave w computes hidden columns
// 32w..32w+31 of a chunk and output blocks w + 4j.  The weight fragments of a chunk form one
// stream -- the KS k-steps of W1 column block 4c + w, then for every output block j the 8 k-steps
// 8c.. of W2 column block w + 4j -- consumed in stages of 8 fragments (NS = 2*KS/8 per chunk, an
// even count) through a two-slot register ring (slot = stage parity), each stage requested one
// stage ahead.  Hidden chunks alternate between two LDS buffers in Hs (2 x TM x HLD): chunk c is
// written to buffer c&1 and one barrier per chunk separates its writers from its readers; buffer
// c&1 is rewritten (chunk c+2) only after every wave passed the barrier of chunk c+1, i.e.
// finished reading chunk c.  The caller orders the first writes to Hs after its earlier readers
// and the next writes to As or Hs after this call.
template <int TM, int D>
struct FfnStream {
  static constexpr int RB = TM / 32, KS = D / 16, OCB = D / 128;
  static constexpr int S1 = KS / 8, NS = S1 + OCB;         // W1 stages, stages per chunk
  static_assert(KS % 8 == 0 && NS % 2 == 0, "unsupported width");
  bf16x8 buf[2][8];
  const bf16x8 *W1l, *W2l;
  int F;
  FE_DEV void load(int c, int t) {      // stage t of chunk c into ring slot t & 1 (compile-time t)
    if (t < S1) {
#pragma unroll
      for (int k = 0; k < 8; ++k) buf[t & 1][k] = W1l[((long long)c * 4 * KS + t * 8 + k) * 64];
    } else {
      const int j = t - S1;
#pragma unroll
      for (int k = 0; k < 8; ++k) buf[t & 1][k] = W2l[((long long)4 * j * (F / 16) + c * 8 + k) * 64];
    }
  }
  // request the stage after stage t of chunk c, if there is one
  FE_DEV void prefetch(int c, int t, int nchunks) {
    if (t + 1 < NS) load(c, t + 1);
    else if (c + 1 < nchunks) load(c + 1, 0);
  }
  // c0: the first hidden chunk this tile streams (its first stage is requested here)
  FE_DEV void start(const void* w1p, const void* w2p, int f, int c0 = 0) {
    const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 3), lane = threadIdx.x & 63;
    F = f;
    W1l = reinterpret_cast<const bf16x8*>(w1p) + (long long)wave * KS * 64 + lane;
    W2l = reinterpret_cast<const bf16x8*>(w2p) + (long long)wave * (f / 16) * 64 + lane;
    load(c0, 0);
  }
  // x += the FFN's contribution of hidden chunks [c0, c1) (c1 < 0: through the last chunk)
  template <class Acc>
  FE_DEV void run(const bf16* As, bf16* Hs, const float* b1, Acc& x, int c0 = 0, int c1 = -1) {
    const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) & 3;
    const int nchunks = c1 < 0 ? F / HC : c1;
    for (int c = c0; c < nchunks; ++c) chunk(c, nchunks, As, Hs, b1, x, lane, wave);
  }
  template <class Acc>
  FE_DEV void chunk(int c, int nchunks, const bf16* As, bf16* Hs, const float* b1, Acc& x, int lane, int wave) {
    constexpr int LD = D + APAD;
    bf16* Hc = Hs + (c & 1) * TM * HLD;
    float4 bias1[4];
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
      bias1[qq] = *reinterpret_cast<const float4*>(&b1[(c * 4 + wave) * 32 + qq * 8 + (lane >> 5) * 4]);
    f32x16 acc_h[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) acc_h[rb] = f32x16{};
#pragma unroll
    for (int t = 0; t < S1; ++t) {
      prefetch(c, t, nchunks);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8 af[4][RB];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) af[k][rb] = a_frag(As, LD, rb * 32, (t * 8 + h * 4 + k) * 16, lane);
        __builtin_amdgcn_sched_barrier(0);   // all reads of the group before its products
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            acc_h[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(buf[t & 1][h * 4 + k], af[k][rb], acc_h[rb], 0, 0, 0);
      }
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const float* bb = reinterpret_cast<const float*>(&bias1[qq]);
        bf16x4 hv;
#pragma unroll
        for (int e = 0; e < 4; ++e) hv[e] = (bf16)fmaxf(acc_h[rb][4 * qq + e] + bb[e], 0.f);
        *reinterpret_cast<bf16x4*>(&Hc[(rb * 32 + (lane & 31)) * HLD + wave * 32 + qq * 8 + (lane >> 5) * 4]) = hv;
      }
    lds_barrier();
#pragma unroll
    for (int j = 0; j < OCB; ++j) {
      const int t = S1 + j;
      prefetch(c, t, nchunks);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8 af[4][RB];
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) af[k][rb] = a_frag(Hc, HLD, rb * 32, (h * 4 + k) * 16, lane);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb)
            x.v[j][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(buf[t & 1][h * 4 + k], af[k][rb], x.v[j][rb], 0, 0, 0);
      }
    }
  }
};

// The same product for a compile-time chunk count (F = 128*NCH), software-pipelined over the
// chunks: between two barriers a wave forms the first-layer block of chunk s and the
// second-layer blocks of chunk s - 1 (two independent MFMA chains), then chunk s's bias + ReLU
// epilogue into hidden buffer s & 1, which the next step reads.  Buffer s & 1 was last read in
// step s - 1 (as chunk s - 2), which ended with a barrier.  Weight stages are consumed, and
// streamed through the DEPTH-slot register ring, in the order
//   W1(0); W1(1) W2(0); W1(2) W2(1); ...; W1(NCH-1) W2(NCH-2); W2(NCH-1).
// Same interface and the same ordering duties for the caller as FfnStream.
template <int TM, int D, int NCH, int DEPTH>
struct FfnPipe {
  static constexpr int RB = TM / 32, KS = D / 16, OCB = D / 128, F = NCH * HC;
  static constexpr int S1 = KS / 8, NS = S1 + OCB, NST = NCH * NS;
  static_assert(KS % 8 == 0 && NCH >= 1 && DEPTH >= 2, "unsupported shape");
  bf16x8 buf[DEPTH][8];
  const bf16x8 *W1l, *W2l;
  static constexpr int g_w1(int c, int t) { return c == 0 ? t : S1 + (c - 1) * NS + t; }
  static constexpr int g_w2(int c, int j) { return S1 + c * NS + (c + 1 < NCH ? S1 : 0) + j; }
  FE_DEV void load(int g) {   // stage g of the consumption order into ring slot g % DEPTH
    bool w1;
    int c, t;
    if (g < S1) {
      w1 = true; c = 0; t = g;
    } else {
      const int r = g - S1, st = r / NS + 1, o = r % NS;
      if (st < NCH) {
        w1 = o < S1; c = w1 ? st : st - 1; t = w1 ? o : o - S1;
      } else {
        w1 = false; c = NCH - 1; t = r - (NCH - 1) * NS;
      }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k)
      buf[g % DEPTH][k] = w1 ? W1l[((long long)c * 4 * KS + t * 8 + k) * 64] : W2l[((long long)4 * t * (F / 16) + c * 8 + k) * 64];
  }
  FE_DEV void fetch(int g) {   // consuming stage g: request stage g + DEPTH - 1
    if (g + DEPTH - 1 < NST) load(g + DEPTH - 1);
  }
  FE_DEV void start(const void* w1p, const void* w2p, int) {
    const int wave = __builtin_amdgcn_readfirstlane((threadIdx.x >> 6) & 3), lane = threadIdx.x & 63;
    W1l = reinterpret_cast<const bf16x8*>(w1p) + (long long)wave * KS * 64 + lane;
    W2l = reinterpret_cast<const bf16x8*>(w2p) + (long long)wave * (F / 16) * 64 + lane;
#pragma unroll
    for (int g = 0; g < DEPTH - 1; ++g)
      if (g < NST) load(g);
  }
  // acc[rb] += the 8 k-steps of ring slot `slot` against the tile At (row stride ld) at k-steps
  // k0..: pairs of k-steps, the LDS reads of pair p + 1 issued before the products of pair p, so
  // the reads stay in flight behind the matrix work
  FE_DEV void steps(const bf16* At, int ld, int k0, int slot, f32x16 (&acc)[RB], int lane) {
    bf16x8 af[2][2][RB];
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) af[0][k][rb] = a_frag(At, ld, rb * 32, (k0 + k) * 16, lane);
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      if (p + 1 < 4) {
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) af[(p + 1) & 1][k][rb] = a_frag(At, ld, rb * 32, (k0 + 2 * p + 2 + k) * 16, lane);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(buf[slot][2 * p + k], af[p & 1][k][rb], acc[rb], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  template <class Acc>
  FE_DEV void run(const bf16* As, bf16* Hs, const float* b1, Acc& x) {
    constexpr int LD = D + APAD;
    const int lane = threadIdx.x & 63, wave = (threadIdx.x >> 6) & 3;
    f32x16 acc_h[RB];
#pragma unroll
    for (int s = 0; s <= NCH; ++s) {
      float4 bias1[4];
      if (s < NCH) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
          bias1[qq] = *reinterpret_cast<const float4*>(&b1[(s * 4 + wave) * 32 + qq * 8 + (lane >> 5) * 4]);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) acc_h[rb] = f32x16{};
#pragma unroll
        for (int t = 0; t < S1; ++t) {
          fetch(g_w1(s, t));
          steps(As, LD, t * 8, g_w1(s, t) % DEPTH, acc_h, lane);
        }
      }
      if (s > 0) {
        const bf16* Hp = Hs + ((s - 1) & 1) * TM * HLD;
#pragma unroll
        for (int j = 0; j < OCB; ++j) {
          fetch(g_w2(s - 1, j));
          f32x16 (&xo)[RB] = x.v[j];
          steps(Hp, HLD, 0, g_w2(s - 1, j) % DEPTH, xo, lane);
        }
      }
      if (s < NCH) {
        bf16* Hc = Hs + (s & 1) * TM * HLD;
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
#pragma unroll
          for (int qq = 0; qq < 4; ++qq) {
            const float* bb = reinterpret_cast<const float*>(&bias1[qq]);
            bf16x4 hv;
#pragma unroll
            for (int e = 0; e < 4; ++e) hv[e] = (bf16)fmaxf(acc_h[rb][4 * qq + e] + bb[e], 0.f);
            *reinterpret_cast<bf16x4*>(&Hc[(rb * 32 + (lane & 31)) * HLD + wave * 32 + qq * 8 + (lane >> 5) * 4]) = hv;
          }
        lds_barrier();
      }
    }
  }
};

// FFN weight stream of a tile: pipelined over a compile-time chunk count (NCH > 0), else the
// runtime-width stream.
template <int TM, int D, int NCH>
using FfnOf = typename std::conditional<(NCH > 0), FfnPipe<TM, D, (NCH > 0 ? NCH : 1), 3>, FfnStream<TM, D>>::type;

template <int TM, int D>
struct ModuleSmem {
  static constexpr int LDA = D + APAD, LDQ = 3 * D + APAD;
  static constexpr int QKV_BYTES = TM * LDQ * 2, HS_BYTES = 2 * TM * HLD * 2;
  static constexpr int BIG = QKV_BYTES > HS_BYTES ? QKV_BYTES : HS_BYTES;
};

// n_layers encoder blocks and the final LayerNorm over a tile of whole groups; one launch per
// module.  Per block: LN1 -> As; q|k|v -> LDS; attention per (group, head) -> As; x += O Wo + bo;
// LN2 -> As; x += FFN.  The fp32 residual x never leaves registers; the result leaves as fp32.
template <int TM, int D, int DH, int NKB, bool CLS, int G, int NCH = 0>
__global__ __launch_bounds__(WG * G, G == 1 ? 2 : 1) void k_module_small(ModuleArgs a) {
  static_assert(G == 1 || !CLS, "the compacted last block runs on one wave group");
  using L = ModuleSmem<TM, D>;
  constexpr int TMG = TM / G, RB = TMG / 32, OCB = D / 128;
  __shared__ __attribute__((aligned(16))) bf16 As[TM * L::LDA];
  __shared__ __attribute__((aligned(16))) char big[L::BIG];
  __shared__ __attribute__((aligned(16))) float2 s_stat[4 * TM];
  __shared__ __attribute__((aligned(16))) float s_vec[2][Vecs<D>::SIZE];   // by layer parity
  __shared__ int s_valid[TM];
  bf16* QKVs = reinterpret_cast<bf16*>(big);
  bf16* Hs = reinterpret_cast<bf16*>(big);
  const int lane = threadIdx.x & 63;
  // wave group gr (waves 4gr .. 4gr+3) owns tile rows gr*TMG .. gr*TMG + TMG - 1 for every
  // row-wise step; attention runs over the whole tile on all 4G waves
  const int gr = G == 1 ? 0 : __builtin_amdgcn_readfirstlane(threadIdx.x >> 8);
  bf16* Ag = As + gr * TMG * L::LDA;
  bf16* QKVg = QKVs + gr * TMG * L::LDQ;
  bf16* Hg = Hs + gr * 2 * TMG * HLD;
  float2* statg = s_stat + gr * 4 * TMG;
  const int* validg = s_valid + gr * TMG;

  const int g0 = xcd_tile(blockIdx.x, gridDim.x) * a.gpt;
  const int ng = min(a.gpt, a.n_groups - g0);
  const long long row0 = (long long)g0 * a.S;
  const int nrows = ng * a.S;

  if (nrows <= 0) return;                              // uniform; the grid has no empty tiles
  if (threadIdx.x < TM) s_valid[threadIdx.x] = (int)threadIdx.x < nrows;
  lds_barrier();                                       // LDS only: nothing outstanding is waited for
  // layer 0's vectors: DMA into LDS, published by the statistics barrier of the first LN1
  vecs_dma<D>(a.layer[0], s_vec[0]);
  Resid<TMG, D> x;
  resid_load<TMG, D>(x, a.Xin, a.xin_f32, row0 + gr * TMG, validg);
  ColGemm<TMG, D, 3 * D / 32> gq;
  gq.start(a.layer[0].wqkv);
  vmem_wait();

  using V = Vecs<D>;
  const int nfull = CLS ? a.n_layers - 1 : a.n_layers;
  for (int l = 0; l < nfull; ++l) {
    const EncW& w = a.layer[l];
    const float* vec = s_vec[l & 1];
    if (l > 0) gq.start(w.wqkv);
    // LN1 -> As.  Past the statistics barrier every wave has left layer l - 1, so the other
    // vector buffer is free for layer l + 1 (waited for at the end of this layer).
    {
      float nm[RB], rstd[RB];
      resid_stats<TMG, D>(x, statg, nm, rstd);
      if (l + 1 < a.n_layers) vecs_dma<D>(a.layer[l + 1], s_vec[(l + 1) & 1]);
      resid_norm_to_lds<TMG, D>(x, nm, rstd, vec + V::G1, vec + V::B1, Ag);
    }
    lds_barrier();
    gq.run(Ag, L::LDA, [&](int, int cb, int rb, const f32x16& acc) {
      block_to_lds_bf16(acc, cb, rb, vec + V::QKV, QKVg, L::LDQ);
    });
    ColGemm<TMG, D, D / 32> go;
    go.start(w.wo);
    lds_barrier();
    group_attention<D, DH, NKB, false, 4 * G>(QKVs, L::LDQ, As, L::LDA, ng, a.S, a.scale * kLog2e);
    FfnOf<TMG, D, NCH> ffn;
    ffn.start(w.w1, w.w2, a.F);
    lds_barrier();
    go.run(Ag, L::LDA, [&](int jj, int, int rb, const f32x16& acc) { resid_add<TMG, D>(x, jj, rb, acc, vec + V::O); });
    resid_ln_to_lds<TMG, D>(x, vec + V::G2, vec + V::B2, statg, Ag);
    lds_barrier();
    ffn.run(Ag, Hg, w.b1, x);
#pragma unroll
    for (int j = 0; j < OCB; ++j)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) resid_add<TMG, D>(x, j, rb, f32x16{}, vec + V::F2);
    vmem_wait();   // this wave's share of the next layer's vectors has landed before the next barrier
  }

  if constexpr (CLS) {
    // Last block when only each group's first row is wanted (the [CLS] rows of the sequence
    // encoder): keys and values still come from every row, but the attention runs for the first
    // query tile of each group only, and the output projection, LN2, FFN and the final LayerNorm
    // run on the first rows alone, compacted into one 32-row block: the attention writes group
    // g's first-row output to row g of As (free once q|k|v are formed), and each wave moves the
    // residual of row g*S to lane g by lane shuffles (same wave, same columns).
    const int last = a.n_layers - 1;
    const EncW& w = a.layer[last];
    const float* vec = s_vec[last & 1];
    if (last > 0) gq.start(w.wqkv);
    {
      float nm[RB], rstd[RB];
      resid_stats<TM, D>(x, s_stat, nm, rstd);
      resid_norm_to_lds<TM, D>(x, nm, rstd, vec + V::G1, vec + V::B1, As);
    }
    lds_barrier();
    gq.run(As, L::LDA, [&](int, int cb, int rb, const f32x16& acc) {
      block_to_lds_bf16(acc, cb, rb, vec + V::QKV, QKVs, L::LDQ);
    });
    ColGemm<32, D, D / 32> go;
    go.start(w.wo);
    lds_barrier();                                   // q|k|v written, every read of As (LN1) retired
    group_attention<D, DH, NKB, true>(QKVs, L::LDQ, As, L::LDA, ng, a.S, a.scale * kLog2e);
    Resid<32, D> xc;
    {
      // lane l of the compact block holds row g = l % 32 (columns of half l / 32), taken from the
      // lane and row block that hold tile row g*S
      const int g = lane & 31, src_row = g * a.S;
      const int src = (src_row & 31) + (lane & 32), src_rb = src_row >> 5;
#pragma unroll
      for (int j = 0; j < D / 128; ++j)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float v = 0.f;
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) {
            const float t = __shfl(x.v[j][rb][i], src, 64);
            if (rb == src_rb) v = t;
          }
          xc.v[j][0][i] = g < ng ? v : 0.f;
        }
    }
    FfnStream<32, D> ffn;
    ffn.start(w.w1, w.w2, a.F);
    lds_barrier();                                   // the compact attention rows are visible
    go.run(As, L::LDA, [&](int jj, int, int rb, const f32x16& acc) { resid_add<32, D>(xc, jj, rb, acc, vec + V::O); });
    // LN2 of the compact rows -> As rows 0..31; its statistics barrier retires the output
    // projection's reads of As, and every wave is past the attention, so the FFN's hidden
    // buffers may take the q|k|v area
    resid_ln_to_lds<32, D>(xc, vec + V::G2, vec + V::B2, s_stat, As);
    lds_barrier();
    ffn.run(As, Hs, w.b1, xc);
#pragma unroll
    for (int j = 0; j < OCB; ++j) resid_add<32, D>(xc, j, 0, f32x16{}, vec + V::F2);
    float4 gg[D / 128][4], bb[D / 128][4];
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        gg[j][q] = *reinterpret_cast<const float4*>(&a.lnfg[resid_col(j, q)]);
        bb[j][q] = *reinterpret_cast<const float4*>(&a.lnfb[resid_col(j, q)]);
      }
    float nm[1], rstd[1];
    resid_stats<32, D>(xc, s_stat, nm, rstd);
    const int r = lane & 31;
    if (r < ng) {
      float* y = a.Y + (long long)(g0 + r) * D;
#pragma unroll
      for (int j = 0; j < D / 128; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const f32x16& v = xc.v[j][0];
          const int rb = 0;
          *reinterpret_cast<float4*>(&y[resid_col(j, q)]) =
              make_float4(fmaf(fmaf(v[4 * q], rstd[rb], nm[rb]), gg[j][q].x, bb[j][q].x),
                          fmaf(fmaf(v[4 * q + 1], rstd[rb], nm[rb]), gg[j][q].y, bb[j][q].y),
                          fmaf(fmaf(v[4 * q + 2], rstd[rb], nm[rb]), gg[j][q].z, bb[j][q].z),
                          fmaf(fmaf(v[4 * q + 3], rstd[rb], nm[rb]), gg[j][q].w, bb[j][q].w));
        }
    }
    return;
  }

  // final LayerNorm, fp32 out: every valid row, or the first row of each group
  float4 gg[D / 128][4], bb[D / 128][4];
#pragma unroll
  for (int j = 0; j < D / 128; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      gg[j][q] = *reinterpret_cast<const float4*>(&a.lnfg[resid_col(j, q)]);
      bb[j][q] = *reinterpret_cast<const float4*>(&a.lnfb[resid_col(j, q)]);
    }
  float nm[RB], rstd[RB];
  resid_stats<TMG, D>(x, statg, nm, rstd);
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = gr * TMG + rb * 32 + (lane & 31);   // tile row
    if (!s_valid[r]) continue;
    long long out;
    if (a.first_row_only) {
      if (r % a.S) continue;
      out = g0 + r / a.S;
    } else {
      out = row0 + r;
    }
    float* y = a.Y + out * D;
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x16& v = x.v[j][rb];
        *reinterpret_cast<float4*>(&y[resid_col(j, q)]) =
            make_float4(fmaf(fmaf(v[4 * q], rstd[rb], nm[rb]), gg[j][q].x, bb[j][q].x),
                        fmaf(fmaf(v[4 * q + 1], rstd[rb], nm[rb]), gg[j][q].y, bb[j][q].y),
                        fmaf(fmaf(v[4 * q + 2], rstd[rb], nm[rb]), gg[j][q].z, bb[j][q].z),
                        fmaf(fmaf(v[4 * q + 3], rstd[rb], nm[rb]), gg[j][q].w, bb[j][q].w));
      }
  }
}

// Residual rows of x to Xout (row stride D; fp32, or bf16 with out_bf16) for valid tile rows.
template <int TM, int D>
FE_DEV void resid_store(const Resid<TM, D>& x, void* Xout, bool out_bf16, long long row0, const int* s_valid) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int rb = 0; rb < TM / 32; ++rb) {
    const int r = rb * 32 + (lane & 31);
    if (!s_valid[r]) continue;
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const f32x16& v = x.v[j][rb];
        const long long o = (row0 + r) * D + resid_col(j, q);
        if (out_bf16) {
          bf16x4 h;
          h[0] = (bf16)v[4 * q]; h[1] = (bf16)v[4 * q + 1]; h[2] = (bf16)v[4 * q + 2]; h[3] = (bf16)v[4 * q + 3];
          *reinterpret_cast<bf16x4*>(static_cast<bf16*>(Xout) + o) = h;
        } else {
          *reinterpret_cast<float4*>(static_cast<float*>(Xout) + o) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
        }
      }
  }
}

// Rows [row0, row0 + TM) of the bf16 output Y that lie below R get zeros (padding rows).
template <int TM, int D>
FE_DEV void zero_rows_bf16(bf16* Y, long long row0, long long R, const int* s_valid) {
  for (int e = threadIdx.x; e < TM * D / 8; e += WG) {
    const int rr = e / (D / 8), c = (e % (D / 8)) * 8;
    if (row0 + rr >= R || (s_valid && s_valid[rr])) continue;
    *reinterpret_cast<bf16x8*>(Y + (row0 + rr) * D + c) = bf16x8{};
  }
}

// The tail of a block whose attention ran in a separate kernel (long groups), bf16 models:
//   x1 = Xin + O Wo + bo (residual in registers), then
//   TAIL 0: x2 = x1 + FFN(LN2(x1)) -> Xout (fp32 or bf16); when Hout is set (last item layer) also
//           Hout = LNf(x2) in bf16, with zero rows for padding rows;
//   TAIL 1: Xout = x1, and the item layers' cross-attention queries Qout = LN2(x1) Wq + bq (bf16).
// NCH > 0 fixes the FFN width at 128*NCH and takes the software-pipelined stream with a
// three-stage weight ring (used at D = 128, where it fits the register budget).
template <int TM, int D, int TAIL, int NCH>
__global__ __launch_bounds__(WG, 2) void k_post(PostArgs a) {
  constexpr int LDA = D + APAD;
  constexpr int HS_BYTES = 2 * TM * HLD * 2, QS_BYTES = 4 * 32 * 40 * 2;
  constexpr int BIG = HS_BYTES > QS_BYTES ? HS_BYTES : QS_BYTES;
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LDA];
  __shared__ __attribute__((aligned(16))) char big[BIG];
  __shared__ __attribute__((aligned(16))) float2 s_stat[4 * TM];
  __shared__ int s_valid[TM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row0 = xcd_tile(blockIdx.x, gridDim.x) * TM;

  if (a.zero && blockIdx.x == 0)
    for (int e = threadIdx.x; e < a.zero_n; e += WG) a.zero[e] = 0;
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) {
    if (TAIL == 0 && a.Hout) zero_rows_bf16<TM, D>(static_cast<bf16*>(a.Hout), row0, a.R, nullptr);
    return;
  }
  ColGemm<TM, D, D / 32> go;
  go.start(a.wo);
  stage_rows<TM, D>(a.O, false, D, row0, s_valid, nullptr, nullptr, As);
  Resid<TM, D> x;
  resid_load<TM, D>(x, a.Xin, a.xin_f32, row0, s_valid);
  FfnOf<TM, D, NCH> ffn;
  // at D = 256 the first FFN stage is requested after the Wo product: held across it, its
  // registers would push the product's operands and accumulators into scratch
  constexpr bool early = D < 256;
  if constexpr (TAIL == 0 && early) ffn.start(a.w1, a.w2, a.F);
  lds_barrier();
  go.run(As, LDA, [&](int jj, int, int rb, const f32x16& acc) { resid_add<TM, D>(x, jj, rb, acc, a.bo); });
  if constexpr (TAIL == 0 && !early) ffn.start(a.w1, a.w2, a.F);
  ColGemm<TM, D, D / 32> gq;
  if constexpr (TAIL == 1) gq.start(a.wq);
  // LN2 -> As (the barrier inside the statistics retires every read of As by the Wo product)
  resid_ln_to_lds<TM, D>(x, a.ln2g, a.ln2b, s_stat, As);
  lds_barrier();
  if constexpr (TAIL == 0) {
    ffn.run(As, reinterpret_cast<bf16*>(big), a.b1, x);
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int rb = 0; rb < TM / 32; ++rb) resid_add<TM, D>(x, j, rb, f32x16{}, a.b2);
    if (a.Xout) resid_store<TM, D>(x, a.Xout, a.xout_bf16, row0, s_valid);
    if (a.Hout) {
      // final LayerNorm of the module into bf16 H; padding rows of the tile become zeros
      float nm[TM / 32], rstd[TM / 32];
      resid_stats<TM, D>(x, s_stat, nm, rstd);
      bf16* H = static_cast<bf16*>(a.Hout);
#pragma unroll
      for (int rb = 0; rb < TM / 32; ++rb) {
        const int r = rb * 32 + (lane & 31);
        if (!s_valid[r]) continue;
#pragma unroll
        for (int j = 0; j < D / 128; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int c = resid_col(j, q);
            const float4 gg = *reinterpret_cast<const float4*>(&a.lnfg[c]);
            const float4 bb = *reinterpret_cast<const float4*>(&a.lnfb[c]);
            const f32x16& v = x.v[j][rb];
            bf16x4 o;
            o[0] = (bf16)(fmaf(fmaf(v[4 * q], rstd[rb], nm[rb]), gg.x, bb.x));
            o[1] = (bf16)(fmaf(fmaf(v[4 * q + 1], rstd[rb], nm[rb]), gg.y, bb.y));
            o[2] = (bf16)(fmaf(fmaf(v[4 * q + 2], rstd[rb], nm[rb]), gg.z, bb.z));
            o[3] = (bf16)(fmaf(fmaf(v[4 * q + 3], rstd[rb], nm[rb]), gg.w, bb.w));
            *reinterpret_cast<bf16x4*>(H + ((long long)row0 + r) * D + c) = o;
          }
      }
      zero_rows_bf16<TM, D>(H, row0, a.R, s_valid);
    }
    if (a.kv) {
      // last context block: the module's final LayerNorm feeds the key/value projections of
      // every item layer (one slab of 2D columns per layer: keys, then values; the slabs are
      // consecutive column blocks of Wkv).  Two item layers run as one weight stream over all
      // 4D columns, requested before the LayerNorm statistics.
      bf16* st = reinterpret_cast<bf16*>(big) + wave * 32 * 40;
      auto kv_store = [&](int cb, int rb, const f32x16& acc) {   // cb: column block over all layers
        const int slab = cb / (D / 32), c0 = (cb % (D / 32)) * 32;   // slab 2l: keys, 2l + 1: values
        bf16* out = static_cast<bf16*>(a.kv) + (long long)slab * a.R * D + (long long)row0 * D + c0;
        store_block_bf16(acc, a.bkv + slab * D + c0, st, out, D, rb, s_valid);
      };
      float nm[TM / 32], rstd[TM / 32];
      if (a.kv_layers == 2) {
        ColGemm<TM, D, 4 * D / 32> gkv;
        gkv.start(a.wkv);
        resid_stats<TM, D>(x, s_stat, nm, rstd);    // also retires the FFN's reads of As and big
        resid_norm_to_lds<TM, D>(x, nm, rstd, a.lnfg, a.lnfb, As);
        lds_barrier();
        gkv.run(As, LDA, [&](int, int cb, int rb, const f32x16& acc) { kv_store(cb, rb, acc); });
      } else {
        resid_stats<TM, D>(x, s_stat, nm, rstd);
        resid_norm_to_lds<TM, D>(x, nm, rstd, a.lnfg, a.lnfb, As);
        lds_barrier();
        for (int l = 0; l < a.kv_layers; ++l) {
          ColGemm<TM, D, 2 * D / 32> gkv;
          gkv.start(static_cast<const bf16x8*>(a.wkv) + (long long)l * (2 * D / 32) * (D / 16) * 64);
          gkv.run(As, LDA, [&](int, int cb, int rb, const f32x16& acc) { kv_store(l * (2 * D / 32) + cb, rb, acc); });
        }
      }
    }
  } else {
    resid_store<TM, D>(x, a.Xout, a.xout_bf16, row0, s_valid);
    bf16* st = reinterpret_cast<bf16*>(big) + wave * 32 * 40;
    bf16* Q = static_cast<bf16*>(a.Qout) + (long long)row0 * D;
    gq.run(As, LDA, [&](int, int cb, int rb, const f32x16& acc) {
      store_block_bf16(acc, a.bq + cb * 32, st, Q + cb * 32, D, rb, s_valid);
    });
  }
}

template <int TM, int D, int DH, bool CLS, int G, int NCH = 0>
hipError_t launch_module_c(const ModuleArgs& a, hipStream_t s) {
  const int tiles = (a.n_groups + a.gpt - 1) / a.gpt;
  const dim3 grid(tiles), block(WG * G);
  switch ((a.S + 15) / 16) {
    case 1: hipLaunchKernelGGL((k_module_small<TM, D, DH, 1, CLS, G, NCH>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_module_small<TM, D, DH, 2, CLS, G, NCH>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((k_module_small<TM, D, DH, 3, CLS, G, NCH>), grid, block, 0, s, a); break;
    case 4: hipLaunchKernelGGL((k_module_small<TM, D, DH, 4, CLS, G, NCH>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// First-row-only modules take the compacted last block.  Launches with few tiles (at most half
// a workgroup per compute unit) take two wave groups per tile, halving each wave's share of
// every row-wise step: there the per-tile latency, not the compute units' throughput, sets the
// time.
template <int TM, int D, int DH>
hipError_t launch_module_t(const ModuleArgs& a, hipStream_t s) {
  if (a.first_row_only) return launch_module_c<TM, D, DH, true, 1>(a, s);
  if constexpr (D == 128) {   // at d = 256 two groups per compute unit would spill registers
    const int tiles = (a.n_groups + a.gpt - 1) / a.gpt;
    // two wave groups leave room in the register budget for the pipelined FFN stream (three-stage
    // weight ring) when the FFN width is fixed at 4d
    if (tiles <= 128 && a.F == 4 * D) return launch_module_c<TM, D, DH, false, 2, 4>(a, s);
    if (tiles <= 128) return launch_module_c<TM, D, DH, false, 2>(a, s);
  }
  return launch_module_c<TM, D, DH, false, 1>(a, s);
}

// The tail of TAIL 0 (no key/value projections) for launches with few row tiles, split by the
// FFN's hidden width over `parts` workgroups per tile so that the weight streams of a tile run on
// several compute units at once.  Workgroup (tile, p) forms x1 = Xin + O Wo + bo and LN2(x1) as
// k_post does, then only hidden chunks [p n / parts, (p + 1) n / parts) of the n, and writes its
// fp32 sums of the tile's valid rows to slab p of a.part ([parts][R][D]): slab 0 holds x1 plus its
// chunks, every other slab its chunks alone.  k_post_reduce finishes the tail.
template <int TM, int D>
__global__ __launch_bounds__(WG, 2) void k_post_part(PostArgs a, int parts) {
  constexpr int LDA = D + APAD, HS_BYTES = 2 * TM * HLD * 2;
  __shared__ __attribute__((aligned(16))) bf16 As[TM * LDA];
  __shared__ __attribute__((aligned(16))) bf16 Hs[HS_BYTES / 2];
  __shared__ __attribute__((aligned(16))) float2 s_stat[4 * TM];
  __shared__ int s_valid[TM];
  const int id = xcd_tile(blockIdx.x, gridDim.x);          // the parts of a tile share an XCD
  const int tile = id / parts, p = id % parts;
  const int row0 = tile * TM;
  if (!mark_rows<TM>(row0, a.R, a.nvalid, a.rows_per_batch, s_valid)) return;
  const int nch = a.F / HC, c0 = p * nch / parts, c1 = (p + 1) * nch / parts;
  ColGemm<TM, D, D / 32> go;
  go.start(a.wo);
  stage_rows<TM, D>(a.O, false, D, row0, s_valid, nullptr, nullptr, As);
  Resid<TM, D> x;
  resid_load<TM, D>(x, a.Xin, a.xin_f32, row0, s_valid);
  FfnStream<TM, D> ffn;
  constexpr bool early = D < 256;                           // as in k_post
  if constexpr (early) ffn.start(a.w1, a.w2, a.F, c0);
  lds_barrier();
  go.run(As, LDA, [&](int jj, int, int rb, const f32x16& acc) { resid_add<TM, D>(x, jj, rb, acc, a.bo); });
  if constexpr (!early) ffn.start(a.w1, a.w2, a.F, c0);
  // LN2 -> As (the barrier inside the statistics retires every read of As by the Wo product)
  resid_ln_to_lds<TM, D>(x, a.ln2g, a.ln2b, s_stat, As);
  lds_barrier();
  if (p > 0) {
#pragma unroll
    for (int j = 0; j < D / 128; ++j)
#pragma unroll
      for (int rb = 0; rb < TM / 32; ++rb) x.v[j][rb] = f32x16{};
  }
  ffn.run(As, Hs, a.b1, x, c0, c1);
  resid_store<TM, D>(x, static_cast<float*>(a.part) + (long long)p * a.R * D, false, row0, s_valid);
}

// Second half of the split tail, one wave per row: x2 = slab 0 + slab 1 + ... (in that order) + b2
// -> Xout (fp32 or bf16); when Hout is set, Hout = LNf(x2) in bf16.  Padding rows are not read;
// their Hout rows become zeros.
template <int D, int PARTS>
__global__ __launch_bounds__(WG) void k_post_reduce(PostArgs a) {
  constexpr int NV = D / 64;                                 // consecutive columns per lane
  typedef float vecf __attribute__((ext_vector_type(NV)));
  const int lane = threadIdx.x & 63;
  const long long r = (long long)blockIdx.x * (WG / 64) + (threadIdx.x >> 6);
  if (r >= a.R) return;
  const int c = lane * NV;
  const bool ok = !a.nvalid || (r % a.rows_per_batch) < a.nvalid[r / a.rows_per_batch];
  if (!ok) {
    if (a.Hout) {
#pragma unroll
      for (int e = 0; e < NV; ++e) static_cast<bf16*>(a.Hout)[r * D + c + e] = (bf16)0.f;
    }
    return;
  }
  const float* P = static_cast<const float*>(a.part) + r * D + c;
  const long long slab = (long long)a.R * D;
  vecf t[PARTS];
#pragma unroll
  for (int q = 0; q < PARTS; ++q) t[q] = *reinterpret_cast<const vecf*>(P + q * slab);
  vecf v = t[0];
#pragma unroll
  for (int q = 1; q < PARTS; ++q) v += t[q];
  const vecf b2 = *reinterpret_cast<const vecf*>(a.b2 + c);
  v += b2;
  if (a.Xout) {
    if (a.xout_bf16) {
      bf16* y = static_cast<bf16*>(a.Xout) + r * D + c;
#pragma unroll
      for (int e = 0; e < NV; ++e) y[e] = (bf16)v[e];
    } else {
      *reinterpret_cast<vecf*>(static_cast<float*>(a.Xout) + r * D + c) = v;
    }
  }
  if (a.Hout) {
    float sum = 0.f;
#pragma unroll
    for (int e = 0; e < NV; ++e) sum += v[e];
    const float mu = wave_sum(sum) * (1.f / D);
    float m2 = 0.f;
#pragma unroll
    for (int e = 0; e < NV; ++e) m2 += (v[e] - mu) * (v[e] - mu);
    const float rstd = rsqrtf(wave_sum(m2) * (1.f / D) + 1e-5f), nm = -mu * rstd;
    const vecf g = *reinterpret_cast<const vecf*>(a.lnfg + c), b = *reinterpret_cast<const vecf*>(a.lnfb + c);
    bf16* h = static_cast<bf16*>(a.Hout) + r * D + c;
#pragma unroll
    for (int e = 0; e < NV; ++e) h[e] = (bf16)fmaf(fmaf(v[e], rstd, nm), g[e], b[e]);
  }
}

// Workgroups per row tile of a TAIL 0 launch without key/value projections (0: the scratch the
// caller lent is missing, too small or misaligned).
template <int TM, int D>
int post_parts(const PostArgs& a) {
  if (a.tail != 0 || a.kv) return 1;
  const int parts = post_split_parts(a.R, D, a.F);
  if (parts == 1) return 1;
  if (!a.part || (reinterpret_cast<uintptr_t>(a.part) & 15) || a.part_bytes < post_part_bytes(a.R, D, a.F)) return 0;
  return parts;
}

template <int TM, int D>
hipError_t launch_post_t(const PostArgs& a, hipStream_t s) {
  dim3 grid((a.R + TM - 1) / TM);
  const int parts = post_parts<TM, D>(a);
  if (parts == 0) return hipErrorInvalidValue;
  if (parts > 1) {
    hipLaunchKernelGGL((k_post_part<TM, D>), dim3(grid.x * parts), dim3(WG), 0, s, a, parts);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 rgrid((a.R + WG / 64 - 1) / (WG / 64));
    if (parts == 2) hipLaunchKernelGGL((k_post_reduce<D, 2>), rgrid, dim3(WG), 0, s, a);
    else if (parts == 4) hipLaunchKernelGGL((k_post_reduce<D, 4>), rgrid, dim3(WG), 0, s, a);
    else hipLaunchKernelGGL((k_post_reduce<D, 8>), rgrid, dim3(WG), 0, s, a);
    return hipGetLastError();
  }
  if (a.tail == 1) hipLaunchKernelGGL((k_post<TM, D, 1, 0>), grid, dim3(WG), 0, s, a);
  else if (D == 128 && a.F == 4 * D) hipLaunchKernelGGL((k_post<TM, D, 0, (D == 128 ? 4 : 0)>), grid, dim3(WG), 0, s, a);
  else hipLaunchKernelGGL((k_post<TM, D, 0, 0>), grid, dim3(WG), 0, s, a);
  return hipGetLastError();
}

}  // namespace

// groups of up to 64 rows (the score blocks of a group are held in registers at once); at
// d = 512 a tile's q|k|v, the double-buffered block vectors and the LN1 tile exceed the LDS of a
// compute unit, so such modules take the separate-attention path
int module_small_tile_rows(int d) { return d >= 512 ? 0 : 64; }

hipError_t launch_module_small(ModuleArgs a, hipStream_t s) {
  if (a.n_groups <= 0) return hipSuccess;
  const int tm = module_small_tile_rows(a.D);
  if (a.S < 1 || a.S > tm || a.n_layers < 1 || a.n_layers > FE_MAX_LAYERS || a.F % HC) return hipErrorInvalidValue;
  a.gpt = tm / a.S;
  const int dh = a.D / a.H;
  switch (a.D) {
    case 128: return dh == 64 ? launch_module_t<64, 128, 64>(a, s) : launch_module_t<64, 128, 32>(a, s);
    case 256: return dh == 64 ? launch_module_t<64, 256, 64>(a, s) : launch_module_t<64, 256, 32>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// A power of two up to 8 that divides the FFN's chunk count when the launch has few row tiles (at
// most 256 workgroups in all), else 1.  A function of the shape alone, so that every caller of a
// shape sums the partial results in the same order.
int post_split_parts(long long R, int D, int F) {
  if (D != 128 && D != 256) return 1;
  const long long tiles = (R + 63) / 64, nch = F / HC;
  if (F % HC) return 1;
  for (int p = 8; p >= 2; p /= 2)
    if (nch % p == 0 && tiles * p <= 256) return p;
  return 1;
}

size_t post_part_bytes(long long R, int D, int F) {
  const int p = post_split_parts(R, D, F);
  return p > 1 ? (size_t)p * R * D * 4 : 0;
}

// d >= 512 models take the tiled products instead of the fused tails
hipError_t launch_post(const PostArgs& a, hipStream_t s) {
  if (a.R <= 0) return hipSuccess;
  switch (a.D) {
    case 128: return launch_post_t<64, 128>(a, s);
    case 256: return launch_post_t<64, 256>(a, s);
    default: return hipErrorInvalidValue;
  }
}
