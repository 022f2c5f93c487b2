// Attention kernels with the neighbouring projections fused in, for bf16 models with d = 128,
// head width 32 and attention groups of at most 256 rows (the context module and the distinct
// items of the RecSys-sized workloads).  A workgroup of 16 waves owns one (batch, head).
//
// k_self_attention (first half of a pre-LN block):
//   1. LN1 of the group's rows -> LDS (bf16), four threads per row;
//   2. q, k, v of head h -- three 32-column blocks of the packed q|k|v weights per 32-row block --
//      on 32x32x16 MFMA, formed transposed as in the row-tile kernels (lane = row, four
//      consecutive columns), written straight into the attention operand layouts: q and k
//      row-major, v transposed;
//   3. one 16-query tile per wave: scores of all keys, one softmax over the whole row, P V, as in
//      the attention kernel with every key resident in LDS.
// k_cross_attention (item layers: self-attention tail + cross-attention):
//   1. x1 = x + O Wo + bo for every row of the request (all heads' O; each head's workgroup
//      forms it, the head-0 workgroup also writes it out as the new residual stream);
//   2. LN2(x1) -> LDS, q of head h = LN2(x1) Wq + bq;
//   3. attention of those queries over the request's context keys/values (the key/value cache).
// No q|k|v or query tensor reaches global memory, and the projections need no launches of their own.
#include "fe_common.h"
#include "fe_dedup.h"
#include "fe_tile.h"
#include "flasheval.h"

namespace {

using fe_tile::APAD;
using fe_tile::a_frag;

constexpr float kLog2e = 1.4426950408889634f;

template <int D, int DH, bool DEDUP>
__global__ __launch_bounds__(1024) void k_self_attention(SelfAttnArgs a) {
  constexpr int NT = 1024, NR = 256, LDA = D + APAD, QLD = DH + 8, VLD = NR + 8;
  constexpr int KS = D / 16, NB = DH / 16, NB32 = NR / 32;
  static_assert(DH == 32, "one 32-column block per head and projection");
  __shared__ __attribute__((aligned(16))) bf16 As[NR * LDA];
  __shared__ __attribute__((aligned(16))) bf16 Qs[NR * QLD];
  __shared__ __attribute__((aligned(16))) bf16 Ks[NR * QLD];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DH * VLD];
  __shared__ __attribute__((aligned(16))) float s_g[D], s_b[D];
  __shared__ int32_t s_uniq[DEDUP ? NR : 1];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = xcd_tile(blockIdx.x, gridDim.x), h = bh % a.n_heads, b = bh / a.n_heads;
  int n = a.per;
  if constexpr (DEDUP) {
    // the request's distinct set; its bitmap and word prefix sums live in As until LN1 overwrites it
    uint32_t* bits = reinterpret_cast<uint32_t*>(As);
    const int W = (a.M + 31) >> 5;
    const bool lead = h == 0;
    int bad = 0;
    const int U = fe_dedup::distinct_set<NT>(a.lists + (long long)b * a.KL, a.KL, a.M, a.per,
                                             lead ? a.uniq + (long long)b * a.per : nullptr,
                                             lead ? a.slot + (long long)b * a.KL : nullptr, &bad, bits, bits + W, s_uniq);
    if (lead && tid == 0) {
      a.n_uniq[b] = U;
      a.status[b] = bad ? FE_DEV_BAD_INDEX : 0;
    }
    n = min(n, U);
    if (n <= 0) {                                    // no valid entry: zero rows only
      if (lead)
        for (int e = tid; e < a.per * (D / 8); e += NT)
          reinterpret_cast<bf16x8*>(a.Xrows)[(long long)b * a.per * (D / 8) + e] = bf16x8{};
      return;                                        // uniform over the workgroup
    }
  } else {
    if (a.nvalid) n = min(n, a.nvalid[b]);
    if (n <= 0) return;                              // uniform over the workgroup
  }
  const int nrb = (n + 31) / 32;                     // 32-row blocks that hold valid rows
  // the weight fragments of this wave's first projection block (step 2), requested now so that
  // their latency hides behind LN1
  const bf16x8* Wqkv = static_cast<const bf16x8*>(a.wqkv);
  bf16x8 wfirst[KS];
  if (wave < 3 * nrb) {
    const int cbg = (wave % 3) * a.n_heads + h;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) wfirst[ks] = Wqkv[((long long)cbg * KS + ks) * 64 + lane];
  }

  // ---- 1. LN1 of rows 0 .. 32*nrb - 1 (rows >= n are zero) -------------------------------
  if (tid < D / 4) {
    reinterpret_cast<float4*>(s_g)[tid] = reinterpret_cast<const float4*>(a.ln_g)[tid];
    reinterpret_cast<float4*>(s_b)[tid] = reinterpret_cast<const float4*>(a.ln_b)[tid];
  }
  {
    constexpr int TPR = NT / NR;                     // four threads per row, D/4 values each
    constexpr int NV = D / TPR;
    const int r = tid / TPR, part = tid % TPR;
    const bool valid = r < n;
    const long long grow = (long long)b * a.per + (valid ? r : 0);
    float v[NV];
    if constexpr (DEDUP) {
      // element rows from the table; the head-0 workgroup also writes them (zero rows from n on)
      const bf16x8* src = reinterpret_cast<const bf16x8*>(static_cast<const bf16*>(a.table) + b * a.table_bs +
                                                          (long long)s_uniq[valid ? r : 0] * D);
      bf16x8* dst = reinterpret_cast<bf16x8*>(static_cast<bf16*>(a.Xrows) + ((long long)b * a.per + r) * D);
#pragma unroll
      for (int i = 0; i < NV / 8; ++i) {
        const bf16x8 t = src[i * TPR + part];
        if (h == 0 && r < a.per) dst[i * TPR + part] = valid ? t : bf16x8{};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[8 * i + e] = (float)t[e];
      }
    } else if (a.x_f32) {
      const float4* src = reinterpret_cast<const float4*>(static_cast<const float*>(a.X) + grow * D);
#pragma unroll
      for (int i = 0; i < NV / 4; ++i) {
        const float4 t = src[i * TPR + part];
        v[4 * i] = t.x; v[4 * i + 1] = t.y; v[4 * i + 2] = t.z; v[4 * i + 3] = t.w;
      }
    } else {
      const bf16x8* src = reinterpret_cast<const bf16x8*>(static_cast<const bf16*>(a.X) + grow * D);
#pragma unroll
      for (int i = 0; i < NV / 8; ++i) {
        const bf16x8 t = src[i * TPR + part];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[8 * i + e] = (float)t[e];
      }
    }
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) sum += v[i];
    sum += __shfl_xor(sum, 1, 64);
    sum += __shfl_xor(sum, 2, 64);
    const float mean = sum * (1.f / D);
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) { const float t = v[i] - mean; q += t * t; }
    q += __shfl_xor(q, 1, 64);
    q += __shfl_xor(q, 2, 64);
    const float rstd = rsqrtf(q * (1.f / D) + 1e-5f), nm = -mean * rstd;
    lds_barrier();                                   // s_g, s_b visible
    if (r < 32 * nrb) {
      // element index of v[i]: fp32 rows hold float4 (i/4)*TPR + part, bf16 rows bf16x8 (i/8)*TPR + part
#pragma unroll
      for (int i = 0; i < NV; i += 4) {
        const int k = (!DEDUP && a.x_f32) ? ((i / 4) * TPR + part) * 4 : ((i / 8) * TPR + part) * 8 + (i % 8);
        const float4 gg = *reinterpret_cast<const float4*>(&s_g[k]);
        const float4 bb = *reinterpret_cast<const float4*>(&s_b[k]);
        bf16x4 o;
        o[0] = (bf16)fmaf(fmaf(v[i], rstd, nm), gg.x, bb.x);
        o[1] = (bf16)fmaf(fmaf(v[i + 1], rstd, nm), gg.y, bb.y);
        o[2] = (bf16)fmaf(fmaf(v[i + 2], rstd, nm), gg.z, bb.z);
        o[3] = (bf16)fmaf(fmaf(v[i + 3], rstd, nm), gg.w, bb.w);
        if (!valid) o = bf16x4{};
        *reinterpret_cast<bf16x4*>(&As[r * LDA + k]) = o;
      }
    }
  }
  lds_barrier();

  // ---- 2. q, k, v of head h: block i = 3*rb + j (j = 0 q, 1 k, 2 v) on wave i % 16 ---------
  {
    for (int i = wave; i < 3 * nrb; i += NT / 64) {
      const int rb = i / 3, j = i % 3;
      const int cbg = j * a.n_heads + h;             // global 32-column block of the projection
      bf16x8 wf[KS], af[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) wf[ks] = i == wave ? wfirst[ks] : Wqkv[((long long)cbg * KS + ks) * 64 + lane];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) af[ks] = a_frag(As, LDA, rb * 32, ks * 16, lane);
      __builtin_amdgcn_sched_barrier(0);   // every operand read issued before the first product
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks], af[ks], acc, 0, 0, 0);
      // lane holds row rb*32 + lane%32, columns 8q + 4*(lane/32) + e of the head in acc[4q + e]
      const int row = rb * 32 + (lane & 31);
      const float* bias = a.bqkv + cbg * 32;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int c = qq * 8 + (lane >> 5) * 4;
        const float4 bb = *reinterpret_cast<const float4*>(&bias[c]);
        const float o0 = acc[4 * qq] + bb.x, o1 = acc[4 * qq + 1] + bb.y;
        const float o2 = acc[4 * qq + 2] + bb.z, o3 = acc[4 * qq + 3] + bb.w;
        if (j == 2) {
          Vt[c * VLD + row] = (bf16)o0;
          Vt[(c + 1) * VLD + row] = (bf16)o1;
          Vt[(c + 2) * VLD + row] = (bf16)o2;
          Vt[(c + 3) * VLD + row] = (bf16)o3;
        } else {
          bf16x4 o;
          o[0] = (bf16)o0; o[1] = (bf16)o1; o[2] = (bf16)o2; o[3] = (bf16)o3;
          *reinterpret_cast<bf16x4*>(&(j == 0 ? Qs : Ks)[row * QLD + c]) = o;
        }
      }
    }
  }
  lds_barrier();

  // ---- 3. attention: query tile `wave`, every key in LDS ----------------------------------
  const int q0 = wave * 16;
  if (q0 >= n) return;                               // uniform over the wave; no barrier follows
  const int g = lane >> 4, r = lane & 15, qrow = q0 + r;
  const float c2 = a.scale * kLog2e;
  const bf16x8 qf = *reinterpret_cast<const bf16x8*>(&Qs[qrow * QLD + g * 8]);
  float p[NB32][8];
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < NB32; ++kb) {
    if (kb >= nrb) continue;                         // uniform
    const int k0 = kb * 32 + (r >> 2) * 8 + (r & 3), k1 = k0 + 4;
    const bf16x8 ka = *reinterpret_cast<const bf16x8*>(&Ks[k0 * QLD + g * 8]);
    const bf16x8 kc = *reinterpret_cast<const bf16x8*>(&Ks[k1 * QLD + g * 8]);
    const f32x4 s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
    const f32x4 s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc, qf, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      p[kb][jj] = s0[jj];
      p[kb][4 + jj] = s1[jj];
    }
    if (kb * 32 + 32 > n) {                          // ragged last block (uniform)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (kb * 32 + g * 8 + jj >= n) p[kb][jj] = -INFINITY;
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) mx = fmaxf(mx, p[kb][jj]);
  }
  const float mc = rows_max(mx) * c2;                // finite: key 0 is always valid
  float l = 0.f;
  bf16x8 pb[NB32];
#pragma unroll
  for (int kb = 0; kb < NB32; ++kb) {
    if (kb >= nrb) continue;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const float e = __builtin_amdgcn_exp2f(fmaf(p[kb][jj], c2, -mc));   // v_exp_f32; exp2(-inf) = 0
      l += e;
      pb[kb][jj] = (bf16)e;
    }
  }
  const float inv = __builtin_amdgcn_rcpf(rows_sum(l));   // v_rcp_f32
  f32x4 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < NB32; ++kb) {
    if (kb >= nrb) continue;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&Vt[(i * 16 + r) * VLD + kb * 32 + g * 8]);
      o[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb[kb], o[i], 0, 0, 0);
    }
  }
  if (qrow >= n) return;
  bf16* Ob = static_cast<bf16*>(a.O) + ((long long)b * a.per + qrow) * D + h * DH;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    bf16x4 w;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) w[jj] = (bf16)(o[i][jj] * inv);
    *reinterpret_cast<bf16x4*>(Ob + i * 16 + g * 4) = w;
  }
}

// Attention of a 16-query tile per wave over keys held in LDS (Ks row-major [key][dh + 8],
// Vt transposed [dh][NR + 8]); keys >= nk are masked.  Q tile rows come from Qs [row][dh + 8].
// O rows q0 + r < nq are written to Ob + row * D (Ob already offset to the head's columns).
template <int D, int DH, int NR>
FE_DEV void tile_attention(const bf16* Qs, const bf16* Ks, const bf16* Vt, int nq, int nk, float c2, bf16* Ob) {
  constexpr int QLD = DH + 8, VLD = NR + 8, NB = DH / 16, NB32 = NR / 32;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int q0 = wave * 16;
  if (q0 >= nq) return;
  const int g = lane >> 4, r = lane & 15, qrow = q0 + r;
  const int nkb = (nk + 31) / 32;
  const bf16x8 qf = *reinterpret_cast<const bf16x8*>(&Qs[qrow * QLD + g * 8]);
  float p[NB32][8];
  float mx = -INFINITY;
#pragma unroll
  for (int kb = 0; kb < NB32; ++kb) {
    if (kb >= nkb) continue;                         // uniform
    const int k0 = kb * 32 + (r >> 2) * 8 + (r & 3), k1 = k0 + 4;
    const bf16x8 ka = *reinterpret_cast<const bf16x8*>(&Ks[k0 * QLD + g * 8]);
    const bf16x8 kc = *reinterpret_cast<const bf16x8*>(&Ks[k1 * QLD + g * 8]);
    const f32x4 s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
    const f32x4 s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc, qf, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      p[kb][jj] = s0[jj];
      p[kb][4 + jj] = s1[jj];
    }
    if (kb * 32 + 32 > nk) {                         // ragged last block (uniform)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj)
        if (kb * 32 + g * 8 + jj >= nk) p[kb][jj] = -INFINITY;
    }
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) mx = fmaxf(mx, p[kb][jj]);
  }
  const float mc = rows_max(mx) * c2;                // finite: key 0 is always valid
  float l = 0.f;
  bf16x8 pb[NB32];
#pragma unroll
  for (int kb = 0; kb < NB32; ++kb) {
    if (kb >= nkb) continue;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const float e = __builtin_amdgcn_exp2f(fmaf(p[kb][jj], c2, -mc));   // v_exp_f32; exp2(-inf) = 0
      l += e;
      pb[kb][jj] = (bf16)e;
    }
  }
  const float inv = __builtin_amdgcn_rcpf(rows_sum(l));   // v_rcp_f32
  f32x4 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < NB32; ++kb) {
    if (kb >= nkb) continue;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&Vt[(i * 16 + r) * VLD + kb * 32 + g * 8]);
      o[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb[kb], o[i], 0, 0, 0);
    }
  }
  if (qrow >= nq) return;
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    bf16x4 w;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) w[jj] = (bf16)(o[i][jj] * inv);
    *reinterpret_cast<bf16x4*>(Ob + (long long)qrow * D + i * 16 + g * 4) = w;
  }
}

template <int D, int DH>
__global__ __launch_bounds__(1024) void k_cross_attention(CrossAttnArgs a) {
  constexpr int NT = 1024, NR = 256, LDA = D + APAD, QLD = DH + 8, VLD = NR + 8, KS = D / 16;
  static_assert(DH == 32 && D == 128, "four 32-column blocks, one per head");
  __shared__ __attribute__((aligned(16))) bf16 As[NR * LDA];       // O rows, then LN2(x1)
  __shared__ __attribute__((aligned(16))) bf16 Qs[NR * QLD];
  __shared__ __attribute__((aligned(16))) bf16 Ks[NR * QLD];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DH * VLD];
  __shared__ __attribute__((aligned(16))) float2 s_stat[4 * NR];   // per column block, per row
  __shared__ __attribute__((aligned(16))) float s_vec[4 * D];       // bo | ln2g | ln2b | bq

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = xcd_tile(blockIdx.x, gridDim.x), h = bh % a.n_heads, b = bh / a.n_heads;
  int n = a.per;
  if (a.nvalid) n = min(n, a.nvalid[b]);
  if (n <= 0) return;                                // uniform over the workgroup
  const int nrb = (n + 31) / 32;
  const int nk = a.T, nkb = (nk + 31) / 32;
  const int cb = wave & 3, rb0 = wave >> 2;
  // Every global load of the prologue is issued before any of them is used -- this wave's Wo
  // fragments, the block's vectors, the head's context keys and values, the attention output rows,
  // the residual rows -- so their latencies overlap; out-of-range rows and keys read a valid row and
  // are zeroed when staged.
  bf16x8 wf[KS];
  {
    const bf16x8* W = static_cast<const bf16x8*>(a.wo);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) wf[ks] = W[((long long)cb * KS + ks) * 64 + lane];
  }
  float4 vec4 = make_float4(0.f, 0.f, 0.f, 0.f);
  if (tid < D) {
    const int v = tid / (D / 4), o = (tid % (D / 4)) * 4;
    const float* src = v == 0 ? a.bo : v == 1 ? a.ln2g : v == 2 ? a.ln2b : a.bq;
    vec4 = *reinterpret_cast<const float4*>(src + o);
  }
  // context keys and values of head h
  constexpr int KV_PER = NR * DH / 8 / NT;           // 16-byte vectors per thread per tensor
  static_assert(KV_PER >= 1, "keys do not split over the workgroup");
  uint4 kr[KV_PER], vr[KV_PER];
  {
    const bf16* Kb = static_cast<const bf16*>(a.Kc) + (long long)b * nk * D + h * DH;
    const bf16* Vb = static_cast<const bf16*>(a.Vc) + (long long)b * nk * D + h * DH;
#pragma unroll
    for (int p = 0; p < KV_PER; ++p) {
      const int e = p * NT + tid, key = e / (DH / 8), d0 = (e % (DH / 8)) * 8;
      const long long kk = key < nk ? key : 0;
      kr[p] = *reinterpret_cast<const uint4*>(Kb + kk * D + d0);
      vr[p] = *reinterpret_cast<const uint4*>(Vb + kk * D + d0);
    }
  }
  // attention output rows O (all heads): row r of the group for vector p
  const long long rbase = (long long)b * a.per;
  constexpr int O_PER = NR * (D / 8) / NT;
  uint4 orow[O_PER];
#pragma unroll
  for (int p = 0; p < O_PER; ++p) {
    const int e = p * NT + tid, r = e / (D / 8), c = (e % (D / 8)) * 8;
    if (r < 32 * nrb)
      orow[p] = *reinterpret_cast<const uint4*>(static_cast<const bf16*>(a.O) + (rbase + (r < n ? r : 0)) * D + c);
  }
  // residual rows: wave w holds column block cb = w % 4 of row blocks w/4 and w/4 + 4, in the
  // transposed accumulator layout (row rb*32 + lane%32, columns cb*32 + 8q + 4(lane/32) + e)
  const int colq = cb * 32 + 4 * (lane >> 5);       // + 8q
  f32x16 x[2];
  if (a.xin_f32) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int rb = rb0 + 4 * i, row = rb * 32 + (lane & 31);
      const bool ok = rb < nrb && row < n;
      const long long grow = rbase + (ok ? row : 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 t = *reinterpret_cast<const float4*>(static_cast<const float*>(a.Xin) + grow * D + colq + 8 * q);
        x[i][4 * q] = ok ? t.x : 0.f;
        x[i][4 * q + 1] = ok ? t.y : 0.f;
        x[i][4 * q + 2] = ok ? t.z : 0.f;
        x[i][4 * q + 3] = ok ? t.w : 0.f;
      }
    }
  }
  bf16x4 xr[2][4];                                   // bf16 residual rows, converted after the staging
  if (!a.xin_f32) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int rb = rb0 + 4 * i, row = rb * 32 + (lane & 31);
      const long long grow = rbase + (rb < nrb && row < n ? row : 0);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        xr[i][q] = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(a.Xin) + grow * D + colq + 8 * q);
    }
  }
  // stage: the vectors, the keys (row-major) and values (transposed; keys nk .. 32*nkb-1 zero),
  // the O rows (rows n .. 32*nrb-1 zero)
  if (tid < D) reinterpret_cast<float4*>(s_vec)[tid] = vec4;
#pragma unroll
  for (int p = 0; p < KV_PER; ++p) {
    const int e = p * NT + tid, key = e / (DH / 8), d0 = (e % (DH / 8)) * 8;
    if (key >= nkb * 32) continue;                   // never read
    const bool ok = key < nk;
    *reinterpret_cast<uint4*>(&Ks[key * QLD + d0]) = ok ? kr[p] : make_uint4(0, 0, 0, 0);
    const bf16* v = reinterpret_cast<const bf16*>(&vr[p]);
#pragma unroll
    for (int i = 0; i < 8; ++i) Vt[(d0 + i) * VLD + key] = ok ? v[i] : (bf16)0.f;
  }
#pragma unroll
  for (int p = 0; p < O_PER; ++p) {
    const int e = p * NT + tid, r = e / (D / 8), c = (e % (D / 8)) * 8;
    if (r < 32 * nrb) *reinterpret_cast<uint4*>(&As[r * LDA + c]) = r < n ? orow[p] : make_uint4(0, 0, 0, 0);
  }
  if (!a.xin_f32) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int rb = rb0 + 4 * i, row = rb * 32 + (lane & 31);
      const bool ok = rb < nrb && row < n;
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) x[i][4 * q + e] = ok ? (float)xr[i][q][e] : 0.f;
    }
  }
  lds_barrier();

  // ---- x1 = x + O Wo + bo ------------------------------------------------------------------
  {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int rb = rb0 + 4 * i;
      if (rb >= nrb) continue;                       // uniform over the wave
      bf16x8 af[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) af[ks] = a_frag(As, LDA, rb * 32, ks * 16, lane);
      __builtin_amdgcn_sched_barrier(0);
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks], af[ks], acc, 0, 0, 0);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 bb = *reinterpret_cast<const float4*>(&s_vec[colq + 8 * q]);
        x[i][4 * q] += acc[4 * q] + bb.x;
        x[i][4 * q + 1] += acc[4 * q + 1] + bb.y;
        x[i][4 * q + 2] += acc[4 * q + 2] + bb.z;
        x[i][4 * q + 3] += acc[4 * q + 3] + bb.w;
      }
    }
  }
  // Wq fragments of head h for the query step, requested before LN2
  bf16x8 wqf[KS];
  if (wave < nrb) {
    const bf16x8* W = static_cast<const bf16x8*>(a.wq);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) wqf[ks] = W[((long long)h * KS + ks) * 64 + lane];
  }
  // the head-0 workgroup writes x1 of the valid rows as the new residual stream
  if (h == 0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int rb = rb0 + 4 * i, row = rb * 32 + (lane & 31);
      if (rb >= nrb || row >= n) continue;
      const long long o = (rbase + row) * D + colq;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if (a.xout_bf16) {
          bf16x4 hv;
          hv[0] = (bf16)x[i][4 * q]; hv[1] = (bf16)x[i][4 * q + 1]; hv[2] = (bf16)x[i][4 * q + 2]; hv[3] = (bf16)x[i][4 * q + 3];
          *reinterpret_cast<bf16x4*>(static_cast<bf16*>(a.Xout) + o + 8 * q) = hv;
        } else {
          *reinterpret_cast<float4*>(static_cast<float*>(a.Xout) + o + 8 * q) =
              make_float4(x[i][4 * q], x[i][4 * q + 1], x[i][4 * q + 2], x[i][4 * q + 3]);
        }
      }
    }
  }
  // ---- LN2(x1) -> As: per-row statistics of the wave's 32 columns (two lanes share a row),
  //      merged across the four column blocks through s_stat (pairwise mean / M2 update) -----
  float nm[2], rstd[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) sum += x[i][k];
    const float m = sum * (1.f / 16);
    float m2 = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) { const float t = x[i][k] - m; m2 += t * t; }
    const auto pm = __builtin_amdgcn_permlane32_swap(__float_as_uint(m), __float_as_uint(m), false, false);
    const auto pq = __builtin_amdgcn_permlane32_swap(__float_as_uint(m2), __float_as_uint(m2), false, false);
    const float ma = __uint_as_float(pm[0]), mb = __uint_as_float(pm[1]), dm = mb - ma;
    const int rb = rb0 + 4 * i;
    if (lane < 32 && rb < nrb)
      s_stat[cb * NR + rb * 32 + lane] =
          make_float2(0.5f * (ma + mb), __uint_as_float(pq[0]) + __uint_as_float(pq[1]) + dm * dm * 8.f);
  }
  lds_barrier();                                     // also retires every read of As (O)
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int rb = rb0 + 4 * i, row = rb * 32 + (lane & 31);
    if (rb >= nrb) continue;
    const float2 p0 = s_stat[row], p1 = s_stat[NR + row], p2 = s_stat[2 * NR + row], p3 = s_stat[3 * NR + row];
    const float mu = 0.25f * ((p0.x + p1.x) + (p2.x + p3.x));
    const float d0 = p0.x - mu, d1 = p1.x - mu, d2 = p2.x - mu, d3 = p3.x - mu;
    const float m2 = (p0.y + p1.y) + (p2.y + p3.y) + (d0 * d0 + d1 * d1 + d2 * d2 + d3 * d3) * 32.f;
    rstd[i] = rsqrtf(m2 * (1.f / D) + 1e-5f);
    nm[i] = -mu * rstd[i];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int c = colq + 8 * q;
      const float4 gg = *reinterpret_cast<const float4*>(&s_vec[D + c]);
      const float4 bb = *reinterpret_cast<const float4*>(&s_vec[2 * D + c]);
      bf16x4 o;
      o[0] = (bf16)fmaf(fmaf(x[i][4 * q], rstd[i], nm[i]), gg.x, bb.x);
      o[1] = (bf16)fmaf(fmaf(x[i][4 * q + 1], rstd[i], nm[i]), gg.y, bb.y);
      o[2] = (bf16)fmaf(fmaf(x[i][4 * q + 2], rstd[i], nm[i]), gg.z, bb.z);
      o[3] = (bf16)fmaf(fmaf(x[i][4 * q + 3], rstd[i], nm[i]), gg.w, bb.w);
      *reinterpret_cast<bf16x4*>(&As[row * LDA + c]) = o;
    }
  }
  lds_barrier();

  // ---- q of head h = LN2(x1) Wq + bq: row block `wave` ------------------------------------
  if (wave < nrb) {
    const int rb = wave, row = rb * 32 + (lane & 31);
    bf16x8 af[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) af[ks] = a_frag(As, LDA, rb * 32, ks * 16, lane);
    __builtin_amdgcn_sched_barrier(0);
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wqf[ks], af[ks], acc, 0, 0, 0);
    const float* bias = s_vec + 3 * D + h * DH;
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      const int c = qq * 8 + (lane >> 5) * 4;
      const float4 bb = *reinterpret_cast<const float4*>(&bias[c]);
      bf16x4 o;
      o[0] = (bf16)(acc[4 * qq] + bb.x);
      o[1] = (bf16)(acc[4 * qq + 1] + bb.y);
      o[2] = (bf16)(acc[4 * qq + 2] + bb.z);
      o[3] = (bf16)(acc[4 * qq + 3] + bb.w);
      *reinterpret_cast<bf16x4*>(&Qs[row * QLD + c]) = o;
    }
  }
  lds_barrier();

  // ---- attention over the context keys ----------------------------------------------------
  tile_attention<D, DH, NR>(Qs, Ks, Vt, n, nk, a.scale * kLog2e,
                            static_cast<bf16*>(a.O2) + rbase * D + h * DH);
}

}  // namespace

bool self_attention_fits(int d, int n_heads, int per) { return d == 128 && d / n_heads == 32 && per >= 1 && per <= 256; }

hipError_t launch_self_attention(const SelfAttnArgs& a, int d, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  if (!self_attention_fits(d, a.n_heads, a.per)) return hipErrorInvalidValue;
  if (a.lists) {
    // the bitmap and its prefix sums live in the 256 x 136 bf16 LN1 tile
    if (a.KL < 1 || a.M < 1 || a.per != min(a.M, a.KL) || 2 * ((a.M + 31) / 32) > 256 * 136 / 2 || !a.table ||
        !a.uniq || !a.n_uniq || !a.slot || !a.status || !a.Xrows)
      return hipErrorInvalidValue;
    hipLaunchKernelGGL((k_self_attention<128, 32, true>), dim3((unsigned)(a.B * a.n_heads)), dim3(1024), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_self_attention<128, 32, false>), dim3((unsigned)(a.B * a.n_heads)), dim3(1024), 0, s, a);
  }
  return hipGetLastError();
}

bool cross_attention_fits(int d, int n_heads, int per, int T) {
  return d == 128 && d / n_heads == 32 && per >= 1 && per <= 256 && T >= 1 && T <= 256;
}

hipError_t launch_cross_attention(const CrossAttnArgs& a, int d, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  if (!cross_attention_fits(d, a.n_heads, a.per, a.T) || a.O2 == a.O || a.Xout == a.Xin) return hipErrorInvalidValue;
  hipLaunchKernelGGL((k_cross_attention<128, 32>), dim3((unsigned)(a.B * a.n_heads)), dim3(1024), 0, s, a);
  return hipGetLastError();
}
