// Self-attention of one head with its q|k|v projection fused in, for bf16 models with d = 128,
// head width 32 and attention groups of at most 256 rows (the context module and the distinct
// items of the RecSys-sized workloads).
//
// A workgroup of 16 waves owns one (batch, head):
//   1. LN1 of the group's rows -> LDS (bf16), four threads per row;
//   2. q, k, v of head h -- three 32-column blocks of the packed q|k|v weights per 32-row block --
//      on 32x32x16 MFMA, formed transposed as in the row-tile kernels (lane = row, four
//      consecutive columns), written straight into the attention operand layouts: q and k
//      row-major, v transposed;
//   3. one 16-query tile per wave: scores of all keys, one softmax over the whole row, P V, as in
//      the attention kernel with every key resident in LDS.
// The q|k|v tensor never reaches global memory, and the projection needs no launch of its own.
#include "fe_common.h"
#include "fe_tile.h"

namespace {

using fe_tile::APAD;
using fe_tile::a_frag;

constexpr float kLog2e = 1.4426950408889634f;

template <int D, int DH>
__global__ __launch_bounds__(1024) void k_self_attention(SelfAttnArgs a) {
  constexpr int NT = 1024, NR = 256, LDA = D + APAD, QLD = DH + 8, VLD = NR + 8;
  constexpr int KS = D / 16, NB = DH / 16, NB32 = NR / 32;
  static_assert(DH == 32, "one 32-column block per head and projection");
  __shared__ __attribute__((aligned(16))) bf16 As[NR * LDA];
  __shared__ __attribute__((aligned(16))) bf16 Qs[NR * QLD];
  __shared__ __attribute__((aligned(16))) bf16 Ks[NR * QLD];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DH * VLD];
  __shared__ __attribute__((aligned(16))) float s_g[D], s_b[D];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int bh = xcd_tile(blockIdx.x, gridDim.x), h = bh % a.n_heads, b = bh / a.n_heads;
  int n = a.per;
  if (a.nvalid) n = min(n, a.nvalid[b]);
  if (n <= 0) return;                                // uniform over the workgroup
  const int nrb = (n + 31) / 32;                     // 32-row blocks that hold valid rows

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
    if (a.x_f32) {
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
    __syncthreads();                                 // s_g, s_b visible
    if (r < 32 * nrb) {
      // element index of v[i]: fp32 rows hold float4 (i/4)*TPR + part, bf16 rows bf16x8 (i/8)*TPR + part
#pragma unroll
      for (int i = 0; i < NV; i += 4) {
        const int k = a.x_f32 ? ((i / 4) * TPR + part) * 4 : ((i / 8) * TPR + part) * 8 + (i % 8);
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
  __syncthreads();

  // ---- 2. q, k, v of head h: block i = 3*rb + j (j = 0 q, 1 k, 2 v) on wave i % 16 ---------
  {
    const bf16x8* W = static_cast<const bf16x8*>(a.wqkv);
    for (int i = wave; i < 3 * nrb; i += NT / 64) {
      const int rb = i / 3, j = i % 3;
      const int cbg = j * a.n_heads + h;             // global 32-column block of the projection
      bf16x8 wf[KS], af[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) wf[ks] = W[((long long)cbg * KS + ks) * 64 + lane];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) af[ks] = a_frag(As, LDA, rb * 32, ks * 16, lane);
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
  __syncthreads();

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

}  // namespace

bool self_attention_fits(int d, int n_heads, int per) { return d == 128 && d / n_heads == 32 && per >= 1 && per <= 256; }

hipError_t launch_self_attention(const SelfAttnArgs& a, int d, hipStream_t s) {
  if (a.B <= 0) return hipSuccess;
  if (!self_attention_fits(d, a.n_heads, a.per)) return hipErrorInvalidValue;
  hipLaunchKernelGGL((k_self_attention<128, 32>), dim3((unsigned)(a.B * a.n_heads)), dim3(1024), 0, s, a);
  return hipGetLastError();
}
