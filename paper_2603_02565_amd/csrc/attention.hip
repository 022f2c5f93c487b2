// Multi-head scaled dot-product attention with a key padding mask and online softmax.
//
// fp32 models (k_attention): one wave owns 16 queries of one (batch, head); a workgroup holds
// WAVES waves that share the
// (batch, head) and walk the keys in blocks of 32.  For each block the wave computes the
// transposed score tile S^T = K Q^T with matrix-core instructions (keys are rows, so every lane
// ends up holding scores of ONE query), updates that query's running max / sum in fp32, and
// multiplies P^T into the transposed output O^T = V^T P^T.  Keeping everything transposed means
// the probabilities produced by one MFMA are already laid out as the B operand of the next, with
// no LDS round trip; only V is transposed through LDS.  The key rows fed to the two score MFMAs
// of a block are permuted so that lane group g holds keys 8g..8g+7 in order, which is exactly the
// k-slot order the P V^T product expects.
#include "fe_common.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;

template <typename T, int WAVES, int DH>
__global__ __launch_bounds__(WAVES * 64) void k_attention(AttnArgs a) {
  constexpr int VPAD = sizeof(T) == 2 ? 8 : 4;
  constexpr int VLD = 32 + VPAD;
  constexpr int NB = DH / 16;            // 16-row blocks of O^T
  __shared__ __attribute__((aligned(16))) T Vt[DH * VLD];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, q_in = lane & 15;
  // flattened grid: x = (query-tile group) + groups * (head + n_heads * batch)
  const int groups = (a.nq + WAVES * 16 - 1) / (WAVES * 16);
  const int qg = blockIdx.x % groups, bh = blockIdx.x / groups;
  const int h = bh % a.n_heads, b = bh / a.n_heads;
  int nq = a.nq, nk = a.nk;
  if (a.q_valid) nq = min(nq, a.q_valid[b]);
  if (a.k_valid) nk = min(nk, a.k_valid[b]);
  if (qg * WAVES * 16 >= nq || nk <= 0) return;   // uniform over the workgroup
  const int q0 = (qg * WAVES + wave) * 16;
  const bool active = q0 < nq;

  const T* Qb = static_cast<const T*>(a.Q) + b * a.q_bs + h * DH;
  const T* Kb = static_cast<const T*>(a.K) + b * a.k_bs + h * DH;
  const T* Vb = static_cast<const T*>(a.V) + b * a.v_bs + h * DH;
  const int qrow = q0 + q_in;
  const bool qok = active && qrow < nq;
  const float sl2 = a.scale * kLog2e;

  // Q^T as the B operand of S^T = K Q^T
  bf16x8 qf8[DH / 32];
  float qf1[DH / 4];
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
      qf8[c] = qok ? *reinterpret_cast<const bf16x8*>(Qb + (long long)qrow * a.q_rs + c * 32 + g * 8) : bf16x8{};
  } else {
#pragma unroll
    for (int s = 0; s < DH / 4; ++s) qf1[s] = qok ? (float)Qb[(long long)qrow * a.q_rs + s * 4 + g] : 0.f;
  }

  float m_run = -INFINITY, l_run = 0.f;
  f32x4 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kb = 0; kb < nk; kb += 32) {
    __syncthreads();
    // ---- V block -> LDS, transposed (zeros past the last valid key)
    constexpr int VEC = 16 / sizeof(T);
    for (int e = threadIdx.x; e < 32 * DH / VEC; e += WAVES * 64) {
      const int key = e / (DH / VEC), d0 = (e % (DH / VEC)) * VEC;
      T v[VEC];
      if (kb + key < nk) {
        *reinterpret_cast<uint4*>(v) = *reinterpret_cast<const uint4*>(Vb + (long long)(kb + key) * a.v_rs + d0);
      } else {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = from_f32<T>(0.f);
      }
#pragma unroll
      for (int i = 0; i < VEC; ++i) Vt[(d0 + i) * VLD + key] = v[i];
    }
    __syncthreads();
    if (!active) continue;

    // ---- S^T for keys kb + kappa_j(r), r = lane row of the A operand
    const int r = lane & 15;
    const int key0 = kb + (r >> 2) * 8 + (r & 3);
    const int key1 = key0 + 4;
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int c = 0; c < DH / 32; ++c) {
        const bf16x8 k0 = key0 < nk ? *reinterpret_cast<const bf16x8*>(Kb + (long long)key0 * a.k_rs + c * 32 + g * 8) : bf16x8{};
        const bf16x8 k1 = key1 < nk ? *reinterpret_cast<const bf16x8*>(Kb + (long long)key1 * a.k_rs + c * 32 + g * 8) : bf16x8{};
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qf8[c], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qf8[c], s1, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int s = 0; s < DH / 4; ++s) {
        const float k0 = key0 < nk ? (float)Kb[(long long)key0 * a.k_rs + s * 4 + g] : 0.f;
        const float k1 = key1 < nk ? (float)Kb[(long long)key1 * a.k_rs + s * 4 + g] : 0.f;
        s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(k0, qf1[s], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(k1, qf1[s], s1, 0, 0, 0);
      }
    }
    // lane now holds scores of query q_in for keys kb + 8g + j, j = 0..7
    float p[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      p[j] = (kb + g * 8 + j < nk) ? s0[j] * sl2 : -INFINITY;
      p[4 + j] = (kb + g * 8 + 4 + j < nk) ? s1[j] * sl2 : -INFINITY;
    }
    float mx = p[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) mx = fmaxf(mx, p[j]);
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) { p[j] = exp2f(p[j] - m_new); psum += p[j]; }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < NB; ++i) o[i] *= alpha;

    // ---- O^T += V^T P^T
    if constexpr (sizeof(T) == 2) {
      bf16x8 pb;
#pragma unroll
      for (int j = 0; j < 8; ++j) pb[j] = (bf16)p[j];
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&Vt[(i * 16 + (lane & 15)) * VLD + g * 8]);
        o[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, o[i], 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int s = 0; s < 8; ++s) {
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          const float vf = Vt[(i * 16 + (lane & 15)) * VLD + g * 8 + s];
          o[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(vf, p[s], o[i], 0, 0, 0);
        }
      }
    }
  }
  if (!active) return;
  float l_tot = l_run + __shfl_xor(l_run, 16, 64);
  l_tot += __shfl_xor(l_tot, 32, 64);
  if (!qok) return;
  const float inv = 1.f / l_tot;
  T* Ob = static_cast<T*>(a.O) + b * a.o_bs + (long long)qrow * a.o_rs + h * DH;
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) Ob[i * 16 + g * 4 + j] = from_f32<T>(o[i][j] * inv);
}

// ------------------------------------------------------------------------------------------
// bf16 models: a workgroup owns one (batch, head) and up to WAVES*QT*16 queries.  Keys are
// walked in chunks of KC that the whole workgroup stages once in LDS (K row-major, V
// transposed) and every query tile of every wave consumes; the next chunk is fetched into
// registers while the current one is in use.  Per 32-key block the wave runs the same
// transposed score / probability / output scheme as above.
// ------------------------------------------------------------------------------------------
template <int DH, int WAVES, int QT, int KC>
__global__ __launch_bounds__(WAVES * 64, WAVES != 4 ? 1 : (DH == 64 && QT >= 2) || QT >= 8 ? 2 : 3) void k_attention_chunked(AttnArgs a) {
  constexpr int NT = WAVES * 64;
  constexpr int KLD = DH + 8, VLD = KC + 8, NB = DH / 16;
  constexpr int PER_T = KC * DH / 8 / NT;         // 16-byte vectors per thread per tensor
  static_assert(PER_T >= 1 && KC * DH / 8 % NT == 0, "chunk does not split over the workgroup");
  __shared__ __attribute__((aligned(16))) bf16 Ks[KC * KLD];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DH * VLD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, q_in = lane & 15;
  const int per_group = WAVES * QT * 16;
  const int groups = (a.nq + per_group - 1) / per_group;
  const int qg = blockIdx.x % groups, bh = blockIdx.x / groups;
  const int h = bh % a.n_heads, b = bh / a.n_heads;
  int nq = a.nq, nk = a.nk;
  if (a.q_valid) nq = min(nq, a.q_valid[b]);
  if (a.k_valid) nk = min(nk, a.k_valid[b]);
  if (qg * per_group >= nq || nk <= 0) return;     // uniform over the workgroup

  const bf16* Qb = static_cast<const bf16*>(a.Q) + b * a.q_bs + h * DH;
  const bf16* Kb = static_cast<const bf16*>(a.K) + b * a.k_bs + h * DH;
  const bf16* Vb = static_cast<const bf16*>(a.V) + b * a.v_bs + h * DH;
  const float sl2 = a.scale * kLog2e;

  // query tile t of this wave: rows q0(t) .. q0(t)+15
  auto q0_of = [&](int t) { return qg * per_group + (t * WAVES + wave) * 16; };
  bf16x8 qf[QT][DH / 32];
  float m_run[QT], l_run[QT];
  f32x4 o[QT][NB];
#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int qrow = q0_of(t) + q_in;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
      qf[t][c] = qrow < nq ? *reinterpret_cast<const bf16x8*>(Qb + (long long)qrow * a.q_rs + c * 32 + g * 8) : bf16x8{};
    m_run[t] = -INFINITY;
    l_run[t] = 0.f;
#pragma unroll
    for (int i = 0; i < NB; ++i) o[t][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  uint4 kreg[PER_T], vreg[PER_T];
  auto load_chunk = [&](int c0) {
#pragma unroll
    for (int p = 0; p < PER_T; ++p) {
      const int e = p * NT + tid, key = e / (DH / 8), d0 = (e % (DH / 8)) * 8;
      const bool ok = c0 + key < nk;
      kreg[p] = ok ? *reinterpret_cast<const uint4*>(Kb + (long long)(c0 + key) * a.k_rs + d0) : make_uint4(0, 0, 0, 0);
      vreg[p] = ok ? *reinterpret_cast<const uint4*>(Vb + (long long)(c0 + key) * a.v_rs + d0) : make_uint4(0, 0, 0, 0);
    }
  };
  load_chunk(0);

  for (int c0 = 0; c0 < nk; c0 += KC) {
    __syncthreads();                                  // the previous chunk is no longer read
#pragma unroll
    for (int p = 0; p < PER_T; ++p) {
      const int e = p * NT + tid, key = e / (DH / 8), d0 = (e % (DH / 8)) * 8;
      *reinterpret_cast<uint4*>(&Ks[key * KLD + d0]) = kreg[p];
      const bf16* v = reinterpret_cast<const bf16*>(&vreg[p]);
#pragma unroll
      for (int i = 0; i < 8; ++i) Vt[(d0 + i) * VLD + key] = v[i];
    }
    __syncthreads();
    if (c0 + KC < nk) load_chunk(c0 + KC);
    const int nkeys = min(KC, nk - c0);

    // 64 keys (two 32-key blocks) per online-softmax step at head width 32 with several query
    // tiles per wave, else 32 (head width 64: a tile's arithmetic is then the same whatever the
    // number of tiles per wave); every key and value fragment of a step is read from LDS once and
    // used by all QT query tiles of the wave.  Keys from nkeys on (zero rows in LDS, up to KC) are
    // masked.
    constexpr int NU = (KC >= 64 && QT >= 2 && DH == 32) ? 2 : 1;   // 32-key blocks per step
    static_assert(KC % (32 * NU) == 0, "whole steps per chunk");
    for (int kb = 0; kb < nkeys; kb += 32 * NU) {
      const int r = lane & 15;
      bf16x8 ka[NU][DH / 32], kc[NU][DH / 32], vf[NU][NB];
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        const int k0 = kb + 32 * u + (r >> 2) * 8 + (r & 3), k1 = k0 + 4;
#pragma unroll
        for (int c = 0; c < DH / 32; ++c) {
          ka[u][c] = *reinterpret_cast<const bf16x8*>(&Ks[k0 * KLD + c * 32 + g * 8]);
          kc[u][c] = *reinterpret_cast<const bf16x8*>(&Ks[k1 * KLD + c * 32 + g * 8]);
        }
#pragma unroll
        for (int i = 0; i < NB; ++i)
          vf[u][i] = *reinterpret_cast<const bf16x8*>(&Vt[(i * 16 + (lane & 15)) * VLD + kb + 32 * u + g * 8]);
      }
#pragma unroll
      for (int t = 0; t < QT; ++t) {
        if (q0_of(t) >= nq) continue;               // uniform
        float p[NU][8];
#pragma unroll
        for (int u = 0; u < NU; ++u) {
          f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < DH / 32; ++c) {
            s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[u][c], qf[t][c], s0, 0, 0, 0);
            s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc[u][c], qf[t][c], s1, 0, 0, 0);
          }
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            p[u][j] = s0[j] * sl2;
            p[u][4 + j] = s1[j] * sl2;
          }
        }
        if (kb + 32 * NU > nkeys) {                 // ragged last step (uniform branch)
#pragma unroll
          for (int u = 0; u < NU; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              if (kb + 32 * u + g * 8 + j >= nkeys) p[u][j] = -INFINITY;
              if (kb + 32 * u + g * 8 + 4 + j >= nkeys) p[u][4 + j] = -INFINITY;
            }
        }
        float mx = p[0][0];
#pragma unroll
        for (int u = 0; u < NU; ++u)
#pragma unroll
          for (int j = 0; j < 8; ++j) mx = fmaxf(mx, p[u][j]);
        mx = rows_max(mx);
        const float m_new = fmaxf(m_run[t], mx);   // finite: every step holds a valid key
        const float alpha = __builtin_amdgcn_exp2f(m_run[t] - m_new);   // v_exp_f32; exp2(-inf) = 0
        float psum = 0.f;
        bf16x8 pb[NU];
#pragma unroll
        for (int u = 0; u < NU; ++u)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const float e = __builtin_amdgcn_exp2f(p[u][j] - m_new);
            psum += e;
            pb[u][j] = (bf16)e;
          }
        l_run[t] = l_run[t] * alpha + psum;
        m_run[t] = m_new;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
          o[t][i] *= alpha;
#pragma unroll
          for (int u = 0; u < NU; ++u) o[t][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[u][i], pb[u], o[t][i], 0, 0, 0);
        }
      }
    }
  }

#pragma unroll
  for (int t = 0; t < QT; ++t) {
    const int qrow = q0_of(t) + q_in;
    if (q0_of(t) >= nq) continue;
    const float l_tot = rows_sum(l_run[t]);
    if (qrow >= nq) continue;
    const float inv = __builtin_amdgcn_rcpf(l_tot);   // v_rcp_f32
    bf16* Ob = static_cast<bf16*>(a.O) + b * a.o_bs + (long long)qrow * a.o_rs + h * DH;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = (bf16)(o[t][i][j] * inv);
      *reinterpret_cast<bf16x4*>(Ob + i * 16 + g * 4) = w;
    }
  }
}

// ------------------------------------------------------------------------------------------
// bf16 models, at most 32*NB32 keys per (batch, head): every key is resident in LDS at once, so
// each 16-query tile takes one softmax over its whole score row (scores of all key blocks held
// in registers) instead of a running rescale.  One workgroup of WAVES waves owns a (batch, head)
// and all its queries (at most 16*WAVES; query tile t on wave t), so its keys are read from
// memory once; they
// are staged behind a single barrier (K row-major, V transposed, rows past nk zero-filled up to
// the next multiple of 32).  Score and output blocks use the same transposed 16x16x32 layout as
// the chunked kernel; the softmax scale is folded into the exponent (exp2(s*c - max(s)*c) with
// c = scale*log2(e) > 0, one FMA per score).
// ------------------------------------------------------------------------------------------
template <int DH, int WAVES, int NB32>
__global__ __launch_bounds__(WAVES * 64) void k_attention_rows(AttnArgs a) {
  constexpr int NT = WAVES * 64, NK = NB32 * 32;
  constexpr int KLD = DH + 8, VLD = NK + 8, NB = DH / 16;
  constexpr int NV = NK * DH / 8;                  // 16-byte vectors per tensor
  constexpr int PER_T = (NV + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) bf16 Ks[NK * KLD];
  __shared__ __attribute__((aligned(16))) bf16 Vt[DH * VLD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, r = lane & 15;
  const int bh = xcd_tile(blockIdx.x, gridDim.x), h = bh % a.n_heads, b = bh / a.n_heads;
  int nq = a.nq, nk = a.nk;
  if (a.q_valid) nq = min(nq, a.q_valid[b]);
  if (a.k_valid) nk = min(nk, a.k_valid[b]);
  if (nq <= 0 || nk <= 0) return;                  // uniform over the workgroup
  const int nb32 = (nk + 31) / 32;

  const bf16* Qb = static_cast<const bf16*>(a.Q) + b * a.q_bs + h * DH;
  const bf16* Kb = static_cast<const bf16*>(a.K) + b * a.k_bs + h * DH;
  const bf16* Vb = static_cast<const bf16*>(a.V) + b * a.v_bs + h * DH;
  const float c2 = a.scale * kLog2e;

  {
    uint4 kr[PER_T], vr[PER_T];
#pragma unroll
    for (int p = 0; p < PER_T; ++p) {
      const int e = p * NT + tid, key = e / (DH / 8), d0 = (e % (DH / 8)) * 8;
      const bool ok = e < NV && key < nk;
      kr[p] = ok ? *reinterpret_cast<const uint4*>(Kb + (long long)key * a.k_rs + d0) : make_uint4(0, 0, 0, 0);
      vr[p] = ok ? *reinterpret_cast<const uint4*>(Vb + (long long)key * a.v_rs + d0) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int p = 0; p < PER_T; ++p) {
      const int e = p * NT + tid, key = e / (DH / 8), d0 = (e % (DH / 8)) * 8;
      if (e >= NV || key >= nb32 * 32) continue;     // never read
      *reinterpret_cast<uint4*>(&Ks[key * KLD + d0]) = kr[p];
      const bf16* v = reinterpret_cast<const bf16*>(&vr[p]);
#pragma unroll
      for (int i = 0; i < 8; ++i) Vt[(d0 + i) * VLD + key] = v[i];
    }
  }
  __syncthreads();

  {
    const int q0 = wave * 16, qrow = q0 + r;
    if (q0 >= nq) return;                            // uniform over the wave; no barrier follows
    bf16x8 qf[DH / 32];
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
      qf[c] = *reinterpret_cast<const bf16x8*>(Qb + (long long)(qrow < nq ? qrow : q0) * a.q_rs + c * 32 + g * 8);
    // raw scores: lane holds, for query r, keys 32*kb + 8*g + j (j < 8)
    float p[NB32][8];
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NB32; ++kb) {
      if (kb >= nb32) continue;                      // uniform
      const int k0 = kb * 32 + (r >> 2) * 8 + (r & 3), k1 = k0 + 4;
      f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < DH / 32; ++c) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(&Ks[k0 * KLD + c * 32 + g * 8]);
        const bf16x8 kc = *reinterpret_cast<const bf16x8*>(&Ks[k1 * KLD + c * 32 + g * 8]);
        s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[c], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kc, qf[c], s1, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        p[kb][j] = s0[j];
        p[kb][4 + j] = s1[j];
      }
      if (kb * 32 + 32 > nk) {                       // ragged last block (uniform)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (kb * 32 + g * 8 + j >= nk) p[kb][j] = -INFINITY;
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) mx = fmaxf(mx, p[kb][j]);
    }
    const float mc = rows_max(mx) * c2;              // finite: key 0 is always valid
    float l = 0.f;
    bf16x8 pb[NB32];
#pragma unroll
    for (int kb = 0; kb < NB32; ++kb) {
      if (kb >= nb32) continue;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float e = __builtin_amdgcn_exp2f(fmaf(p[kb][j], c2, -mc));   // v_exp_f32; exp2(-inf) = 0
        l += e;
        pb[kb][j] = (bf16)e;
      }
    }
    const float inv = __builtin_amdgcn_rcpf(rows_sum(l));   // v_rcp_f32
    f32x4 o[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) o[i] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < NB32; ++kb) {
      if (kb >= nb32) continue;
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const bf16x8 vf = *reinterpret_cast<const bf16x8*>(&Vt[(i * 16 + r) * VLD + kb * 32 + g * 8]);
        o[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb[kb], o[i], 0, 0, 0);
      }
    }
    if (qrow >= nq) return;
    bf16* Ob = static_cast<bf16*>(a.O) + b * a.o_bs + (long long)qrow * a.o_rs + h * DH;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      bf16x4 w;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[j] = (bf16)(o[i][j] * inv);
      *reinterpret_cast<bf16x4*>(Ob + i * 16 + g * 4) = w;
    }
  }
}

template <int DH, int WAVES>
hipError_t launch_rows(const AttnArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((k_attention_rows<DH, WAVES, 8>), dim3((unsigned)(a.n_heads * a.B)), dim3(WAVES * 64), 0, s, a);
  return hipGetLastError();
}

template <int DH, int WAVES, int QT, int KC>
hipError_t launch_chunked(const AttnArgs& a, hipStream_t s) {
  const long long groups = (a.nq + WAVES * QT * 16 - 1) / (WAVES * QT * 16);
  const long long n = groups * a.n_heads * a.B;
  hipLaunchKernelGGL((k_attention_chunked<DH, WAVES, QT, KC>), dim3((unsigned)n), dim3(WAVES * 64), 0, s, a);
  return hipGetLastError();
}

template <int DH>
hipError_t launch_bf16(const AttnArgs& a, hipStream_t s) {
  // all keys in LDS, one workgroup per (batch, head), one query tile per wave (up to 16 waves)
  if (a.nk <= 256 && a.nq > 16 && a.nq <= 256) {
    if (a.nq > 128) return launch_rows<DH, 16>(a, s);
    if (a.nq > 64) return launch_rows<DH, 8>(a, s);
    return launch_rows<DH, 4>(a, s);
  }
  if (a.nq <= 16) {
    // tiny groups (sequence encoder): one wave per (group, head)
    return a.nk <= 32 ? launch_chunked<DH, 1, 1, 32>(a, s) : launch_chunked<DH, 1, 1, 128>(a, s);
  }
  // as many queries per workgroup as still fill the chip, so K/V chunks are shared widely: eight
  // 32-dim query tiles per wave when that makes >= 512 workgroups (two per compute unit, by the
  // variant's registers), four when >= 1024 (three per compute unit), two when >= 512; two
  // 64-dim tiles when >= 512 (two per compute unit; four would not fit the register file)
  const long long bh = (long long)a.n_heads * a.B;
  auto wgs = [&](int qt) { return (a.nq + 64 * qt - 1) / (64 * qt) * bh; };
  if constexpr (DH == 32) {
    if (wgs(8) >= 512) return launch_chunked<DH, 4, 8, 128>(a, s);
    if (wgs(4) >= 1024) return launch_chunked<DH, 4, 4, 128>(a, s);
  }
  if (wgs(2) >= 512) return launch_chunked<DH, 4, 2, 128>(a, s);
  return launch_chunked<DH, 4, 1, 128>(a, s);
}

template <typename T, int DH>
hipError_t launch_t(const AttnArgs& a, hipStream_t s) {
  const int qt = (a.nq + 15) / 16;
  const long long bh = (long long)a.n_heads * a.B;
  if (qt >= 4) {
    hipLaunchKernelGGL((k_attention<T, 4, DH>), dim3((unsigned)(((qt + 3) / 4) * bh)), dim3(256), 0, s, a);
  } else if (qt >= 2) {
    hipLaunchKernelGGL((k_attention<T, 2, DH>), dim3((unsigned)(((qt + 1) / 2) * bh)), dim3(128), 0, s, a);
  } else {
    hipLaunchKernelGGL((k_attention<T, 1, DH>), dim3((unsigned)(qt * bh)), dim3(64), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, bool bf16_model, hipStream_t s) {
  if (a.B <= 0 || a.nq <= 0) return hipSuccess;
  if (bf16_model) return a.dh == 64 ? launch_bf16<64>(a, s) : launch_bf16<32>(a, s);
  return a.dh == 64 ? launch_t<float, 64>(a, s) : launch_t<float, 32>(a, s);
}
