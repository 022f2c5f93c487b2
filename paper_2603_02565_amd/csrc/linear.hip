// Linear (kernelized) attention, the attention the paper's deployment serves both evaluators with
// (Appendix B.3): for a query q and keys k_t with values v_t of one head,
//   out = sum_t (phi(q) . phi(k_t)) v_t / sum_t phi(q) . phi(k_t),   phi(x) = elu(x) + 1,
// with no scale.  By associativity the keys and values of a head fold into a fixed-size state
//   S = sum_t phi(k_t) v_t^T  (dh x dh),   z = sum_t phi(k_t)  (dh),
// and a query attends as (phi(q)^T S) / (phi(q) . z).  That state is the variant's key/value
// cache: computed once per request, it replaces the T x d keys and values of the context.
//
// k_lin_state: the state of every (batch, head), fp32, laid out [B][H][dh + 1][dh] (rows 0..dh-1
//   = S with row i for feature i of phi(k), row dh = z).  bf16 models form S on
//   v_mfma_f32_32x32x16_bf16 from phi(k) and v rounded to bf16 (fp32 accumulation); z and fp32
//   models use fp32 VALU sums.  Every sum runs in a fixed order, so results are reproducible.
// k_lin_apply: the attention output of every valid query row from the state, fp32 arithmetic.
#include <algorithm>

#include "fe_common.h"

namespace {

constexpr float kLog2e = 1.4426950408889634f;

FE_DEV float phi(float x) { return x > 0.f ? x + 1.f : __builtin_amdgcn_exp2f(x * kLog2e); }   // v_exp_f32

// LDS traffic of one wave that its own lanes exchange: wait for the wave's LDS operations and
// keep the compiler from moving memory operations across.
FE_DEV void wave_lds_sync() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// ------------------------------------------------------------------------------------------
// State, bf16 models.  One workgroup (four waves) per (batch, head, key split): split sp of
// nsplit takes the 64-key chunks [sp * cps, (sp + 1) * cps), cps = ceil(chunks / nsplit), and wave w
// of it every fourth of them, starting at the w-th; per chunk every lane loads its share of the keys and values (16-byte
// vectors, the next chunk's loads in flight while the current one is used), forms phi(k) in
// fp32 (accumulating its part of z), and writes phi(k)^T and v^T (bf16) into the wave's LDS
// area, from which the MFMA operands are read: S[i][j] += sum over 16 keys of
// phi(k)^T[i][t] v^T[j][t].  The four waves' partial sums meet in LDS at the end, added in
// wave order.  With nsplit > 1 each split writes its partial state to its own slot of St
// ([B][H][nsplit][dh + 1][dh]) and k_lin_merge adds the splits in order.
// ------------------------------------------------------------------------------------------
template <int DH>
__global__ __launch_bounds__(256) void k_lin_state_bf16(const bf16* __restrict__ K, const bf16* __restrict__ V,
                                                        long long bs, int rs, int nk, const int32_t* __restrict__ nvalid,
                                                        int H, int nsplit, float* __restrict__ St) {
  constexpr int CH = 64, LDT = CH + 8, VPR = DH / 8, NV = CH * VPR / 64, NB = DH / 32;
  constexpr int AREA = 2 * DH * LDT;                       // bf16 elements per wave: phi(k)^T | v^T
  constexpr int RED = 4 * DH * DH;                         // floats of the cross-wave reduction
  constexpr int BYTES = (4 * AREA * 2 > RED * 4) ? 4 * AREA * 2 : RED * 4;
  __shared__ __attribute__((aligned(16))) char smem[BYTES];
  __shared__ float s_z[4][DH];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int id = xcd_tile(blockIdx.x, gridDim.x), bh = id / nsplit, sp = id % nsplit, b = bh / H, h = bh % H;
  const int n = nvalid ? min(nk, nvalid[b]) : nk;
  bf16* fkT = reinterpret_cast<bf16*>(smem) + wave * AREA;   // [DH][LDT]
  bf16* vT = fkT + DH * LDT;                                  // [DH][LDT]
  const bf16* Kb = K + b * bs + h * DH;
  const bf16* Vb = V + b * bs + h * DH;
  // lane's vectors: p-th is vector lane + 64 p of the chunk -> key (lane + 64 p) / VPR, columns
  // 8 * (lane % VPR) .. +7 (the same columns for every p, since 64 is a multiple of VPR)
  const int c8 = (lane % VPR) * 8;
  float zacc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  f32x16 acc[NB][NB];
#pragma unroll
  for (int ib = 0; ib < NB; ++ib)
#pragma unroll
    for (int jb = 0; jb < NB; ++jb) acc[ib][jb] = f32x16{};
  const int nall = (n + CH - 1) / CH, cps = (nall + nsplit - 1) / nsplit;
  const int ch0 = min(nall, sp * cps), nch = min(nall, ch0 + cps);   // this split's chunks [ch0, nch)
  bf16x8 kr[NV], vr[NV];
  auto load = [&](int ch) {
#pragma unroll
    for (int p = 0; p < NV; ++p) {
      const int t = ch * CH + (lane + 64 * p) / VPR;
      kr[p] = bf16x8{};
      vr[p] = bf16x8{};
      if (t < n) {
        kr[p] = *reinterpret_cast<const bf16x8*>(Kb + (long long)t * rs + c8);
        vr[p] = *reinterpret_cast<const bf16x8*>(Vb + (long long)t * rs + c8);
      }
    }
  };
  if (ch0 + wave < nch) load(ch0 + wave);
  for (int ch = ch0 + wave; ch < nch; ch += 4) {
    // phi(k) and v of this chunk -> transposed LDS operands; keys past n are zero rows
#pragma unroll
    for (int p = 0; p < NV; ++p) {
      const int tl = (lane + 64 * p) / VPR, t = ch * CH + tl;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f = t < n ? phi((float)kr[p][e]) : 0.f;
        zacc[e] += f;
        fkT[(c8 + e) * LDT + tl] = (bf16)f;
        vT[(c8 + e) * LDT + tl] = vr[p][e];
      }
    }
    if (ch + 4 < nch) load(ch + 4);
    wave_lds_sync();   // this wave's operand writes are complete before its lanes read them
#pragma unroll
    for (int s = 0; s < CH / 16; ++s) {
      bf16x8 a[NB], bb[NB];
#pragma unroll
      for (int ib = 0; ib < NB; ++ib) {
        a[ib] = *reinterpret_cast<const bf16x8*>(&fkT[(ib * 32 + (lane & 31)) * LDT + 16 * s + 8 * (lane >> 5)]);
        bb[ib] = *reinterpret_cast<const bf16x8*>(&vT[(ib * 32 + (lane & 31)) * LDT + 16 * s + 8 * (lane >> 5)]);
      }
#pragma unroll
      for (int ib = 0; ib < NB; ++ib)
#pragma unroll
        for (int jb = 0; jb < NB; ++jb) acc[ib][jb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[ib], bb[jb], acc[ib][jb], 0, 0, 0);
    }
    wave_lds_sync();   // operand reads are done before the next chunk overwrites them
  }
  // z: lanes with equal lane % VPR hold the same columns; butterfly over the others
#pragma unroll
  for (int e = 0; e < 8; ++e)
#pragma unroll
    for (int o = VPR; o < 64; o <<= 1) zacc[e] += __shfl_xor(zacc[e], o, 64);
  if (lane < VPR)
#pragma unroll
    for (int e = 0; e < 8; ++e) s_z[wave][c8 + e] = zacc[e];
  __syncthreads();   // every wave is past its last LDS operand read: the area becomes the reduction buffer
  float* red = reinterpret_cast<float*>(smem);           // [4][DH][DH]
  // lane holds S[ib*32 + 8q + 4(lane/32) + e][jb*32 + lane%32] in acc[ib][jb][4q + e]
#pragma unroll
  for (int ib = 0; ib < NB; ++ib)
#pragma unroll
    for (int jb = 0; jb < NB; ++jb)
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int i = ib * 32 + 8 * q + 4 * (lane >> 5) + e, j = jb * 32 + (lane & 31);
          red[(wave * DH + i) * DH + j] = acc[ib][jb][4 * q + e];
        }
  __syncthreads();
  float* out = St + ((long long)bh * nsplit + sp) * (DH + 1) * DH;
  for (int x = threadIdx.x; x < DH * DH; x += 256)
    out[x] = ((red[x] + red[DH * DH + x]) + red[2 * DH * DH + x]) + red[3 * DH * DH + x];
  if (threadIdx.x < DH) {
    const int j = threadIdx.x;
    out[DH * DH + j] = ((s_z[0][j] + s_z[1][j]) + s_z[2][j]) + s_z[3][j];
  }
}

// State, fp32 models (small shapes): thread x of the (batch, head) workgroup forms entries
// x, x + 256, ... of the (dh + 1) x dh state, each as one sequential sum over the keys.
__global__ __launch_bounds__(256) void k_lin_state_f32(const float* __restrict__ K, const float* __restrict__ V,
                                                       long long bs, int rs, int nk, const int32_t* __restrict__ nvalid,
                                                       int H, int dh, float* __restrict__ St) {
  const int bh = xcd_tile(blockIdx.x, gridDim.x), b = bh / H, h = bh % H;
  const int n = nvalid ? min(nk, nvalid[b]) : nk;
  const float* Kb = K + b * bs + h * dh;
  const float* Vb = V + b * bs + h * dh;
  float* out = St + (long long)bh * (dh + 1) * dh;
  for (int x = threadIdx.x; x < (dh + 1) * dh; x += 256) {
    const int i = x / dh, j = x % dh;
    float s = 0.f;
    if (i < dh) {
      for (int t = 0; t < n; ++t) s += phi(Kb[(long long)t * rs + i]) * Vb[(long long)t * rs + j];
    } else {
      for (int t = 0; t < n; ++t) s += phi(Kb[(long long)t * rs + j]);
    }
    out[x] = s;
  }
}

// The splits' partial states added in split order: St[bh][x] = sum_sp part[bh][sp][x].
__global__ __launch_bounds__(256) void k_lin_merge(const float* __restrict__ part, int nsplit, long long per_bh,
                                                  long long total, float* __restrict__ St) {
  for (long long i = blockIdx.x * 256ll + threadIdx.x; i < total; i += (long long)gridDim.x * 256) {
    const long long bh = i / per_bh, x = i - bh * per_bh;
    const float* p = part + bh * nsplit * per_bh + x;
    // eight loads in flight at a time; the sum still runs in split order
    float s = 0.f;
    for (int sp0 = 0; sp0 < nsplit; sp0 += 8) {
      float t[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = sp0 + u < nsplit ? p[(long long)(sp0 + u) * per_bh] : 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (sp0 + u < nsplit) s = sp0 + u == 0 ? t[u] : s + t[u];
    }
    St[i] = s;
  }
}

// ------------------------------------------------------------------------------------------
// Apply: one workgroup per (batch, head, tile of RPB query rows), the batch's state of that head
// staged in LDS (fp32).  Thread: one query row, output columns 8c .. 8c + 7 of the head; it
// forms phi(q) of the row in fp32, then out_j = sum_i phi(q)_i S[i][j] / sum_i phi(q)_i z_i.
// Rows r >= rpb or r >= nvalid[b] are not written.
// ------------------------------------------------------------------------------------------
template <typename T, int DH>
__global__ __launch_bounds__(256) void k_lin_apply(const T* __restrict__ Q, int q_rs, const float* __restrict__ St,
                                                   int rpb, const int32_t* __restrict__ nvalid, int H, int tiles,
                                                   T* __restrict__ O, int o_rs) {
  constexpr int TPR = DH / 8, RPB = 256 / TPR;
  __shared__ __attribute__((aligned(16))) float s_st[(DH + 1) * DH];
  const int id = xcd_tile(blockIdx.x, gridDim.x);
  const int tile = id % tiles, bh = id / tiles, h = bh % H, b = bh / H;
  // the query row (any row below rpb: its address needs no valid count), the valid count and the
  // state are all requested before the first of them is used
  const int r = tile * RPB + threadIdx.x / TPR, c = (threadIdx.x % TPR) * 8;
  const T* qrow = Q + ((long long)b * rpb + (r < rpb ? r : 0)) * q_rs + h * DH;
  constexpr int QV = DH * (int)sizeof(T) / 16;               // 16-byte vectors of the row
  uint4 qv[QV];
#pragma unroll
  for (int i = 0; i < QV; ++i) qv[i] = reinterpret_cast<const uint4*>(qrow)[i];
  const int n = nvalid ? min(rpb, nvalid[b]) : rpb;
  const float* src = St + (long long)bh * (DH + 1) * DH;
  for (int x = threadIdx.x; x < (DH + 1) * DH / 4; x += 256)
    reinterpret_cast<float4*>(s_st)[x] = reinterpret_cast<const float4*>(src)[x];
  const bool live = r < n;
  float fq[DH];
#pragma unroll
  for (int i = 0; i < QV; ++i) {
    const T* e = reinterpret_cast<const T*>(&qv[i]);
#pragma unroll
    for (int k = 0; k < 16 / (int)sizeof(T); ++k) fq[i * (16 / (int)sizeof(T)) + k] = phi(to_f32(e[k]));
  }
  __syncthreads();
  if (!live) return;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
#pragma unroll
  for (int i = 0; i < DH; ++i) {
    const float4 s0 = *reinterpret_cast<const float4*>(&s_st[i * DH + c]);
    const float4 s1 = *reinterpret_cast<const float4*>(&s_st[i * DH + c + 4]);
    acc[0] = fmaf(fq[i], s0.x, acc[0]);
    acc[1] = fmaf(fq[i], s0.y, acc[1]);
    acc[2] = fmaf(fq[i], s0.z, acc[2]);
    acc[3] = fmaf(fq[i], s0.w, acc[3]);
    acc[4] = fmaf(fq[i], s1.x, acc[4]);
    acc[5] = fmaf(fq[i], s1.y, acc[5]);
    acc[6] = fmaf(fq[i], s1.z, acc[6]);
    acc[7] = fmaf(fq[i], s1.w, acc[7]);
    den = fmaf(fq[i], s_st[DH * DH + i], den);
  }
  const float inv = 1.f / den;
  T res[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) res[k] = from_f32<T>(acc[k] * inv);
  T* orow = O + ((long long)b * rpb + r) * o_rs + h * DH + c;
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<uint4*>(orow) = *reinterpret_cast<const uint4*>(res);
  } else {
    reinterpret_cast<uint4*>(orow)[0] = reinterpret_cast<const uint4*>(res)[0];
    reinterpret_cast<uint4*>(orow)[1] = reinterpret_cast<const uint4*>(res)[1];
  }
}

template <typename T, int DH>
void apply_as(const void* Q, int q_rs, const float* St, int B, int rpb, const int32_t* nvalid, int H, void* O, int o_rs,
              hipStream_t s) {
  constexpr int RPB = 256 / (DH / 8);
  const int tiles = (rpb + RPB - 1) / RPB;
  hipLaunchKernelGGL((k_lin_apply<T, DH>), dim3(B * H * tiles), dim3(256), 0, s, static_cast<const T*>(Q), q_rs, St,
                     rpb, nvalid, H, tiles, static_cast<T*>(O), o_rs);
}

}  // namespace

int lin_state_splits(int BH, int nk, bool bf16_model) {
  if (!bf16_model || BH <= 0) return 1;
  // enough workgroups to fill the chip (about four per compute unit), at least one 64-key chunk
  // per wave of each split
  const int chunks = (nk + 63) / 64;
  const int want = (1024 + BH - 1) / BH, most = chunks / 4;
  return std::max(1, std::min(want, most));
}

hipError_t launch_lin_state(const void* K, const void* V, long long bs, int rs, int B, int nk, const int32_t* nvalid,
                            int H, int dh, float* St, bool bf16_model, hipStream_t s, float* part) {
  if (B <= 0 || nk <= 0) return hipSuccess;
  if (bf16_model) {
    if ((rs % 8) || (bs % 8)) return hipErrorInvalidValue;   // 16-byte row vectors
    const int ns = part ? lin_state_splits(B * H, nk, true) : 1;
    float* dst = ns > 1 ? part : St;
    const dim3 grid((unsigned)(B * H * ns));
    switch (dh) {
      case 32: hipLaunchKernelGGL(k_lin_state_bf16<32>, grid, dim3(256), 0, s, static_cast<const bf16*>(K),
                                  static_cast<const bf16*>(V), bs, rs, nk, nvalid, H, ns, dst); break;
      case 64: hipLaunchKernelGGL(k_lin_state_bf16<64>, grid, dim3(256), 0, s, static_cast<const bf16*>(K),
                                  static_cast<const bf16*>(V), bs, rs, nk, nvalid, H, ns, dst); break;
      default: return hipErrorInvalidValue;
    }
    if (ns > 1) {
      const long long per_bh = (long long)(dh + 1) * dh, total = (long long)B * H * per_bh;
      const int blocks = (int)std::min<long long>((total + 255) / 256, 4096);
      hipLaunchKernelGGL(k_lin_merge, dim3(blocks), dim3(256), 0, s, part, ns, per_bh, total, St);
    }
  } else {
    hipLaunchKernelGGL(k_lin_state_f32, dim3(B * H), dim3(256), 0, s, static_cast<const float*>(K),
                       static_cast<const float*>(V), bs, rs, nk, nvalid, H, dh, St);
  }
  return hipGetLastError();
}

hipError_t launch_lin_apply(const void* Q, int q_rs, const float* St, int B, int rpb, const int32_t* nvalid, int H,
                            int dh, void* O, int o_rs, bool bf16_model, hipStream_t s) {
  if (B <= 0 || rpb <= 0) return hipSuccess;
  const int esz = bf16_model ? 2 : 4;
  if ((q_rs * esz) % 16 || (o_rs * esz) % 16) return hipErrorInvalidValue;
  if (bf16_model) {
    if (dh == 32) apply_as<bf16, 32>(Q, q_rs, St, B, rpb, nvalid, H, O, o_rs, s);
    else if (dh == 64) apply_as<bf16, 64>(Q, q_rs, St, B, rpb, nvalid, H, O, o_rs, s);
    else return hipErrorInvalidValue;
  } else {
    if (dh == 32) apply_as<float, 32>(Q, q_rs, St, B, rpb, nvalid, H, O, o_rs, s);
    else if (dh == 64) apply_as<float, 64>(Q, q_rs, St, B, rpb, nvalid, H, O, o_rs, s);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}
