// Internal declarations shared by the HIP kernels and the C-ABI layer of libflasheval.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define FE_DEV __device__ __forceinline__

FE_DEV float to_f32(float v) { return v; }
FE_DEV float to_f32(bf16 v) { return (float)v; }
template <typename T> FE_DEV T from_f32(float v);
template <> FE_DEV float from_f32<float>(float v) { return v; }
template <> FE_DEV bf16 from_f32<bf16>(float v) { return (bf16)v; }  // round to nearest even

// Butterflies across the four 16-lane rows of a wave on the gfx950 lane-swap instructions
// (VALU, no LDS round trip).  v_permlane16_swap / v_permlane32_swap applied to (v, v) return,
// in every lane l, the pair {v[l & ~16], v[l | 16]} resp. {v[l & ~32], v[l | 32]}; combining the
// pair gives the xor-16 / xor-32 butterfly, with the same operand order in both partner lanes.
FE_DEV float rows_max(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
FE_DEV float rows_sum(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Tile handled by this workgroup when the tile range is split into eight contiguous parts, one
// per XCD: workgroups are dispatched round-robin over the XCDs (workgroup i to XCD i % 8), so
// XCD x takes tiles x*q + min(x, r) ... of n = 8q + r tiles.  Kernels that walk the same
// batch-major row order then read, on each XCD, rows that the previous kernel wrote through
// that XCD's own L2.  A bijection on [0, n) for every n.
FE_DEV int xcd_tile(int i, int n) {
  const int q = n >> 3, r = n & 7, x = i & 7, y = i >> 3;
  return x * q + min(x, r) + y;
}

// Workgroup barrier for LDS traffic only: waits for this wave's LDS operations, then s_barrier.
// Unlike __syncthreads() it does not wait for outstanding vector-memory operations, so a load
// (or an LDS DMA) issued earlier stays in flight across it; data an LDS DMA writes becomes
// visible to other waves only after the issuing wave's vmem_wait() and a following barrier.
FE_DEV void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
FE_DEV void vmem_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// OR of `pred` over the workgroup of NW waves with an LDS-only barrier: unlike
// __syncthreads_or it neither reads the dispatch packet nor waits for outstanding vector-memory
// loads, so prefetches issued before it stay in flight.  LDS writes made before it are visible to
// the whole workgroup after it.
template <int NW>
FE_DEV bool block_any(int pred) {
  static_assert(NW >= 1 && NW <= 16, "at most 16 waves");
  __shared__ int s_wany[NW];
  const bool w = __any(pred);
  if ((threadIdx.x & 63) == 0) s_wany[threadIdx.x >> 6] = w;
  lds_barrier();
  int r = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) r |= s_wany[i];
  return r != 0;
}

FE_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
FE_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// ------------------------------------------------------------------------------------------
// Host-side launch descriptors (one per kernel family).
// ------------------------------------------------------------------------------------------

enum fe_epi { EPI_STORE = 0, EPI_RELU = 1, EPI_RESID = 2 };

// C = epi( pro(A) x W + bias ).  A is [R][K] with row stride lda (elements); pro(A) is the
// LayerNorm of each A row (over K) when ln_g != nullptr.  W is given transposed, Wt [N][K]
// (k contiguous).  Output column n of row r goes to
//   C + (n / col_block) * col_block_stride + r * ldc + (n % col_block).
// EPI_RESID: C is fp32 and receives res[r*ldr + n] + acc + bias (res may alias C).
// Rows r with (r % rows_per_batch) >= nvalid[r / rows_per_batch] are padding: tiles made
// only of padding are skipped and padding rows are not stored (nvalid == nullptr: all valid).
struct GemmArgs {
  const void* A; int lda; int a_f32;   // a_f32: A holds fp32 values, else act
  int R, K, N;
  const void* Wt;                      // act [N][K]
  const float* bias;                   // [N] or nullptr
  const float* ln_g; const float* ln_b;
  void* C; int ldc; int c_f32;         // c_f32: store fp32, else act
  int col_block; long long col_block_stride;
  int epi;
  const void* res; int ldr; int res_f32;
  const int32_t* nvalid; int rows_per_batch;
  int32_t* zero; int zero_n;           // bf16 projection: zero[0 .. zero_n) is cleared (or nullptr)
};

// O = softmax(Q K^T * scale) V per (batch, head).  Q rows of batch b start at
// Q + b*q_bs (row stride q_rs), likewise K, V, O.  nq/nk rows per batch; the optional
// nvalid[b] caps both the query rows computed and the keys attended (key padding mask).
struct AttnArgs {
  const void* Q; long long q_bs; int q_rs;
  const void* K; long long k_bs; int k_rs;
  const void* V; long long v_bs; int v_rs;
  void* O; long long o_bs; int o_rs;
  int B, nq, nk, n_heads, dh;
  const int32_t* q_valid;   // [B] or nullptr
  const int32_t* k_valid;   // [B] or nullptr
  float scale;
};

// Self-attention of a pre-LN block with the q|k|v projection inside (bf16 models, d = 128,
// head width 32, at most 256 rows per batch): for every batch b and head h,
//   O[b*per + r][h*32 ..] = softmax(q k^T * scale) v over the batch's valid rows,
//   q|k|v = LN1(X) Wqkv + bqkv restricted to head h.
// X is [B*per][d] (fp32 when x_f32, else act); rows r >= nvalid[b] are padding (O not written).
struct SelfAttnArgs {
  const void* X; int x_f32;
  int B, per; const int32_t* nvalid;
  const float *ln_g, *ln_b;
  const void* wqkv; const float* bqkv;
  void* O;
  int n_heads; float scale;
  // With lists != nullptr (the first item layer) the kernel also builds the distinct set of each
  // request from its KL list entries over elements 0..M-1 and reads its rows from `table`
  // (request b's element id at table + b*table_bs + id*D, activation type) instead of X; nvalid
  // and X are then unused.  The head-0 workgroup of request b writes uniq[b][0..per) (ascending,
  // -1 padded), n_uniq[b], slot[b][0..KL), status[b] and the gathered rows Xrows[b][0..per)
  // (zero rows from n_uniq[b] on); per = U_cap = min(M, KL).
  const int32_t* lists; int KL, M;
  const void* table; long long table_bs;
  int32_t *uniq, *n_uniq, *slot, *status;
  void* Xrows;
};
bool self_attention_fits(int d, int n_heads, int per);
hipError_t launch_self_attention(const SelfAttnArgs& a, int d, hipStream_t s);

// Second half of an item layer's attention (bf16 models, d = 128, head width 32, at most 256
// rows per batch and 256 context keys): for every batch b,
//   x1 = Xin + O Wo + bo, written to Xout (fp32) for the valid rows;
//   O2[b*per + r][h*32 ..] = softmax(q k^T * scale) v for every head h, with q = LN2(x1) Wq + bq
//   and k, v the head's columns of Kc, Vc [B][T][d] (act).
// O (act, all heads of the self-attention) and O2 must differ, and so must Xin and Xout: every
// head's workgroup reads the whole rows of O and Xin.
struct CrossAttnArgs {
  const void* O; const void* Xin; int xin_f32; void* Xout;
  int B, per; const int32_t* nvalid;
  const void* wo; const float* bo; const float *ln2g, *ln2b; const void* wq; const float* bq;
  const void* Kc; const void* Vc; int T;
  void* O2;
  int n_heads; float scale;
  int xout_bf16;                        // Xout is bf16 (else fp32)
};
bool cross_attention_fits(int d, int n_heads, int per, int T);
hipError_t launch_cross_attention(const CrossAttnArgs& a, int d, hipStream_t s);

// Tail of a block after attention (bf16 models): x1 = Xin + O Wo + bo, then
//   tail 0: Xout = x1 + FFN(LN2(x1)); with Hout != nullptr also Hout = LayerNorm(x1 + FFN)
//           with gains lnfg, offsets lnfb (bf16), padding rows of Hout below R set to zero
//           (Xout may then be nullptr); with kv != nullptr the key/value projections of the
//           same LayerNorm (see the fields below);
//   tail 1: Xout = x1 and Qout = LN2(x1) Wq + bq (bf16).
// Xout is fp32, or bf16 with xout_bf16 (the residual stream between kernels).
// Rows with (r % rows_per_batch) >= nvalid[r / rows_per_batch] are padding.
struct PostArgs {
  const void* O; const void* Xin; int xin_f32; void* Xout;
  int R, rows_per_batch; const int32_t* nvalid;
  int D, F, tail;
  const void* wo; const float* bo; const float *ln2g, *ln2b;
  const void* w1; const float* b1; const void* w2; const float* b2;
  const void* wq; const float* bq; void* Qout;
  const float *lnfg, *lnfb; void* Hout;
  // tail 0, last context block: with kv != nullptr, for l < kv_layers
  //   kv[(2l + j) * R * D + r * D + c] = (LayerNorm(x1 + FFN) Wkv + bkv)[r][(2l + j) * D + c]
  //   (LayerNorm with lnfg, lnfb; Wkv [D][2 * kv_layers * D] in packed fragment order, bf16 out)
  const void* wkv; const float* bkv; void* kv; int kv_layers;
  int32_t* zero; int zero_n;            // zero[0 .. zero_n) is cleared (or nullptr)
  int xout_bf16;                        // Xout is bf16 (else fp32)
  // tail 0 without kv: scratch of part_bytes bytes (16-byte aligned) that lets a launch with few
  // row tiles split the FFN's hidden width over several workgroups per tile (fp32 partial sums
  // [parts][R][D], added in a fixed order by a second kernel); nullptr: one workgroup per tile
  void* part; size_t part_bytes;
};

// Device pointers of one pre-LN encoder block (matrices of bf16 models in packed fragment order).
struct EncW {
  const float *ln1g, *ln1b; const void* wqkv; const float* bqkv;
  const void* wo; const float* bo;
  const float *ln2g, *ln2b; const void* w1; const float* b1; const void* w2; const float* b2;
};
constexpr int FE_MAX_LAYERS = 8;
constexpr int FE_MAX_OBJECTIVES = 8;   // task heads of fe_score_objectives

// A whole encoder module over short groups (bf16 models): n_layers pre-LN blocks over groups of
// S consecutive rows (attention inside a group), then the module's final LayerNorm.  Y receives
// in fp32 the final LayerNorm of every row (first_row_only = 0, Y [n_groups*S][D]) or of the
// first row of each group (first_row_only = 1, Y [n_groups][D]).
struct ModuleArgs {
  const void* Xin; int xin_f32;
  float* Y; int first_row_only;
  int n_groups, S, gpt;        // gpt: groups per tile (set by the launcher)
  int D, H, F, n_layers; float scale;
  const float *lnfg, *lnfb;
  EncW layer[FE_MAX_LAYERS];
};

int module_small_tile_rows(int d);
hipError_t launch_module_small(ModuleArgs a, hipStream_t s);
hipError_t launch_post(const PostArgs& a, hipStream_t s);
// workgroups per row tile of a tail launch of R rows whose FFN is split by hidden width, and the
// bytes of the fp32 partial sums it needs in PostArgs::part (0 when it is not split)
int post_split_parts(long long R, int D, int F);
size_t post_part_bytes(long long R, int D, int F);
hipError_t launch_gemm(const GemmArgs& a, bool bf16_model, hipStream_t s);   // fp32 models
hipError_t launch_proj(const GemmArgs& a, hipStream_t s);                    // bf16 models, K = d
// bf16 models with d >= 256: 128 x 128 tiles, LDS-staged operands; A bf16 without LayerNorm
// (ln_g == nullptr), K a multiple of 64, N of 128.
bool gemm_tiled_fits(int K, int N);
hipError_t launch_gemm_tiled(const GemmArgs& a, hipStream_t s);
hipError_t launch_attention(const AttnArgs& a, bool bf16_model, hipStream_t s);
hipError_t launch_layernorm(const void* X, int x_f32, long long x_rs, int R, int d, const float* g,
                            const float* b, void* Y, int y_f32, long long y_rs, bool bf16_model,
                            hipStream_t s);
hipError_t launch_layernorm_masked(const void* X, int x_f32, long long x_rs, int R, int d, const float* g,
                                   const float* b, void* Y, int y_f32, long long y_rs, const int32_t* nvalid,
                                   int rpb, bool bf16_model, hipStream_t s);
// Linear attention (phi = elu + 1).  State of keys K and values V (act) per (batch, head):
// St [B][H][dh + 1][dh] fp32 (rows 0..dh-1: sum_t phi(k_t) v_t^T, row dh: sum_t phi(k_t)); key row t
// of batch b at K + b*bs + t*rs + h*dh elements (V likewise), keys t < nvalid[b] (or nk).
hipError_t launch_lin_state(const void* K, const void* V, long long bs, int rs, int B, int nk, const int32_t* nvalid,
                            int H, int dh, float* St, bool bf16_model, hipStream_t s,
                            float* part = nullptr);
// Key splits launch_lin_state uses for BH (batch, head) states over nk keys when given a partial
// buffer `part` of BH * splits * (dh + 1) * dh floats (bf16 models; 1 = no split, no buffer used).
int lin_state_splits(int BH, int nk, bool bf16_model);
// O[b*rpb + r][h*dh + j] = (phi(q) S)_j / (phi(q) . z) for q = Q[b*rpb + r][h*dh ..], rows r < rpb
// and r < nvalid[b] (others untouched); row strides q_rs, o_rs (elements, 16-byte multiples).
hipError_t launch_lin_apply(const void* Q, int q_rs, const float* St, int B, int rpb, const int32_t* nvalid, int H,
                            int dh, void* O, int o_rs, bool bf16_model, hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int n, int32_t v, hipStream_t s);
// dst block b*reps + r = src block b (r < reps); block_bytes a multiple of 4
hipError_t launch_repeat_blocks(const void* src, void* dst, long long block_bytes, int nblk, int reps, hipStream_t s);
// slot_k[q][j] = slot_all[q][q % K][j] (q < BK; slot_all [BK][K][L], slot_k [BK][L])
hipError_t launch_take_list_slots(const int32_t* slot_all, int32_t* slot_k, int BK, int K, int L, hipStream_t s);
hipError_t launch_dedup(const int32_t* lists, int B, int KL, int M, int U_cap, int32_t* uniq,
                        int32_t* n_uniq, int32_t* slot, int32_t* status, hipStream_t s);
// U(z) and the element rows in one launch (one workgroup per request), when
// dedup_gather_fits: out [B][U_cap][d] as launch_gather_rows with idx = uniq, nvalid = n_uniq.
bool dedup_gather_fits(int U_cap, int d, bool bf16_model);
hipError_t launch_dedup_gather(const int32_t* lists, int B, int KL, int M, int U_cap, int32_t* uniq, int32_t* n_uniq,
                               int32_t* slot, int32_t* status, const void* table, long long table_bs, int d,
                               void* out, bool bf16_model, hipStream_t s);
hipError_t launch_gather_rows(const void* table, long long table_bs, int n_rows_table, const int32_t* idx,
                              int idx_bs, const int32_t* nvalid, int B, int rows, int d, void* out,
                              int32_t* status, int status_bit, bool bf16_model, hipStream_t s);
hipError_t launch_assemble(const int32_t* slot, const void* H, int B, int K, int L, int U_cap, int d,
                           const void* cls, const void* pos, void* seq, bool bf16_model, hipStream_t s);
hipError_t launch_score_objectives(const float* Cp, int B, int K, int d, int nobj, const float* W, const float* bias,
                                   const float* alpha, float* obj, float* fused, int32_t* best, hipStream_t s);
hipError_t launch_score_select(const float* Cp, int B, int K, int d, const float* w, const float* bias,
                               float* scores, int32_t* best, hipStream_t s);
