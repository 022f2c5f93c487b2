// C ABI of libflasheval: argument validation, weight packing, workspace layout and the launch
// sequence of each stage.  All device work is in the kernels of gemm.hip, attention.hip and
// index.hip; this file only enqueues them.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "fe_common.h"
#include "flasheval.h"
#include "flasheval_trace.h"

#include <mutex>

namespace {

thread_local std::string g_err;

// ------------------------------------------------------------------------------------------
// Kernel timing (flasheval_trace.h): events recorded around each launch while enabled.
// ------------------------------------------------------------------------------------------
enum Fam { F_GEMM = 0, F_ATTN, F_LN, F_DEDUP, F_GATHER, F_ASSEMBLE, F_SCORE, F_FILL, F_FFN, F_LAYER, F_POST, F_LIN };
const char* const kFamName[FE_TRACE_FAMILIES] = {"gemm", "attention", "layernorm", "dedup", "gather", "assemble",
                                                 "score_select", "fill", "ffn", "layer", "post", "linear"};
struct TraceRec { int fam; hipEvent_t a, b; };
std::mutex g_trace_mu;
bool g_trace_on = false;
std::vector<TraceRec> g_trace;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t take_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <class F>
hipError_t traced(int fam, hipStream_t s, F&& launch) {
  if (!g_trace_on) return launch();
  std::lock_guard<std::mutex> lk(g_trace_mu);
  hipEvent_t a = take_event(), b = take_event();
  if (!a || !b) return hipErrorOutOfMemory;
  hipError_t e = hipEventRecord(a, s);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(b, s);
  if (e != hipSuccess) return e;
  g_trace.push_back({fam, a, b});
  return hipSuccess;
}

#define FE_LAUNCH(fam, stream, call) FE_HIP(traced(fam, stream, [&] { return (call); }))

fe_status fail(fe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define FE_HIP(call)                                                                  \
  do {                                                                                \
    hipError_t e_ = (call);                                                           \
    if (e_ != hipSuccess) return fail(FE_EHIP, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)


struct ItemW {
  const float *ln1g, *ln1b;
  const void* wqkv;
  const float* bqkv;
  const void* wo;
  const float* bo;
  const float *ln2g, *ln2b;
  const void* wq;
  const float* bq;
  const void* wo2;
  const float* bo2;
  const float *ln3g, *ln3b;
  const void* w1;
  const float* b1;
  const void* w2;
  const float* b2;
};

}  // namespace

struct fe_model {
  fe_config cfg;
  bool bf16;
  int device;
  void* dev = nullptr;
  std::vector<EncW> ctx, seq, cross;
  std::vector<ItemW> item;
  const float *ctx_lnf_g, *ctx_lnf_b, *item_lnf_g, *item_lnf_b, *seq_lnf_g, *seq_lnf_b, *cross_lnf_g, *cross_lnf_b;
  const void* wkv;    // [2n*d][d]: rows of block (l, 0) = wk_l^T, block (l, 1) = wv_l^T
  const float* bkv;   // [2n*d]
  const void* cls;
  const void* pos;
  const float* head_w;
  const float* head_b;
  const void* emb;
};

namespace {

// ------------------------------------------------------------------------------------------
// Parameter walk shared by fe_param_count and fe_model_create (host side only).
// ------------------------------------------------------------------------------------------
struct Packer {
  const float* src = nullptr;  // null: count only
  size_t consumed = 0;
  bool bf16 = false;
  std::vector<unsigned char> image;

  size_t place(size_t bytes) {
    size_t off = (image.size() + 255) & ~size_t(255);
    image.resize(off + bytes);
    return off;
  }
  static uint16_t to_bf16(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
  }
  // fp32 vector of n values
  size_t vec(size_t n) {
    const float* p = src + consumed;
    consumed += n;
    if (!src) return 0;
    size_t off = place(n * 4);
    std::memcpy(&image[off], p, n * 4);
    return off;
  }
  // act-type copy of n values in source order
  size_t act(size_t n) {
    const float* p = src + consumed;
    consumed += n;
    if (!src) return 0;
    size_t off = place(n * (bf16 ? 2 : 4));
    if (bf16) {
      uint16_t* dst = reinterpret_cast<uint16_t*>(&image[off]);
      for (size_t i = 0; i < n; ++i) dst[i] = to_bf16(p[i]);
    } else {
      std::memcpy(&image[off], p, n * 4);
    }
    return off;
  }
  // matrix [in][out] -> device layout at byte offset `off`:
  //   fp32 models: transposed, Wt[out][in];
  //   bf16 models: the B-operand fragments of v_mfma_f32_32x32x16_bf16, so that one wave reads
  //   the operand of one instruction as 64 lanes x 16 contiguous bytes.  Block (nb, ks) holds
  //   output columns 32nb..32nb+31 and inputs 16ks..16ks+15; lane l of the block holds
  //   W[16ks + 8(l/32) + j][32nb + l%32] for j = 0..7.  Blocks are ordered nb-major, ks-minor.
  void mat_into(size_t off, size_t in, size_t out) {
    const float* p = src + consumed;
    consumed += in * out;
    if (!src) return;
    if (bf16) {
      uint16_t* dst = reinterpret_cast<uint16_t*>(&image[off]);
      const size_t ksteps = in / 16;
      for (size_t k = 0; k < in; ++k)
        for (size_t n = 0; n < out; ++n) {
          const size_t nb = n / 32, ks = k / 16, lane = ((k % 16) / 8) * 32 + n % 32, j = k % 8;
          dst[((nb * ksteps + ks) * 64 + lane) * 8 + j] = to_bf16(p[k * out + n]);
        }
    } else {
      for (size_t o = 0; o < out; ++o)
        for (size_t i = 0; i < in; ++i) reinterpret_cast<float*>(&image[off])[o * in + i] = p[i * out + o];
    }
  }
  size_t mat(size_t in, size_t out) {
    size_t off = src ? place(in * out * (bf16 ? 2 : 4)) : 0;
    mat_into(off, in, out);
    return off;
  }
  void vec_into(size_t off, size_t n) {
    const float* p = src + consumed;
    consumed += n;
    if (src) std::memcpy(&image[off], p, n * 4);
  }
};

struct EncOff { size_t ln1g, ln1b, wqkv, bqkv, wo, bo, ln2g, ln2b, w1, b1, w2, b2; };
struct ItemOff { size_t ln1g, ln1b, wqkv, bqkv, wo, bo, ln2g, ln2b, wq, bq, wo2, bo2, ln3g, ln3b, w1, b1, w2, b2; };
struct Offsets {
  std::vector<EncOff> ctx, seq, cross;
  std::vector<ItemOff> item;
  size_t ctx_lnf_g, ctx_lnf_b, item_lnf_g, item_lnf_b, seq_lnf_g, seq_lnf_b, cross_lnf_g, cross_lnf_b;
  size_t wkv, bkv, cls, pos, head_w, head_b, emb;
};

EncOff pack_enc(Packer& P, size_t d, size_t F) {
  EncOff o;
  o.ln1g = P.vec(d); o.ln1b = P.vec(d);
  o.wqkv = P.mat(d, 3 * d); o.bqkv = P.vec(3 * d);
  o.wo = P.mat(d, d); o.bo = P.vec(d);
  o.ln2g = P.vec(d); o.ln2b = P.vec(d);
  o.w1 = P.mat(d, F); o.b1 = P.vec(F);
  o.w2 = P.mat(F, d); o.b2 = P.vec(d);
  return o;
}

Offsets pack_all(Packer& P, const fe_config& c) {
  const size_t d = c.d, F = c.ffn_dim, n = c.n_layers;
  const size_t esz = P.bf16 ? 2 : 4;
  Offsets O;
  for (size_t l = 0; l < n; ++l) O.ctx.push_back(pack_enc(P, d, F));
  O.ctx_lnf_g = P.vec(d); O.ctx_lnf_b = P.vec(d);
  O.wkv = P.src ? P.place(2 * n * d * d * esz) : 0;
  O.bkv = P.src ? P.place(2 * n * d * 4) : 0;
  for (size_t l = 0; l < n; ++l) {
    P.mat_into(O.wkv + (2 * l) * d * d * esz, d, d);
    P.vec_into(O.bkv + (2 * l) * d * 4, d);
    P.mat_into(O.wkv + (2 * l + 1) * d * d * esz, d, d);
    P.vec_into(O.bkv + (2 * l + 1) * d * 4, d);
  }
  for (size_t l = 0; l < n; ++l) {
    ItemOff o;
    o.ln1g = P.vec(d); o.ln1b = P.vec(d);
    o.wqkv = P.mat(d, 3 * d); o.bqkv = P.vec(3 * d);
    o.wo = P.mat(d, d); o.bo = P.vec(d);
    o.ln2g = P.vec(d); o.ln2b = P.vec(d);
    o.wq = P.mat(d, d); o.bq = P.vec(d);
    o.wo2 = P.mat(d, d); o.bo2 = P.vec(d);
    o.ln3g = P.vec(d); o.ln3b = P.vec(d);
    o.w1 = P.mat(d, F); o.b1 = P.vec(F);
    o.w2 = P.mat(F, d); o.b2 = P.vec(d);
    O.item.push_back(o);
  }
  O.item_lnf_g = P.vec(d); O.item_lnf_b = P.vec(d);
  for (size_t l = 0; l < n; ++l) O.seq.push_back(pack_enc(P, d, F));
  O.seq_lnf_g = P.vec(d); O.seq_lnf_b = P.vec(d);
  for (size_t l = 0; l < n; ++l) O.cross.push_back(pack_enc(P, d, F));
  O.cross_lnf_g = P.vec(d); O.cross_lnf_b = P.vec(d);
  O.cls = P.act(d);
  O.pos = P.act((size_t)(c.max_L + 1) * d);
  O.head_w = P.vec(d);
  O.head_b = P.vec(1);
  O.emb = c.vocab > 0 ? P.act((size_t)c.vocab * d) : 0;
  return O;
}

fe_status check_config(const fe_config* c) {
  if (!c) return fail(FE_EINVAL, "config is NULL");
  if (c->dtype != FE_F32 && c->dtype != FE_BF16) return fail(FE_EINVAL, "dtype %d is not FE_F32 or FE_BF16", c->dtype);
  if (c->attention != FE_ATTN_SOFTMAX && c->attention != FE_ATTN_LINEAR)
    return fail(FE_EINVAL, "attention %d is not FE_ATTN_SOFTMAX or FE_ATTN_LINEAR", c->attention);
  if (c->d <= 0 || c->n_heads <= 0 || c->n_layers <= 0 || c->ffn_dim <= 0 || c->max_L <= 0 || c->vocab < 0)
    return fail(FE_EINVAL, "config sizes must be positive");
  if (c->d % c->n_heads) return fail(FE_EINVAL, "d=%d is not a multiple of n_heads=%d", c->d, c->n_heads);
  const int dh = c->d / c->n_heads;
  const bool bf = c->dtype == FE_BF16;
  if (!(c->d == 32 || c->d == 64 || c->d == 128 || c->d == 256 || c->d == 512))
    return fail(FE_EUNSUPPORTED, "d=%d not in {32,64,128,256,512}", c->d);
  if (dh != 32 && dh != 64) return fail(FE_EUNSUPPORTED, "head width %d not in {32,64}", dh);
  if (c->n_layers > 8) return fail(FE_EUNSUPPORTED, "n_layers=%d > 8", c->n_layers);
  if (bf && c->d < 128) return fail(FE_EUNSUPPORTED, "bf16 models need d >= 128");
  if (c->ffn_dim % (bf ? 128 : 32) || c->ffn_dim > 4096)
    return fail(FE_EUNSUPPORTED, "ffn_dim=%d must be a multiple of %d and <= 4096", c->ffn_dim, bf ? 128 : 32);
  if (c->max_L > 127) return fail(FE_EUNSUPPORTED, "max_L=%d > 127", c->max_L);
  if (c->vocab > 131072) return fail(FE_EUNSUPPORTED, "vocab=%d > 131072", c->vocab);
  return FE_OK;
}

// ------------------------------------------------------------------------------------------
// Workspace layout
// ------------------------------------------------------------------------------------------
// Wide bf16 models (d >= 512) run their projections and FFNs as tiled products over LDS-staged
// operands (gemm_tiled.hip), with LayerNorms as separate launches: there a row tile of the
// fused kernels would stream whole weight matrices through its compute unit.
constexpr int kWideD = 512;
bool wide(const fe_model* m) { return m->bf16 && m->cfg.d >= kWideD; }

struct Ws {
  size_t status;                                        // int32 [2][B]: items, context
  size_t lin_st;                                        // linear models: fp32 [B][H][dh+1][dh], one module's state
  size_t lin_part;                                      // linear models: the key splits' partial states
  size_t c_kvp;                                         // linear models: act [n][2][B][T][d] item-layer keys/values
  size_t c_xin, c_x, c_qkv, c_o, c_h, c_ln;             // context stage
  size_t i_g0, i_g, i_g1, i_qkv, i_o, i_q, i_h, i_ln;   // item stage
  size_t s_x, s_qkv, s_o, s_h, s_c, s_ln;               // sequence + cross stages
  size_t c_h_bytes, i_h_bytes, s_h_bytes;               // sizes of the FFN hidden buffers
  // *_ln: wide bf16 models only, bf16 [rows][d] LayerNorm outputs feeding the tiled products
  size_t total;
};

struct Bump {
  size_t at;
  size_t take(size_t bytes) {
    size_t off = (at + 255) & ~size_t(255);
    at = off + bytes;
    return off;
  }
};

Ws layout(const fe_model* m, long long B, long long T, long long M, long long K, long long L) {
  const long long d = m->cfg.d, F = m->cfg.ffn_dim;
  const size_t e = m->bf16 ? 2 : 4;
  Ws w{};
  Bump b0{0};
  w.status = b0.take(2 * B * 4);
  const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
  const long long H = m->cfg.n_heads, dh = d / H;
  if (lin) {
    w.lin_st = b0.take(B * H * (dh + 1) * dh * 4);
    const long long ns = std::max(lin_state_splits((int)(B * H), (int)T, m->bf16), lin_state_splits((int)(B * H), (int)K, m->bf16));
    w.lin_part = b0.take(B * H * ns * (dh + 1) * dh * 4);
  }
  size_t base = b0.at, end = base;
  {  // context
    const long long R = B * T;
    Bump b{base};
    if (lin) w.c_kvp = b.take(2 * m->cfg.n_layers * R * d * e);
    w.c_xin = b.take(R * d * e);
    w.c_x = b.take(R * d * 4);
    w.c_qkv = b.take(R * 3 * d * e);
    w.c_o = b.take(R * d * e);
    w.c_h_bytes = std::max((size_t)(R * F * e), post_part_bytes(R, (int)d, (int)F));
    w.c_h = b.take(w.c_h_bytes);
    if (wide(m)) w.c_ln = b.take(R * d * 2);
    end = std::max(end, b.at);
  }
  {  // items
    const long long Ucap = std::min(M, K * L);
    const long long R = B * Ucap;
    Bump b{base};
    w.i_g0 = b.take(R * d * e);
    w.i_g = b.take(R * d * 4);
    w.i_g1 = b.take(R * d * 4);
    w.i_qkv = b.take(R * 3 * d * e);
    w.i_o = b.take(R * d * e);
    w.i_q = b.take(R * d * e);
    w.i_h_bytes = std::max((size_t)(R * F * e), post_part_bytes(R, (int)d, (int)F));
    w.i_h = b.take(w.i_h_bytes);
    if (wide(m)) w.i_ln = b.take(R * d * 2);
    end = std::max(end, b.at);
  }
  {  // sequences (the cross module reuses these buffers; its rows B*K are fewer)
    const long long R = B * K * (L + 1);
    Bump b{base};
    w.s_x = b.take(R * d * 4);
    w.s_qkv = b.take(R * 3 * d * e);
    w.s_o = b.take(R * d * e);
    w.s_h_bytes = std::max({(size_t)(R * F * e), post_part_bytes(R, (int)d, (int)F), post_part_bytes(B * K, (int)d, (int)F)});
    w.s_h = b.take(w.s_h_bytes);
    w.s_c = b.take(B * K * d * 4);
    if (wide(m)) w.s_ln = b.take(R * d * 2);
    end = std::max(end, b.at);
  }
  w.total = (end + 255) & ~size_t(255);
  return w;
}

// Bytes of fe_encode_context's output: the keys and values of every item layer, [n][2][B][T][d]
// act; on linear-attention models their per-head state, [n][B][H][dh+1][dh] fp32.
size_t kv_bytes(const fe_model* m, long long B, long long T) {
  const long long d = m->cfg.d, n = m->cfg.n_layers, H = m->cfg.n_heads, dh = d / H;
  if (m->cfg.attention == FE_ATTN_LINEAR) return (size_t)(n * B * H * (dh + 1) * dh * 4);
  return (size_t)(n * 2 * B * T * d * (m->bf16 ? 2 : 4));
}

// Workspace of the candidate-factorised evaluator: the joint pass's workspace at B*K requests,
// then the per-list copies of the inputs, the per-list key/value caches, the per-list item
// encodings and the assembled sequences.
struct NaiveWs {
  size_t inner, inner_bytes, xin, kv, pool, lists, uniq, n_uniq, slot, H, slot_k, seq, total;
};

NaiveWs naive_layout(const fe_model* m, long long B, long long T, long long M, long long K, long long L, bool ids,
                     bool own_pool) {
  const long long BK = B * K, d = m->cfg.d, n = m->cfg.n_layers, Ucap = std::min(M, K * L);
  const size_t e = m->bf16 ? 2 : 4;
  NaiveWs w{};
  Bump b{0};
  w.inner_bytes = layout(m, BK, T, M, K, L).total;
  w.inner = b.take(w.inner_bytes);
  w.xin = b.take(ids ? BK * T * 4 : BK * T * d * e);
  w.kv = b.take(kv_bytes(m, BK, T));
  w.pool = own_pool ? b.take(BK * M * d * e) : 0;
  w.lists = b.take(BK * K * L * 4);
  w.uniq = b.take(BK * Ucap * 4);
  w.n_uniq = b.take(BK * 4);
  w.slot = b.take(BK * K * L * 4);
  w.H = b.take(BK * Ucap * d * e);
  w.slot_k = b.take(BK * L * 4);
  w.seq = b.take(B * K * (L + 1) * d * e);
  w.total = (b.at + 255) & ~size_t(255);
  return w;
}

template <typename T> T* at(void* base, size_t off) { return reinterpret_cast<T*>(static_cast<char*>(base) + off); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

fe_status check_dims(const fe_model* m, long long B, long long T, long long M, long long K, long long L) {
  if (!m) return fail(FE_EINVAL, "model is NULL");
  if (B < 1 || T < 1 || M < 1 || K < 1 || L < 1) return fail(FE_EINVAL, "B, T, M, K, L must be >= 1");
  if (L > m->cfg.max_L) return fail(FE_EINVAL, "L=%lld exceeds the model's max_L=%d", L, m->cfg.max_L);
  if (T > 8192) return fail(FE_EUNSUPPORTED, "T=%lld > 8192", T);
  if (K > 4096) return fail(FE_EUNSUPPORTED, "K=%lld > 4096", K);
  if (M > 131072) return fail(FE_EUNSUPPORTED, "M=%lld > 131072", M);
  const long long wide = std::max<long long>(3LL * m->cfg.d, m->cfg.ffn_dim);
  const long long rows = std::max({B * T, B * std::min(M, K * L), B * K * (L + 1)});
  if (rows * wide > INT_MAX || 2LL * m->cfg.n_layers * B * T * m->cfg.d > INT_MAX)
    return fail(FE_EINVAL, "batch too large: element counts overflow int32");
  return FE_OK;
}

// ------------------------------------------------------------------------------------------
// Blocks
// ------------------------------------------------------------------------------------------
GemmArgs gemm(const void* A, int lda, bool a_f32, int R, int K, int N, const void* Wt, const float* bias, void* C,
              int ldc, bool c_f32, int epi) {
  GemmArgs g{};
  g.A = A; g.lda = lda; g.a_f32 = a_f32;
  g.R = R; g.K = K; g.N = N;
  g.Wt = Wt; g.bias = bias;
  g.C = C; g.ldc = ldc; g.c_f32 = c_f32;
  g.col_block = N; g.col_block_stride = 0;
  g.epi = epi;
  g.rows_per_batch = 1;
  return g;
}

// One projection launch: packed-weight bf16 kernel or generic fp32 kernel.
// lnbuf: bf16 [R][K] scratch for the LayerNorm of wide models (unused otherwise).
fe_status run_proj(const fe_model* m, const GemmArgs& g, hipStream_t s, void* lnbuf = nullptr);
// X += FFN(LN(X)) on fp32 and wide bf16 models: LN, up-projection + ReLU into Hf, down-projection
// with the residual.
fe_status run_ffn(const fe_model* m, float* X, int R, const float* lng, const float* lnb, const void* w1,
                  const float* b1, const void* w2, const float* b2, void* Hf, const int32_t* nvalid, int rpb,
                  hipStream_t s, void* lnbuf = nullptr);

struct Bufs {
  float* X;      // residual stream [rows][d]: fp32, or bf16 when xbf
  void* qkv;     // act [rows][3d]
  void* O;       // act [rows][d]
  void* Hf;      // act [rows][F]
  void* ln;      // wide bf16 models: bf16 [rows][d] LayerNorm output (else unused)
  bool xbf = false;   // X holds bf16 (the fused tails of bf16 models write it so between kernels)
  size_t hf_bytes = 0;   // bytes of Hf (the fused tails borrow it for the partial sums of split FFNs)
};

// One pre-LN encoder block over nb batches of `per` rows; attention stays inside a batch.
// `xin` is the block input (act or fp32); the output residual stream is written to b.X.
// The key/value projections a bf16 block's tail may also produce from the module's final
// LayerNorm of its output (the last context block; see PostArgs).
struct KvOut {
  const float *lnf_g, *lnf_b;
  const void* wkv; const float* bkv; void* kv; int layers;
  int32_t* zero; int zero_n;   // status words this launch clears (or nullptr)
};

// lin_st != nullptr: the block's attention is linear, through the state buffer lin_st
// (fp32 [nb][H][dh+1][dh]).
fe_status enc_block(const fe_model* m, const EncW& w, int nb, int per, const void* xin, bool xin_f32, const Bufs& b,
                    const int32_t* nvalid, hipStream_t s, const KvOut* kvo = nullptr, float* lin_st = nullptr,
                    float* lin_part = nullptr) {
  const int d = m->cfg.d, F = m->cfg.ffn_dim, R = nb * per;
  const bool bf = m->bf16;
  const size_t e = bf ? 2 : 4;
  const float scale = 1.0f / sqrtf((float)(d / m->cfg.n_heads));
  if (lin_st) {
    // LN1 and q|k|v, the per-head state of the batch's keys and values, then every query row
    GemmArgs g = gemm(xin, d, xin_f32, R, d, 3 * d, w.wqkv, w.bqkv, b.qkv, 3 * d, false, EPI_STORE);
    g.ln_g = w.ln1g; g.ln_b = w.ln1b; g.nvalid = nvalid; g.rows_per_batch = per;
    fe_status st0 = run_proj(m, g, s, b.ln);
    if (st0 != FE_OK) return st0;
    const int H = m->cfg.n_heads, dh = d / H;
    const char* qkv = static_cast<const char*>(b.qkv);
    FE_LAUNCH(F_LIN, s, launch_lin_state(qkv + d * e, qkv + 2 * d * e, (long long)per * 3 * d, 3 * d, nb, per, nvalid,
                                          H, dh, lin_st, bf, s, lin_part));
    FE_LAUNCH(F_LIN, s, launch_lin_apply(qkv, 3 * d, lin_st, nb, per, nvalid, H, dh, b.O, d, bf, s));
  } else if (bf && self_attention_fits(d, m->cfg.n_heads, per)) {
    // LN1, q|k|v of one head and attention in one kernel per (batch, head)
    SelfAttnArgs sa{xin, xin_f32, nb, per, nvalid, w.ln1g, w.ln1b, w.wqkv, w.bqkv, b.O, m->cfg.n_heads, scale};
    FE_LAUNCH(F_ATTN, s, launch_self_attention(sa, d, s));
  } else {
    GemmArgs g = gemm(xin, d, xin_f32, R, d, 3 * d, w.wqkv, w.bqkv, b.qkv, 3 * d, false, EPI_STORE);
    g.ln_g = w.ln1g; g.ln_b = w.ln1b; g.nvalid = nvalid; g.rows_per_batch = per;
    fe_status st0 = run_proj(m, g, s, b.ln);
    if (st0 != FE_OK) return st0;
    AttnArgs a{};
    a.Q = b.qkv; a.q_bs = (long long)per * 3 * d; a.q_rs = 3 * d;
    a.K = static_cast<const char*>(b.qkv) + d * e; a.k_bs = a.q_bs; a.k_rs = 3 * d;
    a.V = static_cast<const char*>(b.qkv) + 2 * d * e; a.v_bs = a.q_bs; a.v_rs = 3 * d;
    a.O = b.O; a.o_bs = (long long)per * d; a.o_rs = d;
    a.B = nb; a.nq = per; a.nk = per; a.n_heads = m->cfg.n_heads; a.dh = d / m->cfg.n_heads;
    a.q_valid = nvalid; a.k_valid = nvalid;
    a.scale = scale;
    FE_LAUNCH(F_ATTN, s, launch_attention(a, bf, s));
  }
  if (bf && !wide(m)) {
    // output projection, residual, LN2 and FFN in one kernel
    PostArgs p{b.O, xin, xin_f32, b.X, R, per, nvalid, d, F, 0, w.wo, w.bo, w.ln2g, w.ln2b,
               w.w1, w.b1, w.w2, w.b2, nullptr, nullptr, nullptr};
    p.xout_bf16 = b.xbf;
    p.part = b.Hf;
    p.part_bytes = b.hf_bytes;
    if (kvo) {
      p.Xout = nullptr;   // nothing reads the module's residual after its key/value projections
      p.lnfg = kvo->lnf_g;
      p.lnfb = kvo->lnf_b;
      p.wkv = kvo->wkv;
      p.bkv = kvo->bkv;
      p.kv = kvo->kv;
      p.kv_layers = kvo->layers;
      p.zero = kvo->zero;
      p.zero_n = kvo->zero_n;
    }
    FE_LAUNCH(F_POST, s, launch_post(p, s));
    return FE_OK;
  }
  GemmArgs g = gemm(b.O, d, false, R, d, d, w.wo, w.bo, b.X, d, true, EPI_RESID);
  g.res = xin; g.ldr = d; g.res_f32 = xin_f32; g.nvalid = nvalid; g.rows_per_batch = per;
  fe_status st = run_proj(m, g, s, b.ln);
  if (st != FE_OK) return st;
  return run_ffn(m, b.X, R, w.ln2g, w.ln2b, w.w1, w.b1, w.w2, w.b2, b.Hf, nvalid, per, s, b.ln);
}

// Whole modules of short groups run as one kernel on bf16 models.
bool module_fits(const fe_model* m, int per) { return m->bf16 && per <= module_small_tile_rows(m->cfg.d); }

// n encoder blocks `ws` over ngroups groups of `per` rows, then the final LayerNorm (lnf_g,
// lnf_b) into fp32 Y: every row, or the first row of each group.
fe_status run_module(const fe_model* m, const std::vector<EncW>& ws, int ngroups, int per, const void* xin, bool xin_f32,
                     const float* lnf_g, const float* lnf_b, float* Y, bool first_row_only, hipStream_t s) {
  ModuleArgs a{};
  a.Xin = xin; a.xin_f32 = xin_f32;
  a.Y = Y; a.first_row_only = first_row_only;
  a.n_groups = ngroups; a.S = per;
  a.D = m->cfg.d; a.H = m->cfg.n_heads; a.F = m->cfg.ffn_dim; a.n_layers = m->cfg.n_layers;
  a.scale = 1.0f / sqrtf((float)(m->cfg.d / m->cfg.n_heads));
  a.lnfg = lnf_g; a.lnfb = lnf_b;
  for (int l = 0; l < m->cfg.n_layers; ++l) a.layer[l] = ws[l];
  FE_LAUNCH(F_LAYER, s, launch_module_small(a, s));
  return FE_OK;
}

// SeqEnc over every list of the batch: c_k = final LayerNorm of each list's [CLS] row (row 0 of
// every (L+1)-row group), fp32 [B*K][d]
fe_status seq_encode(const fe_model* m, int B, int K, int L, const void* seq, float* c, const Bufs& b, hipStream_t s) {
  const int d = m->cfg.d, S = L + 1;
  if (module_fits(m, S)) return run_module(m, m->seq, B * K, S, seq, false, m->seq_lnf_g, m->seq_lnf_b, c, true, s);
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    fe_status st = enc_block(m, m->seq[l], B * K, S, l == 0 ? seq : b.X, l > 0, b, nullptr, s);
    if (st != FE_OK) return st;
  }
  FE_LAUNCH(F_LN, s, launch_layernorm(b.X, 1, (long long)S * d, B * K, d, m->seq_lnf_g, m->seq_lnf_b, c, 1, d, m->bf16, s));
  return FE_OK;
}

// The LayerNorm of a wide model's product input, into lnbuf (bf16), then the tiled product.
fe_status run_wide(const fe_model* m, GemmArgs g, void* lnbuf, hipStream_t s) {
  if (g.ln_g) {
    if (!lnbuf) return fail(FE_EHIP, "internal: no LayerNorm buffer for a wide projection");
    FE_LAUNCH(F_LN, s, launch_layernorm_masked(g.A, g.a_f32, g.lda, g.R, g.K, g.ln_g, g.ln_b, lnbuf, 0, g.K, g.nvalid,
                                               g.rows_per_batch, true, s));
    g.A = lnbuf;
    g.a_f32 = 0;
    g.lda = g.K;
    g.ln_g = g.ln_b = nullptr;
  }
  FE_LAUNCH(F_GEMM, s, launch_gemm_tiled(g, s));
  return FE_OK;
}

fe_status run_proj(const fe_model* m, const GemmArgs& g, hipStream_t s, void* lnbuf) {
  if (wide(m)) return run_wide(m, g, lnbuf, s);
  if (m->bf16) FE_LAUNCH(F_GEMM, s, launch_proj(g, s));
  else FE_LAUNCH(F_GEMM, s, launch_gemm(g, false, s));
  return FE_OK;
}

fe_status run_ffn(const fe_model* m, float* X, int R, const float* lng, const float* lnb, const void* w1,
                  const float* b1, const void* w2, const float* b2, void* Hf, const int32_t* nvalid, int rpb,
                  hipStream_t s, void* lnbuf) {
  const int d = m->cfg.d, F = m->cfg.ffn_dim;
  GemmArgs g = gemm(X, d, true, R, d, F, w1, b1, Hf, F, false, EPI_RELU);
  g.ln_g = lng; g.ln_b = lnb; g.nvalid = nvalid; g.rows_per_batch = rpb;
  if (wide(m)) {
    fe_status st = run_wide(m, g, lnbuf, s);
    if (st != FE_OK) return st;
  } else {
    FE_LAUNCH(F_GEMM, s, launch_gemm(g, false, s));
  }
  g = gemm(Hf, F, false, R, F, d, w2, b2, X, d, true, EPI_RESID);
  g.res = X; g.ldr = d; g.res_f32 = true; g.nvalid = nvalid; g.rows_per_batch = rpb;
  if (wide(m)) return run_wide(m, g, lnbuf, s);
  FE_LAUNCH(F_GEMM, s, launch_gemm(g, false, s));
  return FE_OK;
}

// SeqEnc, then the cross-sequence module, on the buffers b (SeqEnc's separate-block path) and c
// (fp32 [B*K][d], the c_k rows; the cross module's residual when it runs block by block); lin_st:
// linear models' per-head state buffer of one module (fp32 [B][H][dh+1][dh]).
fe_status cross_sequence_run(const fe_model* m, int B, int K, int L, const void* seq, float* Cp, const Bufs& b,
                             float* c, float* lin_st, float* lin_part, hipStream_t s) {
  fe_status st = seq_encode(m, B, K, L, seq, c, b, s);
  if (st != FE_OK) return st;
  const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
  if (!lin && module_fits(m, K))
    return run_module(m, m->cross, B, K, c, true, m->cross_lnf_g, m->cross_lnf_b, Cp, false, s);
  Bufs bc{c, b.qkv, b.O, b.Hf, b.ln};
  bc.hf_bytes = b.hf_bytes;
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    st = enc_block(m, m->cross[l], B, K, c, true, bc, nullptr, s, nullptr, lin ? lin_st : nullptr, lin_part);
    if (st != FE_OK) return st;
  }
  FE_LAUNCH(F_LN, s, launch_layernorm(c, 1, m->cfg.d, B * K, m->cfg.d, m->cross_lnf_g, m->cross_lnf_b, Cp, 1, m->cfg.d,
                                      m->bf16, s));
  return FE_OK;
}

// ------------------------------------------------------------------------------------------
// Library-owned scratch of fe_cross_sequence_noalloc: one copy per device, held until the
// process ends.  Host code never passes the symbol itself to a kernel or copy (on the host it
// is only a stand-in); it uses the device address hipGetSymbolAddress returns for each device.
// ------------------------------------------------------------------------------------------
constexpr size_t kScratchBytes = FE_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "scratch pieces are 256-byte aligned");
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on `device`, looked up once per device with that device current.
fe_status scratch_address(int device, void** out) {
  if (device < 0 || device >= kMaxDevices) return fail(FE_EUNSUPPORTED, "device %d outside [0, %d)", device, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    int cur = -1;
    FE_HIP(hipGetDevice(&cur));
    if (cur != device) FE_HIP(hipSetDevice(device));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != device) (void)hipSetDevice(cur);
    if (e != hipSuccess) return fail(FE_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    if (!p) return fail(FE_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[device] = p;
  }
  *out = g_scratch_ptr[device];
  return FE_OK;
}

// What fe_cross_sequence needs of its workspace, packed: the c rows always; SeqEnc's residual and
// block buffers only when its lists are too long for the module kernel; the block buffers of the
// cross module only when it runs block by block (K > 64, wide or linear models).
struct CrossScratch { size_t c, X, qkv, O, Hf, ln, lin_st, lin_part, total, hf_bytes; };

CrossScratch cross_scratch_layout(const fe_model* m, long long B, long long K, long long L) {
  const long long d = m->cfg.d, F = m->cfg.ffn_dim, S = L + 1, H = m->cfg.n_heads, dh = d / H;
  const size_t e = m->bf16 ? 2 : 4;
  const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
  const bool seq_blocks = !module_fits(m, (int)S), cross_blocks = lin || !module_fits(m, (int)K);
  CrossScratch w{};
  Bump b{0};
  w.c = b.take(B * K * d * 4);
  const long long rows = std::max(seq_blocks ? B * K * S : 0, cross_blocks ? B * K : 0);
  if (seq_blocks) w.X = b.take(B * K * S * d * 4);
  if (rows > 0) {
    w.qkv = b.take(rows * 3 * d * e);
    w.O = b.take(rows * d * e);
    w.hf_bytes = std::max({(size_t)(rows * F * e), seq_blocks ? post_part_bytes(B * K * S, (int)d, (int)F) : size_t(0),
                           cross_blocks ? post_part_bytes(B * K, (int)d, (int)F) : size_t(0)});
    w.Hf = b.take(w.hf_bytes);
    if (wide(m)) w.ln = b.take(rows * d * 2);
  }
  if (lin) {
    w.lin_st = b.take(B * H * (dh + 1) * dh * 4);
    w.lin_part = b.take(B * H * lin_state_splits((int)(B * H), (int)K, m->bf16) * (dh + 1) * dh * 4);
  }
  w.total = (b.at + 255) & ~size_t(255);
  return w;
}

}  // namespace

// Records the error text of a call implemented in another file of the library (the training step).
fe_status fe_report(fe_status st, const char* msg) {
  g_err = msg;
  return st;
}

// ==========================================================================================
// Exported functions
// ==========================================================================================
extern "C" {

const char* fe_last_error(void) { return g_err.c_str(); }

fe_status fe_trace_enable(int on) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  for (auto& r : g_trace) {
    (void)hipEventSynchronize(r.b);
    g_event_pool.push_back(r.a);
    g_event_pool.push_back(r.b);
  }
  g_trace.clear();
  g_trace_on = on != 0;
  return FE_OK;
}

fe_status fe_trace_read(double* total_ms, int64_t* launches) {
  if (!total_ms || !launches) return fail(FE_EINVAL, "NULL output array");
  std::lock_guard<std::mutex> lk(g_trace_mu);
  for (int i = 0; i < FE_TRACE_FAMILIES; ++i) { total_ms[i] = 0.0; launches[i] = 0; }
  fe_status st = FE_OK;
  for (auto& r : g_trace) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess && st == FE_OK) st = fail(FE_EHIP, "trace event: %s", hipGetErrorString(e));
    total_ms[r.fam] += ms;
    launches[r.fam] += 1;
    g_event_pool.push_back(r.a);
    g_event_pool.push_back(r.b);
  }
  g_trace.clear();
  return st;
}

fe_status fe_trace_read_launches(int32_t* family, double* ms, int64_t capacity, int64_t* count) {
  if (!count || (capacity > 0 && (!family || !ms))) return fail(FE_EINVAL, "NULL output array");
  std::lock_guard<std::mutex> lk(g_trace_mu);
  *count = (int64_t)g_trace.size();
  if ((int64_t)g_trace.size() > capacity)
    return fail(FE_EINVAL, "%zu launches recorded, capacity %lld", g_trace.size(), (long long)capacity);
  fe_status st = FE_OK;
  for (size_t i = 0; i < g_trace.size(); ++i) {
    const TraceRec& r = g_trace[i];
    float t = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, r.a, r.b);
    if (e != hipSuccess && st == FE_OK) st = fail(FE_EHIP, "trace event: %s", hipGetErrorString(e));
    family[i] = r.fam;
    ms[i] = t;
    g_event_pool.push_back(r.a);
    g_event_pool.push_back(r.b);
  }
  g_trace.clear();
  return st;
}

const char* fe_trace_family(int i) { return (i >= 0 && i < FE_TRACE_FAMILIES) ? kFamName[i] : ""; }

fe_status fe_param_count(const fe_config* cfg, size_t* n_floats) {
  fe_status st = check_config(cfg);
  if (st != FE_OK) return st;
  if (!n_floats) return fail(FE_EINVAL, "n_floats is NULL");
  Packer P;
  pack_all(P, *cfg);
  *n_floats = P.consumed;
  return FE_OK;
}

fe_status fe_model_create(const fe_config* cfg, const float* params, size_t n_floats, fe_model** out) {
  fe_status st = check_config(cfg);
  if (st != FE_OK) return st;
  if (!params || !out) return fail(FE_EINVAL, "params or out is NULL");
  *out = nullptr;
  size_t need = 0;
  fe_param_count(cfg, &need);
  if (n_floats != need) return fail(FE_EINVAL, "expected %zu parameter floats, got %zu", need, n_floats);
  fe_model* m = new (std::nothrow) fe_model();
  if (!m) return fail(FE_ENOMEM, "host allocation failed");
  m->cfg = *cfg;
  m->bf16 = cfg->dtype == FE_BF16;
  if (hipGetDevice(&m->device) != hipSuccess) {
    delete m;
    return fail(FE_EHIP, "hipGetDevice failed");
  }
  Packer P;
  P.src = params;
  P.bf16 = m->bf16;
  Offsets O = pack_all(P, *cfg);
  hipError_t e = hipMalloc(&m->dev, P.image.size());
  if (e != hipSuccess) {
    delete m;
    return fail(FE_ENOMEM, "hipMalloc(%zu) failed: %s", P.image.size(), hipGetErrorString(e));
  }
  e = hipMemcpy(m->dev, P.image.data(), P.image.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(m->dev);
    delete m;
    return fail(FE_EHIP, "hipMemcpy of weights failed: %s", hipGetErrorString(e));
  }
  char* base = static_cast<char*>(m->dev);
  auto F = [&](size_t off) { return reinterpret_cast<const float*>(base + off); };
  auto A = [&](size_t off) { return static_cast<const void*>(base + off); };
  auto enc = [&](const EncOff& o) {
    return EncW{F(o.ln1g), F(o.ln1b), A(o.wqkv), F(o.bqkv), A(o.wo), F(o.bo), F(o.ln2g), F(o.ln2b),
                A(o.w1), F(o.b1), A(o.w2), F(o.b2)};
  };
  for (auto& o : O.ctx) m->ctx.push_back(enc(o));
  for (auto& o : O.seq) m->seq.push_back(enc(o));
  for (auto& o : O.cross) m->cross.push_back(enc(o));
  for (auto& o : O.item)
    m->item.push_back(ItemW{F(o.ln1g), F(o.ln1b), A(o.wqkv), F(o.bqkv), A(o.wo), F(o.bo), F(o.ln2g), F(o.ln2b),
                            A(o.wq), F(o.bq), A(o.wo2), F(o.bo2), F(o.ln3g), F(o.ln3b), A(o.w1), F(o.b1),
                            A(o.w2), F(o.b2)});
  m->ctx_lnf_g = F(O.ctx_lnf_g); m->ctx_lnf_b = F(O.ctx_lnf_b);
  m->item_lnf_g = F(O.item_lnf_g); m->item_lnf_b = F(O.item_lnf_b);
  m->seq_lnf_g = F(O.seq_lnf_g); m->seq_lnf_b = F(O.seq_lnf_b);
  m->cross_lnf_g = F(O.cross_lnf_g); m->cross_lnf_b = F(O.cross_lnf_b);
  m->wkv = A(O.wkv); m->bkv = F(O.bkv);
  m->cls = A(O.cls); m->pos = A(O.pos);
  m->head_w = F(O.head_w); m->head_b = F(O.head_b);
  m->emb = cfg->vocab > 0 ? A(O.emb) : nullptr;
  *out = m;
  return FE_OK;
}

void fe_model_destroy(fe_model* m) {
  if (!m) return;
  if (m->dev) (void)hipFree(m->dev);
  delete m;
}

fe_status fe_workspace_size(const fe_model* m, int B, int T, int M, int K, int L, size_t* bytes) {
  fe_status st = check_dims(m, B, T, M, K, L);
  if (st != FE_OK) return st;
  if (!bytes) return fail(FE_EINVAL, "bytes is NULL");
  *bytes = layout(m, B, T, M, K, L).total;
  return FE_OK;
}

fe_status fe_kv_size(const fe_model* m, int B, int T, size_t* bytes) {
  fe_status st = check_dims(m, B, T, 1, 1, 1);
  if (st != FE_OK) return st;
  if (!bytes) return fail(FE_EINVAL, "bytes is NULL");
  *bytes = kv_bytes(m, B, T);
  return FE_OK;
}

fe_status fe_read_device_status(const fe_model* m, const void* ws, int B, void* stream, int32_t* host_out) {
  if (!m || !ws || !host_out || B < 1) return fail(FE_EINVAL, "bad arguments to fe_read_device_status");
  std::vector<int32_t> tmp(2 * (size_t)B);
  hipStream_t s = static_cast<hipStream_t>(stream);
  FE_HIP(hipMemcpyAsync(tmp.data(), ws, tmp.size() * 4, hipMemcpyDeviceToHost, s));
  FE_HIP(hipStreamSynchronize(s));
  for (int b = 0; b < B; ++b) host_out[b] = tmp[b] | tmp[B + b];
  return FE_OK;
}

fe_status fe_encode_context(const fe_model* m, int B, int T, const void* x, const int32_t* ctx_ids, void* kv, void* ws,
                            size_t ws_bytes, void* stream) {
  fe_status st = check_dims(m, B, T, 1, 1, 1);
  if (st != FE_OK) return st;
  if ((x == nullptr) == (ctx_ids == nullptr)) return fail(FE_EINVAL, "give exactly one of x and ctx_ids");
  if (ctx_ids && !m->emb) return fail(FE_EINVAL, "ctx_ids given but the model has no vocabulary");
  if (!kv || !ws) return fail(FE_EINVAL, "kv or ws is NULL");
  if (!aligned16(x) || !aligned16(ctx_ids) || !aligned16(kv) || !aligned16(ws))
    return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const Ws w = layout(m, B, T, 1, 1, 1);
  if (ws_bytes < w.total) return fail(FE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, w.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf = m->bf16;
  const int d = m->cfg.d, R = B * T;
  int32_t* status_ctx = at<int32_t>(ws, w.status) + B;
  // the context status words start at zero: cleared before the embedding gather sets bits in
  // them, else by the launch that writes the key/value cache at the end of this call (nothing
  // else writes them)
  const bool clear_late = bf && !ctx_ids;
  if (!clear_late) FE_LAUNCH(F_FILL, s, launch_fill_i32(status_ctx, B, 0, s));
  const void* src = x;
  if (ctx_ids) {
    FE_LAUNCH(F_GATHER, s, launch_gather_rows(m->emb, 0, m->cfg.vocab, ctx_ids, T, nullptr, B, T, d, at<char>(ws, w.c_xin), status_ctx,
                              FE_DEV_BAD_TOKEN, bf, s));
    src = at<char>(ws, w.c_xin);
  }
  Bufs b{at<float>(ws, w.c_x), at<char>(ws, w.c_qkv), at<char>(ws, w.c_o), at<char>(ws, w.c_h), at<char>(ws, w.c_ln)};
  b.hf_bytes = w.c_h_bytes;
  // linear models: the item layers' keys and values go to the workspace first, and kv receives
  // their per-head state
  const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
  float* lin_st = lin ? at<float>(ws, w.lin_st) : nullptr;
  float* lin_part = lin ? at<float>(ws, w.lin_part) : nullptr;
  void* kvp = lin ? at<char>(ws, w.c_kvp) : kv;
  const bool whole = !lin && module_fits(m, T);
  b.xbf = bf && !wide(m) && !whole;   // block by block through the fused tails: bf16 between kernels
  if (whole) {
    st = run_module(m, m->ctx, B, T, src, false, m->ctx_lnf_g, m->ctx_lnf_b, b.X, false, s);
    if (st != FE_OK) return st;
  } else {
    // on bf16 models the last block's tail also applies the final LayerNorm and writes the
    // key/value projections of every item layer
    const KvOut kvo{m->ctx_lnf_g, m->ctx_lnf_b, m->wkv, m->bkv, kvp, m->cfg.n_layers,
                    clear_late ? status_ctx : nullptr, B};
    for (int l = 0; l < m->cfg.n_layers; ++l) {
      const bool last = l + 1 == m->cfg.n_layers;
      st = enc_block(m, m->ctx[l], B, T, l == 0 ? src : b.X, l > 0 && !b.xbf, b, nullptr, s,
                     bf && !wide(m) && last ? &kvo : nullptr, lin_st, lin_part);
      if (st != FE_OK) return st;
    }
  }
  if (!bf || whole || wide(m)) {
    // key/value projections of all item layers, with the context module's final LayerNorm fused
    // into their prologue unless the module kernel already applied it
    GemmArgs g = gemm(b.X, d, true, R, d, 2 * m->cfg.n_layers * d, m->wkv, m->bkv, kvp, d, false, EPI_STORE);
    if (!whole) {
      g.ln_g = m->ctx_lnf_g;
      g.ln_b = m->ctx_lnf_b;
    }
    g.col_block = d; g.col_block_stride = (long long)R * d;
    if (clear_late) {
      g.zero = status_ctx;
      g.zero_n = B;
    }
    st = run_proj(m, g, s, b.ln);
    if (st != FE_OK) return st;
  }
  if (lin) {
    // the linear-attention cache: per item layer and head, sum_t phi(k_t) v_t^T and sum_t phi(k_t)
    const int H = m->cfg.n_heads, dh = d / H;
    const size_t e = bf ? 2 : 4;
    for (int l = 0; l < m->cfg.n_layers; ++l) {
      const char* K = static_cast<const char*>(kvp) + (size_t)(2 * l) * R * d * e;
      const char* V = static_cast<const char*>(kvp) + (size_t)(2 * l + 1) * R * d * e;
      float* out = static_cast<float*>(kv) + (size_t)l * B * H * (dh + 1) * dh;
      FE_LAUNCH(F_LIN, s, launch_lin_state(K, V, (long long)T * d, d, B, T, nullptr, H, dh, out, bf, s, lin_part));
    }
  }
  return FE_OK;
}

fe_status fe_encode_items(const fe_model* m, int B, int M, const void* pool, const int32_t* lists, int K, int L,
                          const void* kv, int T, int32_t* uniq, int32_t* n_uniq, int32_t* slot, void* H, void* ws,
                          size_t ws_bytes, void* stream) {
  fe_status st = check_dims(m, B, T, M, K, L);
  if (st != FE_OK) return st;
  if (!pool && !m->emb) return fail(FE_EINVAL, "pool is NULL and the model has no vocabulary");
  if (!pool && M != m->cfg.vocab) return fail(FE_EINVAL, "token-id items need M == vocab (%d)", m->cfg.vocab);
  if (!lists || !kv || !uniq || !n_uniq || !slot || !H || !ws) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(pool) || !aligned16(lists) || !aligned16(kv) || !aligned16(H) || !aligned16(ws) ||
      !aligned16(uniq) || !aligned16(slot))
    return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const Ws w = layout(m, B, T, M, K, L);
  if (ws_bytes < w.total) return fail(FE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, w.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool bf = m->bf16;
  const int d = m->cfg.d, F = m->cfg.ffn_dim, KL = K * L;
  const int Ucap = std::min(M, KL);
  const int R = B * Ucap;
  const size_t e = bf ? 2 : 4;
  int32_t* status_items = at<int32_t>(ws, w.status);
  const void* table = pool ? pool : m->emb;
  const long long table_bs = pool ? (long long)M * d : 0;
  void* G0 = at<char>(ws, w.i_g0);
  // the first item layer's self-attention kernel builds the distinct set and gathers the rows
  // itself when it covers the set (its bitmap lives in the LN1 tile: M <= 278528)
  const bool set_in_attention = bf && self_attention_fits(d, m->cfg.n_heads, Ucap) && (M + 31) / 32 <= 8704;
  if (set_in_attention) {
    // nothing to launch here
  } else if (dedup_gather_fits(Ucap, d, bf)) {
    FE_LAUNCH(F_DEDUP, s, launch_dedup_gather(lists, B, KL, M, Ucap, uniq, n_uniq, slot, status_items, table, table_bs, d,
                                              G0, bf, s));
  } else {
    FE_LAUNCH(F_DEDUP, s, launch_dedup(lists, B, KL, M, Ucap, uniq, n_uniq, slot, status_items, s));
    FE_LAUNCH(F_GATHER, s, launch_gather_rows(table, table_bs, M, uniq, Ucap, n_uniq, B, Ucap, d, G0, nullptr, 0, bf, s));
  }
  float* G = at<float>(ws, w.i_g);
  float* G1 = at<float>(ws, w.i_g1);
  void* qkv = at<char>(ws, w.i_qkv);
  void* O = at<char>(ws, w.i_o);
  void* Qc = at<char>(ws, w.i_q);
  void* Hf = at<char>(ws, w.i_h);
  void* lnb = wide(m) ? at<char>(ws, w.i_ln) : nullptr;
  const bool fused_tail = bf && !wide(m);     // k_post tails (else separate products)
  const bool rbf = fused_tail;                // G and G1 hold the residual stream in bf16
  const int dh = d / m->cfg.n_heads;
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const ItemW& iw = m->item[l];
    const void* xin = l == 0 ? G0 : static_cast<const void*>(G);
    const bool xin_f32 = l > 0 && !rbf;
    if (bf && self_attention_fits(d, m->cfg.n_heads, Ucap)) {
      SelfAttnArgs sa{xin, xin_f32, B, Ucap, n_uniq, iw.ln1g, iw.ln1b, iw.wqkv, iw.bqkv, O, m->cfg.n_heads,
                      1.0f / sqrtf((float)dh)};
      if (l == 0 && set_in_attention) {
        sa.lists = lists; sa.KL = KL; sa.M = M;
        sa.table = table; sa.table_bs = table_bs;
        sa.uniq = uniq; sa.n_uniq = n_uniq; sa.slot = slot; sa.status = status_items;
        sa.Xrows = G0;
      }
      FE_LAUNCH(F_ATTN, s, launch_self_attention(sa, d, s));   // the distinct set rides in the first launch
    } else {
      GemmArgs g = gemm(xin, d, xin_f32, R, d, 3 * d, iw.wqkv, iw.bqkv, qkv, 3 * d, false, EPI_STORE);
      g.ln_g = iw.ln1g; g.ln_b = iw.ln1b; g.nvalid = n_uniq; g.rows_per_batch = Ucap;
      st = run_proj(m, g, s, lnb);
      if (st != FE_OK) return st;
      AttnArgs a{};
      a.Q = qkv; a.q_bs = (long long)Ucap * 3 * d; a.q_rs = 3 * d;
      a.K = static_cast<const char*>(qkv) + d * e; a.k_bs = a.q_bs; a.k_rs = 3 * d;
      a.V = static_cast<const char*>(qkv) + 2 * d * e; a.v_bs = a.q_bs; a.v_rs = 3 * d;
      a.O = O; a.o_bs = (long long)Ucap * d; a.o_rs = d;
      a.B = B; a.nq = Ucap; a.nk = Ucap; a.n_heads = m->cfg.n_heads; a.dh = dh;
      a.q_valid = n_uniq; a.k_valid = n_uniq;
      a.scale = 1.0f / sqrtf((float)dh);
      FE_LAUNCH(F_ATTN, s, launch_attention(a, bf, s));
    }
    const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
    const void* Kc = static_cast<const char*>(kv) + (size_t)(2 * l) * B * T * d * e;
    const void* Vc = static_cast<const char*>(kv) + (size_t)(2 * l + 1) * B * T * d * e;
    if (!lin && bf && cross_attention_fits(d, m->cfg.n_heads, Ucap, T)) {
      // x1 = x + O Wo + bo -> G1, queries LN2(x1) Wq + bq and the cross-attention in one kernel
      // per (request, head); its output goes to Qc (every head's workgroup reads all of O)
      CrossAttnArgs ca{O, xin, xin_f32, G1, B, Ucap, n_uniq, iw.wo, iw.bo, iw.ln2g, iw.ln2b, iw.wq, iw.bq,
                       Kc, Vc, T, Qc, m->cfg.n_heads, 1.0f / sqrtf((float)dh)};
      ca.xout_bf16 = rbf;
      FE_LAUNCH(F_ATTN, s, launch_cross_attention(ca, d, s));
      const bool last = l + 1 == m->cfg.n_layers;
      PostArgs p{Qc, G1, !rbf, last ? nullptr : G, R, Ucap, n_uniq, d, F, 0, iw.wo2, iw.bo2, iw.ln3g, iw.ln3b,
                 iw.w1, iw.b1, iw.w2, iw.b2, nullptr, nullptr, nullptr,
                 last ? m->item_lnf_g : nullptr, last ? m->item_lnf_b : nullptr, last ? H : nullptr};
      p.xout_bf16 = rbf;
      p.part = Hf;
      p.part_bytes = w.i_h_bytes;
      FE_LAUNCH(F_POST, s, launch_post(p, s));
      continue;
    }
    if (fused_tail) {
      // x1 = x + O Wo + bo -> G, and the cross-attention queries q = LN2(x1) Wq + bq -> Qc
      PostArgs p{O, xin, xin_f32, G, R, Ucap, n_uniq, d, F, 1, iw.wo, iw.bo, iw.ln2g, iw.ln2b,
                 nullptr, nullptr, nullptr, nullptr, iw.wq, iw.bq, Qc};
      p.xout_bf16 = rbf;
      FE_LAUNCH(F_POST, s, launch_post(p, s));
    } else {
      GemmArgs g = gemm(O, d, false, R, d, d, iw.wo, iw.bo, G, d, true, EPI_RESID);
      g.res = xin; g.ldr = d; g.res_f32 = xin_f32; g.nvalid = n_uniq; g.rows_per_batch = Ucap;
      st = run_proj(m, g, s, lnb);
      if (st != FE_OK) return st;
      // cross-attention: the distinct elements are the queries, the context cache the keys/values
      g = gemm(G, d, true, R, d, d, iw.wq, iw.bq, Qc, d, false, EPI_STORE);
      g.ln_g = iw.ln2g; g.ln_b = iw.ln2b; g.nvalid = n_uniq; g.rows_per_batch = Ucap;
      st = run_proj(m, g, s, lnb);
      if (st != FE_OK) return st;
    }
    if (lin) {
      // linear attention of the queries against item layer l's context state
      const float* stl = static_cast<const float*>(kv) + (size_t)l * B * m->cfg.n_heads * (dh + 1) * dh;
      FE_LAUNCH(F_LIN, s, launch_lin_apply(Qc, d, stl, B, Ucap, n_uniq, m->cfg.n_heads, dh, O, d, bf, s));
    } else {
      AttnArgs c{};
      c.Q = Qc; c.q_bs = (long long)Ucap * d; c.q_rs = d;
      c.K = Kc; c.k_bs = (long long)T * d; c.k_rs = d;
      c.V = Vc; c.v_bs = (long long)T * d; c.v_rs = d;
      c.O = O; c.o_bs = (long long)Ucap * d; c.o_rs = d;
      c.B = B; c.nq = Ucap; c.nk = T; c.n_heads = m->cfg.n_heads; c.dh = dh;
      c.q_valid = n_uniq; c.k_valid = nullptr;
      c.scale = 1.0f / sqrtf((float)dh);
      FE_LAUNCH(F_ATTN, s, launch_attention(c, bf, s));
    }
    if (fused_tail) {
      // the last layer also applies the module's final LayerNorm and writes H directly
      const bool last = l + 1 == m->cfg.n_layers;
      PostArgs p{O, G, !rbf, last ? nullptr : G, R, Ucap, n_uniq, d, F, 0, iw.wo2, iw.bo2, iw.ln3g, iw.ln3b,
                 iw.w1, iw.b1, iw.w2, iw.b2, nullptr, nullptr, nullptr,
                 last ? m->item_lnf_g : nullptr, last ? m->item_lnf_b : nullptr, last ? H : nullptr};
      p.xout_bf16 = rbf;
      p.part = Hf;
      p.part_bytes = w.i_h_bytes;
      FE_LAUNCH(F_POST, s, launch_post(p, s));
      continue;
    }
    GemmArgs g = gemm(O, d, false, R, d, d, iw.wo2, iw.bo2, G, d, true, EPI_RESID);
    g.res = G; g.ldr = d; g.res_f32 = true; g.nvalid = n_uniq; g.rows_per_batch = Ucap;
    st = run_proj(m, g, s, lnb);
    if (st != FE_OK) return st;
    st = run_ffn(m, G, R, iw.ln3g, iw.ln3b, iw.w1, iw.b1, iw.w2, iw.b2, Hf, n_uniq, Ucap, s, lnb);
    if (st != FE_OK) return st;
  }
  if (!fused_tail)
    FE_LAUNCH(F_LN, s, launch_layernorm_masked(G, 1, d, R, d, m->item_lnf_g, m->item_lnf_b, H, 0, d, n_uniq, Ucap, bf, s));
  return FE_OK;
}

fe_status fe_assemble(const fe_model* m, int B, int K, int L, int U_cap, const int32_t* slot, const void* H, void* seq,
                      void* stream) {
  fe_status st = check_dims(m, B, 1, U_cap, K, L);
  if (st != FE_OK) return st;
  if (!slot || !H || !seq) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(slot) || !aligned16(H) || !aligned16(seq)) return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  FE_LAUNCH(F_ASSEMBLE, static_cast<hipStream_t>(stream), launch_assemble(slot, H, B, K, L, U_cap, m->cfg.d, m->cls, m->pos, seq, m->bf16,
                         static_cast<hipStream_t>(stream)));
  return FE_OK;
}

fe_status fe_cross_sequence(const fe_model* m, int B, int K, int L, const void* seq, float* Cp, void* ws, size_t ws_bytes,
                            void* stream) {
  fe_status st = check_dims(m, B, 1, 1, K, L);
  if (st != FE_OK) return st;
  if (!seq || !Cp || !ws) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(seq) || !aligned16(Cp) || !aligned16(ws)) return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const Ws w = layout(m, B, 1, 1, K, L);
  if (ws_bytes < w.total) return fail(FE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, w.total);
  Bufs b{at<float>(ws, w.s_x), at<char>(ws, w.s_qkv), at<char>(ws, w.s_o), at<char>(ws, w.s_h), at<char>(ws, w.s_ln)};
  b.hf_bytes = w.s_h_bytes;
  const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
  return cross_sequence_run(m, B, K, L, seq, Cp, b, at<float>(ws, w.s_c), lin ? at<float>(ws, w.lin_st) : nullptr,
                            lin ? at<float>(ws, w.lin_part) : nullptr, static_cast<hipStream_t>(stream));
}

fe_status fe_cross_sequence_noalloc(const fe_model* m, int B, int K, int L, const void* seq, float* Cp, void* stream) {
  fe_status st = check_dims(m, B, 1, 1, K, L);
  if (st != FE_OK) return st;
  if (!seq || !Cp) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(seq) || !aligned16(Cp)) return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const CrossScratch w = cross_scratch_layout(m, B, K, L);
  if (w.total > kScratchBytes)
    return fail(FE_EUNSUPPORTED, "B=%d K=%d L=%d needs %zu bytes of scratch; the static scratch holds %zu", B, K, L,
                w.total, kScratchBytes);
  void* base = nullptr;
  st = scratch_address(m->device, &base);
  if (st != FE_OK) return st;
  Bufs b{at<float>(base, w.X), at<char>(base, w.qkv), at<char>(base, w.O), at<char>(base, w.Hf), at<char>(base, w.ln)};
  b.hf_bytes = w.hf_bytes;
  const bool lin = m->cfg.attention == FE_ATTN_LINEAR;
  return cross_sequence_run(m, B, K, L, seq, Cp, b, at<float>(base, w.c), lin ? at<float>(base, w.lin_st) : nullptr,
                            lin ? at<float>(base, w.lin_part) : nullptr, static_cast<hipStream_t>(stream));
}

fe_status fe_encode_sequences(const fe_model* m, int B, int K, int L, const void* seq, float* C, void* ws,
                              size_t ws_bytes, void* stream) {
  fe_status st = check_dims(m, B, 1, 1, K, L);
  if (st != FE_OK) return st;
  if (!seq || !C || !ws) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(seq) || !aligned16(C) || !aligned16(ws)) return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const Ws w = layout(m, B, 1, 1, K, L);
  if (ws_bytes < w.total) return fail(FE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, w.total);
  Bufs b{at<float>(ws, w.s_x), at<char>(ws, w.s_qkv), at<char>(ws, w.s_o), at<char>(ws, w.s_h), at<char>(ws, w.s_ln)};
  b.hf_bytes = w.s_h_bytes;
  return seq_encode(m, B, K, L, seq, C, b, static_cast<hipStream_t>(stream));
}

fe_status fe_score_objectives(const fe_model* m, int B, int K, const float* Cp, int n_obj, const float* head_w,
                              const float* head_b, const float* fuse_w, float* obj_scores, float* scores, int32_t* best,
                              void* stream) {
  fe_status st = check_dims(m, B, 1, 1, K, 1);
  if (st != FE_OK) return st;
  if (n_obj < 1 || n_obj > FE_MAX_OBJECTIVES) return fail(FE_EUNSUPPORTED, "n_obj=%d outside [1, %d]", n_obj, FE_MAX_OBJECTIVES);
  if (!Cp || !head_w || !head_b || !fuse_w || !obj_scores || !scores || !best)
    return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(Cp) || !aligned16(head_w)) return fail(FE_EINVAL, "Cp and head_w must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  FE_LAUNCH(F_SCORE, s, launch_score_objectives(Cp, B, K, m->cfg.d, n_obj, head_w, head_b, fuse_w, obj_scores, scores,
                                                best, s));
  return FE_OK;
}

fe_status fe_score_select(const fe_model* m, int B, int K, const float* Cp, float* scores, int32_t* best, void* stream) {
  fe_status st = check_dims(m, B, 1, 1, K, 1);
  if (st != FE_OK) return st;
  if (!Cp || !scores || !best) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(Cp)) return fail(FE_EINVAL, "Cp must be 16-byte aligned");
  FE_LAUNCH(F_SCORE, static_cast<hipStream_t>(stream), launch_score_select(Cp, B, K, m->cfg.d, m->head_w, m->head_b, scores, best, static_cast<hipStream_t>(stream)));
  return FE_OK;
}

// ------------------------------------------------------------------------------------------
// Candidate-factorised evaluator on the GPU (a baseline for the joint pass)
// ------------------------------------------------------------------------------------------
fe_status fe_naive_workspace_size(const fe_model* m, int B, int T, int M, int K, int L, int token_ids, size_t* bytes) {
  fe_status st = check_dims(m, B, T, M, K, L);
  if (st != FE_OK) return st;
  st = check_dims(m, (long long)B * K, T, M, K, L);
  if (st != FE_OK) return st;
  if (!bytes) return fail(FE_EINVAL, "bytes is NULL");
  *bytes = naive_layout(m, B, T, M, K, L, token_ids != 0, true).total;
  return FE_OK;
}

fe_status fe_evaluate_naive(const fe_model* m, int B, int T, int M, int K, int L, const void* x, const int32_t* ctx_ids,
                            const void* pool, const int32_t* lists, float* Cp, float* scores, int32_t* best, void* ws,
                            size_t ws_bytes, void* stream) {
  fe_status st = check_dims(m, B, T, M, K, L);
  if (st != FE_OK) return st;
  const long long BKl = (long long)B * K;
  st = check_dims(m, BKl, T, M, K, L);
  if (st != FE_OK) return st;
  if ((x == nullptr) == (ctx_ids == nullptr)) return fail(FE_EINVAL, "give exactly one of x and ctx_ids");
  if (ctx_ids && !m->emb) return fail(FE_EINVAL, "ctx_ids given but the model has no vocabulary");
  if (!pool && !m->emb) return fail(FE_EINVAL, "pool is NULL and the model has no vocabulary");
  if (!pool && M != m->cfg.vocab) return fail(FE_EINVAL, "token-id items need M == vocab (%d)", m->cfg.vocab);
  if (!lists || !Cp || !scores || !best || !ws) return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(x) || !aligned16(ctx_ids) || !aligned16(pool) || !aligned16(lists) || !aligned16(Cp) ||
      !aligned16(ws))
    return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const NaiveWs w = naive_layout(m, B, T, M, K, L, ctx_ids != nullptr, true);
  if (ws_bytes < w.total) return fail(FE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, w.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int BK = (int)BKl, d = m->cfg.d, Ucap = std::min(M, K * L);
  const size_t e = m->bf16 ? 2 : 4;
  void* inner = at<char>(ws, w.inner);
  // the context once per list: request b's context rows copied to each of its K lists
  void* xin = at<char>(ws, w.xin);
  if (ctx_ids) FE_LAUNCH(F_GATHER, s, launch_repeat_blocks(ctx_ids, xin, (long long)T * 4, B, K, s));
  else FE_LAUNCH(F_GATHER, s, launch_repeat_blocks(x, xin, (long long)T * d * e, B, K, s));
  void* kv = at<char>(ws, w.kv);
  st = fe_encode_context(m, BK, T, ctx_ids ? nullptr : xin, ctx_ids ? at<int32_t>(ws, w.xin) : nullptr, kv, inner,
                         w.inner_bytes, stream);
  if (st != FE_OK) return st;
  // every list sees its request's pool and the request's K lists (so the distinct set is U(z))
  const void* pool_k = nullptr;
  if (pool) {
    FE_LAUNCH(F_GATHER, s, launch_repeat_blocks(pool, at<char>(ws, w.pool), (long long)M * d * e, B, K, s));
    pool_k = at<char>(ws, w.pool);
  }
  int32_t* lists_k = at<int32_t>(ws, w.lists);
  FE_LAUNCH(F_GATHER, s, launch_repeat_blocks(lists, lists_k, (long long)K * L * 4, B, K, s));
  // the distinct-element set encoded once per element occurrence: L encodings per list, each
  // against that list's own context cache (every one of them yields the same rows)
  int32_t* slot_all = at<int32_t>(ws, w.slot);
  void* H = at<char>(ws, w.H);
  for (int j = 0; j < L; ++j) {
    st = fe_encode_items(m, BK, M, pool_k, lists_k, K, L, kv, T, at<int32_t>(ws, w.uniq), at<int32_t>(ws, w.n_uniq),
                         slot_all, H, inner, w.inner_bytes, stream);
    if (st != FE_OK) return st;
  }
  // each list assembled from its own encodings, then SeqEnc, cross-sequence module and head
  int32_t* slot_k = at<int32_t>(ws, w.slot_k);
  FE_LAUNCH(F_GATHER, s, launch_take_list_slots(slot_all, slot_k, BK, K, L, s));
  void* seq = at<char>(ws, w.seq);
  st = fe_assemble(m, BK, 1, L, Ucap, slot_k, H, seq, stream);
  if (st != FE_OK) return st;
  st = fe_cross_sequence(m, B, K, L, seq, Cp, inner, w.inner_bytes, stream);
  if (st != FE_OK) return st;
  return fe_score_select(m, B, K, Cp, scores, best, stream);
}

// ------------------------------------------------------------------------------------------
// Pipelined executor: whole passes of independent batches round-robin over its own streams
// ------------------------------------------------------------------------------------------
struct fe_executor {
  const fe_model* m;
  int n = 0, next = 0;
  hipStream_t streams[FE_EXECUTOR_MAX_STREAMS] = {};
  hipEvent_t ready[FE_EXECUTOR_MAX_STREAMS] = {};   // the caller's stream at a submission
  hipEvent_t done[FE_EXECUTOR_MAX_STREAMS] = {};    // stream i after its last pass
  bool used[FE_EXECUTOR_MAX_STREAMS] = {};
};

static void executor_release(fe_executor* ex) {
  for (int i = 0; i < FE_EXECUTOR_MAX_STREAMS; ++i) {
    if (ex->streams[i]) (void)hipStreamSynchronize(ex->streams[i]);
    if (ex->ready[i]) (void)hipEventDestroy(ex->ready[i]);
    if (ex->done[i]) (void)hipEventDestroy(ex->done[i]);
    if (ex->streams[i]) (void)hipStreamDestroy(ex->streams[i]);
  }
  delete ex;
}

fe_status fe_executor_create(const fe_model* m, int n_streams, fe_executor** out) {
  if (!m || !out) return fail(FE_EINVAL, "NULL argument");
  *out = nullptr;
  if (n_streams < 1 || n_streams > FE_EXECUTOR_MAX_STREAMS)
    return fail(FE_EINVAL, "n_streams %d outside 1..%d", n_streams, FE_EXECUTOR_MAX_STREAMS);
  fe_executor* ex = new (std::nothrow) fe_executor;
  if (!ex) return fail(FE_EINVAL, "out of host memory");
  ex->m = m;
  ex->n = n_streams;
  for (int i = 0; i < n_streams; ++i) {
    if (hipStreamCreateWithFlags(&ex->streams[i], hipStreamNonBlocking) != hipSuccess ||
        hipEventCreateWithFlags(&ex->ready[i], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&ex->done[i], hipEventDisableTiming) != hipSuccess) {
      const hipError_t e = hipGetLastError();
      executor_release(ex);
      return fail(FE_EHIP, "stream or event creation failed: %s", hipGetErrorString(e));
    }
  }
  *out = ex;
  return FE_OK;
}

fe_status fe_executor_submit(fe_executor* ex, const fe_pass_args* p, void* stream) {
  if (!ex || !p) return fail(FE_EINVAL, "NULL argument");
  const fe_model* m = ex->m;
  // the whole pass is checked before anything is enqueued, with the rules of the five calls
  fe_status st = check_dims(m, p->B, p->T, p->M, p->K, p->L);
  if (st != FE_OK) return st;
  if ((p->x == nullptr) == (p->ctx_ids == nullptr)) return fail(FE_EINVAL, "give exactly one of x and ctx_ids");
  if (p->ctx_ids && !m->emb) return fail(FE_EINVAL, "ctx_ids given but the model has no vocabulary");
  if (!p->pool && !m->emb) return fail(FE_EINVAL, "pool is NULL and the model has no vocabulary");
  if (!p->pool && p->M != m->cfg.vocab) return fail(FE_EINVAL, "token-id items need M == vocab (%d)", m->cfg.vocab);
  if (!p->lists || !p->kv || !p->uniq || !p->n_uniq || !p->slot || !p->H || !p->seq || !p->Cp || !p->scores ||
      !p->best || !p->ws)
    return fail(FE_EINVAL, "NULL pointer argument");
  if (!aligned16(p->x) || !aligned16(p->ctx_ids) || !aligned16(p->pool) || !aligned16(p->lists) ||
      !aligned16(p->kv) || !aligned16(p->uniq) || !aligned16(p->slot) || !aligned16(p->H) || !aligned16(p->seq) ||
      !aligned16(p->Cp) || !aligned16(p->ws))
    return fail(FE_EINVAL, "pointers must be 16-byte aligned");
  const Ws w = layout(m, p->B, p->T, p->M, p->K, p->L);
  if (p->ws_bytes < w.total) return fail(FE_EINVAL, "workspace of %zu bytes < %zu needed", p->ws_bytes, w.total);
  const int i = ex->next;
  hipStream_t s = ex->streams[i];
  FE_HIP(hipEventRecord(ex->ready[i], static_cast<hipStream_t>(stream)));
  FE_HIP(hipStreamWaitEvent(s, ex->ready[i], 0));
  const int U_cap = std::min(p->M, p->K * p->L);
  st = fe_encode_context(m, p->B, p->T, p->x, p->ctx_ids, p->kv, p->ws, p->ws_bytes, s);
  if (st == FE_OK)
    st = fe_encode_items(m, p->B, p->M, p->pool, p->lists, p->K, p->L, p->kv, p->T, p->uniq, p->n_uniq, p->slot, p->H,
                         p->ws, p->ws_bytes, s);
  if (st == FE_OK) st = fe_assemble(m, p->B, p->K, p->L, U_cap, p->slot, p->H, p->seq, s);
  if (st == FE_OK) st = fe_cross_sequence(m, p->B, p->K, p->L, p->seq, p->Cp, p->ws, p->ws_bytes, s);
  if (st == FE_OK) st = fe_score_select(m, p->B, p->K, p->Cp, p->scores, p->best, s);
  if (st != FE_OK) return st;
  FE_HIP(hipEventRecord(ex->done[i], s));
  ex->used[i] = true;
  ex->next = (i + 1) % ex->n;
  return FE_OK;
}

fe_status fe_executor_join(fe_executor* ex, void* stream) {
  if (!ex) return fail(FE_EINVAL, "NULL argument");
  for (int i = 0; i < ex->n; ++i)
    if (ex->used[i]) FE_HIP(hipStreamWaitEvent(static_cast<hipStream_t>(stream), ex->done[i], 0));
  return FE_OK;
}

void fe_executor_destroy(fe_executor* ex) {
  if (ex) executor_release(ex);
}

}  // extern "C"
