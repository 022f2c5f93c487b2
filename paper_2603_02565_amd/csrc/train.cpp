// The training step (Section 4.5): the joint pass of Sections 4.1-4.4 forward with its
// activations kept in the workspace, the loss with the labels of Appendix B.1, and the backward of
// every step in reverse order, all in fp32 over the flat parameter array of fe_model_create.
//
// Every request of the batch goes through each operation at once: a module's rows are laid out as
// sequences of equal length (context: B x T; item set: B x U_cap, the first n_uniq rows valid;
// SeqEnc: B K x (L+1); cross-sequence: B x K), projections are single products over all rows,
// attention is a batched product over (sequence, head) pairs with the padded keys and queries of
// the item set masked, and weight gradients sum over all rows.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <vector>

#include "fe_common.h"
#include "flasheval_train.h"
#include "train_kernels.h"

static_assert(FE_LOSS_MSE == TRAIN_MSE && FE_LOSS_BCE == TRAIN_BCE && FE_LOSS_CE == TRAIN_CE,
              "the loss kernel takes fe_loss values");

namespace {

fe_status tfail(fe_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  return fe_report(st, buf);
}

#define TRY(call)                          \
  do {                                     \
    hipError_t e_ = (call);                \
    if (e_ != hipSuccess) return e_;       \
  } while (0)

// ------------------------------------------------------------------------------------------
// Offsets (in floats) of every tensor in the flat parameter array
// ------------------------------------------------------------------------------------------
struct EncP { size_t ln1g, ln1b, wqkv, bqkv, wo, bo, ln2g, ln2b, w1, b1, w2, b2; };
struct ItemP { size_t ln1g, ln1b, wqkv, bqkv, wo, bo, ln2g, ln2b, wq, bq, wo2, bo2, ln3g, ln3b, w1, b1, w2, b2; };
struct KvP { size_t wk, bk, wv, bv; };
struct PMap {
  std::vector<EncP> ctx, seq, cross;
  std::vector<KvP> kv;
  std::vector<ItemP> item;
  size_t ctx_g, ctx_b, item_g, item_b, seq_g, seq_b, cross_g, cross_b, cls, pos, head_w, head_b, emb, total;
};

PMap param_map(const fe_config& c) {
  const size_t d = c.d, F = c.ffn_dim, n = c.n_layers;
  size_t o = 0;
  auto take = [&](size_t k) { const size_t r = o; o += k; return r; };
  auto enc = [&]() {
    EncP e;
    e.ln1g = take(d); e.ln1b = take(d); e.wqkv = take(d * 3 * d); e.bqkv = take(3 * d);
    e.wo = take(d * d); e.bo = take(d); e.ln2g = take(d); e.ln2b = take(d);
    e.w1 = take(d * F); e.b1 = take(F); e.w2 = take(F * d); e.b2 = take(d);
    return e;
  };
  PMap P;
  for (size_t l = 0; l < n; ++l) P.ctx.push_back(enc());
  P.ctx_g = take(d); P.ctx_b = take(d);
  for (size_t l = 0; l < n; ++l) {
    KvP k;
    k.wk = take(d * d); k.bk = take(d); k.wv = take(d * d); k.bv = take(d);
    P.kv.push_back(k);
  }
  for (size_t l = 0; l < n; ++l) {
    ItemP e;
    e.ln1g = take(d); e.ln1b = take(d); e.wqkv = take(d * 3 * d); e.bqkv = take(3 * d);
    e.wo = take(d * d); e.bo = take(d); e.ln2g = take(d); e.ln2b = take(d);
    e.wq = take(d * d); e.bq = take(d); e.wo2 = take(d * d); e.bo2 = take(d);
    e.ln3g = take(d); e.ln3b = take(d);
    e.w1 = take(d * F); e.b1 = take(F); e.w2 = take(F * d); e.b2 = take(d);
    P.item.push_back(e);
  }
  P.item_g = take(d); P.item_b = take(d);
  for (size_t l = 0; l < n; ++l) P.seq.push_back(enc());
  P.seq_g = take(d); P.seq_b = take(d);
  for (size_t l = 0; l < n; ++l) P.cross.push_back(enc());
  P.cross_g = take(d); P.cross_b = take(d);
  P.cls = take(d);
  P.pos = take((size_t)(c.max_L + 1) * d);
  P.head_w = take(d);
  P.head_b = take(1);
  P.emb = c.vocab > 0 ? take((size_t)c.vocab * d) : 0;
  P.total = o;
  return P;
}

// ------------------------------------------------------------------------------------------
// Workspace: one bump allocation pass, run without a base to size it
// ------------------------------------------------------------------------------------------
struct Arena {
  char* base;
  size_t off = 0;
  template <class T>
  T* get(size_t n) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

struct Dims {
  int B, T, M, K, L, d, H, dh, F, n, U, S;
  int vocab;
};

// saved activations of one encoder block (pre-LN self-attention + FFN)
struct EncAct {
  const float* x;                 // block input [R][d]
  float *h1, *m1, *r1, *qkv, *P, *o, *x2, *h2, *m2, *r2, *a1, *y;   // a1 = relu(h2 W1 + b1)
};
// saved activations of one item-set layer (self-attention, cross-attention to the context, FFN)
struct ItemAct {
  const float* x;
  float *h1, *m1, *r1, *qkv, *P, *o, *x2, *h2, *m2, *r2, *q, *Pc, *oc, *x3, *h3, *m3, *r3, *a1, *y;
  float *Kl, *Vl;                 // keys and values of the context for this layer [B][T][d]
};
// one encoder stack: nseq sequences of S rows and the final LayerNorm
struct Stack {
  int nseq, S;
  const int32_t* valid;           // per-sequence valid rows (null: all)
  std::vector<EncAct> layer;
  float *out, *mf, *rf;           // final LayerNorm output and its statistics
  bool first_row_only;            // SeqEnc: only the [CLS] row of each sequence is normalised and kept
};

struct Plan {
  Dims D;
  // index work
  int32_t *uniq, *n_uniq, *slot, *status;
  // inputs of the modules
  float *ctx_in, *item_in, *seq;
  Stack ctx, seqs, cross;
  std::vector<ItemAct> item;
  float *item_out, *item_mf, *item_rf;
  float *scores, *dscores;
  // backward scratch
  float *dx_ctx, *dx_item, *dx_seq, *dx_cross, *dQc, *dH, *dCp, *tF, *td, *tq, *dqkv, *dP, *dKl, *dVl;
};

void plan_enc_stack(Arena& A, Stack& st, const Dims& D, int nseq, int S, const int32_t* valid, bool first_row_only) {
  st.nseq = nseq;
  st.S = S;
  st.valid = valid;
  st.first_row_only = first_row_only;
  const size_t R = (size_t)nseq * S, d = D.d, F = D.F;
  st.layer.resize(D.n);
  for (int l = 0; l < D.n; ++l) {
    EncAct& a = st.layer[l];
    a.x = nullptr;
    a.h1 = A.get<float>(R * d); a.m1 = A.get<float>(R); a.r1 = A.get<float>(R);
    a.qkv = A.get<float>(R * 3 * d);
    a.P = A.get<float>((size_t)nseq * D.H * S * S);
    a.o = A.get<float>(R * d); a.x2 = A.get<float>(R * d);
    a.h2 = A.get<float>(R * d); a.m2 = A.get<float>(R); a.r2 = A.get<float>(R);
    a.a1 = A.get<float>(R * F);
    a.y = A.get<float>(R * d);
  }
  const size_t rows_out = first_row_only ? (size_t)nseq : R;
  st.out = A.get<float>(rows_out * d);
  st.mf = A.get<float>(rows_out);
  st.rf = A.get<float>(rows_out);
}

Plan make_plan(Arena& A, const Dims& D) {
  Plan p;
  p.D = D;
  const size_t B = D.B, T = D.T, K = D.K, L = D.L, d = D.d, U = D.U, S = D.S, F = D.F;
  p.uniq = A.get<int32_t>(B * U);
  p.n_uniq = A.get<int32_t>(B);
  p.slot = A.get<int32_t>(B * K * L);
  p.status = A.get<int32_t>(B);
  p.ctx_in = D.vocab ? A.get<float>(B * T * d) : nullptr;
  p.item_in = A.get<float>(B * U * d);
  p.seq = A.get<float>(B * K * S * d);
  plan_enc_stack(A, p.ctx, D, D.B, D.T, nullptr, false);
  p.item.resize(D.n);
  const size_t R = B * U;
  for (int l = 0; l < D.n; ++l) {
    ItemAct& a = p.item[l];
    a.x = nullptr;
    a.h1 = A.get<float>(R * d); a.m1 = A.get<float>(R); a.r1 = A.get<float>(R);
    a.qkv = A.get<float>(R * 3 * d);
    a.P = A.get<float>(B * D.H * U * U);
    a.o = A.get<float>(R * d); a.x2 = A.get<float>(R * d);
    a.h2 = A.get<float>(R * d); a.m2 = A.get<float>(R); a.r2 = A.get<float>(R);
    a.q = A.get<float>(R * d);
    a.Pc = A.get<float>(B * D.H * U * T);
    a.oc = A.get<float>(R * d); a.x3 = A.get<float>(R * d);
    a.h3 = A.get<float>(R * d); a.m3 = A.get<float>(R); a.r3 = A.get<float>(R);
    a.a1 = A.get<float>(R * F);
    a.y = A.get<float>(R * d);
    a.Kl = A.get<float>(B * T * d);
    a.Vl = A.get<float>(B * T * d);
  }
  p.item_out = A.get<float>(R * d);
  p.item_mf = A.get<float>(R);
  p.item_rf = A.get<float>(R);
  plan_enc_stack(A, p.seqs, D, D.B * D.K, D.S, nullptr, true);
  plan_enc_stack(A, p.cross, D, D.B, D.K, nullptr, false);
  p.scores = A.get<float>(B * K);
  p.dscores = A.get<float>(B * K);
  // backward scratch: sized for the largest module
  const size_t Rc = B * T, Rs = B * K * S, Rx = B * K;
  const size_t Rmax = std::max(std::max(Rc, R), std::max(Rs, Rx));
  const size_t Pmax = std::max(std::max(B * D.H * T * T, B * D.H * U * std::max(U, T)),
                               std::max(B * K * D.H * S * S, B * D.H * K * K));
  p.dx_ctx = A.get<float>(Rc * d);
  p.dx_item = A.get<float>(R * d);
  p.dx_seq = A.get<float>(Rs * d);
  p.dx_cross = A.get<float>(Rx * d);
  p.dQc = A.get<float>(Rc * d);
  p.dH = A.get<float>(R * d);
  p.dCp = A.get<float>(Rx * d);
  p.tF = A.get<float>(Rmax * F);
  p.td = A.get<float>(Rmax * d);
  p.tq = A.get<float>(R * d);
  p.dqkv = A.get<float>(Rmax * 3 * d);
  p.dP = A.get<float>(Pmax);
  p.dKl = A.get<float>(Rc * d);
  p.dVl = A.get<float>(Rc * d);
  return p;
}

// ------------------------------------------------------------------------------------------
// Products
// ------------------------------------------------------------------------------------------
TGemm gemm0() {
  TGemm g;
  std::memset(&g, 0, sizeof g);
  g.nbatch = 1;
  g.nb2 = 1;
  g.alpha = 1.f;
  return g;
}

// Y = [relu](X W + b [+ resid]), X [R][din] rows of stride x_rs, W [din][dout] row-major, resid
// laid out as Y
hipError_t linear(const float* X, long long x_rs, int R, int din, const float* W, const float* b, int dout, float* Y,
                  long long y_rs, const float* resid, bool relu, hipStream_t s) {
  TGemm g = gemm0();
  g.A = X; g.a_rs = x_rs; g.a_cs = 1;
  g.B = W; g.b_rs = dout; g.b_cs = 1;
  g.C = Y; g.c_rs = y_rs;
  g.bias = b;
  g.R = resid;
  g.relu = relu;
  g.M = R; g.N = dout; g.K = din;
  return t_gemm(g, s);
}

// dX (=, or += when accumulate) dY W^T, zeroed where mask <= 0 (the backward of a ReLU whose
// output is mask; null: none)
hipError_t linear_dx(const float* dY, long long dy_rs, int R, int dout, const float* W, int din, float* dX,
                     long long dx_rs, bool accumulate, const float* mask, hipStream_t s) {
  TGemm g = gemm0();
  g.A = dY; g.a_rs = dy_rs; g.a_cs = 1;
  g.B = W; g.b_rs = 1; g.b_cs = dout;
  g.C = dX; g.c_rs = dx_rs;
  g.mask = mask;
  g.M = R; g.N = din; g.K = dout;
  g.beta = accumulate ? 1.f : 0.f;
  return t_gemm(g, s);
}

// dW += X^T dY over the R rows, db += column sums of dY (db may be null; summed by the same launch)
hipError_t linear_dw(const float* X, long long x_rs, int R, int din, const float* dY, long long dy_rs, int dout,
                     float* dW, float* db, hipStream_t s) {
  TGemm g = gemm0();
  g.A = X; g.a_rs = 1; g.a_cs = x_rs;
  g.B = dY; g.b_rs = dy_rs; g.b_cs = 1;
  g.C = dW; g.c_rs = dout;
  g.M = din; g.N = dout; g.K = R;
  g.beta = 1.f;
  // enough (row chunk x output tile) workgroups to fill the chip; chunks of at least 256 rows
  const long long tiles = (long long)((din + 63) / 64) * ((dout + 63) / 64);
  long long chunks = std::max(1LL, 2048 / tiles);
  long long ks = std::max(256LL, (R + chunks - 1) / chunks);
  g.ksplit = (int)((ks + 31) / 32 * 32);
  g.colsum = db;
  return t_gemm(g, s);
}

// Multi-head attention over nseq sequences, all heads at once.  Query rows of sequence z start at
// q + z*q_bs (row stride q_rs, head h in columns h*dh..), likewise keys and values; Sq queries and
// Sk keys per sequence; P [nseq][H][Sq][Sk]; o rows at o + z*o_bs (stride o_rs).
struct AttnIO {
  const float *q, *k, *v;
  long long q_rs, k_rs, v_rs, q_bs, k_bs, v_bs;
  int nseq, Sq, Sk;
  const int32_t *qlen, *klen;
};

hipError_t attn_fwd(const AttnIO& a, const Dims& D, float* P, float* o, long long o_rs, long long o_bs, hipStream_t s) {
  const long long pz = (long long)a.Sq * a.Sk;
  TGemm g = gemm0();
  g.A = a.q; g.a_rs = a.q_rs; g.a_cs = 1; g.a_b1 = a.q_bs; g.a_b2 = D.dh;
  g.B = a.k; g.b_rs = 1; g.b_cs = a.k_rs; g.b_b1 = a.k_bs; g.b_b2 = D.dh;
  g.C = P; g.c_rs = a.Sk; g.c_b1 = D.H * pz; g.c_b2 = pz;
  g.M = a.Sq; g.N = a.Sk; g.K = D.dh;
  g.nbatch = a.nseq * D.H; g.nb2 = D.H;
  TRY(t_gemm(g, s));
  TRY(t_softmax_fwd(P, P, a.nseq * D.H, D.H, a.Sq, a.Sk, 1.f / std::sqrt((float)D.dh), a.qlen, a.klen, s));
  TGemm h = gemm0();
  h.A = P; h.a_rs = a.Sk; h.a_cs = 1; h.a_b1 = D.H * pz; h.a_b2 = pz;
  h.B = a.v; h.b_rs = a.v_rs; h.b_cs = 1; h.b_b1 = a.v_bs; h.b_b2 = D.dh;
  h.C = o; h.c_rs = o_rs; h.c_b1 = o_bs; h.c_b2 = D.dh;
  h.M = a.Sq; h.N = D.dh; h.K = a.Sk;
  h.nbatch = a.nseq * D.H; h.nb2 = D.H;
  return t_gemm(h, s);
}

// dq, dk, dv (overwritten; same strides as q, k, v) from dO and the saved P; dP is scratch.
hipError_t attn_bwd(const AttnIO& a, const Dims& D, const float* P, const float* dO, long long do_rs, long long do_bs,
                    float* dq, float* dk, float* dv, float* dP, hipStream_t s) {
  const long long pz = (long long)a.Sq * a.Sk;
  const int nb = a.nseq * D.H;
  // dP = dO V^T
  TGemm g = gemm0();
  g.A = dO; g.a_rs = do_rs; g.a_cs = 1; g.a_b1 = do_bs; g.a_b2 = D.dh;
  g.B = a.v; g.b_rs = 1; g.b_cs = a.v_rs; g.b_b1 = a.v_bs; g.b_b2 = D.dh;
  g.C = dP; g.c_rs = a.Sk; g.c_b1 = D.H * pz; g.c_b2 = pz;
  g.M = a.Sq; g.N = a.Sk; g.K = D.dh;
  g.nbatch = nb; g.nb2 = D.H;
  TRY(t_gemm(g, s));
  // dV = P^T dO
  g = gemm0();
  g.A = P; g.a_rs = 1; g.a_cs = a.Sk; g.a_b1 = D.H * pz; g.a_b2 = pz;
  g.B = dO; g.b_rs = do_rs; g.b_cs = 1; g.b_b1 = do_bs; g.b_b2 = D.dh;
  g.C = dv; g.c_rs = a.v_rs; g.c_b1 = a.v_bs; g.c_b2 = D.dh;
  g.M = a.Sk; g.N = D.dh; g.K = a.Sq;
  g.nbatch = nb; g.nb2 = D.H;
  TRY(t_gemm(g, s));
  // dS = scale P (dP - rowsum(P dP))
  TRY(t_softmax_bwd(P, dP, (long long)nb * a.Sq, a.Sk, 1.f / std::sqrt((float)D.dh), s));
  // dQ = dS K
  g = gemm0();
  g.A = dP; g.a_rs = a.Sk; g.a_cs = 1; g.a_b1 = D.H * pz; g.a_b2 = pz;
  g.B = a.k; g.b_rs = a.k_rs; g.b_cs = 1; g.b_b1 = a.k_bs; g.b_b2 = D.dh;
  g.C = dq; g.c_rs = a.q_rs; g.c_b1 = a.q_bs; g.c_b2 = D.dh;
  g.M = a.Sq; g.N = D.dh; g.K = a.Sk;
  g.nbatch = nb; g.nb2 = D.H;
  TRY(t_gemm(g, s));
  // dK = dS^T Q
  g = gemm0();
  g.A = dP; g.a_rs = 1; g.a_cs = a.Sk; g.a_b1 = D.H * pz; g.a_b2 = pz;
  g.B = a.q; g.b_rs = a.q_rs; g.b_cs = 1; g.b_b1 = a.q_bs; g.b_b2 = D.dh;
  g.C = dk; g.c_rs = a.k_rs; g.c_b1 = a.k_bs; g.c_b2 = D.dh;
  g.M = a.Sk; g.N = D.dh; g.K = a.Sq;
  g.nbatch = nb; g.nb2 = D.H;
  return t_gemm(g, s);
}

// self-attention of the rows of a qkv buffer [nseq][S][3d]
AttnIO self_io(const float* qkv, const Dims& D, int nseq, int S, const int32_t* valid) {
  AttnIO a;
  const long long rs = 3LL * D.d;
  a.q = qkv; a.k = qkv + D.d; a.v = qkv + 2 * D.d;
  a.q_rs = a.k_rs = a.v_rs = rs;
  a.q_bs = a.k_bs = a.v_bs = rs * S;
  a.nseq = nseq; a.Sq = a.Sk = S;
  a.qlen = a.klen = valid;
  return a;
}

// ------------------------------------------------------------------------------------------
// Encoder block (pre-LN): x2 = x + MHA(LN1 x) Wo + bo;  y = x2 + relu(LN2 x2 W1 + b1) W2 + b2
// ------------------------------------------------------------------------------------------
hipError_t enc_fwd(const float* W, const EncP& p, EncAct& a, const Dims& D, int nseq, int S, const int32_t* valid,
                   hipStream_t s) {
  const int R = nseq * S, d = D.d, F = D.F;
  TRY(t_ln_fwd(a.x, d, R, d, W + p.ln1g, W + p.ln1b, a.h1, d, a.m1, a.r1, s));
  TRY(linear(a.h1, d, R, d, W + p.wqkv, W + p.bqkv, 3 * d, a.qkv, 3 * d, nullptr, false, s));
  TRY(attn_fwd(self_io(a.qkv, D, nseq, S, valid), D, a.P, a.o, d, (long long)S * d, s));
  TRY(linear(a.o, d, R, d, W + p.wo, W + p.bo, d, a.x2, d, a.x, false, s));
  TRY(t_ln_fwd(a.x2, d, R, d, W + p.ln2g, W + p.ln2b, a.h2, d, a.m2, a.r2, s));
  TRY(linear(a.h2, d, R, d, W + p.w1, W + p.b1, F, a.a1, F, nullptr, true, s));
  return linear(a.a1, F, R, F, W + p.w2, W + p.b2, d, a.y, d, a.x2, false, s);
}

// dx holds d loss / d y on entry and d loss / d x on return; parameter gradients are added to G.
hipError_t enc_bwd(const float* W, float* G, const EncP& p, const EncAct& a, const Dims& D, int nseq, int S,
                   const int32_t* valid, float* dx, Plan& pl, hipStream_t s) {
  const int R = nseq * S, d = D.d, F = D.F;
  // FFN
  TRY(linear_dw(a.a1, F, R, F, dx, d, d, G + p.w2, G + p.b2, s));
  TRY(linear_dx(dx, d, R, d, W + p.w2, F, pl.tF, F, false, a.a1, s));
  TRY(linear_dw(a.h2, d, R, d, pl.tF, F, F, G + p.w1, G + p.b1, s));
  TRY(linear_dx(pl.tF, F, R, F, W + p.w1, d, pl.td, d, false, nullptr, s));
  TRY(t_ln_bwd(a.x2, d, R, d, W + p.ln2g, a.m2, a.r2, pl.td, d, dx, d, G + p.ln2g, G + p.ln2b, s));
  // self-attention
  TRY(linear_dw(a.o, d, R, d, dx, d, d, G + p.wo, G + p.bo, s));
  TRY(linear_dx(dx, d, R, d, W + p.wo, d, pl.td, d, false, nullptr, s));
  const AttnIO io = self_io(a.qkv, D, nseq, S, valid);
  TRY(attn_bwd(io, D, a.P, pl.td, d, (long long)S * d, pl.dqkv, pl.dqkv + d, pl.dqkv + 2 * d, pl.dP, s));
  TRY(linear_dw(a.h1, d, R, d, pl.dqkv, 3 * d, 3 * d, G + p.wqkv, G + p.bqkv, s));
  TRY(linear_dx(pl.dqkv, 3 * d, R, 3 * d, W + p.wqkv, d, pl.td, d, false, nullptr, s));
  return t_ln_bwd(a.x, d, R, d, W + p.ln1g, a.m1, a.r1, pl.td, d, dx, d, G + p.ln1g, G + p.ln1b, s);
}

hipError_t stack_fwd(const float* W, const std::vector<EncP>& ps, size_t g_off, size_t b_off, Stack& st, const float* in,
                     const Dims& D, hipStream_t s) {
  const float* x = in;
  for (int l = 0; l < D.n; ++l) {
    st.layer[l].x = x;
    TRY(enc_fwd(W, ps[l], st.layer[l], D, st.nseq, st.S, st.valid, s));
    x = st.layer[l].y;
  }
  if (st.first_row_only)
    return t_ln_fwd(x, (long long)st.S * D.d, st.nseq, D.d, W + g_off, W + b_off, st.out, D.d, st.mf, st.rf, s);
  return t_ln_fwd(x, D.d, st.nseq * st.S, D.d, W + g_off, W + b_off, st.out, D.d, st.mf, st.rf, s);
}

// dout: d loss / d (stack output); dx receives d loss / d (stack input) (overwritten)
hipError_t stack_bwd(const float* W, float* G, const std::vector<EncP>& ps, size_t g_off, size_t b_off, const Stack& st,
                     const float* dout, float* dx, const Dims& D, Plan& pl, hipStream_t s) {
  const long long R = (long long)st.nseq * st.S;
  TRY(t_fill(dx, R * D.d, 0.f, s));
  const float* xl = st.layer[D.n - 1].y;
  if (st.first_row_only)
    TRY(t_ln_bwd(xl, (long long)st.S * D.d, st.nseq, D.d, W + g_off, st.mf, st.rf, dout, D.d, dx, (long long)st.S * D.d,
                 G + g_off, G + b_off, s));
  else
    TRY(t_ln_bwd(xl, D.d, (int)R, D.d, W + g_off, st.mf, st.rf, dout, D.d, dx, D.d, G + g_off, G + b_off, s));
  for (int l = D.n - 1; l >= 0; --l) TRY(enc_bwd(W, G, ps[l], st.layer[l], D, st.nseq, st.S, st.valid, dx, pl, s));
  return hipSuccess;
}

// ------------------------------------------------------------------------------------------
// Item-set layer (Section 4.2): set self-attention, cross-attention of the items to the encoded
// context through this layer's key/value projections, FFN; all pre-LN with residuals
// ------------------------------------------------------------------------------------------
AttnIO cross_io(const ItemAct& a, const Dims& D, const int32_t* n_uniq) {
  AttnIO io;
  io.q = a.q; io.q_rs = D.d; io.q_bs = (long long)D.U * D.d;
  io.k = a.Kl; io.k_rs = D.d; io.k_bs = (long long)D.T * D.d;
  io.v = a.Vl; io.v_rs = D.d; io.v_bs = (long long)D.T * D.d;
  io.nseq = D.B; io.Sq = D.U; io.Sk = D.T;
  io.qlen = n_uniq;
  io.klen = nullptr;
  return io;
}

hipError_t item_fwd(const float* W, const ItemP& p, const KvP& kv, ItemAct& a, const float* Qc, const Dims& D,
                    const int32_t* n_uniq, hipStream_t s) {
  const int R = D.B * D.U, d = D.d, F = D.F, Rc = D.B * D.T;
  TRY(linear(Qc, d, Rc, d, W + kv.wk, W + kv.bk, d, a.Kl, d, nullptr, false, s));
  TRY(linear(Qc, d, Rc, d, W + kv.wv, W + kv.bv, d, a.Vl, d, nullptr, false, s));
  TRY(t_ln_fwd(a.x, d, R, d, W + p.ln1g, W + p.ln1b, a.h1, d, a.m1, a.r1, s));
  TRY(linear(a.h1, d, R, d, W + p.wqkv, W + p.bqkv, 3 * d, a.qkv, 3 * d, nullptr, false, s));
  TRY(attn_fwd(self_io(a.qkv, D, D.B, D.U, n_uniq), D, a.P, a.o, d, (long long)D.U * d, s));
  TRY(linear(a.o, d, R, d, W + p.wo, W + p.bo, d, a.x2, d, a.x, false, s));
  TRY(t_ln_fwd(a.x2, d, R, d, W + p.ln2g, W + p.ln2b, a.h2, d, a.m2, a.r2, s));
  TRY(linear(a.h2, d, R, d, W + p.wq, W + p.bq, d, a.q, d, nullptr, false, s));
  TRY(attn_fwd(cross_io(a, D, n_uniq), D, a.Pc, a.oc, d, (long long)D.U * d, s));
  TRY(linear(a.oc, d, R, d, W + p.wo2, W + p.bo2, d, a.x3, d, a.x2, false, s));
  TRY(t_ln_fwd(a.x3, d, R, d, W + p.ln3g, W + p.ln3b, a.h3, d, a.m3, a.r3, s));
  TRY(linear(a.h3, d, R, d, W + p.w1, W + p.b1, F, a.a1, F, nullptr, true, s));
  return linear(a.a1, F, R, F, W + p.w2, W + p.b2, d, a.y, d, a.x3, false, s);
}

// dx: d / d (layer output) in, d / d (layer input) out; d / d (encoded context) added to dQc
hipError_t item_bwd(const float* W, float* G, const ItemP& p, const KvP& kv, const ItemAct& a, const float* Qc,
                    const Dims& D, const int32_t* n_uniq, float* dx, Plan& pl, hipStream_t s) {
  const int R = D.B * D.U, d = D.d, F = D.F, Rc = D.B * D.T;
  // FFN
  TRY(linear_dw(a.a1, F, R, F, dx, d, d, G + p.w2, G + p.b2, s));
  TRY(linear_dx(dx, d, R, d, W + p.w2, F, pl.tF, F, false, a.a1, s));
  TRY(linear_dw(a.h3, d, R, d, pl.tF, F, F, G + p.w1, G + p.b1, s));
  TRY(linear_dx(pl.tF, F, R, F, W + p.w1, d, pl.td, d, false, nullptr, s));
  TRY(t_ln_bwd(a.x3, d, R, d, W + p.ln3g, a.m3, a.r3, pl.td, d, dx, d, G + p.ln3g, G + p.ln3b, s));
  // cross-attention to the context
  TRY(linear_dw(a.oc, d, R, d, dx, d, d, G + p.wo2, G + p.bo2, s));
  TRY(linear_dx(dx, d, R, d, W + p.wo2, d, pl.td, d, false, nullptr, s));
  TRY(attn_bwd(cross_io(a, D, n_uniq), D, a.Pc, pl.td, d, (long long)D.U * d, pl.tq, pl.dKl, pl.dVl, pl.dP, s));
  TRY(linear_dw(a.h2, d, R, d, pl.tq, d, d, G + p.wq, G + p.bq, s));
  TRY(linear_dx(pl.tq, d, R, d, W + p.wq, d, pl.td, d, false, nullptr, s));
  TRY(t_ln_bwd(a.x2, d, R, d, W + p.ln2g, a.m2, a.r2, pl.td, d, dx, d, G + p.ln2g, G + p.ln2b, s));
  TRY(linear_dw(Qc, d, Rc, d, pl.dKl, d, d, G + kv.wk, G + kv.bk, s));
  TRY(linear_dw(Qc, d, Rc, d, pl.dVl, d, d, G + kv.wv, G + kv.bv, s));
  TRY(linear_dx(pl.dKl, d, Rc, d, W + kv.wk, d, pl.dQc, d, true, nullptr, s));
  TRY(linear_dx(pl.dVl, d, Rc, d, W + kv.wv, d, pl.dQc, d, true, nullptr, s));
  // set self-attention
  TRY(linear_dw(a.o, d, R, d, dx, d, d, G + p.wo, G + p.bo, s));
  TRY(linear_dx(dx, d, R, d, W + p.wo, d, pl.td, d, false, nullptr, s));
  TRY(attn_bwd(self_io(a.qkv, D, D.B, D.U, n_uniq), D, a.P, pl.td, d, (long long)D.U * d, pl.dqkv, pl.dqkv + d,
               pl.dqkv + 2 * d, pl.dP, s));
  TRY(linear_dw(a.h1, d, R, d, pl.dqkv, 3 * d, 3 * d, G + p.wqkv, G + p.bqkv, s));
  TRY(linear_dx(pl.dqkv, 3 * d, R, 3 * d, W + p.wqkv, d, pl.td, d, false, nullptr, s));
  return t_ln_bwd(a.x, d, R, d, W + p.ln1g, a.m1, a.r1, pl.td, d, dx, d, G + p.ln1g, G + p.ln1b, s);
}

// ------------------------------------------------------------------------------------------
// The whole step
// ------------------------------------------------------------------------------------------
struct Inputs {
  const float *x, *pool;
  const int32_t *ctx_ids, *lists, *relevant;
  int kind;
  float *loss, *scores_out;
};

hipError_t run_step(const float* W, float* G, const PMap& pm, Plan& pl, const Inputs& in, size_t n_params,
                    hipStream_t s) {
  const Dims& D = pl.D;
  const int d = D.d;
  TRY(t_fill(G, (long long)n_params, 0.f, s));
  TRY(t_fill(in.loss, 1, 0.f, s));
  // ---- forward
  // context rows (Section 4.1): given rows, or the embedding rows of the token ids
  const float* x0 = in.x;
  if (D.vocab) {
    TRY(t_gather(W + pm.emb, 0, D.vocab, in.ctx_ids, D.T, nullptr, D.B, D.T, d, pl.ctx_in, s));
    x0 = pl.ctx_in;
  }
  TRY(stack_fwd(W, pm.ctx, pm.ctx_g, pm.ctx_b, pl.ctx, x0, D, s));
  const float* Qc = pl.ctx.out;
  // distinct elements of each request, in ascending id, and every list entry's slot among them
  TRY(launch_dedup(in.lists, D.B, D.K * D.L, D.M, D.U, pl.uniq, pl.n_uniq, pl.slot, pl.status, s));
  if (D.vocab)
    TRY(t_gather(W + pm.emb, 0, D.vocab, pl.uniq, D.U, pl.n_uniq, D.B, D.U, d, pl.item_in, s));
  else
    TRY(t_gather(in.pool, (long long)D.M * d, D.M, pl.uniq, D.U, pl.n_uniq, D.B, D.U, d, pl.item_in, s));
  const float* g = pl.item_in;
  for (int l = 0; l < D.n; ++l) {
    pl.item[l].x = g;
    TRY(item_fwd(W, pm.item[l], pm.kv[l], pl.item[l], Qc, D, pl.n_uniq, s));
    g = pl.item[l].y;
  }
  const int Ri = D.B * D.U;
  TRY(t_ln_fwd(g, d, Ri, d, W + pm.item_g, W + pm.item_b, pl.item_out, d, pl.item_mf, pl.item_rf, s));
  // candidate sequences (Section 4.3) and SeqEnc: the [CLS] row of each list
  TRY(t_assemble(pl.item_out, D.B, D.U, pl.slot, D.K, D.L, d, W + pm.cls, W + pm.pos, pl.seq, s));
  TRY(stack_fwd(W, pm.seq, pm.seq_g, pm.seq_b, pl.seqs, pl.seq, D, s));
  // cross-sequence module over the K lists of each request (Section 4.4) and the linear head
  TRY(stack_fwd(W, pm.cross, pm.cross_g, pm.cross_b, pl.cross, pl.seqs.out, D, s));
  const int Rx = D.B * D.K;
  TRY(linear(pl.cross.out, d, Rx, d, W + pm.head_w, W + pm.head_b, 1, pl.scores, 1, nullptr, false, s));
  if (in.scores_out)
    TRY(t_copy(pl.scores, in.scores_out, (long long)Rx, s));
  // ---- loss (Section 4.5) with the labels of Appendix B.1
  TRY(t_loss(pl.scores, in.lists, in.relevant, D.M, D.B, D.K, D.L, in.kind, in.loss, pl.dscores, s));
  // ---- backward
  // head: s = Cp w + b
  {
    TGemm gg = gemm0();  // dCp = ds w^T
    gg.A = pl.dscores; gg.a_rs = 1; gg.a_cs = 1;
    gg.B = W + pm.head_w; gg.b_rs = d; gg.b_cs = 1;
    gg.C = pl.dCp; gg.c_rs = d;
    gg.M = Rx; gg.N = d; gg.K = 1;
    TRY(t_gemm(gg, s));
    TRY(linear_dw(pl.cross.out, d, Rx, d, pl.dscores, 1, 1, G + pm.head_w, G + pm.head_b, s));
  }
  TRY(stack_bwd(W, G, pm.cross, pm.cross_g, pm.cross_b, pl.cross, pl.dCp, pl.dx_cross, D, pl, s));
  TRY(stack_bwd(W, G, pm.seq, pm.seq_g, pm.seq_b, pl.seqs, pl.dx_cross, pl.dx_seq, D, pl, s));
  TRY(t_fill(pl.dH, (long long)Ri * d, 0.f, s));
  TRY(t_assemble_bwd(pl.dx_seq, D.B, D.U, pl.slot, D.K, D.L, d, pl.dH, G + pm.cls, G + pm.pos, s));
  TRY(t_fill(pl.dx_item, (long long)Ri * d, 0.f, s));
  TRY(t_ln_bwd(pl.item[D.n - 1].y, d, Ri, d, W + pm.item_g, pl.item_mf, pl.item_rf, pl.dH, d, pl.dx_item, d,
               G + pm.item_g, G + pm.item_b, s));
  TRY(t_fill(pl.dQc, (long long)D.B * D.T * d, 0.f, s));
  for (int l = D.n - 1; l >= 0; --l)
    TRY(item_bwd(W, G, pm.item[l], pm.kv[l], pl.item[l], Qc, D, pl.n_uniq, pl.dx_item, pl, s));
  if (D.vocab)
    TRY(t_scatter_add(pl.dx_item, pl.uniq, D.U, pl.n_uniq, D.B, D.U, d, G + pm.emb, 0, D.vocab, s));
  TRY(stack_bwd(W, G, pm.ctx, pm.ctx_g, pm.ctx_b, pl.ctx, pl.dQc, pl.dx_ctx, D, pl, s));
  if (D.vocab) TRY(t_scatter_add(pl.dx_ctx, in.ctx_ids, D.T, nullptr, D.B, D.T, d, G + pm.emb, 0, D.vocab, s));
  return hipSuccess;
}

fe_status check(const fe_config* cfg, int B, int T, int M, int K, int L, Dims* D) {
  size_t n = 0;
  const fe_status st = fe_param_count(cfg, &n);  // the model envelope
  if (st != FE_OK) return st;
  if (cfg->dtype != FE_F32) return tfail(FE_EUNSUPPORTED, "the training step runs FE_F32 models");
  if (cfg->attention != FE_ATTN_SOFTMAX) return tfail(FE_EUNSUPPORTED, "the training step covers softmax attention");
  if (B < 1 || T < 1 || M < 1 || K < 1 || L < 1) return tfail(FE_EINVAL, "B, T, M, K, L must be >= 1");
  if (L > cfg->max_L) return tfail(FE_EINVAL, "L=%d exceeds max_L=%d", L, cfg->max_L);
  if (T > 8192) return tfail(FE_EUNSUPPORTED, "T=%d > 8192", T);
  if (K > 1024) return tfail(FE_EUNSUPPORTED, "K=%d > 1024", K);
  if (M > 131072) return tfail(FE_EUNSUPPORTED, "M=%d > 131072", M);
  if (cfg->vocab > 0 && M != cfg->vocab) return tfail(FE_EINVAL, "token-id items need M = vocab (%d), got %d", cfg->vocab, M);
  const long long U = std::min<long long>(M, (long long)K * L), rows_max = 0x7fffffffLL / 4;
  if ((long long)B * K * (L + 1) > rows_max || (long long)B * T > rows_max || (long long)B * U > rows_max)
    return tfail(FE_EUNSUPPORTED, "B=%d gives more than %lld rows in a module", B, rows_max);
  D->B = B; D->T = T; D->M = M; D->K = K; D->L = L;
  D->d = cfg->d; D->H = cfg->n_heads; D->dh = cfg->d / cfg->n_heads; D->F = cfg->ffn_dim; D->n = cfg->n_layers;
  D->U = (int)std::min<long long>(M, (long long)K * L);
  D->S = L + 1;
  D->vocab = cfg->vocab;
  return FE_OK;
}

}  // namespace

extern "C" {

fe_status fe_train_workspace_size(const fe_config* cfg, int B, int T, int M, int K, int L, size_t* bytes) {
  Dims D;
  const fe_status st = check(cfg, B, T, M, K, L, &D);
  if (st != FE_OK) return st;
  if (!bytes) return tfail(FE_EINVAL, "bytes is NULL");
  Arena A{nullptr};
  make_plan(A, D);
  *bytes = (A.off + 255) & ~size_t(255);
  return FE_OK;
}

fe_status fe_train_grads(const fe_config* cfg, const float* params, int B, int T, int M, int K, int L,
                         const float* x, const int32_t* ctx_ids, const float* pool, const int32_t* lists,
                         const int32_t* relevant, int loss_kind, float* loss, float* scores, float* grads, void* ws,
                         size_t ws_bytes, void* stream) {
  Dims D;
  fe_status st = check(cfg, B, T, M, K, L, &D);
  if (st != FE_OK) return st;
  if (!params || !grads || !lists || !relevant || !loss || !ws) return tfail(FE_EINVAL, "a required pointer is NULL");
  if (cfg->vocab > 0 ? !ctx_ids : (!x || !pool))
    return tfail(FE_EINVAL, cfg->vocab > 0 ? "ctx_ids is NULL" : "x or pool is NULL");
  if (loss_kind < FE_LOSS_MSE || loss_kind > FE_LOSS_CE) return tfail(FE_EINVAL, "loss_kind %d out of range", loss_kind);
  if (reinterpret_cast<uintptr_t>(ws) % 256) return tfail(FE_EINVAL, "workspace is not 256-byte aligned");
  Arena probe{nullptr};
  make_plan(probe, D);
  if (ws_bytes < probe.off) return tfail(FE_EINVAL, "workspace of %zu bytes < %zu needed", ws_bytes, probe.off);
  Arena A{static_cast<char*>(ws)};
  Plan pl = make_plan(A, D);
  const PMap pm = param_map(*cfg);
  Inputs in{x, pool, ctx_ids, lists, relevant, loss_kind, loss, scores};
  const hipError_t e = run_step(params, grads, pm, pl, in, pm.total, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return tfail(FE_EHIP, "training step launch failed: %s", hipGetErrorString(e));
  return FE_OK;
}

}  // extern "C"
