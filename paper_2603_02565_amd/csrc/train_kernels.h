// Launchers of the fp32 training kernels (train_kernels.hip), used by the training step (train.cpp).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>
#include <type_traits>

#include "flasheval.h"

// sets the text fe_last_error returns and passes st through
fe_status fe_report(fe_status st, const char* msg);

enum { TRAIN_MSE = 0, TRAIN_BCE = 1, TRAIN_CE = 2 };
constexpr int TRAIN_COL_ROWS = 64;   // rows per workgroup of a column reduction

// C[z] = alpha * A[z] B[z] + beta * C[z] + bias (bias[j] over columns, may be null), z < nbatch,
// z = z1 * nb2 + z2.  Element (i, k) of A[z] is A[z1*a_b1 + z2*a_b2 + i*a_rs + k*a_cs]; B (k, j)
// and C (i, j) likewise (C with unit column stride).  ksplit > 0: the K range is cut into chunks
// of ksplit (a multiple of 32) and each chunk adds alpha * its partial product into C atomically (beta must be 1,
// bias and the epilogue null); the sum order then varies from run to run.
struct TGemm {
  const float* A;
  const float* B;
  float* C;
  const float* bias;
  // epilogue, in this order after alpha and bias: + R (residual, laid out as C); relu; times
  // [mask > 0] (mask laid out as C).  Null / 0: not applied.  Not with ksplit.
  const float* R;
  int relu;
  const float* mask;
  // colsum (k_gemm only, nbatch 1): colsum[j] += alpha * sum_k B[k][j] over this launch's k range (the
  // bias gradient when B is dY and k runs over rows); null: not computed.
  float* colsum;
  int M, N, K;
  long long a_rs, a_cs, b_rs, b_cs, c_rs;
  long long a_b1, a_b2, b_b1, b_b2, c_b1, c_b2;
  int nbatch, nb2;
  float alpha, beta;
  int ksplit;
};

hipError_t t_gemm(const TGemm& g, hipStream_t s);
// Y = LN(X) * g + b per row of d values (eps 1e-5); mean and 1/std per row saved
hipError_t t_ln_fwd(const float* X, long long x_rs, int rows, int d, const float* g, const float* b, float* Y,
                    long long y_rs, float* mean, float* rstd, hipStream_t s);
// dX += the LayerNorm input gradient of dY; dg, db += the parameter gradients (atomically)
hipError_t t_ln_bwd(const float* X, long long x_rs, int rows, int d, const float* g, const float* mean,
                    const float* rstd, const float* dY, long long dy_rs, float* dX, long long dx_rs, float* dg,
                    float* db, hipStream_t s);
// P = softmax(scale * S) per row of nk keys; rows of batch z (z1 = z / nb2) use keys j < klen[z1]
// and are zero for query rows i >= qlen[z1] (null: no bound)
hipError_t t_softmax_fwd(const float* S, float* P, int nbatch, int nb2, int nq, int nk, float scale,
                         const int32_t* qlen, const int32_t* klen, hipStream_t s);
// dP <- scale * P * (dP - rowsum(P * dP)): the gradient of the pre-scale scores, in place
hipError_t t_softmax_bwd(const float* P, float* dP, long long rows, int nk, float scale, hipStream_t s);
hipError_t t_copy(const float* x, float* y, long long n, hipStream_t s);
hipError_t t_fill(float* y, long long n, float v, hipStream_t s);
// Y[b][r] = row idx[b*idx_bs + r] of the table at T + b*t_bs, for r < nvalid[b] (all rows if null)
// and ids in [0, n_table); other rows are zero
hipError_t t_gather(const float* T, long long t_bs, int n_table, const int32_t* idx, int idx_bs, const int32_t* nvalid,
                    int B, int rows, int d, float* Y, hipStream_t s);
// its backward: the rows of dY added into the rows of dT the gather read (atomically)
hipError_t t_scatter_add(const float* dY, const int32_t* idx, int idx_bs, const int32_t* nvalid, int B, int rows, int d,
                         float* dT, long long t_bs, int n_table, hipStream_t s);
// seq [B][K][L+1][d] from H [B][U_cap][d] by slot [B][K][L]; row 0 = cls + pos[0]
hipError_t t_assemble(const float* H, int B, int U_cap, const int32_t* slot, int K, int L, int d, const float* cls,
                      const float* pos, float* seq, hipStream_t s);
hipError_t t_assemble_bwd(const float* dseq, int B, int U_cap, const int32_t* slot, int K, int L, int d, float* dH,
                          float* dcls, float* dpos, hipStream_t s);
// batch loss (added to *loss) and dloss/dscores; K <= 1024
hipError_t t_loss(const float* scores, const int32_t* lists, const int32_t* relevant, int M, int B, int K, int L, int kind,
                  float* loss, float* dscores, hipStream_t s);
