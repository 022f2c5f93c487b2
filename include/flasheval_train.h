/*
 * flasheval_train.h -- the training step of the evaluator: loss and gradient of every parameter
 * for one batch, on the GPU, in fp32.
 *
 * Section 4.5 trains the evaluator end to end on list-level targets built from item-level
 * feedback.  fe_train_grads runs the joint pass of Sections 4.1-4.4 (context encoder, item-set
 * encoder with its cross-attention to the context, candidate assembly, SeqEnc, cross-sequence
 * module, linear head) forward with its activations kept, then the loss, then the backward of
 * every step, and writes d loss / d theta for the whole flat parameter array.
 *
 * Labels (Appendix B.1): with a_{k,j} = relevant[b][lists[b][k][j]] the binary feedback of the
 * j-th element of list k, r_k = sum_j a_{k,j}, and y = the smallest k with the largest r_k.
 * Losses per request (Section 4.5), averaged over the B requests of the batch:
 *   FE_LOSS_MSE  (1/K) sum_k (s_k - r_k)^2                        (scalar target r_k)
 *   FE_LOSS_BCE  (1/K) sum_k BCE(sigmoid(s_k), r_k / L)           (probabilistic target r_k / L)
 *   FE_LOSS_CE   -log softmax(s)_y                                (listwise, target list y)
 *
 * All arithmetic is fp32 (products accumulate in fp32; LayerNorm eps 1e-5; softmax attention
 * with scale 1/sqrt(dh)).  The step is written for correctness and generality first: plain tiled
 * fp32 products and separate launches per operation.
 */
#ifndef FLASHEVAL_TRAIN_H
#define FLASHEVAL_TRAIN_H

#include <stddef.h>
#include <stdint.h>

#include "flasheval.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { FE_LOSS_MSE = 0, FE_LOSS_BCE = 1, FE_LOSS_CE = 2 } fe_loss;

/*
 * Workspace bytes fe_train_grads needs for B requests with T context rows, pools of M elements
 * (M = vocab for token-id items) and K lists of length L.  The workspace holds every saved
 * activation of the forward (all layers of the four modules, the attention probabilities
 * included) and the backward's scratch, so it grows with B * (T^2 + U^2 + U T + K L^2 + K^2),
 * U = min(M, K L).
 *
 * Errors: FE_EINVAL (NULL pointer, sizes < 1, L > max_L), FE_EUNSUPPORTED (a config outside the
 * fe_model_create envelope, dtype other than FE_F32, attention other than FE_ATTN_SOFTMAX,
 * T > 8192, K > 1024, M > 131072).
 */
fe_status fe_train_workspace_size(const fe_config* cfg, int B, int T, int M, int K, int L, size_t* bytes);

/*
 * One training step's forward and backward on `stream` (a hipStream_t; NULL = the null stream),
 * asynchronous with respect to the host.  Every pointer but cfg is DEVICE memory of the current
 * HIP device; nothing is allocated.
 *
 *   params    fp32 [n_floats]: the flat parameter array in the fe_model_create order
 *             (n_floats from fe_param_count)
 *   x         fp32 [B][T][d] context rows (vocab == 0), else NULL
 *   ctx_ids   int32 [B][T] context token ids (vocab > 0), else NULL; ids outside [0, vocab) embed
 *             as zero rows
 *   pool      fp32 [B][M][d] element embeddings (vocab == 0), else NULL (items are rows of emb)
 *   lists     int32 [B][K][L] element indices in [0, M); an entry outside that range is left out
 *             of the distinct set and contributes a zero row without a position (as in
 *             fe_assemble), no feedback and no gradient; such entries are not reported (the
 *             inference calls report them in their status word)
 *   relevant  int32 [B][M] binary item-level feedback (0 or 1)
 *   loss_kind fe_loss
 *   loss      fp32 [1], overwritten with the batch loss
 *   scores    fp32 [B][K] list scores of the forward, or NULL
 *   grads     fp32 [n_floats], overwritten with d loss / d params in the same flat layout
 *             (d / d pool and d / d x are not produced: they are inputs, not parameters)
 *   ws        workspace of ws_bytes >= fe_train_workspace_size bytes, 256-byte aligned
 *
 * The gradient sums are accumulated with atomics in places, so their last bits vary between runs.
 * Errors: those of fe_train_workspace_size; FE_EINVAL for a missing input, a workspace that is too
 * small or misaligned, or loss_kind out of range; FE_EHIP for a failed launch.
 */
fe_status fe_train_grads(const fe_config* cfg, const float* params, int B, int T, int M, int K, int L,
                         const float* x, const int32_t* ctx_ids, const float* pool, const int32_t* lists,
                         const int32_t* relevant, int loss_kind, float* loss, float* scores, float* grads, void* ws,
                         size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* FLASHEVAL_TRAIN_H */
