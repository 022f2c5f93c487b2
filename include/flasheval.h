/*
 * flasheval.h -- C ABI of the FlashEvaluator joint-evaluation forward pass on
 * AMD Instinct MI355X (gfx950).
 *
 * The pass scores K candidate lists of one request jointly (paper, Section 3:
 * an instance z = (x, C(x), L_1..L_K) is mapped to a score vector in R^K and
 * the selected list is its argmax, eq. (1)).  It runs as five stream-ordered
 * calls, each a sequence of HIP kernels:
 *
 *   fe_encode_context   encode the request context once; emit the key/value
 *                       cache of every item layer             (Section 4.2)
 *   fe_encode_items     distinct element set U(z) with occurrence ranks,
 *                       then one encoding per distinct element (Sections 4.1, 4.2)
 *   fe_assemble         index-based assembly of [CLS; H[L_k]] + positions (Section 4.3)
 *   fe_cross_sequence   intra-sequence encoder -> c_k, then cross-sequence
 *                       self-attention over c_1..c_K           (Sections 4.3, 4.4)
 *   fe_score_select     linear score head and argmax           (Section 4.4, eq. (1))
 *
 * Network readings where the paper leaves details open (all blocks pre-LN with
 * residuals, LayerNorm eps 1e-5 with biased variance, multi-head attention with
 * biases and scale 1/sqrt(d_head), ReLU FFN, [CLS] at position 0, positions
 * added after the gather, smallest index wins an argmax tie, NaN never wins,
 * all-NaN selects -1) are the same as in the CPU oracle that tests this library.
 *
 * Conventions
 *   - Every tensor argument of the five calls is a DEVICE pointer owned by the
 *     caller; the library never allocates, frees or synchronises inside them.
 *     Scratch memory is the caller's workspace (size from fe_workspace_size).
 *   - Calls are asynchronous on `stream` (a hipStream_t, NULL = default
 *     stream) and return once their kernels are enqueued.  One workspace must
 *     not be used by two streams at the same time.  The model is read-only
 *     after creation: calls on different streams may run concurrently on one
 *     model when they share no output and no workspace (fe_executor_* below
 *     orders whole passes that way).
 *   - Tensors are dense and row-major with the model width d innermost.  Head
 *     h of an attention module owns columns h*dh .. h*dh+dh-1, dh = d/n_heads.
 *   - "act" is the model's activation type: float (FE_F32) or bfloat16
 *     (FE_BF16, stored as 16-bit patterns).  Matrix products on FE_BF16 models
 *     multiply bf16 operands with fp32 accumulation; LayerNorm statistics,
 *     softmax and the residual stream inside a module are kept in fp32.
 *   - Indices are int32.  U_cap = min(M, K*L) distinct elements per request.
 *   - Pointers must be 16-byte aligned and d*sizeof(act) a multiple of 16.
 *
 * Errors
 *   - FE_EINVAL: null or misaligned pointer, non-positive size, L > max_L,
 *     x and ctx_ids both or neither given, pool NULL on a model without a
 *     vocabulary, workspace too small, size products that overflow int32.
 *   - FE_EUNSUPPORTED: shape outside the envelope documented at fe_model_create.
 *   - FE_EHIP: a HIP launch failed; fe_last_error() returns the message.
 *   Host-side validation happens before any launch: on a non-OK status
 *   nothing was enqueued.  Data errors found on the device (an element index
 *   outside [0, M), a context token outside [0, vocab)) set bits of the per-
 *   request status words in the workspace; read them with
 *   fe_read_device_status.  Outputs are unspecified for a request whose status
 *   is not zero.  No C++ exception crosses this interface.
 */
#ifndef FLASHEVAL_H
#define FLASHEVAL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FE_OK = 0,
  FE_EINVAL = 1,
  FE_EUNSUPPORTED = 2,
  FE_ENOMEM = 3,
  FE_EHIP = 4
} fe_status;

typedef enum { FE_F32 = 0, FE_BF16 = 1 } fe_dtype;

/*
 * Attention form.  FE_ATTN_SOFTMAX: scaled dot-product attention everywhere (Section 4).
 * FE_ATTN_LINEAR: the deployment setting of Appendix B.3, which serves the evaluator with
 * linear (kernelized) attention: in the context self-attention, the items' cross-attention to
 * the context and the cross-sequence attention -- the attentions over sets that grow with the
 * workload (T context rows, K lists) -- the weight of key k for query q is phi(q) . phi(k)
 * with phi(x) = elu(x) + 1, no scale, and the output is the weighted sum of the values over
 * the sum of the weights.  The item-set self-attention and SeqEnc keep softmax.  The context-side
 * cache then becomes a fixed-size per-head state (see fe_encode_context).
 */
typedef enum { FE_ATTN_SOFTMAX = 0, FE_ATTN_LINEAR = 1 } fe_attention;

/* Device status bits (per request). */
#define FE_DEV_BAD_INDEX 1  /* a list entry outside [0, M): its slot is -1, fe_assemble writes a zero row */
#define FE_DEV_BAD_TOKEN 2  /* a context token id outside [0, vocab): its row is embedded as zeros */

typedef struct {
  int32_t d;         /* model width */
  int32_t n_heads;   /* attention heads in every module */
  int32_t n_layers;  /* blocks in each of the four modules */
  int32_t ffn_dim;   /* FFN hidden width */
  int32_t max_L;     /* longest list; the position table has max_L + 1 rows */
  int32_t vocab;     /* > 0: the model owns an embedding table E[vocab][d]; 0: none */
  int32_t dtype;     /* fe_dtype of activations and matrices */
  int32_t attention; /* fe_attention */
} fe_config;

typedef struct fe_model fe_model; /* opaque; immutable after creation */

/* Number of floats in the flat parameter array that fe_model_create takes. */
fe_status fe_param_count(const fe_config* cfg, size_t* n_floats);

/*
 * Create a model on the current HIP device.  `params` is a HOST array of
 * `n_floats` floats holding every parameter, concatenated in this order
 * (matrices in [in][out] orientation, i.e. y = x W + b, row-major):
 *
 *   for l in 0..n-1:  ctx.l   = ENC block
 *   ctx.lnf.g [d], ctx.lnf.b [d]
 *   for l in 0..n-1:  ctx.kv.l: wk [d][d], bk [d], wv [d][d], bv [d]
 *                     (key/value projections used by item layer l's
 *                      cross-attention, applied to the encoded context)
 *   for l in 0..n-1:  item.l  = ln1.g, ln1.b, wqkv [d][3d], bqkv [3d], wo [d][d], bo,
 *                               ln2.g, ln2.b, wq [d][d], bq, wo2 [d][d], bo2,
 *                               ln3.g, ln3.b, w1 [d][F], b1 [F], w2 [F][d], b2
 *   item.lnf.g, item.lnf.b
 *   for l in 0..n-1:  seq.l   = ENC block;    seq.lnf.g, seq.lnf.b
 *   for l in 0..n-1:  cross.l = ENC block;    cross.lnf.g, cross.lnf.b
 *   cls [d], pos [max_L+1][d], head.w [d], head.b [1]
 *   if vocab > 0:     emb [vocab][d]
 *
 *   ENC block = ln1.g [d], ln1.b [d], wqkv [d][3d], bqkv [3d], wo [d][d], bo [d],
 *               ln2.g [d], ln2.b [d], w1 [d][F], b1 [F], w2 [F][d], b2 [d]
 *   wqkv holds the query, key and value projections as consecutive column
 *   blocks of width d.
 *
 * On FE_BF16 models matrices, [CLS], positions and the embedding table are
 * rounded to bfloat16 on upload (exact if the values already are bf16);
 * biases, LayerNorm parameters and the head stay fp32.  The model owns its
 * device copies (allocated here, freed by fe_model_destroy).
 *
 * Supported envelope (else FE_EUNSUPPORTED): d in {32, 64, 128, 256, 512}, dh = d/n_heads in
 * {32, 64}, 1 <= n_layers <= 8, ffn_dim <= 4096, max_L <= 127, vocab <= 131072.  FE_BF16
 * models need d >= 128 and ffn_dim a multiple of 128; FE_F32 models need ffn_dim a multiple
 * of 32.
 */
fe_status fe_model_create(const fe_config* cfg, const float* params, size_t n_floats, fe_model** out);
void fe_model_destroy(fe_model* m);

/*
 * Workspace bytes needed for a batch of B requests with T context rows, pools
 * of M elements (M = vocab for token-id items) and K lists of length L.  The
 * same workspace serves all five calls of one pass; it starts with the per-
 * request device status words.  Envelope: T <= 8192, K <= 4096, M <= 131072.
 */
fe_status fe_workspace_size(const fe_model* m, int B, int T, int M, int K, int L, size_t* bytes);

/*
 * Bytes of fe_encode_context's output kv for B requests of T context rows:
 *   FE_ATTN_SOFTMAX  n_layers * 2 * B * T * d * sizeof(act)   ([n][2][B][T][d] act)
 *   FE_ATTN_LINEAR   n_layers * B * H * (dh + 1) * dh * 4     ([n][B][H][dh+1][dh] fp32)
 */
fe_status fe_kv_size(const fe_model* m, int B, int T, size_t* bytes);

/* Message of the last non-OK status returned on this thread ("" if none). */
const char* fe_last_error(void);

/*
 * Copy the B per-request status words (FE_DEV_* bits) from workspace `ws` to
 * host memory `host_out` [B].  Synchronises `stream`.
 */
fe_status fe_read_device_status(const fe_model* m, const void* ws, int B, void* stream, int32_t* host_out);

/*
 * Section 4.2, Query Context Module plus the context-side key/value cache:
 * per request, the context rows pass n encoder blocks and a final LayerNorm;
 * for every item layer l, K_l and V_l are that result times ctx.kv.l.wk / wv
 * plus bias.  Exactly one of
 *   x       [B][T][d] act  -- context vectors, or
 *   ctx_ids [B][T] int32   -- token ids embedded through the model's table
 * is non-NULL.  Output kv (fe_kv_size bytes):
 *   FE_ATTN_SOFTMAX  [n_layers][2][B][T][d] act (index 0 = keys, 1 = values);
 *   FE_ATTN_LINEAR   [n_layers][B][H][dh + 1][dh] fp32: for item layer l, request b and head h,
 *                    rows i < dh hold sum_t phi(K_l[t])_i V_l[t] over the head's columns and row
 *                    dh holds sum_t phi(K_l[t]) -- everything the items' linear cross-attention
 *                    needs, independent of T.
 */
fe_status fe_encode_context(const fe_model* m, int B, int T, const void* x, const int32_t* ctx_ids, void* kv,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * Sections 4.1-4.2: distinct elements and their shared encoding.
 *   pool   [B][M][d] act, or NULL on a model with a vocabulary (then the
 *          elements are token ids and M must equal vocab).
 *   lists  [B][K][L] int32 element indices into the pool (0-based).
 *   kv     output of fe_encode_context for the same B and T (and model).
 * Outputs:
 *   uniq   [B][U_cap] int32  distinct indices of each request, ascending,
 *                            padded with -1;
 *   n_uniq [B] int32         U of each request;
 *   slot   [B][K][L] int32   rank of each occurrence in uniq (-1 if the index
 *                            was out of range);
 *   H      [B][U_cap][d] act row u = encoding of element uniq[u]: n blocks of
 *                            [masked self-attention over the U distinct
 *                            elements, cross-attention with the elements as
 *                            queries and kv as keys/values, FFN], then a final
 *                            LayerNorm.  Rows >= U are zero.
 */
fe_status fe_encode_items(const fe_model* m, int B, int M, const void* pool, const int32_t* lists, int K, int L,
                          const void* kv, int T, int32_t* uniq, int32_t* n_uniq, int32_t* slot, void* H,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * Section 4.3, index-based assembly with positions added after indexing:
 *   seq[b][k][0]   = cls + pos[0]
 *   seq[b][k][j+1] = H[b][slot[b][k][j]] + pos[j+1]      (j < L)
 * A slot outside [0, U_cap) gives a zero row.  seq is [B][K][L+1][d] act; the
 * sum is formed in fp32 and rounded once to act.
 */
fe_status fe_assemble(const fe_model* m, int B, int K, int L, int U_cap, const int32_t* slot, const void* H,
                      void* seq, void* stream);

/*
 * Sections 4.3-4.4: SeqEnc (n encoder blocks over each list's L+1 rows, no
 * mask; c_k = final-LayerNorm of the [CLS] row), then the cross-sequence
 * module (n encoder blocks over the K vectors c_1..c_K of a request, no
 * positions, no mask, final LayerNorm).  seq [B][K][L+1][d] act in,
 * Cp [B][K][d] fp32 out.
 */
fe_status fe_cross_sequence(const fe_model* m, int B, int K, int L, const void* seq, float* Cp, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): fe_cross_sequence without a workspace argument.  Same
 * computation and kernels, same arguments otherwise (seq [B][K][L+1][d] act in, Cp [B][K][d]
 * fp32 out, caller-owned device pointers), bit-identical results.  Its scratch (the c_k rows and,
 * for long lists, many lists, wide or linear models, the block buffers) lives in a static device
 * array of FE_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs on until the
 * process ends; the call allocates and frees nothing.  A shape whose scratch exceeds that size
 * returns FE_EUNSUPPORTED before any launch (e.g. B=64, K=50, L=10 at d=128 needs 1.6 MB).
 * Every call on one device uses that device's single array: calls that overlap on one device
 * (concurrent streams or threads) race and give undefined results; calls ordered on one stream
 * are safe.  Nothing in the array needs to start at zero.
 */
#define FE_NOALLOC_SCRATCH_BYTES (32u << 20)
fe_status fe_cross_sequence_noalloc(const fe_model* m, int B, int K, int L, const void* seq, float* Cp,
                                    void* stream);

/*
 * Section 4.4 and eq. (1): scores[b][k] = Cp[b][k] . head.w + head.b (fp32),
 * best[b] = smallest k with the maximal score, NaN scores skipped, -1 if all
 * are NaN.  Cp [B][K][d] fp32, scores [B][K] fp32, best [B] int32.
 */
fe_status fe_score_select(const fe_model* m, int B, int K, const float* Cp, float* scores, int32_t* best,
                          void* stream);

/*
 * Section 4.4 variant without cross-sequence interaction (the "- CrossSeq"
 * ablation of Appendix B.4): SeqEnc only, C[b][k] = c_k, the final-LayerNorm
 * [CLS] row of list k, so every list is scored on its own representation
 * (pass C to fe_score_select or fe_score_objectives in place of Cp).  seq
 * [B][K][L+1][d] act in, C [B][K][d] fp32 out; ws as for fe_cross_sequence.
 */
fe_status fe_encode_sequences(const fe_model* m, int B, int K, int L, const void* seq, float* C, void* ws,
                              size_t ws_bytes, void* stream);

/*
 * Section 4.4, multi-objective form: n_obj task-specific linear heads on the
 * shared C'_k and a fusion of their predictions.  The paper leaves the fusion
 * open; here it is the weighted sum with caller weights:
 *   obj_scores[b][k][t] = Cp[b][k] . head_w[t] + head_b[t]          (fp32)
 *   scores[b][k]        = sum_t fuse_w[t] * obj_scores[b][k][t]     (t = 0, 1, ...)
 *   best[b]             = smallest k with the largest fused score (NaN skipped,
 *                         -1 if all NaN), as in fe_score_select.
 * head_w [n_obj][d], head_b [n_obj], fuse_w [n_obj] are caller-owned fp32
 * device arrays (they are not model parameters); 1 <= n_obj <= 8
 * (FE_EUNSUPPORTED otherwise).  Cp [B][K][d] fp32 (or C of
 * fe_encode_sequences), obj_scores [B][K][n_obj], scores [B][K], best [B].
 */
fe_status fe_score_objectives(const fe_model* m, int B, int K, const float* Cp, int n_obj, const float* head_w,
                              const float* head_b, const float* fuse_w, float* obj_scores, float* scores,
                              int32_t* best, void* stream);

/*
 * Baseline, outside the joint pass: the candidate-factorised evaluator (E^ind,
 * Section 3) of the same network on the GPU, with every reuse taken out.  The
 * context is encoded once per list (B*K context encodings, each list with its
 * own key/value cache) and the distinct-element set once per element
 * occurrence (L set encodings per list, against that list's cache), the cost
 * structure of Appendix A.3 extended to the context side.  Each list is then
 * assembled from its own encodings; SeqEnc, the cross-sequence module and the
 * head run as in the joint pass.  QKV-Cache reuses exact results (Section
 * 4.2), so the outputs equal those of the five calls; only the work differs.
 *
 * Arguments are those of the five calls: x [B][T][d] act or ctx_ids [B][T]
 * int32 (exactly one), pool [B][M][d] act or NULL on a vocabulary model,
 * lists [B][K][L] int32.  Outputs Cp [B][K][d] fp32, scores [B][K] fp32,
 * best [B] int32 (device, caller-owned).  ws is a device workspace of at least
 * fe_naive_workspace_size bytes (token_ids = 1 when ctx_ids will be given);
 * it holds the joint pass's workspace for B*K requests, per-list copies of
 * the inputs and per-list caches, so B*K must pass the same envelope and
 * int32 limits as a batch of B*K requests (FE_EINVAL / FE_EUNSUPPORTED
 * otherwise).  Asynchronous on `stream`; errors as for the five calls.
 */
fe_status fe_naive_workspace_size(const fe_model* m, int B, int T, int M, int K, int L, int token_ids,
                                  size_t* bytes);
fe_status fe_evaluate_naive(const fe_model* m, int B, int T, int M, int K, int L, const void* x,
                            const int32_t* ctx_ids, const void* pool, const int32_t* lists, float* Cp,
                            float* scores, int32_t* best, void* ws, size_t ws_bytes, void* stream);

/*
 * Pipelined executor for serving many batches: not a step of the method, it orders the five
 * calls of independent batches on several streams so that their kernels share the GPU.  At
 * serving batch sizes the pass's kernels are latency-bound (one workgroup per compute unit and
 * long dependent chains inside each), so a second or third batch in flight fills compute units
 * that one batch leaves idle.
 *
 * fe_executor_create: n_streams (1 .. FE_EXECUTOR_MAX_STREAMS) HIP streams on the model's device,
 *   non-blocking and at the default priority, with two events each.  Allocates no device memory.
 *   Call with the model's device current.
 * fe_executor_submit: one whole pass -- fe_encode_context, fe_encode_items, fe_assemble,
 *   fe_cross_sequence and fe_score_select with the arguments in `p` -- on the executor's next
 *   stream in round-robin order, after that stream has waited for the work enqueued so far on
 *   `stream` (the caller's stream, NULL = default, whose work produced the inputs).  Returns once
 *   the kernels are enqueued.  The whole pass is validated first, with the rules of the five
 *   calls (p->ws_bytes >= fe_workspace_size(B, T, M, K, L)); on FE_EINVAL or FE_EUNSUPPORTED
 *   nothing was enqueued (FE_EHIP, a failed launch, may leave the pass's earlier kernels
 *   enqueued, as for the five calls).  A submission must not share any output (kv, uniq,
 *   n_uniq, slot, H, seq, Cp, scores, best) or the workspace with a submission still in flight;
 *   one buffer set per stream, submission i using set i mod n_streams, satisfies this.  Inputs
 *   may be shared.
 * fe_executor_join: makes `stream` wait (on the device) for every pass submitted so far; the
 *   outputs are valid for work enqueued on `stream` after it.
 * fe_executor_destroy: waits on the host for the submitted passes, then releases the streams and
 *   events.  One executor must not be used by two host threads at once.
 */
#define FE_EXECUTOR_MAX_STREAMS 8
typedef struct fe_executor fe_executor; /* opaque */
typedef struct {
  int B, T, M, K, L;
  const void* x;          /* [B][T][d] act, or NULL when ctx_ids is given */
  const int32_t* ctx_ids; /* [B][T] int32, or NULL when x is given */
  const void* pool;       /* [B][M][d] act, or NULL on a vocabulary model */
  const int32_t* lists;   /* [B][K][L] int32 */
  void* kv;               /* fe_kv_size bytes */
  int32_t* uniq;          /* [B][U_cap] */
  int32_t* n_uniq;        /* [B] */
  int32_t* slot;          /* [B][K][L] */
  void* H;                /* [B][U_cap][d] act */
  void* seq;              /* [B][K][L+1][d] act */
  float* Cp;              /* [B][K][d] */
  float* scores;          /* [B][K] */
  int32_t* best;          /* [B] */
  void* ws;
  size_t ws_bytes;
} fe_pass_args;
fe_status fe_executor_create(const fe_model* m, int n_streams, fe_executor** out);
fe_status fe_executor_submit(fe_executor* ex, const fe_pass_args* p, void* stream);
fe_status fe_executor_join(fe_executor* ex, void* stream);
void fe_executor_destroy(fe_executor* ex);

#ifdef __cplusplus
}
#endif

#endif /* FLASHEVAL_H */
