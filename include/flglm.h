/*
 * flglm.h - C ABI of the FL-GLM server-stack library (MI355X / gfx950).
 *
 * What it computes.  In FL-GLM the model is split into three parts; the
 * server holds the middle blocks 1..N-2 and maps the clients' smashed data
 * h_0 to h_{N-2} = Block_(1,N-2)(h_0) (Section 3.1, Model Split).  With
 * client-batch parallel training the server stacks the smashed data of M
 * clients into one batch (Section 3.3, Parallel Acceleration); here the
 * stacked batch is packed without padding: rows of client 0's sequences,
 * then client 1's, and so on, with per-sequence offsets.  In the backward
 * pass the server receives dL/dh_{N-2}, returns dL/dh_0 to every client and
 * accumulates the gradients of its own weights (split learning, Section 1
 * and Section 3.1).
 *
 * Each block is a pre-LayerNorm transformer layer (Section 3.1: multi-head
 * self-attention followed by a feed-forward network; Appendix A: scores
 * softmax(Q K^T / sqrt(d_h))):
 *     u = LN1(x);  [q|k|v] = u W_qkv^T + b_qkv;  q, k rotated on the first
 *     rotary_dim dims of every head (pairs (i, i + rotary_dim/2), angle
 *     p * rope_base^(-2i/rotary_dim), p = position inside the sequence);
 *     h = x + Attn(q, k, v) W_o^T + b_o;   w = LN2(h);
 *     y = h + gelu_tanh(w W_1^T + b_1) W_2^T + b_2.
 * Attention never crosses a sequence boundary (hence never a client
 * boundary).  Mask: causal, or prefix-LM where key j is visible to query i
 * iff j <= max(i, P_s - 1).
 *
 * Conventions (all entry points):
 *   - Return 0 (FL_OK) or a negative FL_ERR_* code; fl_last_error() gives a
 *     thread-local message for the last failure.  Nothing is enqueued and no
 *     output is written when an entry point returns an error from its
 *     validation step.
 *   - "host" pointers are read during the call only; "device" pointers are
 *     caller-owned device memory (hipMalloc / torch), 16-byte aligned.
 *   - `stream` is a hipStream_t (NULL = the default stream).  All device work
 *     is asynchronous on that stream; execution errors surface at the
 *     caller's next synchronisation.  One stream per handle at a time.
 *   - A handle is not thread-safe: its upload ring and launch records are
 *     unsynchronised host state, so calls on one handle must not run
 *     concurrently from several threads (use one handle per thread).
 *   - Element type of activations and weights is the handle's dtype (bf16 or
 *     fp32); statistics, softmax and all accumulation are fp32; weight
 *     gradients are fp32 and are accumulated (+=), never zeroed.
 *   - Results are deterministic: identical inputs give bitwise-identical
 *     outputs (no atomics).
 */
#ifndef FLGLM_H_
#define FLGLM_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FL_OK 0
#define FL_ERR_NULL (-1)        /* a required pointer is NULL */
#define FL_ERR_SHAPE (-2)       /* unsupported or inconsistent stack shape */
#define FL_ERR_SEQLENS (-3)     /* cu_seqlens / total_tokens / max_seqlen inconsistent, or an empty sequence */
#define FL_ERR_CLIENTS (-4)     /* client_seq_ptr inconsistent, or a client without sequences */
#define FL_ERR_PREFIX (-5)      /* bad mask kind or prefix length */
#define FL_ERR_WORKSPACE (-6)   /* workspace or saved buffer too small */
#define FL_ERR_ALIAS (-7)       /* an output overlaps an input it must not overlap */
#define FL_ERR_ALIGN (-8)       /* a device pointer is not 16-byte aligned */
#define FL_ERR_HIP (-9)         /* a HIP runtime call or kernel launch failed */
#define FL_ERR_ARG (-10)        /* other invalid argument */
#define FL_ERR_NOMEM (-11)      /* a host allocation for a handle failed */

#define FL_BF16 0
#define FL_F32 1

#define FL_MASK_CAUSAL 0
#define FL_MASK_PREFIX 1

/* Shape of the server-held stack; all blocks are identical.  Supported:
 * hidden % 256 == 0, hidden / num_heads in {64, 128}, ffn_hidden % 256 == 0,
 * rotary_dim % 32 == 0 and <= head dim, hidden <= 4096, ln_eps > 0.
 *
 * num_prefix > 0 selects P-tuning v2 (Section 3.1 and Appendix A, P-tuning
 * v2): every block has num_prefix learned key and value rows ([L_p, H],
 * head h at columns h*d, not rotated) spliced in front of each sequence's
 * own keys and values, K' = [prefix_key; key], V' = [prefix_value; value],
 * and visible to every query of every sequence.  bf16 only; at most 4096.
 *
 * ChatGLM-6B's own block (the paper's base model; these details are
 * ChatGLM-6B's, not the paper's), for loading its weights:
 *   residual_alpha > 0: the residual carries the normalised input scaled by
 *     alpha (ChatGLM-6B: sqrt(2 * 28)): h = alpha u + Attn(...) W_o^T + b_o,
 *     y = alpha w + gelu(...) W_2^T + b_2; 0 = the plain x + f(LN(x)).
 *   rotary_2d = 1: GLM 2-D positions (needs rotary_dim = head dim / 2).  A
 *     sequence's context is its prefix-LM prefix (the whole sequence in a
 *     causal batch) ending with the [gMASK] token at M = max(P - 1, 0);
 *     dims [0, r) of each head are rotated by p1 = t in the context, M after
 *     it, and dims [r, 2r) by the block position p2 = 0 in the context,
 *     t - P + 1 after it. */
typedef struct fl_stack_desc {
  int32_t num_layers;   /* N server blocks (26 for ChatGLM-6B's server part) */
  int32_t hidden;       /* H */
  int32_t num_heads;    /* n_h; head dim d = H / n_h */
  int32_t ffn_hidden;   /* F */
  int32_t rotary_dim;   /* r: leading dims of each head that are rotated */
  float rope_base;      /* 10000 */
  float ln_eps;         /* 1e-5 */
  int32_t dtype;        /* FL_BF16 or FL_F32 */
  int32_t num_prefix;   /* L_p, P-tuning v2 prefix length; 0 = no prefix */
  float residual_alpha; /* 0: plain residual; > 0: ChatGLM-6B's alpha-scaled residual */
  int32_t rotary_2d;    /* 0: 1-D positions; 1: GLM 2-D positions */
} fl_stack_desc;

/* A packed batch of clients (host arrays).  Sequence s covers packed rows
 * [cu_seqlens[s], cu_seqlens[s+1]); client c owns sequences
 * [client_seq_ptr[c], client_seq_ptr[c+1]), i.e. rows
 * [cu_seqlens[client_seq_ptr[c]], cu_seqlens[client_seq_ptr[c+1]]). */
typedef struct fl_batch_desc {
  int32_t num_clients;            /* C >= 1 */
  int32_t num_seqs;               /* S >= C */
  int64_t total_tokens;           /* T = cu_seqlens[S] */
  int32_t max_seqlen;             /* max_s (cu_seqlens[s+1] - cu_seqlens[s]) */
  const int32_t* cu_seqlens;      /* host [S+1]: cu[0] = 0, strictly increasing */
  const int32_t* client_seq_ptr;  /* host [C+1]: csp[0] = 0, strictly increasing, csp[C] = S */
  int32_t mask_kind;              /* FL_MASK_CAUSAL or FL_MASK_PREFIX */
  const int32_t* prefix_len;      /* host [S], 0 <= P_s <= L_s; NULL unless FL_MASK_PREFIX */
} fl_batch_desc;

/* One block's parameters (device, handle dtype).  Weights are
 * out-features-major (y = x W^T + b): w_qkv [3H, H] (rows [0,H) query,
 * [H,2H) key, [2H,3H) value; head h owns rows h*d .. h*d+d-1 of each),
 * b_qkv [3H], w_o [H, H], b_o [H], w_1 [F, H], b_1 [F], w_2 [H, F], b_2 [H],
 * ln1_g, ln1_b, ln2_g, ln2_b [H].  prefix_k, prefix_v [L_p, H]: the
 * P-tuning v2 prefix (required when num_prefix > 0, ignored otherwise). */
typedef struct fl_layer_params {
  const void *w_qkv, *b_qkv, *w_o, *b_o, *w_1, *b_1, *w_2, *b_2;
  const void *ln1_g, *ln1_b, *ln2_g, *ln2_b;
  const void *prefix_k, *prefix_v;
} fl_layer_params;

/* One block's gradient accumulators (device fp32, same shapes as the
 * parameters).  The backward adds into them.  The twelve weight pointers
 * are either all set (full fine-tuning) or all NULL: frozen weights, as in
 * P-tuning v2, where no weight gradient is formed at all.  prefix_k and
 * prefix_v are required when num_prefix > 0 (the sum over every sequence of
 * every client), ignored otherwise. */
typedef struct fl_layer_grads {
  float *w_qkv, *b_qkv, *w_o, *b_o, *w_1, *b_1, *w_2, *b_2;
  float *ln1_g, *ln1_b, *ln2_g, *ln2_b;
  float *prefix_k, *prefix_v;
} fl_layer_grads;

typedef struct fl_stack fl_stack;

/* Creates a handle for a stack shape (validated; FL_ERR_SHAPE if
 * unsupported; FL_ERR_NOMEM if the handle cannot be allocated).  Host-only:
 * no HIP call.  On its first device call the
 * handle creates a few events and a small pinned host staging area used to
 * upload per-call batch descriptors; it never owns device memory. */
int fl_stack_create(const fl_stack_desc* desc, fl_stack** out);
/* Releases the handle.  Waits for uploads still in flight. NULL is a no-op. */
int fl_stack_destroy(fl_stack* stack);

/* Bytes of the `saved` buffer fl_server_stack_forward fills for the
 * backward: with recompute = 0 every block's intermediates; with
 * recompute = 1 only the inputs of blocks 2..N (the backward recomputes each
 * block's forward from its input). */
int fl_stack_saved_bytes(const fl_stack* stack, const fl_batch_desc* batch, int recompute, size_t* bytes);
/* Bytes of device workspace needed by forward / backward / pack calls for
 * this batch (one size serves all of them).  In bf16 it includes room for
 * the backward's attention softmax gradient dS (Appendix A form of the
 * attention), stored once and read by the dq pass: one 64 x 64 bf16 tile per
 * head and per pair of 64-row query / key tiles with a visible pair, when
 * that totals at most 8 GiB (beyond, dq recomputes it and nothing is
 * stored). */
int fl_stack_workspace_bytes(const fl_stack* stack, const fl_batch_desc* batch, int recompute, size_t* bytes);

/* Forward through the N server blocks (Section 3.1, h_{N-2} =
 * Block_(1,N-2)(h_0)) over the packed client batch.
 *   x  device [T, H]  packed smashed data h_0 (not modified)
 *   y  device [T, H]  output h_{N-2}; must not overlap x
 *   saved  device, fl_stack_saved_bytes(recompute) bytes, or NULL for a
 *          forward-only (inference) call
 *   workspace  device, >= fl_stack_workspace_bytes bytes, contents scratch */
int fl_server_stack_forward(fl_stack* stack, const fl_batch_desc* batch, const fl_layer_params* layers,
                            const void* x, void* y, void* saved, int recompute, void* workspace,
                            size_t workspace_bytes, void* stream);

/* Allocation-free inference forward, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  Computes what fl_server_stack_forward
 * computes with saved = NULL (the same kernels in the same order: the same
 * bits), with two differences:
 *   - the workspace is a static device array of FL_NOALLOC_SCRATCH_BYTES
 *     that the library holds on every GPU it runs on until the process ends
 *     (its address is looked up on the first call on each device); a batch
 *     whose forward needs more (at the ChatGLM-6B block shape, about 1800
 *     tokens) gets FL_ERR_WORKSPACE;
 *   - the batch plan travels in kernel arguments, not through pinned
 *     staging: at most FL_NOALLOC_MAX_SEQS sequences, else FL_ERR_ARG.
 * It calls no hipMalloc, hipFree, hipHostMalloc or event creation; launch
 * timing (fl_stack_profile) is off for its launches.  Every call on one GPU
 * shares that GPU's array and leaves it holding the last call's
 * intermediates: calls that overlap on one GPU (other streams, threads or
 * handles) race, so callers serialise them.  Validation errors are returned
 * before anything is enqueued, as for the other entry points.
 *   x  device [T, H]  (not modified);  y  device [T, H], not overlapping x */
#define FL_NOALLOC_SCRATCH_BYTES (256u << 20)
#define FL_NOALLOC_MAX_SEQS 256
int fl_server_stack_forward_noalloc(fl_stack* stack, const fl_batch_desc* batch, const fl_layer_params* layers,
                                    const void* x, void* y, void* stream);

/* Backward through blocks N..1 after a forward with the same batch, params,
 * x and recompute flag that filled `saved`.
 *   dy  device [T, H]  dL/dh_{N-2} from the clients (not modified)
 *   dx  device [T, H]  dL/dh_0, returned to the clients; must not overlap dy or x
 *   grads  [N] accumulators (+=) */
int fl_server_stack_backward(fl_stack* stack, const fl_batch_desc* batch, const fl_layer_params* layers,
                             const fl_layer_grads* grads, const void* x, const void* saved, const void* dy,
                             void* dx, int recompute, void* workspace, size_t workspace_bytes, void* stream);

/* Host only: packed row range [begin, end) of client `client`. */
int fl_client_token_range(const fl_batch_desc* batch, int32_t client, int64_t* begin, int64_t* end);

/* Client batching (Section 3.3): gather the clients' sequence-first tensors
 * client_bufs[c] (device [Lmax_c, B_c, H], Lmax_c = the client's longest
 * sequence, B_c = its number of sequences; positions beyond a sequence's
 * length are ignored) into the packed [T, H] buffer, or scatter the packed
 * buffer back (unpack zero-fills the padded positions).  Byte copies: exact. */
int fl_pack_clients(fl_stack* stack, const fl_batch_desc* batch, const void* const* client_bufs, void* packed,
                    void* workspace, size_t workspace_bytes, void* stream);
int fl_unpack_clients(fl_stack* stack, const fl_batch_desc* batch, const void* packed, void* const* client_bufs,
                      void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Client side of the split model (Section 3.1, Model Split): the client
 * holds the embedding layer, block 0, block N-1 and the final linear layer;
 * it computes h_0 = Block_0(Embedding(x)), receives the server's h_{N-2}, and
 * finishes with y' = Linear(Block_{N-1}(h_{N-2})) and the cross-entropy loss
 * against the next-token labels.  Blocks 0 and N-1 are one-block stacks
 * (fl_stack_create with num_layers = 1); the entry points below are the
 * embedding and the final linear layer with the loss.
 *
 * The final linear layer has no bias and no normalisation in front of it
 * (the paper applies Linear directly to Block_{N-1}'s output).  Its weight
 * is [vocab, hidden] (out-features-major, like the block weights).
 * Token ids and labels are host arrays (the client's own tokens), copied to
 * the device through pinned staging during the call.
 * ------------------------------------------------------------------------ */
typedef struct fl_client fl_client;

typedef struct {
  int64_t vocab;   /* multiple of 8, <= 2^24 (ChatGLM-6B: 130528) */
  int32_t hidden;  /* multiple of 256, <= 16384 */
  int32_t dtype;   /* FL_BF16 | FL_F32: element type of tables, weights, activations */
  float ln_eps;    /* eps of the optional final LayerNorm (> 0 when one is used; ChatGLM-6B: 1e-5) */
} fl_client_desc;

/* FL_ERR_SHAPE for an unsupported descriptor, FL_ERR_NOMEM if the handle
 * cannot be allocated. */
int fl_client_create(const fl_client_desc* desc, fl_client** out);
int fl_client_destroy(fl_client* client);
/* Workspace for T tokens (1 <= T <= 2^26): the logits [T, vocab rounded up
 * to 256] in the element type, per-token log-sum-exp, labels, ids, the
 * embedding-gradient plan, the final LayerNorm's output, statistics and
 * gradient partials, and the GEMM's split-reduction scratch.
 * Caller-allocated device memory, 16-byte aligned. */
int fl_client_workspace_bytes(const fl_client* client, int64_t T, size_t* bytes);

/* Embedding(x): out [T, hidden] (device) = rows ids[t] (host [T], each in
 * [0, vocab), else FL_ERR_ARG) of table [vocab, hidden] (device).  Copies:
 * exact. */
int fl_embedding_forward(fl_client* client, const void* table, const int32_t* ids, int64_t T, void* out,
                         void* workspace, size_t workspace_bytes, void* stream);
/* Gradient of the table: dtable [vocab, hidden] (device fp32) += for every
 * token t, dout[t] (device [T, hidden]) into row ids[t] (host).  Tokens of one
 * id are added in token order (deterministic, no atomics). */
int fl_embedding_backward(fl_client* client, const int32_t* ids, int64_t T, const void* dout, float* dtable,
                          void* workspace, size_t workspace_bytes, void* stream);

/* y' = LN(h) W^T and the cross-entropy: for every token t with labels[t]
 * >= 0 (host [T]; a negative label marks a token without target; labels >=
 * vocab give FL_ERR_ARG), loss_tok[t] = logsumexp(y'_t) - y'_t[labels[t]],
 * else 0; loss_sum = the sum of loss_tok in a fixed order.  h [T, hidden],
 * W [vocab, hidden] device; loss_tok [T] and loss_sum [1] device fp32.
 * ln_g / ln_b [hidden] (device, both or neither): ChatGLM-6B's final
 * LayerNorm (eps = the descriptor's ln_eps, hidden <= 4096); NULL = no
 * normalisation, the paper's y' = Linear(Block_{N-1}(h_{N-2})).  The
 * logits, log-sum-exp and normalised input stay in the workspace for
 * fl_lm_head_backward. */
int fl_lm_head_forward(fl_client* client, const void* h, const void* ln_g, const void* ln_b, const void* w,
                       const int32_t* labels, int64_t T, float* loss_tok, float* loss_sum, void* workspace,
                       size_t workspace_bytes, void* stream);
/* Backward of grad_scale * loss_sum (grad_scale = 1 / labelled tokens gives
 * the mean): dlogits = grad_scale (softmax - onehot) on labelled tokens, 0
 * on the others (computed in place in the workspace, which must still hold
 * the forward's logits: same T, no other head call in between); dh [T,
 * hidden] = dlogits W, taken back through the final LayerNorm when ln_g is
 * given (the same ln_g as the forward); dln_g / dln_b fp32 [hidden] +=
 * its gain / shift gradients (NULL: frozen); dw [vocab, hidden] fp32 +=
 * dlogits^T LN(h), or NULL when the weight is frozen (P-tuning v2). */
int fl_lm_head_backward(fl_client* client, const void* h, const void* ln_g, const void* w, int64_t T,
                        float grad_scale, void* dh, float* dln_g, float* dln_b, float* dw, void* workspace,
                        size_t workspace_bytes, void* stream);

/* Server update (Section 4.1.4, Parameter Settings: Adam, learning rate
 * 2e-2, batch size 1, no warmup, no weight decay).  One step of Algorithm 1
 * of the Adam paper (Kingma & Ba) over n fp32 elements, elementwise in
 * fp32:  m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2;
 * param -= lr (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps).
 * The hyper-parameters are doubles: 1 - beta and the bias corrections
 * 1 - beta^step are formed in double on the host and rounded to fp32 once
 * (subtracting a beta near 1 in fp32 would lose digits).  The paper gives no betas or eps; the Adam paper's
 * defaults (0.9, 0.999, 1e-8) are the usual choice.
 *   param, grad, exp_avg, exp_avg_sq: device fp32 [n], caller-owned, updated
 *     in place (grad only read unless zero_grad); exp_avg / exp_avg_sq start
 *     at zero before step 1.
 *   param_bf16: device bf16 [n] or NULL; when set, receives the updated
 *     parameters rounded to nearest even (the compute copy the stack reads).
 *   step: the 1-based time step t.  zero_grad = 1 also clears grad, ready
 *     for the next backward's accumulation (the stack accumulates, += ).
 * Any layout works as long as the five buffers index the same parameters
 * element by element: one flat arena per role updates a whole stack (or
 * every block's P-tuning prefix) in one launch.
 * Errors: FL_ERR_NULL, FL_ERR_ALIGN (16 bytes), FL_ERR_ALIAS (buffers
 * overlap), FL_ERR_ARG (n < 0, step < 1, lr < 0 or not finite, beta outside
 * [0, 1), eps < 0); nothing is enqueued then.  n = 0 is a no-op. */
int fl_adam_step(float* param, float* grad, float* exp_avg, float* exp_avg_sq, void* param_bf16, int64_t n,
                 int64_t step, double lr, double beta1, double beta2, double eps, int zero_grad, void* stream);

/* Server-hierarchical aggregation (Section 3.3, Parallel Acceleration: one
 * server-side model per client, parameters averaged at the end of each
 * training period; the paper's periods are 50 or 100 steps).  params is a
 * host array of num_replicas (1..32) device pointers to fp32 [n]; every
 * replica is overwritten with the elementwise mean (sum in replica order,
 * divided by num_replicas, fp32).  params_bf16: NULL, or a host array of
 * num_replicas device pointers to bf16 [n] compute copies that receive the
 * mean rounded to nearest even.  Only parameters are averaged; optimizer
 * moments stay with their replica.  No two buffers may overlap
 * (FL_ERR_ALIAS); FL_ERR_NULL / FL_ERR_ALIGN / FL_ERR_ARG as above. */
int fl_average_replicas(int32_t num_replicas, float* const* params, void* const* params_bf16, int64_t n,
                        void* stream);

/* Launch timing (off by default).  While enabled, every kernel launch the
 * handle enqueues is bracketed by two HIP events on the call's stream and
 * tagged with its class and its algorithmic work (flops of the contraction,
 * minimal HBM bytes).  Enabling clears earlier records.  The overhead is two
 * event records per launch. */
#define FL_PROF_PLAN 0              /* positions + rotary table */
#define FL_PROF_LAYERNORM_FWD 1
#define FL_PROF_GEMM_NT_BIAS 2      /* QKV projection */
#define FL_PROF_ROPE 3
#define FL_PROF_ATTN_FWD 4
#define FL_PROF_GEMM_NT_BIAS_RES 5  /* output projection, FFN2 (+ residual) */
#define FL_PROF_GEMM_NT_BIAS_GELU 6 /* FFN1 + GeLU */
#define FL_PROF_GEMM_TN_ACC 7       /* weight gradients (fp32 +=) */
#define FL_PROF_GEMM_NN_GELU_BWD 8  /* FFN2 input gradient x GeLU' */
#define FL_PROF_GEMM_NN 9           /* other input gradients */
#define FL_PROF_LAYERNORM_BWD 10
#define FL_PROF_COLSUM 11           /* bias and LayerNorm parameter gradients */
#define FL_PROF_ATTN_BWD 12
#define FL_PROF_PREFIX_GRAD 13      /* P-tuning v2 prefix gradients: sum over sequences */
#define FL_PROF_NUM_CLASSES 14
int fl_stack_profile(fl_stack* stack, int enable);
/* The same for a subset of the classes: bit c of class_mask times the
 * launches of class c (the others run without events); 0 turns timing off.
 * fl_stack_profile(stack, 1) times every class. */
int fl_stack_profile_classes(fl_stack* stack, uint32_t class_mask);
/* Totals for one class over the records since profiling was enabled:
 * launch count, summed event time (ms), algorithmic flops and bytes.
 * Waits for the recorded events. */
int fl_stack_profile_read(fl_stack* stack, int cls, int64_t* launches, double* milliseconds, double* flops,
                          double* bytes);
/* Name of a profiling class ("" when out of range). */
const char* fl_profile_class_name(int cls);

/* Thread-local description of the last error returned on this thread. */
const char* fl_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* FLGLM_H_ */
