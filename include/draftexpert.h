/*
 * draftexpert.h - C ABI of the MoE draft/verify hot path of DraftExpert
 * (expansion-aware self-speculative decoding for expert-offloaded MoE
 * inference), hand-written HIP for gfx950 (MI355X).
 *
 * Conventions shared by every call
 *   - All tensor pointers are DEVICE pointers unless a parameter says "host".
 *     The caller owns every buffer; the layer calls never allocate device
 *     memory: their scratch comes in through (ws, ws_bytes), sized by
 *     de_workspace_bytes().
 *   - Activations (x, y, logits, gates) are fp32, row-major [T, H] etc.
 *     Router weights are fp32 [N, H].  Expert weights are fp32 or bf16
 *     (raw uint16 bit patterns) as de_moe_desc.wdtype says.
 *   - An expert block is one contiguous region [G: I x H][U: I x H][D: H x I],
 *     each matrix row-major [out, in].  The shared path of a layer is one
 *     block whose I is the concatenated n_shared * I_shared (a sum of SwiGLU
 *     experts equals one SwiGLU over the concatenated intermediate).
 *     Weight pointers and strides must be 16-byte aligned.
 *   - Every call enqueues work on `stream` and returns without synchronising
 *     the host.  Data-dependent sizes (the union size) stay in device memory.
 *   - Argument checks run on the host before any HIP call, so an invalid call
 *     returns DE_ERR_INVALID / DE_ERR_UNSUPPORTED / DE_ERR_WORKSPACE and
 *     enqueues nothing.  Device pointers are only checked for NULL and
 *     alignment.  A launch failure returns DE_ERR_HIP.
 *   - Limits: 1 <= T <= 64 block positions; 1 <= k <= min(N, 32);
 *     1 <= N <= 256; H, I multiples of 8 for bf16 and of 4 for fp32 weights.
 *
 * Notation follows the paper: TopK_l(h) (Eq. 1), the block union U_l(B)
 * (Eq. 2, Eq. 3), the target MoE output y* (Eq. 4) and the fixed-footprint
 * draft output y^d (Eq. 5); acceptance follows Algorithm 1.
 */
#ifndef DRAFTEXPERT_H
#define DRAFTEXPERT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DE_ABI_VERSION 2

/* Return codes. */
#define DE_OK 0
#define DE_ERR_INVALID (-1)      /* NULL / misaligned pointer, size out of range */
#define DE_ERR_UNSUPPORTED (-2)  /* dtype or option combination not implemented */
#define DE_ERR_HIP (-3)          /* a HIP launch or runtime call failed */
#define DE_ERR_WORKSPACE (-4)    /* ws NULL or smaller than de_workspace_bytes() */
#define DE_ERR_NOT_RESIDENT (-5) /* a needed routed expert had no valid slot (Section 3.5:
                                    a missed expert must be loaded, never dropped) */

/* Router score functions (the router distribution R_l of Section 3.2). */
#define DE_SOFTMAX 0 /* scores softmax(z + b); selection key z + b */
#define DE_SIGMOID 1 /* scores sigmoid(z); selection key sigmoid(z) + b */

/* Expert weight element types.  An expert block is [G][U][D], G and U
 * [I, H], D [H, I], each matrix row-major [out, in]:
 *   DE_F32 / DE_BF16: rows * cols elements of 4 / 2 bytes;
 *   DE_Q4_0: the 4.5-bit block format of the paper's mobile platform
 *     (Section 4.1): each row in blocks of 32 weights, a block being 16 bytes
 *     of 4-bit codes q (byte j: weight j in the low nibble, weight j + 16 in
 *     the high nibble) and an fp16 scale d, weight = d (q - 8).  A matrix
 *     stores every row's codes first (cols / 2 bytes per row, block b of a row
 *     at byte 16 b), then every row's scales (cols / 16 bytes per row): 18
 *     bytes per 32 weights, rows * cols * 9 / 16 bytes per matrix.  H, I and
 *     the shared and draft I must be multiples of 32.  Applies to the routed,
 *     shared and draft experts of a layer; embedding, LM head and the dense
 *     layer stay bf16. */
#define DE_F32 0
#define DE_BF16 1
#define DE_Q4_0 2

/* Shape and options of one MoE layer. */
typedef struct de_moe_desc {
  int32_t hidden;       /* H */
  int32_t n_experts;    /* N routed experts */
  int32_t top_k;        /* k */
  int32_t inter;        /* I of each routed expert */
  int32_t shared_inter; /* concatenated shared intermediate (0: no shared path) */
  int32_t draft_inter;  /* I_d of the draft expert (0: none) */
  int32_t score_func;   /* DE_SOFTMAX or DE_SIGMOID */
  int32_t norm_topk;    /* 1: divide the k gates by their sum */
  float routed_scale;   /* multiplies every routed gate */
  int32_t wdtype;       /* DE_F32, DE_BF16 or DE_Q4_0 expert weights */
} de_moe_desc;

/* Where routed expert e lives: base + slot_of_expert[e] * slot_stride_bytes.
 * slot_of_expert NULL means slot e (all experts resident, in order).
 * A slot < 0 or >= n_slots marks an expert that is not resident.  The paper's
 * runtime loads a missed expert on demand and never drops it (Section 3.5,
 * Algorithm 1); the expert cache below does so before it launches.  A layer
 * call that meets a needed expert without a valid slot cannot load it: that
 * expert's term is left out of y (its partials are zero, nothing stale is
 * summed) and the workspace's status word records it, so that the next
 * de_layer_status (de_model_status for the model calls) returns
 * DE_ERR_NOT_RESIDENT. */
typedef struct de_expert_table {
  const void* base;              /* device: slot 0 */
  int64_t slot_stride_bytes;     /* >= 3*I*H*elem, multiple of 16 */
  const int32_t* slot_of_expert; /* device [N] or NULL */
  int32_t n_slots;               /* number of valid slots */
} de_expert_table;

/* Optional fused epilogue of a layer call.  With residual != NULL the layer
 * writes y = residual + layer(x) (the pre-norm residual stack); with
 * normed != NULL it also writes RMSNorm(y) = y / sqrt(mean(y^2) + eps), the
 * next layer's input.  residual may alias y (one block per position writes
 * each row after reading it); normed must not alias residual. */
typedef struct de_epilogue {
  const float* residual; /* device [T, H] or NULL */
  float* normed;         /* device [T, H] or NULL */
  float eps;
} de_epilogue;

int de_abi_version(void);
const char* de_error_string(int code);
/* The HIP runtime's message for the last failed HIP call the library saw on
 * this host thread ("" if none): the detail behind DE_ERR_HIP. */
const char* de_hip_error_detail(void);

/* Host-only validation of a layer descriptor (DE_OK or an error code). */
int de_check_desc(const de_moe_desc* d);

/* Scratch bytes needed by de_route_topk, de_grouped_swiglu, de_draft_layer
 * and de_verify_layer for blocks of up to T positions (0 on an invalid desc). */
size_t de_workspace_bytes(const de_moe_desc* d, int T);

/* Zeroes the control words at the start of a freshly allocated workspace
 * (enqueued on `stream`).  Required once per allocation before its first use
 * by a layer call; every layer call leaves its counters zero again.  Calls
 * that share one workspace must not run concurrently. */
int de_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

/* Device-side conditions of the layer calls made on workspace ws (a
 * de_workspace_bytes workspace), surfaced on the host: waits for `stream`,
 * reads the workspace's status word and clears it.  Returns DE_OK,
 * DE_ERR_NOT_RESIDENT when some call since the last check met a needed routed
 * expert whose slot is outside [0, n_slots) (its term was dropped; see
 * de_expert_table), DE_ERR_WORKSPACE for a bad ws, DE_ERR_HIP on a failed
 * copy.  Host-synchronous by design; the layer calls themselves never wait. */
int de_layer_status(void* ws, size_t ws_bytes, hipStream_t stream);

/* Router scoring and top-k selection (Eq. 1) with the gates of Eq. (4).
 *   x [T, H], w_router [N, H], bias [N] or NULL.
 *   topk_idx [T, k] int32: expert ids in descending selection key, ties to the
 *   lower id.  topk_gate [T, k]: softmax probability (or unbiased sigmoid) of
 *   each chosen expert, divided by the k-sum if norm_topk, times routed_scale.
 * Logits are accumulated in fp32. */
int de_route_topk(const de_moe_desc* d, int T, const float* x, const float* w_router,
                  const float* bias, int32_t* topk_idx, float* topk_gate, void* ws,
                  size_t ws_bytes, hipStream_t stream);

/* Union of the block's top-k sets with per-expert token lists (Eq. 2, Eq. 3).
 * Integer only, so deterministic.
 *   n_union [1]: |U|; union_ids [N]: members ascending, the tail set to -1;
 *   offsets [N+1]: list bounds, offsets[u]..offsets[u+1] for member u, entries
 *   past n_union equal to T*k; tok_list [T*k]: block positions, ascending
 *   within each member; gate_list [T*k]: the matching gates; pair_pos [T, k]:
 *   where (topk_idx[t,j], t) sits in the lists.
 * An id outside [0, N) or repeated within one position makes n_union = -1 and
 * leaves the other outputs unspecified. */
int de_expert_union(int T, int k, int N, const int32_t* topk_idx, const float* topk_gate,
                    int32_t* n_union, int32_t* union_ids, int32_t* offsets, int32_t* tok_list,
                    float* gate_list, int32_t* pair_pos, hipStream_t stream);

/* Grouped SwiGLU over the union plus the shared path (Eq. 4 without routing):
 *   y[t] = S(x_t) + sum_j gate[t,j] E_{idx[t,j]}(x_t),   E(v) = D(silu(Gv) * (Uv)).
 * Each union expert's weights are streamed from HBM once for all of its
 * positions.  Inputs are de_expert_union's outputs; shared_w may be NULL
 * when desc.shared_inter is 0.  Partial sums are combined in a fixed order
 * (no float atomics), so repeated calls are bitwise identical. */
int de_grouped_swiglu(const de_moe_desc* d, int T, const float* x, const de_expert_table* routed,
                      const int32_t* n_union, const int32_t* union_ids, const int32_t* offsets,
                      const int32_t* tok_list, const float* gate_list, const int32_t* pair_pos,
                      const void* shared_w, float* y, const de_epilogue* epi, void* ws,
                      size_t ws_bytes, hipStream_t stream);

/* Fixed-footprint draft layer (Eq. 5):
 *   y^d_t = S(x_t) + g_{t,e1} E_{e1}(x_t) + gamma * E^d(x_t),
 * e1 the top-1 expert and g_{t,e1} its target gate.  Only e1 of the routed
 * experts is read.  pred_idx / pred_gate [T, k] (may be NULL) receive the full
 * top-k of the draft router: the predicted verifier experts (Section 3.4).
 * draft_w NULL (or desc.draft_inter 0) drops the draft-expert term.
 * With bf16 weights and T = 1 the whole layer runs as one launch of the
 * persistent draft kernel (routing, gate/up, down and the combine with its
 * epilogue), with the same bits as the separate launches; the environment
 * variable DE_PD_SINGLE set to "0" keeps the separate launches.  The
 * epilogue's residual may be y itself. */
int de_draft_layer(const de_moe_desc* d, int T, const float* x, const float* w_router,
                   const float* bias, const de_expert_table* routed, const void* shared_w,
                   const void* draft_w, float gamma, float* y, int32_t* pred_idx,
                   float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                   hipStream_t stream);

/* The same layer with the r (1 <= r <= k) leading experts of each position
 * in the routed term, each with its target gate:
 *   y^d_t = S(x_t) + sum_{j<r} g_{t,j} E_{idx[t,j]}(x_t) + gamma * E^d(x_t).
 * r = 1 is de_draft_layer; draft_w NULL with r > 1 is the shared + top-r
 * self-drafter the paper compares with (Section 1, Table 3).  Only the r
 * experts are read.  DE_ERR_INVALID for r outside [1, k]. */
int de_draft_layer_topr(const de_moe_desc* d, int T, const float* x, const float* w_router,
                        const float* bias, const de_expert_table* routed, const void* shared_w,
                        const void* draft_w, float gamma, int r, float* y, int32_t* pred_idx,
                        float* pred_gate, const de_epilogue* epi, void* ws, size_t ws_bytes,
                        hipStream_t stream);

/* Target MoE layer over a verify block of T positions (Eq. 4): routing,
 * union build and the grouped SwiGLU in one call.  Every intermediate output
 * pointer (topk_idx .. pair_pos) may be NULL; non-NULL ones receive the same
 * values as de_route_topk / de_expert_union. */
int de_verify_layer(const de_moe_desc* d, int T, const float* x, const float* w_router,
                    const float* bias, const de_expert_table* routed, const void* shared_w,
                    float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                    int32_t* union_ids, int32_t* offsets, int32_t* tok_list, float* gate_list,
                    int32_t* pair_pos, const de_epilogue* epi, void* ws, size_t ws_bytes,
                    hipStream_t stream);

/* de_verify_layer for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels and results, with the layer's scratch taken from a
 * file-scope device array of de_noalloc_scratch_bytes() bytes (16 MiB) that
 * each GPU holds until the process ends, instead of a caller workspace.  The
 * call allocates nothing.  DE_ERR_WORKSPACE when de_workspace_bytes(d, T)
 * exceeds that size.  Every call on one GPU shares that GPU's array: calls
 * that overlap on one GPU (other streams, other host threads) race.  A needed
 * routed expert without a valid slot has its term dropped as in
 * de_verify_layer, but nothing reports it (use de_verify_layer and
 * de_layer_status for that). */
size_t de_noalloc_scratch_bytes(void);
int de_verify_layer_noalloc(const de_moe_desc* d, int T, const float* x, const float* w_router,
                            const float* bias, const de_expert_table* routed, const void* shared_w,
                            float* y, int32_t* topk_idx, float* topk_gate, int32_t* n_union,
                            int32_t* union_ids, int32_t* offsets, int32_t* tok_list,
                            float* gate_list, int32_t* pair_pos, const de_epilogue* epi,
                            hipStream_t stream);

/* Greedy exact acceptance (Algorithm 1, verify and accept):
 *   target_argmax[j] = argmax_v target_logits[j, v] (ties to the lowest v,
 *   NaN treated as -inf), j = 0..K; out[0] = n = largest m <= K with
 *   draft_tokens[i-1] == target_argmax[i-1] for all i <= m; out[1] =
 *   target_argmax[n] (the bonus token).  K = 0 gives the argmax of one row.
 *   draft_tokens may be NULL when K is 0.  One launch: rows are split in
 *   4096-logit chunks reduced in a fixed order (deterministic).  Scratch: ws
 *   of de_accept_workspace_bytes(K, V) bytes, zero-filled once by
 *   de_workspace_init. */
size_t de_accept_workspace_bytes(int K, int V);
int de_accept_len(int K, int V, const float* target_logits, const int32_t* draft_tokens,
                  int32_t* target_argmax, int32_t* out, void* ws, size_t ws_bytes,
                  hipStream_t stream);

/* ---- Stacked-model glue (a pre-norm residual stack without attention) ---- */

/* logits [T, V] = x [T, H] . W^T with W bf16 [V, H] (the LM head). */
int de_lm_head(int T, int H, int V, const float* x, const void* w_lm, float* logits,
               hipStream_t stream);

/* out [T, H] = x / sqrt(mean(x^2) + eps) per row (unit gain). out may alias x. */
int de_rmsnorm(int T, int H, const float* x, float eps, float* out, hipStream_t stream);

/* h [T, H] = fp32(emb[tokens[t]]) with emb bf16 [V, H]; tokens is a device
 * int32 array.  normed (may be NULL) receives RMSNorm(h).  A token id outside
 * [0, V) reads nothing: its rows of h and normed are NaN, and status (a device
 * int32, may be NULL) gets bit 2 set (OR-ed in, never cleared here). */
int de_embed_gather(int T, int H, int V, const int32_t* tokens, const void* emb, float* h,
                    float* normed, float eps, int32_t* status, hipStream_t stream);

/* Dense SwiGLU layer y = E(x) of intermediate I (layer 0 of the stack), with
 * the optional epilogue.  Scratch: de_dense_workspace_bytes(T, H, I).  The
 * down projection runs in up to three intermediate chunks whose partials are
 * summed in chunk order. */
size_t de_dense_workspace_bytes(int T, int H, int I);
int de_dense_swiglu(int T, int H, int I, int wdtype, const float* x, const void* w, float* y,
                    const de_epilogue* epi, void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- The stacked model and one draft-then-verify step (Algorithm 1) ---- */

/* Weights of one MoE layer of the stack. */
typedef struct de_layer_weights {
  const float* w_router;  /* fp32 [N, H] */
  const float* bias;      /* fp32 [N] or NULL */
  de_expert_table routed; /* routed experts (resident, or the slots of a cache) */
  const void* shared_w;   /* shared-path block; NULL when moe.shared_inter is 0 */
  const void* draft_w;    /* draft-expert block or NULL (drops the gamma term) */
  float gamma;            /* scale of the draft-expert term of Eq. (5) */
} de_layer_weights;

/* A pre-norm residual stack without attention (attention and its KV cache
 * stay resident and are outside this path):
 *   h = Emb[token];  h += Dense(RMSNorm(h))          (layer 0, if dense_inter > 0)
 *   h += MoE_l(RMSNorm(h)),  l = 1..n_layers          (Eq. 4 target / Eq. 5 draft)
 *   logits = W_lm RMSNorm(h).
 * All RMSNorms have unit gain and epsilon eps.  Without attention a block
 * position depends only on its own token. */
typedef struct de_model {
  de_moe_desc moe;                /* shape of every MoE layer */
  int32_t n_layers;               /* MoE layers (0..4096) */
  int32_t vocab;                  /* V */
  int32_t dense_inter;            /* I of the dense layer 0 (0: no dense layer) */
  int32_t dense_wdtype;           /* DE_F32 or DE_BF16 */
  float eps;                      /* RMSNorm epsilon (>= 0) */
  const void* emb;                /* bf16 [V, H] */
  const void* dense_w;            /* dense block [G|U|D]; NULL when dense_inter is 0 */
  const void* lm_head;            /* bf16 [V, H] */
  const de_layer_weights* layers; /* HOST array [n_layers]; read during the call only */
  int32_t draft_topr;             /* routed experts of every draft layer: 1 (Eq. 5, also
                                     when 0) .. top_k (de_draft_layer_topr) */
} de_model;

/* Forward modes: the MoE layers as the target (Eq. 4) or the drafter (Eq. 5). */
#define DE_TARGET 0
#define DE_DRAFT 1

/* Scratch bytes of the model calls for blocks of up to T positions (0 on an
 * invalid model).  A fresh allocation is zero-filled once with
 * de_workspace_init; every model call leaves its control words zero again.
 * Calls that share one workspace must not run concurrently. */
size_t de_model_workspace_bytes(const de_model* m, int T);

/* Host-only validation of a model (DE_OK or an error code).  Checks the MoE
 * shape, every layer's pointers and table, and the glue's sizes. */
int de_check_model(const de_model* m);

/* Device-side conditions of the model calls made on workspace ws, as
 * de_layer_status: DE_ERR_NOT_RESIDENT when a MoE layer met a needed routed
 * expert without a valid slot (a table of m->layers marks it absent),
 * DE_ERR_INVALID when a token id outside [0, vocab) reached the embedding.
 * Waits for `stream` and clears the word. */
int de_model_status(const de_model* m, void* ws, size_t ws_bytes, hipStream_t stream);

/* Logits of T independent positions (each a token id, device int32 [T]):
 * logits [T, V] fp32; argmax [T] (may be NULL) the row argmax, ties to the
 * lowest id; n_union [n_layers] (may be NULL; DE_TARGET only) the union size
 * of every MoE layer over the T positions (Eq. 3). */
int de_model_forward(const de_model* m, int T, const int32_t* tokens, int mode, float* logits,
                     int32_t* argmax, int32_t* n_union, void* ws, size_t ws_bytes,
                     hipStream_t stream);

/* One exact draft-then-verify step with K drafts (Algorithm 1, fixed K):
 *   block [K+1] int32: block[0] = the last committed token (input);
 *     block[i+1] = argmax of the drafter's logits at block[i], i = 0..K-1
 *     (output: the drafts);
 *   the target then scores the K+1 positions of block in one pass:
 *   target_argmax [K+1] its row argmax; out [2] = (n, bonus) as
 *   de_accept_len, so the step emits block[1..n] followed by the bonus token;
 *   n_union [n_layers] (may be NULL) the verify union size per MoE layer;
 *   pred_idx [K, n_layers, k] (may be NULL) the drafter's router top-k at
 *   draft position i in layer l: the experts predicted for verify position i.
 * Every launch is enqueued on `stream`; nothing synchronises the host.
 * Scratch: de_model_workspace_bytes(m, K + 1). */
int de_spec_step(const de_model* m, int K, int32_t* block, int32_t* target_argmax, int32_t* out,
                 int32_t* n_union, int32_t* pred_idx, void* ws, size_t ws_bytes,
                 hipStream_t stream);

/* Plain greedy decoding with the target, one position per pass:
 * tokens [n_steps + 1], tokens[0] the input, tokens[i+1] = argmax of the
 * target logits at tokens[i].  Scratch: de_model_workspace_bytes(m, 1). */
int de_greedy_decode(const de_model* m, int n_steps, int32_t* tokens, void* ws, size_t ws_bytes,
                     hipStream_t stream);

/* ---- Expert cache over a pinned host pool (Section 3.5, Algorithm 1) ----
 *
 * Routed experts live in a pinned host pool; each MoE layer has n_slots HBM
 * slots.  The cache keeps the accelerator expert set C (which expert is in
 * which slot), starts copies on its own streams (prefetches of predicted
 * verifier experts, on-demand loads of misses), and hands the kernels a
 * per-layer slot table in which exactly the experts of the current request
 * are marked resident.  Bookkeeping is host-side and deterministic; only the
 * stall time depends on timing.
 *
 * Policy (the paper names the sets but no eviction rule):
 *   - a free slot (lowest index) is used first; otherwise the least recently
 *     used slot (ties: lowest index) whose expert is neither needed by the
 *     current request nor predicted for the current block; a demand load may
 *     fall back to a predicted, unneeded expert; a prefetch may not, and is
 *     skipped when no slot qualifies;
 *   - an expert in flight counts as resident: a request for it waits on its
 *     copy (hits include such waits);
 *   - "use" (LRU time) is a request or a copy; a prefetch of a resident
 *     expert changes nothing but the predicted set. */
typedef struct de_cache de_cache; /* opaque */

typedef struct de_cache_cfg {
  int32_t n_layers;          /* L */
  int32_t n_experts;         /* N routed experts per layer */
  int32_t n_slots;           /* HBM slots per layer, 1..N */
  int32_t fake_copies;       /* 1: copies are host memcpy and every pointer below is
                                host memory (bookkeeping without a GPU) */
  int64_t expert_bytes;      /* bytes of one expert block, multiple of 16 */
  int64_t slot_stride_bytes; /* >= expert_bytes, multiple of 256 */
  const void* host_pool;     /* pinned host [L][N] blocks, stride expert_bytes */
  void* slot_pool;           /* device [L][n_slots] blocks, stride slot_stride_bytes */
  int32_t* slot_map;         /* device int32 [L][N]: the slot tables the kernels read */
} de_cache_cfg;

typedef struct de_cache_counts {
  int64_t prefetch_issued;  /* copies started by de_cache_prefetch */
  int64_t prefetch_used;    /* ... needed by a verify request of the same block */
  int64_t prefetch_wasted;  /* ... evicted, or left when their block ended, unused */
  int64_t prefetch_skipped; /* predictions dropped for want of an evictable slot */
  int64_t draft_needed;     /* experts requested by the draft path (top-1) */
  int64_t draft_hits;       /* ... found resident or in flight */
  int64_t verify_needed;    /* experts requested by verify chunks */
  int64_t verify_hits;      /* ... found resident or in flight */
  int64_t demand_loads;     /* copies started by de_cache_ensure (misses) */
  int64_t evictions;
  int64_t bytes_copied;     /* host-to-device bytes of all copies */
  double stall_us;          /* time the compute stream waited for copies */
  int64_t draft_layers;     /* MoE layers run by de_spec_step_cached on the draft path */
  double draft_layer_us;    /* ... their summed duration on the compute stream */
  int64_t verify_layers;    /* verify MoE layers run by de_spec_step_cached */
  double verify_layer_us;   /* ... their summed duration (routing, readback, copies
                               waited for, every chunk, combine) */
} de_cache_counts;

#define DE_NEED_DRAFT 0  /* the draft path's top-1 expert (Eq. 5) */
#define DE_NEED_VERIFY 1 /* a chunk of the verify union (Eq. 3) */

/* Creates a cold cache (every slot empty; slot_map filled with -1).  The
 * caller owns the three memory regions; the cache owns two copy streams
 * (default priority), per-slot events and a small pinned scratch. */
int de_cache_create(const de_cache_cfg* cfg, de_cache** out);
/* Waits for outstanding copies and frees the cache's own objects. */
int de_cache_destroy(de_cache* c);
/* Empties every slot and zeroes the statistics (waits for copies first). */
int de_cache_reset(de_cache* c);
/* Starts a new draft/verify block: prefetched experts the ending block's
 * verify never requested count as wasted; every predicted set is cleared. */
int de_cache_begin_block(de_cache* c);
/* Records experts_host[0..n) (host array) as predicted verifier experts of
 * `layer` for the current block and starts a copy for each that is neither
 * resident nor in flight (Algorithm 1: prefetch of the newly predicted set
 * minus C and P).  Returns without waiting. */
int de_cache_prefetch(de_cache* c, int layer, const int32_t* experts_host, int n);
/* Makes the n distinct experts needed_host[0..n) (n <= n_slots) resident in
 * `layer`, starting on-demand copies for misses; `compute` waits for every
 * copy they depend on; then the layer's slot table is rewritten on `compute`
 * with exactly these n experts resident (-1 elsewhere).  Host-synchronous
 * bookkeeping; the GPU work is enqueued. */
int de_cache_ensure(de_cache* c, int layer, const int32_t* needed_host, int n, int purpose,
                    hipStream_t compute);
/* The work enqueued on `compute` so far is the last to read `layer`'s slots:
 * later copies into them wait for it. */
int de_cache_release(de_cache* c, int layer, hipStream_t compute);
/* The expert table of `layer` (base = its first slot, slot_of_expert = its
 * row of slot_map). */
int de_cache_table(const de_cache* c, int layer, de_expert_table* table);
/* Statistics since creation or the last reset (waits for every copy and
 * event it reads). */
int de_cache_stats(de_cache* c, de_cache_counts* stats);
/* Host view of which slot holds each expert of `layer` (-1: none), into
 * slot_of_expert_host [N]. */
int de_cache_slots(const de_cache* c, int layer, int32_t* slot_of_expert_host);

/* de_spec_step with the routed experts behind the cache (Algorithm 1 with
 * offload).  At every draft position and MoE layer the drafter's router runs
 * first; its top-k is read back to the host, the top-1 expert is requested
 * (DE_NEED_DRAFT) and the whole top-k is prefetched for verification; then
 * the layer's grouped part runs on the cached slots.  Verification reads each
 * layer's union back, requests it in chunks of at most n_slots members
 * (members resident or in flight first, then the rest, each part in
 * ascending id), and combines after the last chunk, which gives the same
 * bits as the resident step.  The routed tables of m->layers are not used.
 * Synchronises the host with `stream` once per layer and position.
 * Arguments as de_spec_step; pred_idx [K, n_layers, k] may be NULL. */
int de_spec_step_cached(const de_model* m, de_cache* cache, int K, int32_t* block,
                        int32_t* target_argmax, int32_t* out, int32_t* n_union, int32_t* pred_idx,
                        void* ws, size_t ws_bytes, hipStream_t stream);

/* ---- Confidence-expansion truncation (Section 3.4, Eqs. 12-14; Algorithm 1) ----
 *
 * Drafting stops before appending draft token i when the token is uncertain
 * and would grow the predicted verifier set too much: q_i < tau and
 * Delta_i > B_i.  q_i is the largest softmax probability of the token's draft
 * logits; the predicted verifier experts of the token in layer l are the
 * drafter's router top-k there; the block-level predicted set is the union of
 * those (layer, expert) pairs over the kept tokens and Delta_i is how many
 * pairs token i would add.  B_i is a fixed count of layer-experts, or, with
 * DE_BUDGET_CACHE, the room the predicted set still has in the expert cache:
 * sum over layers of max(0, slots - pairs of the set in that layer). */
#define DE_BUDGET_CACHE (-1)

/* q [T] fp32 (device) = 1 / sum_v exp(l_v - max_v l_v) for each row of
 * logits [T, V] fp32 (device, row-major).  A NaN logit counts as -infinity;
 * a row with no logit above -infinity gives NaN.  One launch on `stream`. */
int de_confidence(int T, int V, const float* logits, float* q, hipStream_t stream);

/* Eq. 12-14 for one draft token, in one launch on `stream` (all pointers
 * device):
 *   pred_idx [L, k] int32: the token's predicted experts per layer (ids in
 *     [0, N), N <= 256; an id outside is skipped and counted in out[4]);
 *   uhat [L, ceil(N / 64)] uint64 (8-byte aligned): the block-level set,
 *     bit e of layer l's words = pair (l, e); read as empty when `first` is
 *     nonzero (no clearing needed before a block's first token); grown by
 *     the token's pairs only when the token is kept;
 *   q [1] fp32: the token's confidence (e.g. from de_confidence);
 *   tau: the confidence threshold (not NaN);
 *   budget: B_i >= 0, or DE_BUDGET_CACHE to derive it from `slots` per layer;
 *   out [5] int32 = (Delta_i, stop (0/1), B_i used, set size after,
 *     ids out of range).
 * DE_ERR_INVALID on bad sizes or pointers. */
int de_expansion(int L, int k, int N, const int32_t* pred_idx, uint64_t* uhat, int first,
                 const float* q, float tau, int budget, int slots, int32_t* out,
                 hipStream_t stream);

typedef struct {
  float tau;         /* confidence threshold */
  int32_t budget;    /* B_i: a fixed count of layer-experts, or DE_BUDGET_CACHE */
  int32_t slots;     /* slots per layer for DE_BUDGET_CACHE; 0 with a cache: its n_slots */
  int32_t prefetch;  /* with a cache: nonzero starts the kept tokens' verifier prefetches */
} de_trunc_cfg;

/* One exact draft-then-verify step with truncation (Algorithm 1): up to
 * k_max drafts, each kept or stopped by Eq. 14 after its draft pass; the
 * kept drafts d_1..d_n_drafted are verified as de_spec_step verifies K of
 * them.  With `cache` (may be NULL) the routed experts come through it as in
 * de_spec_step_cached, except that a draft token's verifier prefetches (its
 * top-k in every layer) are started after the token is kept (only with
 * cfg->prefetch), and a stopped token starts none.  tau = 0 never stops:
 * the fixed-K step.
 *   block [k_max+1]: block[0] input; block[1..n_drafted] the kept drafts
 *     (entries after them unspecified);
 *   target_argmax [k_max+1] (first n_drafted+1 written), out [2] = (n, bonus)
 *     against the kept drafts, n_union [n_layers] (may be NULL);
 *   n_drafted: HOST int32, the number of kept drafts;
 *   pred_idx [k_max, n_layers, k] (required): the drafter's top-k per
 *     evaluated token and layer;
 *   q [k_max] fp32 (required): the confidence of every evaluated token;
 *   trace [k_max, 4] int32 (may be NULL): per evaluated token
 *     (Delta_i, stop, B_i, set size after).
 * Tokens after the stopped one are not evaluated (their entries untouched).
 * Synchronises the host with `stream` once per evaluated token (and, with a
 * cache, once per layer and position).  Scratch:
 * de_model_workspace_bytes(m, k_max + 1). */
int de_spec_step_trunc(const de_model* m, de_cache* cache, int k_max, const de_trunc_cfg* cfg,
                       int32_t* block, int32_t* target_argmax, int32_t* out, int32_t* n_drafted,
                       int32_t* n_union, int32_t* pred_idx, float* q, int32_t* trace, void* ws,
                       size_t ws_bytes, hipStream_t stream);

/* ---- Self-distillation signals (Section 3.3, Eqs. 6-10) ----
 *
 * Training the draft experts is outside this library; these calls emit what
 * it consumes, from passes the runtime already makes. */

/* The residual target of Eq. 6 for the last de_verify_layer (or
 * de_grouped_swiglu) call made with the same desc, T and workspace on
 * `stream`: m_star [T, H] fp32 (device) = y* - S(x) - g_e1 E_e1(x), i.e. the
 * sum of each position's routed partials ranked 2..k, in list order. */
int de_residual_target(const de_moe_desc* d, int T, const void* ws, size_t ws_bytes,
                       float* m_star, hipStream_t stream);

/* The router logits z = W_r x [T, N] fp32 of the last layer call made with
 * the same desc, T and workspace (device copy on `stream`). */
int de_layer_router_logits(const de_moe_desc* d, int T, const void* ws, size_t ws_bytes,
                           float* z, hipStream_t stream);

/* Row divergences (one launch; all pointers device): for each row r of a
 * (target) [rows, lda] and b (draft) [rows, ldb], first n values:
 *   sigmoid = 0: p = softmax((a_r + bias) / tau), q = softmax((b_r + bias) / tau),
 *     kl[r] = tau^2 KL(p || q) (Eq. 8 with temperature tau; Eq. 10 with tau 1
 *     and the router bias), and, when ce is not NULL, ce[r] =
 *     -log softmax(b_r + bias)[argmax (a_r + bias)] (Eq. 9; ties to the lowest
 *     index, NaN as -infinity);
 *   sigmoid = 1 (sigmoid routers, Eq. 10): p and q the sigmoid scores
 *     normalised to sum one, kl[r] = KL(p || q); bias and ce must be NULL and
 *     tau 1.
 * bias [n] may be NULL. */
int de_row_kl(int rows, int n, const float* a, int lda, const float* b, int ldb,
              const float* bias, int sigmoid, float tau, float* kl, float* ce,
              hipStream_t stream);

/* The self-distillation signals of T teacher-forced positions (tokens [T],
 * device), from one target pass and one draft pass over them (without
 * attention a position depends only on its token):
 *   m_star [n_layers, T, H]: the residual target of Eq. 6 at every MoE layer;
 *   router_kl [n_layers, T]: Eq. 10, KL from the target's router distribution
 *     at the target's layer input to the router distribution at the draft
 *     path's layer input (softmax(z + b); sigmoid routers: normalised scores);
 *   logit_kl [T]: Eq. 8 at temperature tau; token_ce [T]: Eq. 9.
 * m_star and router_kl are both given or both NULL, likewise logit_kl and
 * token_ce.  All device fp32.  Scratch: de_model_workspace_bytes(m, T). */
int de_distill_signals(const de_model* m, int T, const int32_t* tokens, float tau,
                       float* m_star, float* router_kl, float* logit_kl, float* token_ce,
                       void* ws, size_t ws_bytes, hipStream_t stream);

/* Pure streaming read of `bytes` (multiple of 16) from buf: the measured HBM
 * read ceiling.  sink [1] receives a value that depends on every byte. */
int de_stream_probe(const void* buf, size_t bytes, float* sink, hipStream_t stream);

/* ---- Instrumentation ---- */

/* Kernel phases that can be bracketed by caller-owned HIP events. */
#define DE_PHASE_GATEUP 0 /* the grouped gate/up kernel (Eq. 4 first half) */
#define DE_PHASE_DOWN 1   /* the grouped down-projection kernel */
#define DE_PHASE_LAYER 2  /* the verify layer's single launch (de_verify_single_launch) */
#define DE_PHASE_DRAFT_PASS 3 /* the persistent launch that runs a draft position's MoE
                               * layers (the first launch, for stacks of more than 32) */

/* Arms a one-shot timer: the next layer or model call (de_grouped_swiglu,
 * de_draft_layer, de_verify_layer, de_dense_swiglu, the model forward and
 * step calls) made on this host thread
 * records `start` on its stream right before launching the kernel of `phase`
 * and `stop` right after it, then disarms.  Either event may be NULL.  The
 * events are created and read by the caller (e.g. hipEventElapsedTime). */
int de_time_next_phase(int phase, hipEvent_t start, hipEvent_t stop);

/* 1 when de_verify_layer (and the verify passes of the model calls without a
 * chained router) runs the layer of this shape as one launch, else 0.  That launch covers Eq. 4 over the block's union (top-k selection
 * from the router logits, union, grouped gate/up and down, shared path and
 * the combine with its epilogue) and gives the same bits as the separate
 * launches; every armed phase timer then brackets it.  It serves bf16
 * weights and blocks of 2 or more positions whose staged rows fit a CU's LDS
 * (the V2-Lite layer at T = 2..9).  It is off unless the environment
 * variable DE_VERIFY_FUSED is "1": on MI355X it measures slower than the
 * separate launches (235 against 158 us at T = 9). */
int de_verify_single_launch(const de_moe_desc* d, int T);

#ifdef __cplusplus
}
#endif

#endif /* DRAFTEXPERT_H */
