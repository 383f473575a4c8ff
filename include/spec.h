/*
 * spec.h -- C ABI of the SpeContext decode-step hot path for MI355X (gfx950).
 *
 * SpeContext (arXiv 2512.00722) runs a lightweight retrieval head before the
 * LLM: it keeps a full key cache K_r, forms attention weights for the current
 * query after the Q/K projection, and selects the important tokens once per
 * decode step (Sec. 4.3, "Implementation Details").  The LLM then attends
 * only to the K/V rows at those tokens, gathered per KV head (Sec. 4.3,
 * "Support for MHA"/"Support for GQA"); the same selection serves every layer
 * (Sec. 7.2.1).  Elastic loading keeps the previous selection S_last and
 * loads only S_now - S_last into the places of S_last - S_now (Sec. 5.4).
 *
 * Conventions for every entry point
 * ---------------------------------
 *  - bf16 tensors are passed as uint16_t bit patterns.  All tensor pointers
 *    are DEVICE pointers; `spec_dims` and `spec_elastic` are host structs.
 *  - Layouts are token-major and row-major:
 *        q_r     [B][H_r][d_r]
 *        K_r     [B][L_cap][H_r][d_r]        (sequence stride kr_stride_b)
 *        q       [n_layers][B][H_q][d]
 *        K, V    [n_layers][B][L_cap][H_kv][d] (strides kv_stride_layer,
 *                                              kv_stride_b; the inner
 *                                              [token][head][dim] block is
 *                                              contiguous)
 *        scores  [B][n_sets][L_max] fp32
 *        idx     [B][n_sets][k_max] int32, counts [B] int32,
 *        out     [n_layers][B][H_q][d] fp32, lse [n_layers][B][H_q] fp32.
 *  - Token sets (spec_dims.n_sets): n_sets = 1 is the batch-level mapping of
 *    Sec. 4.2, one set per sequence from the retrieval heads' softmax weights
 *    summed over heads, shared by every KV head and layer.  n_sets = H_kv is
 *    the head-level mapping of Sec. 4.2/4.3 ("Support for GQA"): set g is
 *    chosen from the element-wise maximum, per token, of the weights of
 *    retrieval heads g*H_r/H_kv .. (g+1)*H_r/H_kv - 1, and KV head g (with
 *    its G query heads) attends over set g only.  Every set of a sequence has
 *    the same size k_b.
 *  - Per-sequence lengths live on the device and are clamped in the kernels,
 *    not validated: L_b = min(seq_lens[b], L_max) (negative -> 0) and
 *    k_b = min(ks[b], L_b, k_max) (negative -> 0).
 *  - Ownership: the caller allocates every buffer, including the workspace
 *    sized by spec_workspace_size().  The library never allocates, frees or
 *    synchronises; every call only enqueues work on `stream` (a hipStream_t,
 *    NULL = the null stream).  Outputs are valid once the stream reaches them.
 *  - Alignment: bf16 tensors, `out` and the workspace must be 16-byte
 *    aligned; int32/fp32 arrays (seq_lens, ks, scores, idx, counts, lse,
 *    slot_tok, n_changed) 4-byte aligned.
 *  - Errors: every argument check is done on the host BEFORE any HIP call,
 *    so on error nothing is enqueued.  SPEC_ERR_INVALID: null pointer,
 *    non-positive dimension, H_q % H_kv != 0, L_max > L_cap, k_max > L_max,
 *    a misaligned pointer, a negative or non-finite scale, a stride not a
 *    multiple of 8 elements or smaller than the block it steps over, a
 *    non-zero `reserved`.  SPEC_ERR_UNSUPPORTED:
 *    d != 128, d_r not 64 or 128, H_r > 16, G = H_q/H_kv not a power of
 *    two up to 128, H_kv > 16, n_sets not 1 or H_kv, n_sets = H_kv with H_r
 *    not a multiple of H_kv or B*n_sets > 65535, B or n_layers > 65535, and
 *    for elastic loading L_cap > 245760 or n_sets != 1.  SPEC_ERR_WORKSPACE: ws_bytes
 *    below spec_workspace_size() (SPEC_ERR_TOO_LARGE: above the static scratch
 *    of spec_step_noalloc).  SPEC_ERR_HIP: a launch failed; the HIP
 *    error code is kept (per thread) for spec_last_hip_error().
 *  - Calls are reentrant; concurrent calls must not share a workspace.
 *  - Debugging: with the environment variable SPEC_DEBUG=1 (read at every
 *    call) each entry point first copies the device-resident lengths and
 *    indices it is given to the host and returns SPEC_ERR_INVALID, with
 *    nothing enqueued, for values the kernels would otherwise clamp:
 *    seq_lens outside [0, L_max], negative ks, counts outside [0, k_max],
 *    idx entries below counts outside [0, L_cap), token ids outside the
 *    vocabulary; after the launch it synchronises the stream and reports an
 *    asynchronous failure as SPEC_ERR_HIP.  The calls then synchronise and
 *    cannot be captured in a graph.
 *  - Schedule switches (environment, read at every call; results are the
 *    same bit for bit, only the kernels' schedule changes):
 *    SPEC_TOPK_PATH=tiles takes the tiled selection kernels for short rows
 *    too; SPEC_ATTN_SCHEDULE=cold starts every attention work unit cold (no
 *    pipelining across units); SPEC_ATTN_ORDER=perm keeps the permuted work
 *    order on ragged batches; SPEC_ELASTIC_PATH=copy or =fused takes one
 *    elastic-loading path for every sequence of spec_step.
 */
#ifndef SPEC_H_
#define SPEC_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPEC_API __attribute__((visibility("default")))

typedef enum spec_status {
  SPEC_OK = 0,
  SPEC_ERR_INVALID = 1,
  SPEC_ERR_UNSUPPORTED = 2,
  SPEC_ERR_WORKSPACE = 3,
  SPEC_ERR_HIP = 4,
  SPEC_ERR_TOO_LARGE = 5  /* spec_step_noalloc: the step needs more workspace
                             than its static scratch holds                   */
} spec_status;

typedef enum spec_op {
  SPEC_OP_SCORE = 0,
  SPEC_OP_TOPK = 1,
  SPEC_OP_GATHER = 2,
  SPEC_OP_ATTN = 3,
  SPEC_OP_DELTA = 4,
  SPEC_OP_STEP = 5,
  SPEC_OP_FRONTEND = 6,
  SPEC_OP_OFFLOAD = 7     /* spec_step_offload */
} spec_op;

/* A hipStream_t handle; NULL selects the null stream. */
typedef void* spec_stream;

/* Problem dimensions (host struct). */
typedef struct spec_dims {
  int32_t B;        /* sequences in the batch                                 */
  int32_t L_cap;    /* token capacity of every cache row                      */
  int32_t L_max;    /* host upper bound on seq_lens (sizes grids), <= L_cap   */
  int32_t k_max;    /* host upper bound on ks (row length of idx), <= L_max   */
  int32_t H_r;      /* retrieval-head heads                                   */
  int32_t d_r;      /* retrieval-head head dimension (64 or 128)              */
  int32_t n_layers; /* LLM layers attended with one selection                 */
  int32_t H_q;      /* LLM query heads                                        */
  int32_t H_kv;     /* LLM KV heads; query head h reads KV head h / (H_q/H_kv) */
  int32_t d;        /* LLM head dimension (128)                               */
  int64_t kr_stride_b;     /* elements between sequences of K_r; 0 = L_cap*H_r*d_r */
  int64_t kv_stride_layer; /* elements between layers of K/V; 0 = B*kv_stride_b   */
  int64_t kv_stride_b;     /* elements between sequences of K/V; 0 = L_cap*H_kv*d */
  float scale_r;    /* retrieval softmax scale; 0 = 1/sqrt(d_r)               */
  float scale;      /* LLM attention scale; 0 = 1/sqrt(d)                     */
  int32_t n_sets;   /* token sets per sequence: 1 (one set for every KV head,
                       summed heads) or H_kv (one per KV head, group maximum) */
  int32_t reserved; /* must be 0                                              */
} spec_dims;

/* Device-resident elastic-loading state (host struct of device pointers).
 *   slot_tok  [B][k_max] int32: token held by each slot, -1 = empty (S_last);
 *   kbuf,vbuf [n_layers][B][k_max][H_kv][d] bf16: the rows held by the slots;
 *   n_changed [B] int32 (output): rows loaded by the last update;
 *   slot_src  [B][k_max] int32 (output): per slot, the token the last update
 *             loaded into it, or -1 (kept or left empty).                   */
typedef struct spec_elastic {
  int32_t* slot_tok;
  uint16_t* kbuf;
  uint16_t* vbuf;
  int32_t* n_changed;
  int32_t* slot_src;
} spec_elastic;

/* Retrieval scoring (Sec. 4.3 "Implementation Details"; Eq. 1 per head;
 * the mappings of Sec. 4.2).  For t < L_b:
 *     l[h,t] = scale_r * dot(q_r[b,h,:], K_r[b,t,h,:]),
 *     p[h,t] = exp(l[h,t] - M_h) / Z_h
 * with M_h = max_t l[h,t] and Z_h = sum_t exp(l[h,t] - M_h) (softmax per head
 * over all cached tokens), then
 *     n_sets = 1:    scores[b,0,t] = sum_h p[h,t]
 *     n_sets = H_kv: scores[b,g,t] = max over the heads h of group g of p[h,t].
 * scores[b,g,t] = -inf for L_b <= t < L_max.  Computed in fp32 from bf16
 * inputs.  Needs workspace spec_workspace_size(SPEC_OP_SCORE).             */
SPEC_API spec_status spec_score(const spec_dims* dm, const uint16_t* q_r,
                       const uint16_t* k_r, const int32_t* seq_lens,
                       float* scores, void* ws, size_t ws_bytes,
                       spec_stream stream);

/* Token selection (Sec. 4.3: the important tokens are selected from the
 * attention weights).  For each sequence b and set g, the k_b tokens t < L_b
 * with the largest scores[b,g,t]; among equal scores the lower token index
 * wins.  idx[b,g, 0..k_b) receives them in ascending token order and
 * idx[b,g, k_b..k_max) is set to -1.  counts (nullable) receives k_b.  The
 * selection is exact on the fp32 keys.  Needs workspace
 * spec_workspace_size(SPEC_OP_TOPK).                                          */
SPEC_API spec_status spec_topk(const spec_dims* dm, const float* scores,
                      const int32_t* seq_lens, const int32_t* ks,
                      int32_t* idx, int32_t* counts, void* ws, size_t ws_bytes,
                      spec_stream stream);

/* Materialised KV gather (Sec. 4.3 "Support for MHA": the selected KV is
 * loaded per head).  For every layer, sequence, KV head g and j < counts[b]:
 *     k_sel[l,b,j,g,:] = K[l,b,idx[b,s,j],g,:],  v_sel likewise,
 * with s = 0 (n_sets = 1: whole rows move) or s = g (n_sets = H_kv: each
 * head's piece comes from its own set), a bit-exact copy.  k_sel/v_sel are
 * dense [n_layers][B][k_max][H_kv][d], the layout compact-mode attention
 * reads; rows j >= counts[b] are left unchanged.  idx entries must lie in
 * [0, L_b); out-of-range entries are clamped into [0, L_cap).  No workspace. */
SPEC_API spec_status spec_gather(const spec_dims* dm, const uint16_t* k_cache,
                        const uint16_t* v_cache, const int32_t* idx,
                        const int32_t* counts, uint16_t* k_sel,
                        uint16_t* v_sel, spec_stream stream);

/* Sparse GQA decode attention (Eq. 1 over the selected rows; Sec. 4.3
 * "Support for GQA": the G = H_q/H_kv query heads of a group share KV head
 * g = h / G).  For every layer l, sequence b and query head h:
 *     s_j = scale * dot(q[l,b,h,:], Kj[g,:]),   j < counts[b]
 *     out[l,b,h,:] = sum_j softmax_j(s) * Vj[g,:],  lse[l,b,h] = log sum_j e^{s_j}
 * Indexed mode (idx != NULL): Kj = K[l,b,idx[b,s,j]] read from the caches,
 * s = 0 for n_sets = 1 and s = g for n_sets = H_kv (the gather is fused;
 * indices outside [0, L_cap) are clamped into it).
 * Compact mode (idx == NULL): k/v are dense [n_layers][B][k_max][H_kv][d]
 * buffers and Kj = k[l,b,j].  With counts[b] = 0 the output is 0 and lse is
 * -inf.  fp32 accumulation and output; lse is nullable.  For one layer of a
 * model, pass n_layers = 1 with layer-offset pointers.  Needs workspace
 * spec_workspace_size(SPEC_OP_ATTN).                                        */
SPEC_API spec_status spec_sparse_decode_attn(const spec_dims* dm, const uint16_t* q,
                                    const uint16_t* k, const uint16_t* v,
                                    const int32_t* idx, const int32_t* counts,
                                    float* out, float* lse, void* ws,
                                    size_t ws_bytes, spec_stream stream);

/* Sparse decode attention over the slots of an elastic state whose last
 * update has not been copied yet (Sec. 5.4's loads fused into Eq. 1's
 * reads).  As compact-mode spec_sparse_decode_attn over slots
 * [0, counts[b]) of el->kbuf/vbuf, except that a slot with
 * el->slot_src[b,s] = t >= 0 is read from the caches at token t (clamped into
 * [0, L_cap)), and that row, K and V of every layer, is written into the slot
 * on the way, bit for bit.  After the call the slot buffers hold what the
 * update's copy would have written; calling it again with the same slot_src
 * rewrites the same rows (same outputs).  el->slot_tok and el->n_changed are
 * not used.  Needs workspace spec_workspace_size(SPEC_OP_ATTN).             */
SPEC_API spec_status spec_sparse_decode_attn_elastic(const spec_dims* dm,
                                    const uint16_t* q, const uint16_t* k_cache,
                                    const uint16_t* v_cache, const spec_elastic* el,
                                    const int32_t* counts, float* out, float* lse,
                                    void* ws, size_t ws_bytes, spec_stream stream);

/* Elastic loading on the device (Sec. 5.4).  S_now = idx_now[b, 0..c) with
 * c = min(counts[b], k_max): distinct tokens in ascending order, as spec_topk
 * writes them.  S_last = the tokens held in el->slot_tok[b, 0..k_max).  Slots
 * whose token is not in S_now are freed; the tokens of S_now - S_last are
 * copied, for every layer, K and V, from the caches into freed slots (the
 * i-th smallest freed slot receives the i-th smallest new token); freed
 * slots left over are set to -1.  With the budget c kept fixed between calls
 * (the paper's |S_last| = |S_now|) slots [0, c) hold exactly S_now afterwards
 * and the rest are -1; if c shrank so that a kept token sits at a slot >= c,
 * the sequence is reloaded in full to restore that layout.
 * el->n_changed[b] = number of rows loaded; el->slot_src[b,s] = the token
 * loaded into slot s, or -1.  Start from slot_tok = -1 everywhere for a full
 * load.  Needs workspace spec_workspace_size(SPEC_OP_DELTA).               */
SPEC_API spec_status spec_delta_gather(const spec_dims* dm, const int32_t* idx_now,
                              const int32_t* counts, const uint16_t* k_cache,
                              const uint16_t* v_cache, const spec_elastic* el,
                              void* ws, size_t ws_bytes, spec_stream stream);

/* One fused decode step: spec_score -> spec_topk -> spec_sparse_decode_attn
 * indexed over the caches; or, when el != NULL, spec_score -> spec_topk ->
 * the elastic update's slot plan -> spec_sparse_decode_attn_elastic (the
 * update's rows are read from the caches once, by the attention, which also
 * writes them into their slots: the state afterwards is spec_delta_gather's).
 * All enqueued on `stream` with no host synchronisation.  idx_out [B][n_sets][k_max] and counts_out [B] receive
 * the selection; out/lse as for spec_sparse_decode_attn (lse nullable);
 * scores_out [B][n_sets][L_max] (nullable) receives the retrieval scores.
 * Elastic loading needs n_sets = 1.  Needs workspace
 * spec_workspace_size(SPEC_OP_STEP).                                        */
SPEC_API spec_status spec_step(const spec_dims* dm, const uint16_t* q_r,
                      const uint16_t* k_r, const int32_t* seq_lens,
                      const int32_t* ks, const uint16_t* q,
                      const uint16_t* k_cache, const uint16_t* v_cache,
                      int32_t* idx_out, int32_t* counts_out, float* out,
                      float* lse, float* scores_out, const spec_elastic* el,
                      void* ws, size_t ws_bytes, spec_stream stream);

/* KV of offloaded layers held in host memory (host struct).  k and v are
 * host pointers into pinned memory allocated with hipHostMalloc (the GPU
 * reads it directly over the host link); layout as the device cache:
 * [n_off][B][L_cap][H_kv][d] bf16 with the strides below.                   */
typedef struct spec_host_kv {
  const uint16_t* k;
  const uint16_t* v;
  int64_t stride_layer;  /* elements between layers; 0 = B * stride_b        */
  int64_t stride_b;      /* elements between sequences; 0 = L_cap * H_kv * d */
} spec_host_kv;

/* Elastic loading from host memory with an asynchronous per-layer dataflow
 * (Sec. 5.1: the selection is known before the LLM runs, so the loads of
 * every layer are issued at once on their own stream and overlap the
 * computation; Sec. 5.4: only S_now - S_last is loaded, into the slots freed
 * by S_last - S_now).  dm->n_layers = the offloaded layers (those of `host`
 * and of el->kbuf/vbuf).  On `stream`: the slot plan of spec_delta_gather
 * (same pairing, same full reload when the budget shrinks, n_changed), then
 * layer_ready[n_layers] is recorded (the fork point).  On `copy_stream`,
 * after waiting for that event, for each layer l in order: the K and V rows
 * of the new tokens copied from `host` into their slots of layer l, then
 * layer_ready[l] recorded.  A consumer of layer l waits for layer_ready[l]
 * only.  layer_ready: n_layers + 1 caller-created hipEvent_t handles; it may
 * be NULL only when copy_stream is NULL, in which case every copy runs on
 * `stream` after the plan.  The host pointers must be pinned host memory
 * (SPEC_ERR_INVALID otherwise, before anything is enqueued).  Needs
 * workspace spec_workspace_size(SPEC_OP_DELTA).                            */
SPEC_API spec_status spec_offload_load(const spec_dims* dm, const int32_t* idx_now,
                              const int32_t* counts, const spec_host_kv* host,
                              const spec_elastic* el, void* ws, size_t ws_bytes,
                              spec_stream stream, spec_stream copy_stream,
                              void* const* layer_ready);

/* One decode step with part of the KV offloaded to host memory (Sec. 5.1,
 * 5.4; the offloaded layers are the last ones, as the paper's adaptive
 * memory management offloads them first).  Layers [0, n_dev_layers) are in
 * the device caches k_cache/v_cache (layout and strides of dm, as for
 * spec_step); layers [n_dev_layers, dm->n_layers) are in `host`, and el's
 * slot buffers hold their selected rows ([n_off][B][k_max][H_kv][d], n_off =
 * n_layers - n_dev_layers; start from slot_tok = -1 for a full load).  On
 * `stream`: spec_score, spec_topk, the slot plan, then the attention of the
 * device layers (one launch, indexed over the caches) while the host loads
 * run on `copy_stream` (spec_offload_load with layer_ready[0..n_off]), then,
 * for each offloaded layer, a wait for its layer_ready event and its
 * attention over its slots.  Outputs as spec_step (idx, counts, out for all
 * layers, lse and scores nullable).  One token set per sequence (n_sets = 1).
 * copy_stream NULL runs everything on `stream`.  0 <= n_dev_layers <
 * n_layers.  Needs workspace spec_workspace_size(SPEC_OP_OFFLOAD).         */
SPEC_API spec_status spec_step_offload(const spec_dims* dm, const uint16_t* q_r,
                              const uint16_t* k_r, const int32_t* seq_lens,
                              const int32_t* ks, const uint16_t* q,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              int32_t n_dev_layers, const spec_host_kv* host,
                              int32_t* idx_out, int32_t* counts_out, float* out,
                              float* lse, float* scores_out, const spec_elastic* el,
                              void* ws, size_t ws_bytes, spec_stream stream,
                              spec_stream copy_stream, void* const* layer_ready);

/* The fused decode step of spec_step without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that forbid allocation).  Arguments, outputs and errors are
 * those of spec_step.  The workspace is a static device array of
 * spec_step_noalloc_max_bytes() bytes (64 MiB) that every GPU the library
 * runs on holds from the first call until the process ends; the call itself
 * allocates nothing.  A step whose spec_workspace_size(SPEC_OP_STEP)
 * exceeds it returns SPEC_ERR_TOO_LARGE before any HIP call (the five
 * benchmark workloads need 0.3-53 MB with one set per sequence).  All calls
 * on one GPU share that GPU's array, which keeps the last call's contents
 * (no part of it needs to start zeroed): calls that overlap on one GPU
 * (concurrent streams or threads) race and must be serialised by the
 * caller.  The first call on a GPU looks the array's device address up
 * (hipGetSymbolAddress), so make it once outside any graph capture.      */
SPEC_API spec_status spec_step_noalloc(const spec_dims* dm, const uint16_t* q_r,
                              const uint16_t* k_r, const int32_t* seq_lens,
                              const int32_t* ks, const uint16_t* q,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              int32_t* idx_out, int32_t* counts_out, float* out,
                              float* lse, float* scores_out, const spec_elastic* el,
                              spec_stream stream);

/* Size in bytes of spec_step_noalloc's static scratch (per GPU).            */
SPEC_API size_t spec_step_noalloc_max_bytes(void);

/* Retrieval-head front end parameters (host struct).                        */
typedef struct spec_frontend {
  int32_t vocab;         /* rows of the embedding table                       */
  int32_t hidden;        /* embedding width = input width of W_q and W_k; a
                            multiple of 128                                   */
  float rope_base;       /* rotary base: theta_i = rope_base^(-2i/d_r), > 0   */
  float yarn_scale;      /* YaRN context-extension factor s; <= 1 = no scaling */
  int32_t yarn_orig_ctx; /* context the model was trained at (> 0 if s > 1)   */
  float yarn_alpha;      /* YaRN ramp bounds, in rotations over yarn_orig_ctx; */
  float yarn_beta;       /* alpha = beta = 0 selects 1 and 32                  */
  int32_t reserved;      /* must be 0                                         */
} spec_frontend;

/* Retrieval-head front end for the new token of every sequence (Sec. 4.3:
 * the retrieval head is the distilled model's embedding and Q/K projection,
 * with its 2K context extended by YaRN).  For each sequence b, with
 * x = emb[tokens[b]] (ids clamped into [0, vocab)) and p = pos[b]:
 *     q = W_q x,  k = W_k x                 (fp32 accumulation, [H_r][d_r])
 *     q_r[b,h]        = m * rot(q[h], p)    bf16 (round to nearest even)
 *     K_r[b, p, h]    = m * rot(k[h], p)    bf16, only when 0 <= p < L_cap
 * rot turns dimension pair (i, i + d_r/2) by the angle p * theta'_i, with
 * theta_i = rope_base^(-2i/d_r) and, when yarn_scale = s > 1 (YaRN), the
 * pair's r_i = yarn_orig_ctx * theta_i / (2 pi) rotations over the original
 * context giving gamma_i = clamp((r_i - alpha) / (beta - alpha), 0, 1) and
 *     theta'_i = (1 - gamma_i) * theta_i / s + gamma_i * theta_i,
 *     m = 0.1 ln(s) + 1;
 * without scaling theta' = theta and m = 1.  Angles are formed in fp64.
 * Layouts: tokens, pos [B] int32; emb [vocab][hidden] bf16; w_q, w_k
 * [H_r * d_r][hidden] bf16 (a linear layer's [out][in], feature h*d_r + i
 * being dimension i of head h); q_r [B][H_r][d_r]; K_r as for spec_score
 * (dm->B, H_r, d_r, L_cap and kr_stride_b are used; the other dimensions
 * are validated as everywhere).  In a decode step, p is the new token's
 * index, so that seq_lens = p + 1 afterwards makes the scoring include it.
 * SPEC_ERR_INVALID also for a null fe, vocab or hidden <= 0, a non-finite
 * or non-positive rope_base, a non-finite yarn_scale, and with s > 1
 * yarn_orig_ctx <= 0 or alpha >= beta; SPEC_ERR_UNSUPPORTED for hidden not
 * a multiple of 128.  The result is deterministic (fixed summation order).
 * Needs workspace spec_workspace_size(SPEC_OP_FRONTEND) (fp32 partial sums
 * of the projection; any contents on entry).                                */
SPEC_API spec_status spec_retrieval_qk(const spec_dims* dm, const spec_frontend* fe,
                              const int32_t* tokens, const int32_t* pos,
                              const uint16_t* emb, const uint16_t* w_q,
                              const uint16_t* w_k, uint16_t* q_r, uint16_t* k_r,
                              void* ws, size_t ws_bytes, spec_stream stream);

/* MLA problem dimensions (host struct).  The MLA models this serves
 * (DeepSeek-V3/R1 and Kimi-K2 style) have d_c = 512, d_rope = 64,
 * d_nope = d_v = 128; those values are the supported ones.                  */
typedef struct spec_mla_dims {
  int32_t B;         /* sequences in the batch                                */
  int32_t L_cap;     /* token capacity of every cache row                     */
  int32_t k_max;     /* row length of idx, <= L_cap, <= 32768                 */
  int32_t n_layers;  /* layers attended with one selection                    */
  int32_t H;         /* query heads (64 or 128)                               */
  int32_t d_c;       /* latent width (512)                                    */
  int32_t d_rope;    /* rotary key width, shared by the heads (64)            */
  int32_t d_nope;    /* per-head query/key width without position (128)      */
  int32_t d_v;       /* per-head value width (128)                            */
  int32_t reserved;  /* must be 0                                             */
  int64_t ckv_stride_layer; /* elements between layers of ckv; 0 = B*ckv_stride_b */
  int64_t ckv_stride_b;     /* elements between sequences; 0 = L_cap*(d_c+d_rope) */
  float scale;       /* softmax scale; 0 = 1/sqrt(d_nope + d_rope)            */
  int32_t reserved2; /* must be 0                                             */
} spec_mla_dims;

/* Sparse decode attention of an MLA model over the selected tokens (Sec. 4.3,
 * "Support for MLA": the cache holds a low-dimensional latent per token and
 * only the selected latents are raised to the heads' dimension).  For every
 * layer l, sequence b and head h, with j over idx[b, 0..counts[b]):
 *     key_j   = [W_UK[l,h] c_j ; r_j],   value_j = W_UV[l,h] c_j,
 *     s_j     = scale * dot(q[l,b,h,:], key_j),
 *     out[l,b,h,:] = sum_j softmax_j(s) value_j,  lse[l,b,h] = log sum_j e^{s_j}
 * where the cache row of token t is ckv[l,b,t,:] = [c_t (d_c) ; r_t (d_rope)]
 * and q[l,b,h,:] = [q_nope (d_nope) ; q_rope (d_rope)].  The result is
 * computed in the absorbed form (W_UK folded into the query, W_UV applied to
 * the weighted sum of latents), equal in exact arithmetic: the per-head keys
 * and values are never formed.  Layouts (bf16 unless noted):
 *     q      [n_layers][B][H][d_nope + d_rope]
 *     ckv    [n_layers][B][L_cap][d_c + d_rope]  (strides in dm; rows dense)
 *     w_uk   [n_layers][H][d_nope][d_c],  w_uv [n_layers][H][d_v][d_c]
 *            (each maps a latent to one head's part: a linear layer's [out][in])
 *     idx    [B][k_max] int32 (indices outside [0, L_cap) are clamped),
 *     counts [B] int32 (clamped into [0, k_max]),
 *     out    [n_layers][B][H][d_v] fp32, lse [n_layers][B][H] fp32 (nullable).
 * counts[b] = 0 gives out = 0 and lse = -inf.  fp32 accumulation; the
 * absorbed query and the latent output enter the matrix cores as bf16 high +
 * low pairs (~2^-16 relative), the softmax weights as a truncated pair
 * (2^-14).
 * SPEC_ERR_INVALID: null pointer, non-positive dimension, k_max > L_cap,
 * misaligned pointer (16 bytes for tensors, 4 for idx/counts/lse), a stride
 * below the block it steps over or not a multiple of 8, a negative or
 * non-finite scale, non-zero reserved fields.  SPEC_ERR_UNSUPPORTED: other
 * widths than the ones above, H not 64 or 128, k_max > 32768, B > 65535.
 * SPEC_ERR_WORKSPACE: ws_bytes below spec_mla_workspace_size().             */
SPEC_API spec_status spec_mla_sparse_decode_attn(const spec_mla_dims* dm, const uint16_t* q,
                                        const uint16_t* ckv, const uint16_t* w_uk,
                                        const uint16_t* w_uv, const int32_t* idx,
                                        const int32_t* counts, float* out, float* lse,
                                        void* ws, size_t ws_bytes, spec_stream stream);

/* Workspace bytes of spec_mla_sparse_decode_attn (the absorbed queries and
 * the partial results of split selections).                                 */
SPEC_API spec_status spec_mla_workspace_size(const spec_mla_dims* dm, size_t* bytes);

/* Workspace bytes needed by `op` for dimensions `dm` (0 for SPEC_OP_GATHER).
 * Returns the same validation status as the op itself.                      */
SPEC_API spec_status spec_workspace_size(const spec_dims* dm, spec_op op,
                                size_t* bytes);

/* Static description of a status code (never NULL).                         */
SPEC_API const char* spec_status_string(spec_status s);

/* HIP error code of the last SPEC_ERR_HIP on the calling thread (0 = none). */
SPEC_API int spec_last_hip_error(void);

/* Library version string.                                                   */
SPEC_API const char* spec_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SPEC_H_ */
