/*
 * war.h -- C ABI of the MI355X speculative-verification decode step.
 *
 * The operation (WAR, arXiv 2607.17299):
 *  - Rollout is batched LLM inference over multi-turn trajectories whose KV
 *    cache is kept and reused from turn to turn (Background, "Rollout
 *    Bottlenecks"; System Design, "Overview of WAR").
 *  - Under low load the model-free suffix drafter proposes draft tokens.  The
 *    target model verifies them in one forward pass and advances several tokens
 *    when they are accepted (System Design, "SuffixDecoding").
 *  - Under high load speculation is off and the same step is plain batched
 *    decode (System Design, "SuffixDecoding": adaptive enabling, stateless
 *    mode switching).
 *  - Speculation must be lossless (Introduction; Background, "Why Workload
 *    Matters").  Here that means greedy verification:
 *      - row 0 of request b is its pending token x_b at position ctx_b;
 *      - rows 1..n_b are its drafts d_1..d_n;
 *      - g_i is the argmax of row i (ties go to the lowest id);
 *      - accept_b is the largest a with d_m == g_{m-1} for all m <= a;
 *      - next_b is g_{accept_b}.
 *    war_kv_commit then keeps the KV of rows 0..accept_b, sets
 *    ctx_b += accept_b + 1, and returns the pages reserved for rejected
 *    slots (rollback).
 *
 * Conventions
 *  - Every array argument is a DEVICE pointer owned by the caller, unless its
 *    comment says "host".  The library never frees caller memory.
 *  - Every call is ordered on the given HIP stream (a hipStream_t passed as
 *    void*; NULL = the null stream).  Nothing waits for the device unless the
 *    comment says so.
 *  - Calls on one model or one pool are not thread-safe: use one stream per
 *    model and pool.
 *  - Arguments are checked on the host before anything is enqueued.  On error
 *    the call returns a negative status, enqueues nothing and changes no
 *    state.  war_last_error() describes the last failure of the calling
 *    thread.
 */
#ifndef WAR_H
#define WAR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t war_status;
#define WAR_OK                0
#define WAR_ERR_INVALID_ARG  (-1)
#define WAR_ERR_OUT_OF_PAGES (-2)
#define WAR_ERR_HIP          (-3)
#define WAR_ERR_UNSUPPORTED  (-4)
#define WAR_ERR_DEVICE       (-5) /* the device flagged bad input (war_pool_state) */

/* Decoder shape.
 * Layers: RMSNorm -> QKV -> rotate-half RoPE -> grouped-query attention -> O-proj,
 * then residual -> RMSNorm -> SwiGLU FFN -> residual; final RMSNorm; untied LM head.
 * Constraints: d_model, ffn_dim, vocab and (n_q_heads + 2 n_kv_heads) * head_dim
 * are multiples of 128; head_dim is 64 or 128; n_q_heads / n_kv_heads is 1..8;
 * page_size is 16. */
typedef struct war_model_config {
  int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, ffn_dim, vocab;
  float rms_eps;     /* RMSNorm epsilon                                        */
  float rope_base;   /* RoPE base: pair j of a head turns by pos * base^(-2j/D) */
  int32_t page_size; /* KV tokens per page (16)                                */
  int32_t max_rows;  /* most rows one forward pass holds (verify: B*(k_max+1)) */
} war_model_config;

typedef struct war_model war_model;     /* opaque: owned weight copy + owned workspace */
typedef struct war_kv_pool war_kv_pool; /* opaque: owned allocator state, borrowed KV */

/* Number of weight pointers a model takes: 3 + 7 * n_layers. */
int32_t war_weight_count(const war_model_config* cfg);

/* Create a model over caller-owned bf16 weights (device pointers, row-major [out, in]).
 * Canonical order:
 *   embed [V, d];
 *   then for each layer:
 *     attn_norm [d];
 *     w_qkv [(nq + 2 nkv) * hd, d]  (query rows head-major, then key rows, then value rows);
 *     w_o [d, nq * hd];
 *     ffn_norm [d];
 *     w_gate [F, d];
 *     w_up [F, d];
 *     w_down [d, F];
 *   then final_norm [d];
 *   then w_lm [V, d].
 * The model copies every weight into device memory it owns, the projection
 * and LM-head matrices repacked into the order its GEMM kernel streams
 * (16-row by 64-column MFMA fragments, each 16-byte lane chunk contiguous), so
 * the caller's buffers are not read after this call returns and may be freed.
 * The copy costs as much device memory as the weights themselves.  The model
 * also allocates its own device workspace (sized by max_rows).  Returns WAR_ERR_UNSUPPORTED for shapes
 * outside the constraints above. */
war_status war_model_create(const war_model_config* cfg, const void* const* weights,
                            int32_t n_weights, war_model** out);
void war_model_destroy(war_model* m);

/* Create a KV page pool over caller-owned storage.
 *   kv_pages     bf16, n_layers * num_pages * n_kv_heads * 2 * page_size * head_dim
 *                elements.  Page p of layer l, kv-head h starts at element
 *                ((l * num_pages + p) * n_kv_heads + h) * 2 * page_size * head_dim.
 *                It holds the keys (page_size * head_dim elements, in the
 *                fragment order below), then the values transposed as
 *                [head_dim][page_size].  page_size is 16.  Key slot s, dim d
 *                sits at element ((t * head_dim/32 + d/32) * 8 + s8) * 32 + d%32
 *                of the key region, with t = (s/4) % 2 and s8 = 4 (s/8) + s%4:
 *                one 512-byte run per (slot group t, 32-dim step), which is
 *                what one attention operand load reads.
 *   block_tables int32 [max_seqs][max_pages_per_seq].  Entry [s][j] is the
 *                physical page of sequence s's logical page j, or -1.
 *                Initialised to -1 here.
 * The pool owns its free stack, reference counts and per-sequence page counts.
 * Free pages pop as 0, 1, 2, ...  Pops go in batch order, logical pages
 * ascending.  Pushes go in reverse batch order, logical pages descending.  So
 * reserving and then discarding a step restores the stack exactly. */
war_status war_kv_pool_create(const war_model_config* cfg, void* kv_pages, int32_t num_pages,
                              int32_t* block_tables, int32_t max_seqs, int32_t max_pages_per_seq,
                              void* stream, war_kv_pool** out);
void war_kv_pool_destroy(war_kv_pool* p);

/* Ensure capacity for n_tokens[i] slots for sequence seq_ids[i] (host arrays,
 * distinct ids).  A trajectory's KV cache grows with its length and stays
 * resident from turn to turn, so KV memory is the pressure point of rollout
 * (Background, "Rollout Bottlenecks"; System Design, "Overview of WAR").
 * Pages are popped from the free stack; nothing changes when they do not
 * suffice (WAR_ERR_OUT_OF_PAGES).  Synchronises the stream. */
war_status war_kv_alloc(war_kv_pool* p, int32_t n, const int32_t* seq_ids_host,
                        const int32_t* n_tokens_host, void* stream);

/* dst shares the first n_tokens (a multiple of page_size) of src.  dst must hold no
 * pages.  The shared pages' reference counts rise.  The caller sets dst's
 * ctx_len to n_tokens.  Cache reuse across sibling rollouts (System Design,
 * "Overview of WAR"). */
war_status war_kv_fork(war_kv_pool* p, int32_t src_seq, int32_t dst_seq, int32_t n_tokens,
                       void* stream);

/* Drop every page of each listed sequence (host array, distinct ids); a page
 * returns to the free stack when its reference count reaches 0.  A finished
 * trajectory releases the KV memory it held (Background, "Rollout
 * Bottlenecks": KV footprint limits how many requests a replica keeps).
 * Synchronises the stream. */
war_status war_kv_free(war_kv_pool* p, int32_t n, const int32_t* seq_ids_host, void* stream);

/* Write precomputed keys/values of tokens [pos0, pos0 + n) of one layer of one
 * sequence into its pages (capacity must already be there, e.g. war_kv_alloc).
 * src: bf16 [2][n_kv_heads][n][head_dim] (0 = keys after RoPE, 1 = values).
 * Imports a cached context computed elsewhere: the scheduler places a
 * request on the replica whose cache already holds its prefix, and a
 * trajectory's KV is reused across turns instead of recomputed (System
 * Design, "Overview of WAR" and the cache-aware scheduler).  Reads the
 * sequence's page count (one stream synchronisation). */
war_status war_kv_load(war_kv_pool* p, int32_t seq_id, int32_t layer, int32_t pos0, int32_t n,
                       const void* src, void* stream);

/* Append a new turn to cached trajectories (System Design, "Overview of WAR";
 * Background, "Rollout Bottlenecks").
 *   seq_ids     device int32 [n]
 *   ctx_lens    device int32 [n]; read, then += n_new
 *   n_new_host  HOST int32 [n], >= 1
 *   new_tokens  device int32, packed: sequence i's tokens at offset sum_{j<i} n_new[j]
 *   next_tokens device int32 [n]: argmax after each sequence's last new token
 *   last_logits device fp32 [n][vocab], or NULL
 * Reserves pages for ctx + n_new slots and computes the new tokens' KV (causal,
 * against the cached context).  This call synchronises the stream once to read
 * ctx_lens. */
war_status war_prefill_append(war_model* m, war_kv_pool* p, int32_t n, const int32_t* seq_ids,
                              int32_t* ctx_lens, const int32_t* n_new_host,
                              const int32_t* new_tokens, int32_t* next_tokens,
                              float* last_logits, void* stream);

/* One speculative-verification step over B requests (k_max = 0: plain decode).
 *   seq_ids      device int32 [B], distinct (checked on the device)
 *   ctx_lens     device int32 [B]  cached tokens per request (not changed here)
 *   last_tokens  device int32 [B]  pending token (previous step's next_tokens)
 *   draft_tokens device int32 [B][k_max] (may be NULL when k_max == 0)
 *   draft_lens   device int32 [B]  in [0, k_max] (NULL: all k_max)
 *   accept_lens  device int32 [B]  out
 *   next_tokens  device int32 [B]  out
 *   logits       device fp32 [B * (k_max + 1)][vocab] or NULL.  Row b*(k_max+1)+i
 *                holds request b's row i; rows with i > draft_len are unspecified.
 * Reserves the pages for ctx + draft_len + 1 slots, writes the KV of all rows,
 * and leaves the pool waiting for war_kv_commit.  Until that commit the pool
 * accepts no other call that changes pages.
 * The device checks what the host cannot see without waiting: ids in range
 * and distinct, ctx_len >= 0, ctx + draft_len + 1 within max_pages_per_seq,
 * token ids in [0, vocab), enough free pages.  On a bad id, length or page
 * count the whole step fails on the device: no page moves, accept_lens and
 * next_tokens are -1 for every request, the following war_kv_commit changes
 * nothing, and war_pool_state returns WAR_ERR_DEVICE (a bad token id is
 * flagged the same way but the step runs with token 0 in its place).  The
 * host never waits for the device here while its lower bound on the free
 * pages (kept from each commit's report) covers B * ceil((k_max+1)/16)
 * pages; otherwise it reads the exact count once. */
war_status war_verify_step(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                           const int32_t* ctx_lens, const int32_t* last_tokens,
                           const int32_t* draft_tokens, const int32_t* draft_lens, int32_t k_max,
                           int32_t* accept_lens, int32_t* next_tokens, float* logits,
                           void* stream);

/* The verify step with sampled verification instead of greedy acceptance (the
 * paper's rollouts sample: Evaluation, temperature 1.0, top-k 200; speculation
 * stays lossless: Introduction; Background, "Why Workload Matters").  Same
 * arguments and pool protocol as war_verify_step, plus:
 *   uniforms     device fp32 [B * (k_max + 1)][2], each in [0, 1): for row
 *                b*(k_max+1)+i, [0] is the acceptance test of draft i+1 and [1]
 *                the draw made at that row.  The caller owns the randomness.
 *   temperature  > 0
 *   top_k        in [1, vocab]
 * Row i's target distribution keeps the top_k largest logits (value
 * descending, ties to the lowest token id) and takes softmax(logit / T) over
 * them.  Draft i+1 is accepted iff uniform[0] < p_i(draft); at the first
 * rejection next_token is drawn from p_i without the rejected draft, and after
 * the last accepted draft from p_n; a draw with uniform v is the smallest token
 * id whose cumulative weight (in id order) exceeds v times the total.  The
 * logits are written to `logits` when it is not NULL, else to a workspace the
 * model allocates on first use ([B * (k_max + 1)][vocab] fp32).  Decisions are
 * taken in fp32. */
war_status war_verify_step_sampled(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                                   const int32_t* ctx_lens, const int32_t* last_tokens,
                                   const int32_t* draft_tokens, const int32_t* draft_lens, int32_t k_max,
                                   const float* uniforms, float temperature, int32_t top_k,
                                   int32_t* accept_lens, int32_t* next_tokens, float* logits, void* stream);

/* The verify step with a draft TREE per request (SuffixDecoding proposes
 * speculation trees; the paper counts their tree-mask handling among the
 * verification costs: Evaluation).  Greedy acceptance.  Same arguments and
 * pool protocol as war_verify_step, plus:
 *   draft_parents device int32 [B][k_max]: node 0 is last_token, node i
 *                 (1..draft_len) carries draft_tokens[b][i-1] and has parent
 *                 draft_parents[b][i-1] in [0, i).  A parent outside that range
 *                 sets the device error flag (war_pool_state) and is read as i-1.
 *   accept_path   device int32 [B][k_max] out, or NULL: the accepted nodes in
 *                 depth order, -1 beyond accept_lens[b].
 *   k_max         + 1 <= 32.
 * Node i is scored on its root-to-node path: position ctx + depth(i), and it
 * sees the cached context and the nodes of that path.  Its logits are row
 * b*(k_max+1)+i.  A node is accepted when its parent is (the root always is)
 * and its token is the parent's greedy token; the accepted path ends at the
 * deepest accepted node (lowest index among equals), accept_lens[b] is its
 * depth and next_tokens[b] its greedy token.  Before returning, the step moves
 * the KV of the accepted nodes to slots ctx + 1 .. ctx + accept_lens[b], so
 * war_kv_commit keeps exactly the accepted path. */
war_status war_verify_step_tree(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                                const int32_t* ctx_lens, const int32_t* last_tokens,
                                const int32_t* draft_tokens, const int32_t* draft_parents,
                                const int32_t* draft_lens, int32_t k_max, int32_t* accept_lens,
                                int32_t* next_tokens, int32_t* accept_path, float* logits, void* stream);

/* war_verify_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, pool protocol and results as war_verify_step (greedy chain
 * drafts); the step's workspace (activations, split-K partials, attention
 * work list and partials, counters) is laid over a static device array of
 * 64 MiB that the library holds on each GPU it runs on until the process
 * ends, instead of the model's own workspace.  This call allocates nothing:
 * no hipMalloc, hipFree or allocating library routine, and no host buffers.
 * It returns WAR_ERR_UNSUPPORTED (enqueuing nothing) when the step does not
 * fit: the rows B*(k_max+1) with their partials, plus the attention items of
 * B requests of max_pages_per_seq pages (longer attention chunks are taken
 * first to fit).  When the host's lower bound on free pages does not cover
 * B*ceil((k_max+1)/16) pages it reads the exact count (one stream
 * synchronisation) and returns WAR_ERR_OUT_OF_PAGES if that does not cover
 * it either.  Every call on one GPU shares that GPU's array: calls that
 * overlap on one GPU (other streams, other threads) race; the array keeps the
 * last call's contents, and the step clears what must start at zero. */
war_status war_verify_step_noalloc(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                                   const int32_t* ctx_lens, const int32_t* last_tokens,
                                   const int32_t* draft_tokens, const int32_t* draft_lens, int32_t k_max,
                                   int32_t* accept_lens, int32_t* next_tokens, float* logits,
                                   void* stream);

/* Commit the pending verify step.
 *   accept_lens device int32 [B]; -1 discards the step.  Values are clamped
 *               to [-1, reserved capacity].
 * Effects:
 *   ctx_lens[b] += accept_lens[b] + 1;
 *   the pages the step reserved beyond the new length go back to the free
 *   stack, and their block-table entries become -1.
 * After a step that failed on the device nothing changes.  Use the same B,
 * seq_ids and ctx_lens as the verify step (an id out of range is flagged and
 * skipped).  When the kernel ends it writes its sequence number and the free
 * page count to a host-mapped word of the pool, which later verify steps read
 * instead of waiting. */
war_status war_kv_commit(war_kv_pool* p, int32_t B, const int32_t* seq_ids, int32_t* ctx_lens,
                         const int32_t* accept_lens, void* stream);

/* Synchronise the stream.  Copy the allocator state to HOST buffers (each may
 * be NULL):
 *   free_stack      [num_pages]  (only the first *free_count entries are meaningful)
 *   refcount        [num_pages]
 *   held            [max_seqs]   pages held per sequence
 *   step_base       [max_seqs]   pages held before the last reservation
 * Returns WAR_ERR_DEVICE if a kernel flagged bad device-side input since the
 * last call (a token id outside [0, vocab), a sequence id out of range or
 * repeated within one step, a negative or too long context, a tree parent out
 * of range, or a device page shortage); the flags are then cleared. */
war_status war_pool_state(war_kv_pool* p, int32_t* free_count, int32_t* free_stack,
                          int32_t* refcount, int32_t* held, int32_t* step_base, void* stream);

/* Thread-local description of the last non-OK status ("" if none). */
const char* war_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* WAR_H */
