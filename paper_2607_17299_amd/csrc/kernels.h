// Internal launch interface between the C-ABI runtime and the gfx950 kernels.
#pragma once

#include <algorithm>

#include "common.h"

// Geometry of the paged KV storage:
//   element offset of page `page`, layer `layer`, kv-head `kvh`, kind (0 = K, 1 = V^T)
//   = ((((layer * num_pages + page) * n_kv_heads + kvh) * 2 + kind) * page_size * head_dim
// V is stored transposed, [head_dim][page_size].  K (page_size = 16) is stored
// in the order the attention's MFMA fragments read it, so that every K load of
// a wave reads 512 contiguous bytes of a page: key slot s, dim d sits at
// key_elem(s, d) (below).
struct KvGeom {
  bf16_t* kv;
  int64_t num_pages;
  int n_kv_heads, head_dim, page_size;
  __host__ __device__ int64_t page_elems(int layer, int page, int kvh, int kind) const {
    return ((((int64_t)layer * num_pages + page) * n_kv_heads + kvh) * 2 + kind) *
           (int64_t)page_size * head_dim;
  }
};

// Element offset of key slot s (0..15), dim d in a page's K region.  The slots
// form two groups of eight, t = (s / 4) % 2 (slots 0-3, 8-11 and 4-7, 12-15:
// the two 16-key S^T tiles of a 32-key block take one group from each of the
// block's two pages), and the dims 32-wide k-steps j = d / 32; group t, k-step
// j is one 512-byte run of eight 64-byte rows (member s8 = 4 (s / 8) + s % 4),
// which is what one MFMA operand load of a wave reads from the page.
__host__ __device__ inline int key_elem(int s, int d, int head_dim) {
  const int t = (s >> 2) & 1, s8 = ((s >> 3) << 2) | (s & 3);
  return ((t * (head_dim >> 5) + (d >> 5)) * 8 + s8) * 32 + (d & 31);
}

struct VerifySetupArgs {
  int B, k_max, vocab;
  int32_t* unit_ctr;  // attention work counters [8], cleared here
  int chunk;         // keys per attention item; doubled when that still leaves
  int items_double;  // at least this many items (enough to fill the attention grid)
  int G;        // query heads per kv-head
  int rb;       // attention row block of the step (rows per unit)
  int cascade;  // 1: plan shared-prefix attention units for forked siblings
  const int32_t* seq_ids;
  const int32_t* ctx_lens;
  const int32_t* last_tokens;
  const int32_t* draft_tokens;
  const int32_t* draft_lens;
  const int32_t* draft_parents;  // nullable: tree drafts [B][k_max], parent of node i+1
};

// C[m][n] = sum_k A[arow(m)][k] * W[n][k]   (bf16 in, fp32 accumulate)
// W rows n < n_split come from W1, rows >= n_split from W2 (row n - n_split).
struct GemmArgs {
  const bf16_t* A;
  int lda;
  const int32_t* a_rows;  // nullable: A row m -> a_rows[m]
  const bf16_t* Wp;  // weights in MFMA fragment order (launch_pack_weights)
  int M, N, K, kper;
  bf16_t* out;       // EPI_SWIGLU: silu(gate) * up, bf16 [M][ld_out]
  int64_t ld_out;
  float* P;  // partial sums [split][M][N]
  // argmax epilogue (split == 1): per (row, 128-column block) best value and index
  float* logits;  // nullable [M][ld_logits]
  int64_t ld_logits;
  float* amax_v;
  int32_t* amax_i;
};

enum { EPI_PARTIAL = 0, EPI_ARGMAX = 1, EPI_SWIGLU = 2 };

struct AttnArgs {
  const bf16_t* q;  // [rows][n_q_heads * head_dim]
  int q_stride;
  KvGeom kv;
  int layer;
  const int32_t* table;
  int max_pages;
  StepMeta meta;
  int G, TB, n_kv_heads;
  int prb;           // rows per (item, kv-head) in the partials (the step's row block)
  float scale_log2;  // log2(e) / sqrt(head_dim)
  float* pm;         // [item][kvh][RB]
  float* pl;         // [item][kvh][RB]
  float* po;         // [item][kvh][RB][head_dim]
  bf16_t* o;         // combine output [rows][n_q_heads * head_dim]
  int32_t* unit_ctr; // [8] attention work counters; zero before each attention
                     // launch (the combine kernel resets them)
};

// allocator / setup (alloc.hip)
void launch_pool_init(const PoolDev& p, hipStream_t st);
void launch_grow(const PoolDev& p, int n, const int32_t* seq, const int32_t* a, const int32_t* b,
                 int mode, hipStream_t st);
void launch_verify_setup(const PoolDev& p, const VerifySetupArgs& a, const StepMeta& m,
                         hipStream_t st);
void launch_commit(const PoolDev& p, int B, const int32_t* seq, int32_t* ctx, const int32_t* acc,
                   uint32_t commit_seq, hipStream_t st);
void launch_free(const PoolDev& p, int n, const int32_t* seq, hipStream_t st);
void launch_fork(const PoolDev& p, int src, int dst, int npg, hipStream_t st);
void launch_kv_load(const PoolDev& p, const KvGeom& g, int seq, int layer, int pos0, int n,
                    const bf16_t* src, hipStream_t st);
void launch_add_ctx(int n, int32_t* ctx, const int32_t* add, hipStream_t st);

// GEMM (gemm.hip)
int gemm_mt(int M);             // 16-row tiles per m-block for M rows
int gemm_mw(int M);             // m-blocks per workgroup
int gemm_mblock_groups(int M);  // workgroups per 128-column block and split
void launch_gemm(const GemmArgs& g, int epi, int splits, hipStream_t st);
// W [N][K] row-major -> dst in MFMA fragment order; N % 16 == 0, K % 64 == 0
// Repack [N][K] weights (N % 128 == 0) into the GEMM's grouped fragment order;
// W2 non-null: W and W2 are the gate and up halves ([N/2][K] each) of a SwiGLU
// pair, interleaved in groups of 4 + 4 tiles.
void launch_pack_weights(const bf16_t* W, const bf16_t* W2, int N, int K, bf16_t* dst, hipStream_t st);

// sampled verification (sample.hip)
struct SampleArgs {
  const float* logits;     // [B * kp1][V] fp32
  int V;
  const int32_t* ntok;     // per request: drafts + 1 (0: no rows)
  const int32_t* drafts;   // [B][k_max]
  int k_max, kp1, B;
  const float* uniforms;   // [B * kp1][2]: acceptance test, draw
  float temperature;
  int top_k;
  int32_t* row_out;        // [B * kp1][3]: accepted?, token if rejected here, token if last
};
void launch_sample(const SampleArgs& s, int32_t* accept_lens, int32_t* next_tokens, hipStream_t st);

// attention (attn.hip)
int attn_rows_per_block(int G, int k_rows);  // RB (16, 32 or 48)
void launch_attn(const AttnArgs& a, int RB, int head_dim, int grid, hipStream_t st);
void launch_attn_combine(const AttnArgs& a, int RB, int head_dim, int n_segs, hipStream_t st);

// elementwise / row kernels (rows.hip)
struct ModelDims {
  int d, nq, nkv, hd, F, V, qkv;
  float eps;
};
void launch_rope_table(int rows, const int32_t* pos, const double* inv_freq, int half, float* cos_t,
                       float* sin_t, hipStream_t st);
void launch_embed_norm(int rows, const int32_t* tok, const bf16_t* E, const bf16_t* g, int d,
                       float eps, float* h, bf16_t* u, hipStream_t st);
void launch_residual_norm(int rows, int splits, const float* P, int d, const bf16_t* g, float eps,
                          float* h, bf16_t* u, hipStream_t st);
void launch_qkv_rope(int rows, int splits, const float* P, const ModelDims& md,
                     const float* cos_t, const float* sin_t, const StepMeta& meta,
                     const int32_t* row_req, const int32_t* table, int max_pages, const KvGeom& kv,
                     int layer, bf16_t* q, hipStream_t st);
// parents (nullable): tree drafts; accept_path [n_req][k_max] then receives the
// accepted nodes in depth order, -1 beyond the accept length
void launch_argmax_accept(int n_req, const int32_t* ntok, int row_stride, int n_blocks,
                          const float* amax_v, const int32_t* amax_i, const int32_t* draft_tokens,
                          const int32_t* parents, int k_max, int32_t* accept_lens, int32_t* next_tokens,
                          int32_t* accept_path, hipStream_t st);
// Tree drafts: move the KV of each request's accepted nodes (slots ctx + node)
// to slots ctx + 1 .. ctx + accept_len, every layer.
void launch_kv_compact(const KvGeom& kv, int n_layers, int B, const StepMeta& meta, const int32_t* table,
                       int max_pages, const int32_t* accept_lens, const int32_t* accept_path, int k_max,
                       hipStream_t st);
