// C-ABI runtime: model and KV-pool objects, argument checks, page-capacity
// tracking, and the orchestration of the verify step, commit and prefill-append
// as sequences of gfx950 kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_set>
#include <vector>

#include "../../include/war.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

war_status fail(war_status code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIPCHK(x)                                                            \
  do {                                                                       \
    hipError_t e_ = (x);                                                     \
    if (e_ != hipSuccess)                                                    \
      return fail(WAR_ERR_HIP, std::string(#x) + ": " + hipGetErrorString(e_)); \
  } while (0)

#define CHECK(cond, msg)                          \
  do {                                            \
    if (!(cond)) return fail(WAR_ERR_INVALID_ARG, msg); \
  } while (0)

// Grow-only device buffer.
struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
  hipError_t ensure(size_t n) {
    if (n <= bytes) return hipSuccess;
    if (p) {
      hipError_t e = hipFree(p);
      if (e != hipSuccess) return e;
      p = nullptr;
      bytes = 0;
    }
    hipError_t e = hipMalloc(&p, n);
    if (e == hipSuccess) bytes = n;
    return e;
  }
  void release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    bytes = 0;
  }
  template <class T>
  T* as() const {
    return static_cast<T*>(p);
  }
};

// Pointers into the model's own weight copy; the matrices are in MFMA fragment
// order (w_gate_up = gate rows then up rows, one N = 2F matrix).
struct LayerW {
  const bf16_t *attn_norm, *w_qkv, *w_o, *ffn_norm, *w_gate_up, *w_down;
};

constexpr int kMaxBatch = 1024;

// Opt-in per-kernel timing: HIP events recorded on the launch stream around
// every kernel launch, summed per kernel name when read back.
struct Profiler {
  bool on = false;
  std::vector<hipEvent_t> pool;
  size_t used = 0;
  std::vector<std::pair<std::string, std::pair<size_t, size_t>>> marks;
  hipEvent_t next() {
    if (used == pool.size()) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      pool.push_back(e);
    }
    return pool[used++];
  }
};
constexpr int kPrefillChunk = 4096;  // keys per attention item when prefilling (chunk-major: L2 serves the row blocks)
constexpr int kPrefillRows = 128;    // attention rows per prefill row block (k_attn_rows)
constexpr int kMaxItemsPerSeq = 512;  // attention chunks one combine merges
constexpr int kAttnGrid = 512;        // persistent attention grid: 2 workgroups per CU
constexpr int64_t kPartialCap = int64_t(64) << 20;  // fp32 split-K partial elements

// Everything a forward pass's kernels use besides the caller's arrays and the
// model's weights, as views of ONE device allocation: activations, split-K
// partials, RoPE table, LM-head argmax partials, step metadata and the
// attention work list and partials.  The model owns one such allocation
// (grown on demand); a verify step may lay the same views over a fixed
// region instead.
struct Workspace {
  float* h;          // residual [R][d] fp32
  bf16_t* u;         // norm output [R][d]
  bf16_t* q;         // rotated queries [R][nq*hd]
  bf16_t* o;         // attention output [R][nq*hd]
  bf16_t* y;         // SwiGLU output [R][F]
  float* P;          // split-K partials [p_elems]
  float *cos_t, *sin_t;          // [R][hd/2]
  float* amax_v;                 // [R][V/128]
  int32_t* amax_i;               // [R][V/128]
  int32_t* rows;                 // tok, pos, active, row_req [4][R]
  int32_t* tree;                 // kvpos, tmask [2][R]
  int32_t* reqs;                 // seq, pos0, ntok, row0 [4][n_req_cap]
  int32_t* segs;                 // begin, count, req, rb [4][n_seg_cap]
  int32_t* n_items;              // [4]
  int32_t* unit_ctr;             // [8], zero between attention launches
  int32_t* a_rows;               // [kMaxBatch] LM-head rows of a prefill chunk
  int4* items;                   // [items_cap]
  int4* udesc;                   // [2 * items_cap]
  int32_t* order;                // [items_cap]
  float *pm, *pl, *po;           // [items_cap][nkv][rb_cap] (po: x hd)
  int R = 0, n_req_cap = 0, n_seg_cap = 0, rb_cap = 0;
  int64_t items_cap = 0, p_elems = 0;
  bool tree_step = false;        // the metadata describes tree drafts

  StepMeta meta() const {
    StepMeta m;
    m.tok = rows;
    m.pos = rows + R;
    m.active = rows + 2 * R;
    m.row_req = rows + 3 * R;
    m.req_seq = reqs;
    m.req_pos0 = reqs + n_req_cap;
    m.req_ntok = reqs + 2 * n_req_cap;
    m.req_row0 = reqs + 3 * n_req_cap;
    m.items = items;
    m.udesc = udesc;
    m.order = order;
    m.n_items = n_items;
    m.seg_begin = segs;
    m.seg_count = segs + n_seg_cap;
    m.seg_req = segs + 2 * n_seg_cap;
    m.seg_rb = segs + 3 * n_seg_cap;
    m.kvpos = tree_step ? tree : nullptr;
    m.tmask = tree_step ? reinterpret_cast<uint32_t*>(tree + R) : nullptr;
    return m;
  }
};

// Lays a workspace out from `base` (nullptr: measure only); returns its bytes.
size_t ws_layout(const ModelDims& md, int R, int64_t items, int rb, int64_t p_elems, char* base,
                 Workspace* w) {
  size_t off = 0;
  auto take = [&](size_t bytes) -> char* {
    char* at = base ? base + off : nullptr;
    off += (bytes + 255) & ~size_t(255);
    return at;
  };
  Workspace v;
  v.R = R;
  v.n_req_cap = std::max(R, kMaxBatch);
  v.n_seg_cap = R + kMaxBatch;
  v.items_cap = std::max<int64_t>(items, 1);
  v.rb_cap = rb;
  v.p_elems = p_elems;
  const size_t nqhd = (size_t)md.nq * md.hd, nb = (size_t)md.V / 128;
  v.h = reinterpret_cast<float*>(take((size_t)R * md.d * 4));
  v.u = reinterpret_cast<bf16_t*>(take((size_t)R * md.d * 2));
  v.q = reinterpret_cast<bf16_t*>(take((size_t)R * nqhd * 2));
  v.o = reinterpret_cast<bf16_t*>(take((size_t)R * nqhd * 2));
  v.y = reinterpret_cast<bf16_t*>(take((size_t)R * md.F * 2));
  v.P = reinterpret_cast<float*>(take((size_t)p_elems * 4));
  v.cos_t = reinterpret_cast<float*>(take((size_t)R * md.hd / 2 * 4));
  v.sin_t = reinterpret_cast<float*>(take((size_t)R * md.hd / 2 * 4));
  v.amax_v = reinterpret_cast<float*>(take((size_t)R * nb * 4));
  v.amax_i = reinterpret_cast<int32_t*>(take((size_t)R * nb * 4));
  v.rows = reinterpret_cast<int32_t*>(take((size_t)4 * R * 4));
  v.tree = reinterpret_cast<int32_t*>(take((size_t)2 * R * 4));
  v.reqs = reinterpret_cast<int32_t*>(take((size_t)4 * v.n_req_cap * 4));
  v.segs = reinterpret_cast<int32_t*>(take((size_t)4 * v.n_seg_cap * 4));
  v.n_items = reinterpret_cast<int32_t*>(take(16));
  v.unit_ctr = reinterpret_cast<int32_t*>(take(8 * 4));
  v.a_rows = reinterpret_cast<int32_t*>(take((size_t)kMaxBatch * 4));
  v.items = reinterpret_cast<int4*>(take((size_t)v.items_cap * sizeof(int4)));
  v.udesc = reinterpret_cast<int4*>(take((size_t)v.items_cap * 2 * sizeof(int4)));
  v.order = reinterpret_cast<int32_t*>(take((size_t)v.items_cap * 4));
  const size_t pr = (size_t)v.items_cap * md.nkv * rb;
  v.pm = reinterpret_cast<float*>(take(pr * 4));
  v.pl = reinterpret_cast<float*>(take(pr * 4));
  v.po = reinterpret_cast<float*>(take(pr * md.hd * 4));
  if (w) *w = v;
  return off;
}

// ---- static device scratch (war_verify_step_noalloc)
// A fixed array in device memory that every GPU the library runs on holds
// until the process ends.  Host code never uses its name as an address: the
// name is a host-side stand-in.  scratch_address() asks the runtime for the
// current device's copy once (hipGetSymbolAddress) and keeps it per device.
constexpr size_t kScratchBytes = size_t(64) << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// The current device's copy of `scratch` (out may be null: set-up only).
war_status scratch_address(void** out) {
  int dev = 0;
  HIPCHK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(WAR_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    HIPCHK(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return fail(WAR_ERR_HIP, "hipGetSymbolAddress returned no address for the scratch array");
    g_scratch_ptr[dev] = ptr;
  }
  if (out) *out = g_scratch_ptr[dev];
  return WAR_OK;
}

}  // namespace

struct war_model {
  war_model_config cfg;
  ModelDims md;
  const bf16_t* embed;
  std::vector<LayerW> layers;
  const bf16_t* final_norm;
  const bf16_t* w_lm;
  DevBuf wts;  // owned copy of every weight (matrices packed)
  int max_rows;
  DevBuf inv_freq;  // RoPE frequencies [hd/2] fp64
  DevBuf ws_buf;    // the model's own workspace allocation
  Workspace ws;     // views into ws_buf
  DevBuf logits_ws, row_out;  // sampled verification: full logits, per-row outcomes
  DevBuf path_ws;             // tree drafts: accepted path when the caller passes none
  std::vector<int32_t> h_stage;  // host staging for prefill metadata
  DevBuf stage_dev;              // device copy of per-prefill host arrays
  int32_t* pinned = nullptr;     // pinned host staging
  size_t pinned_ints = 0;
  Profiler prof;
};

// Host view of the pool's free pages.  A verify step needs a lower bound of
// the device's free count without waiting for the device:
//  - an exact count is known after every call that synchronises (base_fc,
//    with total_need and commit_issued at that time);
//  - every verify step adds the most pages it can take to total_need;
//  - every commit kernel, when it ends, writes (its sequence number, the free
//    count) to a host-mapped word; need_at[j % kRing] is total_need when
//    commit j was issued, so fc_j - (total_need - need_at[j]) bounds the count
//    after every step issued since.
constexpr int kRing = 1024;

struct war_kv_pool {
  war_model_config cfg;
  KvGeom geom;
  PoolDev dev;
  DevBuf state;    // stack | refcount | held | base | scalars
  DevBuf tmp;      // device copies of host id arrays
  int32_t* pinned = nullptr;
  size_t pinned_ints = 0;
  unsigned long long* report = nullptr;  // host-mapped (commit sequence << 32) | free count
  int64_t base_fc = 0, base_total = 0;
  uint32_t base_seq = 0, commit_issued = 0;
  int64_t total_need = 0;
  int64_t need_at[kRing] = {};
  int64_t exact_waits = 0;  // verify steps that read the exact count
  bool pending = false;
  int pending_B = 0;
  bool forked = false;  // some sequences may share pages (war_kv_fork was called)
};

namespace {

hipError_t ensure_pinned(int32_t*& p, size_t& cap, size_t n) {
  if (n <= cap) return hipSuccess;
  if (p) (void)hipHostFree(p);
  p = nullptr;
  cap = 0;
  hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&p), n * sizeof(int32_t), hipHostMallocDefault);
  if (e == hipSuccess) cap = n;
  return e;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

war_status check_config(const war_model_config* c) {
  if (!c) return fail(WAR_ERR_INVALID_ARG, "null config");
  if (c->n_layers < 1 || c->d_model < 1 || c->n_q_heads < 1 || c->n_kv_heads < 1 ||
      c->head_dim < 1 || c->ffn_dim < 1 || c->vocab < 1 || c->max_rows < 1)
    return fail(WAR_ERR_INVALID_ARG, "non-positive dimension in config");
  if (c->n_q_heads % c->n_kv_heads) return fail(WAR_ERR_INVALID_ARG, "n_q_heads % n_kv_heads != 0");
  const int G = c->n_q_heads / c->n_kv_heads;
  const int qkv = (c->n_q_heads + 2 * c->n_kv_heads) * c->head_dim;
  if (c->d_model % 128 || c->ffn_dim % 128 || c->vocab % 128 || qkv % 128 ||
      (c->n_q_heads * c->head_dim) % 128)
    return fail(WAR_ERR_UNSUPPORTED, "d_model, ffn_dim, vocab and projection widths must be multiples of 128");
  {
    // the GEMM addresses a packed matrix with 32-bit byte offsets
    const int64_t d = c->d_model, big = std::max({(int64_t)c->vocab * d, 2 * (int64_t)c->ffn_dim * d,
                                                   (int64_t)qkv * d, (int64_t)c->n_q_heads * c->head_dim * d});
    if (big * 2 > 0x7fffffffLL - (1 << 16))
      return fail(WAR_ERR_UNSUPPORTED, "a weight matrix of 2 GiB or more");
  }
  if (c->head_dim != 64 && c->head_dim != 128) return fail(WAR_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (G > 8) return fail(WAR_ERR_UNSUPPORTED, "more than 8 query heads per kv head");
  if (c->page_size != 16) return fail(WAR_ERR_UNSUPPORTED, "page_size must be 16");
  if (c->max_rows > 65536) return fail(WAR_ERR_UNSUPPORTED, "max_rows > 65536");
  if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f)) return fail(WAR_ERR_INVALID_ARG, "bad eps or rope base");
  return WAR_OK;
}

bool same_shape(const war_model_config& a, const war_model_config& b) {
  return a.n_layers == b.n_layers && a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim &&
         a.page_size == b.page_size;
}

struct Split {
  int s, kper;
};

// Records an event pair around the launches in its scope when profiling is on.
struct Timed {
  Profiler& p;
  hipStream_t st;
  size_t i0 = 0;
  const char* name;
  bool act;
  Timed(Profiler& pr, hipStream_t s, const char* n) : p(pr), st(s), name(n), act(pr.on) {
    if (act) {
      i0 = p.used;
      hipEvent_t e = p.next();
      if (e) (void)hipEventRecord(e, st);
      else act = false;
    }
  }
  ~Timed() {
    if (act) {
      const size_t i1 = p.used;
      hipEvent_t e = p.next();
      if (e) {
        (void)hipEventRecord(e, st);
        p.marks.push_back({name, {i0, i1}});
      }
    }
  }
};

// Split-K: the fewest splits that divide K exactly, give >= 192 workgroups and
// leave at most 48 steps of 64 per split; the fully unrolled kernels need exact
// splits.  Fewer splits mean fewer fp32 partial sums to write and to add up
// afterwards; below ~192 workgroups too few CUs stream W (measured on the
// 4096- and 6144-wide projections: 192-256 is the optimum); at 512-1024 rows
// (prefill chunks) splits of 64-192 steps ran 6-25% slower than 32-48.
Split pick_split(int M, int N, int K, int64_t cap_elems) {
  const int base = (N / 128) * gemm_mblock_groups(M);  // workgroups per split
  for (int s = 1; s <= 64; ++s) {
    if (K % (s * 64)) continue;
    if ((int64_t)base * s >= 192 && K / (s * 64) <= 48 && (int64_t)s * M * N <= cap_elems) return {s, K / s};
  }
  // fall back: one split per 1024 of K (runtime-loop kernel)
  int s = std::max(1, K / 1024);
  while (s > 1 && (int64_t)s * M * N > cap_elems) --s;
  const int kper = cdiv_i(cdiv_i(K, s), 64) * 64;
  return {cdiv_i(K, kper), kper};
}

// Split-K partial elements the projections of an R-row pass write at most.
int64_t partials_needed(const ModelDims& md, int R) {
  int64_t n = 1;
  const int shapes[3][2] = {{md.qkv, md.d}, {md.d, md.nq * md.hd}, {md.d, md.F}};
  for (const auto& nk : shapes) {
    const Split sp = pick_split(R, nk[0], nk[1], kPartialCap);
    n = std::max<int64_t>(n, (int64_t)sp.s * R * nk[0]);
  }
  return n;
}

// One projection: P[split][M][N] = A x W^T (or the LM-head argmax epilogue).
war_status gemm(const Workspace& w, const bf16_t* A, int lda, const int32_t* a_rows, const bf16_t* Wp,
                int M, int N, int K, int* splits_out, hipStream_t st, bool argmax = false,
                float* logits = nullptr, bf16_t* swiglu_out = nullptr) {
  GemmArgs g{};
  g.A = A;
  g.lda = lda;
  g.a_rows = a_rows;
  g.Wp = Wp;
  g.M = M;
  g.N = N;
  g.K = K;
  // the paired gate/up layout is only read by the SwiGLU epilogue: one split
  Split sp{1, K};
  if (!argmax && !swiglu_out) {
    sp = pick_split(M, N, K, kPartialCap);
    if ((int64_t)sp.s * M * N > w.p_elems) return fail(WAR_ERR_INVALID_ARG, "internal: split-K partials exceed the workspace");
  }
  g.kper = sp.kper;
  const bool fuse = swiglu_out != nullptr;
  g.out = swiglu_out;
  g.ld_out = N / 2;
  g.P = w.P;
  g.logits = logits;
  g.ld_logits = N;
  g.amax_v = w.amax_v;
  g.amax_i = w.amax_i;
  launch_gemm(g, argmax ? EPI_ARGMAX : fuse ? EPI_SWIGLU : EPI_PARTIAL, sp.s, st);
  if (splits_out) *splits_out = sp.s;
  return WAR_OK;
}

#define WARCHK(x)                      \
  do {                                 \
    war_status s_ = (x);               \
    if (s_ != WAR_OK) return s_;       \
  } while (0)

// The decoder body over `R` rows whose metadata is in w.meta(); the final
// normalised hidden state ends in w.u.
war_status run_layers(war_model* m, const Workspace& w, war_kv_pool* p, int R, const AttnArgs& attn_base,
                      int RB, int attn_grid, int n_segs, hipStream_t st) {
  const ModelDims& md = m->md;
  const StepMeta meta = w.meta();
  Profiler& pf = m->prof;
  {
    Timed t(pf, st, "rope_table");
    launch_rope_table(R, meta.pos, m->inv_freq.as<double>(), md.hd / 2, w.cos_t, w.sin_t, st);
  }
  {
    Timed t(pf, st, "embed_norm");
    launch_embed_norm(R, meta.tok, m->embed, m->layers[0].attn_norm, md.d, md.eps, w.h, w.u, st);
  }
  for (int l = 0; l < m->cfg.n_layers; ++l) {
    const LayerW& L = m->layers[l];
    int s = 1;
    {
      Timed t(pf, st, "gemm_qkv");
      WARCHK(gemm(w, w.u, md.d, nullptr, L.w_qkv, R, md.qkv, md.d, &s, st));
    }
    {
      Timed t(pf, st, "qkv_rope_kvwrite");
      launch_qkv_rope(R, s, w.P, md, w.cos_t, w.sin_t, meta, meta.row_req, p->dev.table, p->dev.max_pages,
                      p->geom, l, w.q, st);
    }
    AttnArgs a = attn_base;
    a.layer = l;
    {
      Timed t(pf, st, "attention");
      launch_attn(a, RB, md.hd, attn_grid, st);
    }
    {
      Timed t(pf, st, "attn_combine");
      launch_attn_combine(a, RB, md.hd, n_segs, st);
    }
    {
      Timed t(pf, st, "gemm_o");
      WARCHK(gemm(w, w.o, md.nq * md.hd, nullptr, L.w_o, R, md.d, md.nq * md.hd, &s, st));
    }
    {
      Timed t(pf, st, "residual_norm");
      launch_residual_norm(R, s, w.P, md.d, L.ffn_norm, md.eps, w.h, w.u, st);
    }
    {
      Timed t(pf, st, "gemm_gate_up_swiglu");
      WARCHK(gemm(w, w.u, md.d, nullptr, L.w_gate_up, R, 2 * md.F, md.d, &s, st, false, nullptr, w.y));
    }
    {
      Timed t(pf, st, "gemm_down");
      WARCHK(gemm(w, w.y, md.F, nullptr, L.w_down, R, md.d, md.F, &s, st));
    }
    const bf16_t* gnext = l + 1 < m->cfg.n_layers ? m->layers[l + 1].attn_norm : m->final_norm;
    {
      Timed t(pf, st, "residual_norm");
      launch_residual_norm(R, s, w.P, md.d, gnext, md.eps, w.h, w.u, st);
    }
  }
  HIPCHK(hipGetLastError());
  return WAR_OK;
}

AttnArgs attn_args(war_model* m, const Workspace& w, war_kv_pool* p, int TB) {
  AttnArgs a{};
  a.q = w.q;
  a.q_stride = m->md.nq * m->md.hd;
  a.kv = p->geom;
  a.table = p->dev.table;
  a.max_pages = p->dev.max_pages;
  a.meta = w.meta();
  a.G = m->md.nq / m->md.nkv;
  a.TB = TB;
  a.n_kv_heads = m->md.nkv;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)m->md.hd));
  a.pm = w.pm;
  a.pl = w.pl;
  a.po = w.po;
  a.o = w.o;
  a.unit_ctr = w.unit_ctr;
  return a;
}

// Grow the model's own workspace to hold n_items attention items of RB rows
// (rows: max_rows; partials: kPartialCap or what max_rows needs).  A new
// allocation starts with the attention work counters at zero.
war_status ensure_ws(war_model* m, int64_t n_items, int RB) {
  Workspace& w = m->ws;
  if (w.R && n_items <= w.items_cap && RB <= w.rb_cap) return WAR_OK;
  const int64_t items = std::max<int64_t>(n_items, w.items_cap);
  const int rb = std::max(RB, w.rb_cap);
  const int64_t pel = std::max<int64_t>(kPartialCap, partials_needed(m->md, m->max_rows));
  const size_t bytes = ws_layout(m->md, m->max_rows, items, rb, pel, nullptr, nullptr);
  const bool tree = w.tree_step;
  HIPCHK(m->ws_buf.ensure(bytes));
  ws_layout(m->md, m->max_rows, items, rb, pel, m->ws_buf.as<char>(), &w);
  w.tree_step = tree;
  HIPCHK(hipMemset(w.unit_ctr, 0, 8 * 4));
  return WAR_OK;
}

// ---- host lower bound of the pool's free pages (see war_kv_pool)
void set_exact_free(war_kv_pool* p, int64_t fc) {
  p->base_fc = fc;
  p->base_total = p->total_need;
  p->base_seq = p->commit_issued;
}

int64_t free_lower_bound(war_kv_pool* p) {
  int64_t lb = p->base_fc - (p->total_need - p->base_total);
  const unsigned long long r = __atomic_load_n(p->report, __ATOMIC_ACQUIRE);
  const uint32_t seq = (uint32_t)(r >> 32);
  const int64_t fc = (int64_t)(uint32_t)r;
  // a commit newer than the exact count, still in the ring
  if ((int32_t)(seq - p->base_seq) > 0 && (int32_t)(p->commit_issued - seq) >= 0 &&
      p->commit_issued - seq < (uint32_t)kRing)
    lb = std::max(lb, fc - (p->total_need - p->need_at[seq % kRing]));
  return lb;
}

// Read the pool's device scalars (syncs the stream).
war_status read_free_count(war_kv_pool* p, hipStream_t st, int32_t* fc, int32_t* err) {
  int32_t sc[2];
  HIPCHK(hipMemcpyAsync(sc, p->dev.scalars, sizeof(sc), hipMemcpyDeviceToHost, st));
  HIPCHK(hipStreamSynchronize(st));
  *fc = sc[0];
  if (err) *err = sc[1];
  set_exact_free(p, sc[0]);
  return WAR_OK;
}

war_status upload_ids(war_kv_pool* p, int n, const int32_t* a, const int32_t* b, hipStream_t st) {
  HIPCHK(ensure_pinned(p->pinned, p->pinned_ints, 2 * (size_t)n));
  HIPCHK(p->tmp.ensure(2 * (size_t)std::max(n, 1) * sizeof(int32_t)));
  std::memcpy(p->pinned, a, n * sizeof(int32_t));
  if (b) std::memcpy(p->pinned + n, b, n * sizeof(int32_t));
  HIPCHK(hipMemcpyAsync(p->tmp.p, p->pinned, (b ? 2 : 1) * n * sizeof(int32_t), hipMemcpyHostToDevice, st));
  return WAR_OK;
}

war_status check_ids(const war_kv_pool* p, int n, const int32_t* ids) {
  std::unordered_set<int32_t> seen;
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= p->dev.max_seqs) return fail(WAR_ERR_INVALID_ARG, "sequence id out of range");
    if (!seen.insert(ids[i]).second) return fail(WAR_ERR_INVALID_ARG, "duplicate sequence id");
  }
  return WAR_OK;
}

}  // namespace

// ===================================================================== C ABI
extern "C" {

const char* war_last_error(void) { return g_err.c_str(); }

int32_t war_weight_count(const war_model_config* cfg) { return cfg ? 3 + 7 * cfg->n_layers : -1; }

war_status war_model_create(const war_model_config* cfg, const void* const* weights, int32_t n_weights,
                            war_model** out) {
  if (!out) return fail(WAR_ERR_INVALID_ARG, "null out");
  *out = nullptr;
  war_status st = check_config(cfg);
  if (st != WAR_OK) return st;
  if (!weights || n_weights != war_weight_count(cfg))
    return fail(WAR_ERR_INVALID_ARG, "expected 3 + 7*n_layers weight pointers");
  for (int i = 0; i < n_weights; ++i)
    if (!weights[i] || !aligned16(weights[i])) return fail(WAR_ERR_INVALID_ARG, "null or unaligned weight");
  war_model* m = new war_model();
  m->cfg = *cfg;
  ModelDims& md = m->md;
  md.d = cfg->d_model;
  md.nq = cfg->n_q_heads;
  md.nkv = cfg->n_kv_heads;
  md.hd = cfg->head_dim;
  md.F = cfg->ffn_dim;
  md.V = cfg->vocab;
  md.qkv = (md.nq + 2 * md.nkv) * md.hd;
  md.eps = cfg->rms_eps;
  // One owned allocation: embedding (row-major), norm gains, and every matrix
  // repacked into MFMA fragment order.  The caller's buffers are read here
  // (stream-ordered on the null stream, then synchronised) and never again.
  const int64_t d = md.d, F = md.F, V = md.V, nqhd = (int64_t)md.nq * md.hd;
  const int64_t per_layer = 2 * d + (int64_t)md.qkv * d + d * nqhd + 2 * F * d + d * F;
  const int64_t total = 2 * V * d + d + cfg->n_layers * per_layer;
  if (hipError_t e0 = m->wts.ensure((size_t)total * 2); e0 != hipSuccess) {
    delete m;
    return fail(WAR_ERR_HIP, std::string("weight allocation: ") + hipGetErrorString(e0));
  }
  bf16_t* dst = m->wts.as<bf16_t>();
  int k = 0;
  auto src = [&]() { return static_cast<const bf16_t*>(weights[k++]); };
  hipError_t ecopy = hipSuccess;
  auto copy = [&](int64_t n) {
    bf16_t* at = dst;
    const hipError_t ec = hipMemcpyAsync(at, src(), (size_t)n * 2, hipMemcpyDeviceToDevice, nullptr);
    if (ecopy == hipSuccess) ecopy = ec;
    dst += n;
    return at;
  };
  auto pack = [&](int64_t N, int64_t K) {
    bf16_t* at = dst;
    launch_pack_weights(src(), nullptr, (int)N, (int)K, at, nullptr);
    dst += N * K;
    return at;
  };
  auto pack_pair = [&](int64_t F2, int64_t K) {  // gate [F2][K], then up [F2][K]
    bf16_t* at = dst;
    const bf16_t* gate = src();
    const bf16_t* up = src();
    launch_pack_weights(gate, up, (int)(2 * F2), (int)K, at, nullptr);
    dst += 2 * F2 * K;
    return at;
  };
  m->embed = copy(V * d);
  for (int l = 0; l < cfg->n_layers; ++l) {
    LayerW L;
    L.attn_norm = copy(d);
    L.w_qkv = pack(md.qkv, d);
    L.w_o = pack(d, nqhd);
    L.ffn_norm = copy(d);
    L.w_gate_up = pack_pair(F, d);
    L.w_down = pack(d, F);
    m->layers.push_back(L);
  }
  m->final_norm = copy(d);
  m->w_lm = pack(V, d);
  if (ecopy == hipSuccess) ecopy = hipGetLastError();
  if (hipError_t e0 = hipDeviceSynchronize(); e0 != hipSuccess || ecopy != hipSuccess) {
    if (e0 == hipSuccess) e0 = ecopy;
    war_model_destroy(m);
    return fail(WAR_ERR_HIP, std::string("weight copy: ") + hipGetErrorString(e0));
  }
  m->max_rows = cfg->max_rows;
  hipError_t e = m->inv_freq.ensure((size_t)md.hd / 2 * 8);
  if (e == hipSuccess) {
    std::vector<double> inv(md.hd / 2);
    for (int j = 0; j < md.hd / 2; ++j) inv[j] = std::pow((double)cfg->rope_base, -2.0 * j / md.hd);
    e = hipMemcpy(m->inv_freq.p, inv.data(), inv.size() * 8, hipMemcpyHostToDevice);
  }
  if (e != hipSuccess) {
    war_model_destroy(m);
    return fail(WAR_ERR_HIP, std::string("workspace allocation: ") + hipGetErrorString(e));
  }
  if (war_status ws = ensure_ws(m, 1, 16); ws != WAR_OK) {
    const std::string msg = g_err;
    war_model_destroy(m);
    return fail(ws, msg);
  }
  // this device's copy of the static scratch array, for war_verify_step_noalloc
  if (war_status ss = scratch_address(nullptr); ss != WAR_OK) {
    const std::string msg = g_err;
    war_model_destroy(m);
    return fail(ss, msg);
  }
  *out = m;
  return WAR_OK;
}

void war_model_destroy(war_model* m) {
  if (!m) return;
  for (DevBuf* b : {&m->wts, &m->inv_freq, &m->ws_buf, &m->path_ws, &m->logits_ws, &m->row_out, &m->stage_dev})
    b->release();
  if (m->pinned) (void)hipHostFree(m->pinned);
  for (hipEvent_t e : m->prof.pool) (void)hipEventDestroy(e);
  delete m;
}

war_status war_kv_pool_create(const war_model_config* cfg, void* kv_pages, int32_t num_pages,
                              int32_t* block_tables, int32_t max_seqs, int32_t max_pages_per_seq,
                              void* stream, war_kv_pool** out) {
  if (!out) return fail(WAR_ERR_INVALID_ARG, "null out");
  *out = nullptr;
  war_status s0 = check_config(cfg);
  if (s0 != WAR_OK) return s0;
  CHECK(kv_pages && block_tables, "null kv_pages or block_tables");
  CHECK(aligned16(kv_pages), "kv_pages must be 16-byte aligned");
  CHECK(num_pages > 0 && max_seqs > 0 && max_pages_per_seq > 0, "non-positive pool size");
  CHECK((int64_t)max_pages_per_seq * cfg->page_size <= (1 << 24), "max_pages_per_seq too large");
  hipStream_t st = static_cast<hipStream_t>(stream);
  war_kv_pool* p = new war_kv_pool();
  p->cfg = *cfg;
  p->geom.kv = static_cast<bf16_t*>(kv_pages);
  p->geom.num_pages = num_pages;
  p->geom.n_kv_heads = cfg->n_kv_heads;
  p->geom.head_dim = cfg->head_dim;
  p->geom.page_size = cfg->page_size;
  const size_t words = (size_t)2 * num_pages + 2 * (size_t)max_seqs + 4;
  hipError_t e = p->state.ensure(words * 4);
  if (e != hipSuccess) {
    delete p;
    return fail(WAR_ERR_HIP, std::string("pool state allocation: ") + hipGetErrorString(e));
  }
  int32_t* w = p->state.as<int32_t>();
  p->dev.stack = w;
  p->dev.refcount = w + num_pages;
  p->dev.held = w + 2 * (size_t)num_pages;
  p->dev.base = p->dev.held + max_seqs;
  p->dev.scalars = p->dev.base + max_seqs;
  p->dev.table = block_tables;
  p->dev.num_pages = num_pages;
  p->dev.max_seqs = max_seqs;
  p->dev.max_pages = max_pages_per_seq;
  p->dev.page_size = cfg->page_size;
  // the commit kernel's report word: pinned, mapped into the device's address space
  e = hipHostMalloc(reinterpret_cast<void**>(&p->report), sizeof(unsigned long long),
                    hipHostMallocMapped | hipHostMallocCoherent);
  if (e == hipSuccess) {
    *p->report = (unsigned long long)(uint32_t)num_pages;  // commit 0, every page free
    e = hipHostGetDevicePointer(reinterpret_cast<void**>(&p->dev.report), p->report, 0);
  } else {
    p->report = nullptr;
  }
  if (e != hipSuccess) {
    war_kv_pool_destroy(p);
    return fail(WAR_ERR_HIP, std::string("pool report word: ") + hipGetErrorString(e));
  }
  p->base_fc = num_pages;
  launch_pool_init(p->dev, st);
  e = hipGetLastError();
  if (e != hipSuccess) {
    war_kv_pool_destroy(p);
    return fail(WAR_ERR_HIP, std::string("pool init: ") + hipGetErrorString(e));
  }
  *out = p;
  return WAR_OK;
}

void war_kv_pool_destroy(war_kv_pool* p) {
  if (!p) return;
  p->state.release();
  p->tmp.release();
  if (p->pinned) (void)hipHostFree(p->pinned);
  if (p->report) (void)hipHostFree(p->report);
  delete p;
}

war_status war_pool_state(war_kv_pool* p, int32_t* free_count, int32_t* free_stack, int32_t* refcount,
                          int32_t* held, int32_t* step_base, void* stream) {
  CHECK(p, "null pool");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t fc, err;
  war_status s = read_free_count(p, st, &fc, &err);
  if (s != WAR_OK) return s;
  if (free_count) *free_count = fc;
  if (free_stack) HIPCHK(hipMemcpy(free_stack, p->dev.stack, (size_t)p->dev.num_pages * 4, hipMemcpyDeviceToHost));
  if (refcount) HIPCHK(hipMemcpy(refcount, p->dev.refcount, (size_t)p->dev.num_pages * 4, hipMemcpyDeviceToHost));
  if (held) HIPCHK(hipMemcpy(held, p->dev.held, (size_t)p->dev.max_seqs * 4, hipMemcpyDeviceToHost));
  if (step_base) HIPCHK(hipMemcpy(step_base, p->dev.base, (size_t)p->dev.max_seqs * 4, hipMemcpyDeviceToHost));
  if (err) {
    // reported once: the flags start again from zero
    HIPCHK(hipMemsetAsync(p->dev.scalars + 1, 0, 4, st));
    HIPCHK(hipStreamSynchronize(st));
    return fail(WAR_ERR_DEVICE, err & ERR_NO_PAGES     ? "device page shortage"
                                : err & ERR_DUP_SEQ    ? "a sequence id appears twice in one verify step"
                                : err & ERR_BAD_PARENT ? "tree parent out of range on device"
                                                       : "bad token id, sequence id or context length on device");
  }
  return WAR_OK;
}

war_status war_kv_alloc(war_kv_pool* p, int32_t n, const int32_t* seq_ids_host, const int32_t* n_tokens_host,
                        void* stream) {
  CHECK(p, "null pool");
  CHECK(!p->pending, "a verify step is waiting for war_kv_commit");
  CHECK(n >= 0 && n <= kMaxBatch, "n out of range [0, 1024]");
  if (n == 0) return WAR_OK;
  CHECK(seq_ids_host && n_tokens_host, "null array");
  war_status s = check_ids(p, n, seq_ids_host);
  if (s != WAR_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int64_t bound = 0;
  for (int i = 0; i < n; ++i) {
    CHECK(n_tokens_host[i] >= 0, "negative token count");
    const int pg = cdiv_i(n_tokens_host[i], p->dev.page_size);
    CHECK(pg <= p->dev.max_pages, "n_tokens exceeds max_pages_per_seq");
    bound += pg;
  }
  if (bound > free_lower_bound(p)) {
    int32_t fc;
    s = read_free_count(p, st, &fc, nullptr);
    if (s != WAR_OK) return s;
    std::vector<int32_t> held(p->dev.max_seqs);
    HIPCHK(hipMemcpy(held.data(), p->dev.held, held.size() * 4, hipMemcpyDeviceToHost));
    int64_t need = 0;
    for (int i = 0; i < n; ++i)
      need += std::max(0, cdiv_i(n_tokens_host[i], p->dev.page_size) - held[seq_ids_host[i]]);
    if (need > fc) return fail(WAR_ERR_OUT_OF_PAGES, "not enough free KV pages");
  }
  s = upload_ids(p, n, seq_ids_host, n_tokens_host, st);
  if (s != WAR_OK) return s;
  const int32_t* d = p->tmp.as<int32_t>();
  launch_grow(p->dev, n, d, d + n, nullptr, 0, st);
  HIPCHK(hipGetLastError());
  int32_t fc;
  return read_free_count(p, st, &fc, nullptr);  // waits: the pinned staging buffer is reused
}

war_status war_kv_fork(war_kv_pool* p, int32_t src_seq, int32_t dst_seq, int32_t n_tokens, void* stream) {
  CHECK(p, "null pool");
  CHECK(!p->pending, "a verify step is waiting for war_kv_commit");
  CHECK(src_seq >= 0 && src_seq < p->dev.max_seqs && dst_seq >= 0 && dst_seq < p->dev.max_seqs &&
            src_seq != dst_seq, "bad sequence ids");
  CHECK(n_tokens >= 0 && n_tokens % p->dev.page_size == 0, "fork length must be a multiple of the page size");
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t hs, hd;
  HIPCHK(hipMemcpyAsync(&hs, p->dev.held + src_seq, 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipMemcpyAsync(&hd, p->dev.held + dst_seq, 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipStreamSynchronize(st));
  const int npg = n_tokens / p->dev.page_size;
  CHECK(hd == 0, "fork destination already holds pages");
  CHECK(hs >= npg, "fork source holds fewer pages");
  launch_fork(p->dev, src_seq, dst_seq, npg, st);
  HIPCHK(hipGetLastError());
  if (npg > 0) p->forked = true;
  int32_t fc;
  return read_free_count(p, st, &fc, nullptr);
}

war_status war_kv_free(war_kv_pool* p, int32_t n, const int32_t* seq_ids_host, void* stream) {
  CHECK(p, "null pool");
  CHECK(!p->pending, "a verify step is waiting for war_kv_commit");
  CHECK(n >= 0 && n <= kMaxBatch, "n out of range [0, 1024]");
  if (n == 0) return WAR_OK;
  CHECK(seq_ids_host, "null array");
  war_status s = check_ids(p, n, seq_ids_host);
  if (s != WAR_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = upload_ids(p, n, seq_ids_host, nullptr, st);
  if (s != WAR_OK) return s;
  launch_free(p->dev, n, p->tmp.as<int32_t>(), st);
  HIPCHK(hipGetLastError());
  int32_t fc;
  return read_free_count(p, st, &fc, nullptr);  // waits: the pinned staging buffer is reused
}

war_status war_kv_load(war_kv_pool* p, int32_t seq_id, int32_t layer, int32_t pos0, int32_t n,
                       const void* src, void* stream) {
  CHECK(p && src, "null pool or src");
  CHECK(seq_id >= 0 && seq_id < p->dev.max_seqs, "sequence id out of range");
  CHECK(layer >= 0 && layer < p->cfg.n_layers, "layer out of range");
  CHECK(pos0 >= 0 && n >= 0, "negative position or count");
  if (n == 0) return WAR_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int32_t hs;
  HIPCHK(hipMemcpyAsync(&hs, p->dev.held + seq_id, 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipStreamSynchronize(st));
  CHECK((int64_t)pos0 + n <= (int64_t)hs * p->dev.page_size, "tokens beyond the sequence's pages");
  launch_kv_load(p->dev, p->geom, seq_id, layer, pos0, n, static_cast<const bf16_t*>(src), st);
  HIPCHK(hipGetLastError());
  return WAR_OK;
}

}  // extern "C"

namespace {

// Sampling parameters of war_verify_step_sampled (nullptr uniforms: greedy).
struct SampleParams {
  const float* uniforms = nullptr;
  float temperature = 1.f;
  int top_k = 1;
};

// A fixed device region to lay the step's workspace over instead of the
// model's own workspace (which grows on demand); nothing is allocated then.
struct StaticWs {
  char* base;
  size_t bytes;
};

war_status verify_impl(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                       const int32_t* ctx_lens, const int32_t* last_tokens, const int32_t* draft_tokens,
                       const int32_t* draft_lens, int32_t k_max, int32_t* accept_lens,
                       int32_t* next_tokens, float* logits, void* stream, const SampleParams& sp,
                       const int32_t* draft_parents = nullptr, int32_t* accept_path = nullptr,
                       const StaticWs* fixed = nullptr) {
  CHECK(m && p, "null model or pool");
  CHECK(same_shape(m->cfg, p->cfg), "model and pool shapes differ");
  CHECK(!p->pending, "previous verify step not committed");
  CHECK(B >= 1 && B <= kMaxBatch && B <= p->dev.max_seqs, "B out of range");
  CHECK(k_max >= 0, "negative k_max");
  const int G = m->md.nq / m->md.nkv;
  if (G * (k_max + 1) > 48) return fail(WAR_ERR_UNSUPPORTED, "n_q/n_kv * (k_max+1) must be <= 48");
  CHECK((int64_t)B * (k_max + 1) <= m->max_rows, "B*(k_max+1) exceeds max_rows");
  CHECK(seq_ids && ctx_lens && last_tokens && accept_lens && next_tokens, "null array");
  CHECK(k_max == 0 || draft_tokens, "draft_tokens required when k_max > 0");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int P = p->dev.page_size;
  const bool tree = draft_parents != nullptr && k_max > 0;
  if (tree && k_max + 1 > 32) return fail(WAR_ERR_UNSUPPORTED, "tree drafts: k_max + 1 must be <= 32");
  if (tree && sp.uniforms) return fail(WAR_ERR_UNSUPPORTED, "tree drafts are verified greedily");

  const int kp1 = k_max + 1;
  const int R = B * kp1;
  const int RB = attn_rows_per_block(G, kp1);
  // keys per attention item: long enough that each wave streams 8+ blocks
  int chunk = 1024;
  while (cdiv_i(p->dev.max_pages * P, chunk) > kMaxItemsPerSeq) chunk *= 2;
  int64_t max_items = (int64_t)B * cdiv_i(p->dev.max_pages * P, chunk);
  Workspace wsv;
  if (fixed) {
    // a fixed region: rows exactly R; the attention items bound shrinks by
    // longer chunks until the layout fits (the step setup may still double it)
    const int64_t pel = partials_needed(m->md, R);
    size_t bytes = ws_layout(m->md, R, max_items, RB, pel, nullptr, nullptr);
    while (bytes > fixed->bytes && chunk < (1 << 20)) {
      chunk *= 2;
      max_items = (int64_t)B * cdiv_i(p->dev.max_pages * P, chunk);
      bytes = ws_layout(m->md, R, max_items, RB, pel, nullptr, nullptr);
    }
    if (bytes > fixed->bytes)
      return fail(WAR_ERR_UNSUPPORTED, "the step's workspace (" + std::to_string(bytes) +
                                           " bytes) exceeds the static scratch (" +
                                           std::to_string(fixed->bytes) + " bytes)");
    ws_layout(m->md, R, max_items, RB, pel, fixed->base, &wsv);
  } else {
    war_status s = ensure_ws(m, max_items, RB);
    if (s != WAR_OK) return s;
    wsv = m->ws;
  }
  wsv.tree_step = tree;
  if (!fixed) m->ws.tree_step = tree;
  const Workspace& w = wsv;

  // capacity: ctx + draft + 1 slots need at most cdiv(k_max+1, P) new pages per request
  const int64_t bound = (int64_t)B * cdiv_i(k_max + 1, P);
  int64_t need = bound;
  if (bound > free_lower_bound(p)) {
    int32_t fc;
    ++p->exact_waits;
    war_status s = read_free_count(p, st, &fc, nullptr);
    if (s != WAR_OK) return s;
    if (bound > fc) {
      // with a fixed region no per-request state is read (it would need host buffers)
      if (fixed) return fail(WAR_ERR_OUT_OF_PAGES, "fewer free KV pages than B * ceil((k_max+1)/page_size)");
      std::vector<int32_t> sid(B), ctx(B), dl(B, k_max), held(p->dev.max_seqs);
      HIPCHK(hipMemcpy(sid.data(), seq_ids, B * 4, hipMemcpyDeviceToHost));
      HIPCHK(hipMemcpy(ctx.data(), ctx_lens, B * 4, hipMemcpyDeviceToHost));
      if (draft_lens) HIPCHK(hipMemcpy(dl.data(), draft_lens, B * 4, hipMemcpyDeviceToHost));
      HIPCHK(hipMemcpy(held.data(), p->dev.held, held.size() * 4, hipMemcpyDeviceToHost));
      need = 0;
      for (int b = 0; b < B; ++b) {
        CHECK(sid[b] >= 0 && sid[b] < p->dev.max_seqs, "sequence id out of range");
        const int d = std::min(std::max(dl[b], 0), k_max);
        need += std::max(0, cdiv_i(std::max(ctx[b], 0) + d + 1, P) - held[sid[b]]);
      }
      if (need > fc) return fail(WAR_ERR_OUT_OF_PAGES, "not enough free KV pages for the draft slots");
    }
  }

  VerifySetupArgs va;
  va.B = B;
  va.k_max = k_max;
  va.vocab = m->md.V;
  va.unit_ctr = w.unit_ctr;
  va.chunk = chunk;
  va.items_double = cdiv_i(2 * kAttnGrid, m->md.nkv);  // 2+ units per workgroup of a full grid
  va.seq_ids = seq_ids;
  va.ctx_lens = ctx_lens;
  va.last_tokens = last_tokens;
  va.draft_tokens = draft_tokens;
  va.draft_lens = draft_lens;
  va.G = G;
  va.rb = RB;
  va.cascade = p->forked && B > 1 ? 1 : 0;  // shared-prefix units for forked siblings
  va.draft_parents = tree ? draft_parents : nullptr;
  if (tree && !accept_path) {
    HIPCHK(m->path_ws.ensure((size_t)B * k_max * 4));
    accept_path = m->path_ws.as<int32_t>();
  }
  const StepMeta meta = w.meta();
  {
    Timed t(m->prof, st, "verify_setup");
    launch_verify_setup(p->dev, va, meta, st);
  }

  AttnArgs a = attn_args(m, w, p, kp1);
  a.prb = RB;
  // persistent grid = resident capacity: 2 workgroups per CU
  const int grid = (int)std::min<int64_t>(max_items * m->md.nkv, kAttnGrid);
  war_status s = run_layers(m, w, p, R, a, RB, grid, B, st);
  if (s != WAR_OK) return s;
  int sdummy;
  if (sp.uniforms) {
    // the full logits are needed: the caller's buffer, else the workspace
    float* lg = logits;
    if (!lg) {
      HIPCHK(m->logits_ws.ensure((size_t)R * m->md.V * 4));
      lg = m->logits_ws.as<float>();
    }
    HIPCHK(m->row_out.ensure((size_t)R * 3 * 4));
    {
      Timed t(m->prof, st, "gemm_lm_head");
      WARCHK(gemm(w, w.u, m->md.d, nullptr, m->w_lm, R, m->md.V, m->md.d, &sdummy, st, true, lg));
    }
    SampleArgs sa{};
    sa.logits = lg;
    sa.V = m->md.V;
    sa.ntok = meta.req_ntok;
    sa.drafts = draft_tokens;
    sa.k_max = k_max;
    sa.kp1 = kp1;
    sa.B = B;
    sa.uniforms = sp.uniforms;
    sa.temperature = sp.temperature;
    sa.top_k = sp.top_k;
    sa.row_out = m->row_out.as<int32_t>();
    Timed t(m->prof, st, "sample_accept");
    launch_sample(sa, accept_lens, next_tokens, st);
  } else {
    {
      Timed t(m->prof, st, "gemm_lm_head_argmax");
      WARCHK(gemm(w, w.u, m->md.d, nullptr, m->w_lm, R, m->md.V, m->md.d, &sdummy, st, true, logits));
    }
    Timed t(m->prof, st, "argmax_accept");
    launch_argmax_accept(B, meta.req_ntok, kp1, m->md.V / 128, w.amax_v, w.amax_i, draft_tokens,
                         tree ? draft_parents : nullptr, k_max, accept_lens, next_tokens, accept_path, st);
  }
  if (tree) {
    Timed t(m->prof, st, "kv_compact");
    launch_kv_compact(p->geom, m->cfg.n_layers, B, meta, p->dev.table, p->dev.max_pages, accept_lens,
                      accept_path, k_max, st);
  }
  HIPCHK(hipGetLastError());
  p->total_need += need;
  p->pending = true;
  p->pending_B = B;
  return WAR_OK;
}

}  // namespace

extern "C" {

war_status war_verify_step(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                           const int32_t* ctx_lens, const int32_t* last_tokens, const int32_t* draft_tokens,
                           const int32_t* draft_lens, int32_t k_max, int32_t* accept_lens,
                           int32_t* next_tokens, float* logits, void* stream) {
  return verify_impl(m, p, B, seq_ids, ctx_lens, last_tokens, draft_tokens, draft_lens, k_max, accept_lens,
                     next_tokens, logits, stream, SampleParams{});
}

war_status war_verify_step_sampled(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                                   const int32_t* ctx_lens, const int32_t* last_tokens,
                                   const int32_t* draft_tokens, const int32_t* draft_lens, int32_t k_max,
                                   const float* uniforms, float temperature, int32_t top_k,
                                   int32_t* accept_lens, int32_t* next_tokens, float* logits, void* stream) {
  CHECK(m, "null model");
  CHECK(uniforms, "null uniforms");
  CHECK(std::isfinite(temperature) && temperature > 0.f, "temperature must be positive and finite");
  CHECK(top_k >= 1 && top_k <= m->md.V, "top_k out of range [1, vocab]");
  SampleParams sp;
  sp.uniforms = uniforms;
  sp.temperature = temperature;
  sp.top_k = top_k;
  return verify_impl(m, p, B, seq_ids, ctx_lens, last_tokens, draft_tokens, draft_lens, k_max, accept_lens,
                     next_tokens, logits, stream, sp);
}

war_status war_verify_step_tree(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                                const int32_t* ctx_lens, const int32_t* last_tokens,
                                const int32_t* draft_tokens, const int32_t* draft_parents,
                                const int32_t* draft_lens, int32_t k_max, int32_t* accept_lens,
                                int32_t* next_tokens, int32_t* accept_path, float* logits, void* stream) {
  CHECK(k_max == 0 || draft_parents, "draft_parents required when k_max > 0");
  return verify_impl(m, p, B, seq_ids, ctx_lens, last_tokens, draft_tokens, draft_lens, k_max, accept_lens,
                     next_tokens, logits, stream, SampleParams{}, draft_parents, accept_path);
}

war_status war_verify_step_noalloc(war_model* m, war_kv_pool* p, int32_t B, const int32_t* seq_ids,
                                   const int32_t* ctx_lens, const int32_t* last_tokens,
                                   const int32_t* draft_tokens, const int32_t* draft_lens, int32_t k_max,
                                   int32_t* accept_lens, int32_t* next_tokens, float* logits, void* stream) {
  CHECK(m, "null model");
  void* base = nullptr;
  war_status s = scratch_address(&base);
  if (s != WAR_OK) return s;
  const StaticWs fixed{static_cast<char*>(base), kScratchBytes};
  const bool prof = m->prof.on;  // the profiler creates events: off for this call
  m->prof.on = false;
  s = verify_impl(m, p, B, seq_ids, ctx_lens, last_tokens, draft_tokens, draft_lens, k_max, accept_lens,
                  next_tokens, logits, stream, SampleParams{}, nullptr, nullptr, &fixed);
  m->prof.on = prof;
  return s;
}

war_status war_kv_commit(war_kv_pool* p, int32_t B, const int32_t* seq_ids, int32_t* ctx_lens,
                         const int32_t* accept_lens, void* stream) {
  CHECK(p, "null pool");
  CHECK(p->pending, "no verify step to commit");
  CHECK(B == p->pending_B, "B differs from the verify step's");
  CHECK(seq_ids && ctx_lens && accept_lens, "null array");
  const uint32_t seq = p->commit_issued + 1;
  launch_commit(p->dev, B, seq_ids, ctx_lens, accept_lens, seq, static_cast<hipStream_t>(stream));
  HIPCHK(hipGetLastError());
  p->commit_issued = seq;
  p->need_at[seq % kRing] = p->total_need;
  p->pending = false;
  return WAR_OK;
}

war_status war_prefill_append(war_model* m, war_kv_pool* p, int32_t n, const int32_t* seq_ids,
                              int32_t* ctx_lens, const int32_t* n_new_host, const int32_t* new_tokens,
                              int32_t* next_tokens, float* last_logits, void* stream) {
  CHECK(m && p, "null model or pool");
  CHECK(same_shape(m->cfg, p->cfg), "model and pool shapes differ");
  CHECK(!p->pending, "a verify step is waiting for war_kv_commit");
  CHECK(n >= 1 && n <= kMaxBatch, "n out of range [1, 1024]");
  CHECK(seq_ids && ctx_lens && n_new_host && new_tokens && next_tokens, "null array");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int P = p->dev.page_size;
  const int G = m->md.nq / m->md.nkv;
  int64_t total = 0;
  for (int i = 0; i < n; ++i) {
    CHECK(n_new_host[i] >= 1, "n_new must be >= 1");
    total += n_new_host[i];
  }
  CHECK(total <= (int64_t)1 << 30, "too many new tokens");
  // read ids, lengths and held pages (one synchronisation)
  std::vector<int32_t> sid(n), ctx(n), held(p->dev.max_seqs), toks(total);
  HIPCHK(hipMemcpyAsync(toks.data(), new_tokens, total * 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipMemcpyAsync(sid.data(), seq_ids, n * 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipMemcpyAsync(ctx.data(), ctx_lens, n * 4, hipMemcpyDeviceToHost, st));
  HIPCHK(hipMemcpyAsync(held.data(), p->dev.held, held.size() * 4, hipMemcpyDeviceToHost, st));
  int32_t fc;
  war_status s = read_free_count(p, st, &fc, nullptr);
  if (s != WAR_OK) return s;
  s = check_ids(p, n, sid.data());
  if (s != WAR_OK) return s;
  for (int64_t i = 0; i < total; ++i)
    CHECK(toks[i] >= 0 && toks[i] < m->md.V, "token id outside [0, vocab)");
  int64_t need = 0;
  for (int i = 0; i < n; ++i) {
    CHECK(ctx[i] >= 0, "negative ctx_len");
    const int64_t pages = cdiv_i(ctx[i] + n_new_host[i], P);
    CHECK(pages <= p->dev.max_pages, "sequence would exceed max_pages_per_seq");
    CHECK(ctx[i] <= (int64_t)held[sid[i]] * P, "ctx_len beyond the sequence's pages");
    need += std::max<int64_t>(0, pages - held[sid[i]]);
  }
  if (need > fc) return fail(WAR_ERR_OUT_OF_PAGES, "not enough free KV pages for the new tokens");

  // reserve: targets = ctx + n_new
  HIPCHK(m->stage_dev.ensure((size_t)n * 4));
  HIPCHK(ensure_pinned(m->pinned, m->pinned_ints, (size_t)n));
  std::memcpy(m->pinned, n_new_host, n * 4);
  int32_t* d_new = m->stage_dev.as<int32_t>();
  HIPCHK(hipMemcpyAsync(d_new, m->pinned, n * 4, hipMemcpyHostToDevice, st));
  launch_grow(p->dev, n, seq_ids, ctx_lens, d_new, 1, st);
  HIPCHK(hipGetLastError());
  set_exact_free(p, fc - need);

  // forward over chunks of at most max_rows packed rows; attention in row
  // blocks of kPrefillRows rows (k_attn_rows)
  const int RB = kPrefillRows;
  CHECK(RB % G == 0, "internal: query heads per kv head must divide the prefill row block");
  const int TB = RB / G;
  int chunk = kPrefillChunk;
  while (cdiv_i(p->dev.max_pages * P, chunk) > kMaxItemsPerSeq) chunk *= 2;
  std::vector<int64_t> cu(n + 1, 0);
  for (int i = 0; i < n; ++i) cu[i + 1] = cu[i] + n_new_host[i];
  const int R_cap = m->max_rows;
  for (int64_t r0 = 0; r0 < total; r0 += R_cap) {
    const int64_t r1 = std::min<int64_t>(total, r0 + R_cap);
    const int R = (int)(r1 - r0);
    // requests of this chunk
    std::vector<int32_t> rq_seq, rq_pos0, rq_ntok, rq_row0, rq_idx;
    for (int i = 0; i < n; ++i) {
      const int64_t a = std::max<int64_t>(r0, cu[i]), b = std::min<int64_t>(r1, cu[i + 1]);
      if (a >= b) continue;
      rq_idx.push_back(i);
      rq_seq.push_back(sid[i]);
      rq_pos0.push_back((int32_t)(ctx[i] + (a - cu[i])));
      rq_ntok.push_back((int32_t)(b - a));
      rq_row0.push_back((int32_t)(a - r0));
    }
    const int nr = (int)rq_seq.size();
    std::vector<int32_t> pos(R), act(R, 1), rreq(R);
    std::vector<int32_t> sg_b, sg_c, sg_r, sg_rb;
    std::vector<int4> items, udesc;
    for (int j = 0; j < nr; ++j) {
      for (int t = 0; t < rq_ntok[j]; ++t) {
        pos[rq_row0[j] + t] = rq_pos0[j] + t;
        rreq[rq_row0[j] + t] = j;
      }
      // items (and so the merge order) row block by row block; the work order
      // chunk by chunk, so that the units reading one key chunk for different
      // row blocks run together and find it in their XCD's L2
      const int nrb = cdiv_i(rq_ntok[j], TB);
      const int seg0 = (int)sg_b.size();
      for (int rb = 0; rb < nrb; ++rb) {
        const int S = rq_pos0[j] + std::min(rq_ntok[j], (rb + 1) * TB);
        const int nch = cdiv_i(S, chunk);
        sg_b.push_back((int32_t)items.size());
        sg_c.push_back(nch);
        sg_r.push_back(j);
        sg_rb.push_back(rb);
        for (int c = 0; c < nch; ++c) items.push_back(make_int4(j, rb, c, 0));
      }
      const int max_nch = sg_c.back();  // the last row block sees the most keys
      for (int c = 0; c < max_nch; ++c)
        for (int rb = 0; rb < nrb; ++rb) {
          if (c >= sg_c[seg0 + rb]) continue;
          const int t0 = rb * TB, ntk = std::min(TB, rq_ntok[j] - t0);
          udesc.push_back(make_int4(sg_b[seg0 + rb] + c, j, c, t0 | (ntk << 16)));
          udesc.push_back(make_int4(0, rq_seq[j], rq_pos0[j], rq_row0[j]));
        }
    }
    const int nseg = (int)sg_b.size();
    CHECK(nseg <= m->ws.n_seg_cap && nr <= m->ws.n_req_cap, "internal: prefill chunk too fragmented");
    // previous chunk's kernels read the metadata buffers: wait before overwriting
    // (and before ensure_ws may reallocate the workspace)
    HIPCHK(hipStreamSynchronize(st));
    s = ensure_ws(m, (int64_t)items.size(), RB);
    if (s != WAR_OK) return s;
    m->ws.tree_step = false;  // prefill rows are a causal chain
    const Workspace& w = m->ws;
    const StepMeta meta = w.meta();  // after any reallocation
    auto h2d = [&](void* dst, const void* src, size_t bytes) {
      return hipMemcpyAsync(dst, src, bytes, hipMemcpyHostToDevice, st);
    };
    HIPCHK(h2d(meta.pos, pos.data(), R * 4));
    HIPCHK(h2d(meta.active, act.data(), R * 4));
    HIPCHK(h2d(meta.row_req, rreq.data(), R * 4));
    HIPCHK(hipMemcpyAsync(meta.tok, new_tokens + r0, R * 4, hipMemcpyDeviceToDevice, st));
    HIPCHK(h2d(meta.req_seq, rq_seq.data(), nr * 4));
    HIPCHK(h2d(meta.req_pos0, rq_pos0.data(), nr * 4));
    HIPCHK(h2d(meta.req_ntok, rq_ntok.data(), nr * 4));
    HIPCHK(h2d(meta.req_row0, rq_row0.data(), nr * 4));
    HIPCHK(h2d(meta.seg_begin, sg_b.data(), nseg * 4));
    HIPCHK(h2d(meta.seg_count, sg_c.data(), nseg * 4));
    HIPCHK(h2d(meta.seg_req, sg_r.data(), nseg * 4));
    HIPCHK(h2d(meta.seg_rb, sg_rb.data(), nseg * 4));
    HIPCHK(h2d(meta.items, items.data(), items.size() * sizeof(int4)));
    HIPCHK(h2d(meta.udesc, udesc.data(), udesc.size() * sizeof(int4)));
    // prefill: the work order is the item list
    const int32_t ni4[4] = {(int32_t)items.size(), (int32_t)items.size(), 0, chunk};
    const int32_t ni = ni4[0];
    HIPCHK(h2d(meta.n_items, ni4, 16));
    HIPCHK(hipStreamSynchronize(st));  // host vectors go out of scope below

    AttnArgs a = attn_args(m, w, p, TB);
    a.meta.order = nullptr;  // prefill items run in list order
    a.prb = RB;
    const int grid = (int)std::min<int64_t>((int64_t)ni * m->md.nkv, kAttnGrid);
    s = run_layers(m, w, p, R, a, RB, std::max(grid, 1), nseg, st);
    if (s != WAR_OK) return s;
    // LM head on the rows that end a sequence inside this chunk
    std::vector<int32_t> last_rows;
    int first_seq = -1;
    for (int j = 0; j < nr; ++j) {
      const int i = rq_idx[j];
      if (cu[i + 1] <= r1 && cu[i + 1] > r0) {
        if (first_seq < 0) first_seq = i;
        last_rows.push_back((int32_t)(cu[i + 1] - 1 - r0));
      }
    }
    if (!last_rows.empty()) {
      const int nl = (int)last_rows.size();
      HIPCHK(hipMemcpyAsync(w.a_rows, last_rows.data(), nl * 4, hipMemcpyHostToDevice, st));
      int sd;
      WARCHK(gemm(w, w.u, m->md.d, w.a_rows, m->w_lm, nl, m->md.V, m->md.d, &sd, st, true,
                  last_logits ? last_logits + (int64_t)first_seq * m->md.V : nullptr));
      launch_argmax_accept(nl, nullptr, 1, m->md.V / 128, w.amax_v, w.amax_i, nullptr, nullptr, 0, nullptr,
                           next_tokens + first_seq, nullptr, st);
      HIPCHK(hipGetLastError());
      HIPCHK(hipStreamSynchronize(st));  // last_rows goes out of scope
    }
  }
  launch_add_ctx(n, ctx_lens, d_new, st);
  HIPCHK(hipGetLastError());
  return read_free_count(p, st, &fc, nullptr);  // waits for the whole append
}

war_status war_profile(war_model* m, int32_t enable) {
  CHECK(m, "null model");
  m->prof.on = enable != 0;
  m->prof.used = 0;
  m->prof.marks.clear();
  return WAR_OK;
}

war_status war_profile_read(war_model* m, char* out, int32_t out_len) {
  CHECK(m && out && out_len > 0, "null argument");
  HIPCHK(hipDeviceSynchronize());
  std::vector<std::string> names;
  std::vector<double> ms;
  std::vector<int> calls;
  for (auto& mk : m->prof.marks) {
    float t = 0.f;
    HIPCHK(hipEventElapsedTime(&t, m->prof.pool[mk.second.first], m->prof.pool[mk.second.second]));
    size_t i = 0;
    while (i < names.size() && names[i] != mk.first) ++i;
    if (i == names.size()) {
      names.push_back(mk.first);
      ms.push_back(0.0);
      calls.push_back(0);
    }
    ms[i] += t;
    calls[i] += 1;
  }
  std::string text;
  for (size_t i = 0; i < names.size(); ++i)
    text += names[i] + " " + std::to_string(calls[i]) + " " + std::to_string(ms[i]) + "\n";
  std::strncpy(out, text.c_str(), (size_t)out_len - 1);
  out[out_len - 1] = 0;
  m->prof.used = 0;
  m->prof.marks.clear();
  return (int64_t)text.size() < out_len ? WAR_OK : fail(WAR_ERR_INVALID_ARG, "profile text truncated");
}

war_status war_debug_sample(const float* logits, int32_t V, int32_t B, int32_t k_max, const int32_t* ntok,
                            const int32_t* drafts, const float* uniforms, float temperature, int32_t top_k,
                            int32_t* accept_lens, int32_t* next_tokens, void* stream) {
  CHECK(logits && ntok && uniforms && next_tokens && (k_max == 0 || drafts), "null array");
  CHECK(V >= 1 && B >= 1 && k_max >= 0, "bad sizes");
  CHECK(std::isfinite(temperature) && temperature > 0.f, "temperature must be positive and finite");
  CHECK(top_k >= 1 && top_k <= V, "top_k out of range [1, V]");
  hipStream_t st = static_cast<hipStream_t>(stream);
  DevBuf rows;
  HIPCHK(rows.ensure((size_t)B * (k_max + 1) * 3 * 4));
  SampleArgs sa{};
  sa.logits = logits;
  sa.V = V;
  sa.ntok = ntok;
  sa.drafts = drafts;
  sa.k_max = k_max;
  sa.kp1 = k_max + 1;
  sa.B = B;
  sa.uniforms = uniforms;
  sa.temperature = temperature;
  sa.top_k = top_k;
  sa.row_out = rows.as<int32_t>();
  launch_sample(sa, accept_lens, next_tokens, st);
  const hipError_t e = hipStreamSynchronize(st);
  rows.release();
  HIPCHK(e);
  return WAR_OK;
}

war_status war_debug_pool_waits(war_kv_pool* p, int64_t* waits) {
  CHECK(p && waits, "null argument");
  *waits = p->exact_waits;
  return WAR_OK;
}

war_status war_debug_workspace(war_model* m, const char* name, void** ptr, int64_t* bytes) {
  CHECK(m && name && ptr && bytes, "null argument");
  const std::string n(name);
  const Workspace& w = m->ws;
  const ModelDims& md = m->md;
  const int64_t R = w.R, nqhd = (int64_t)md.nq * md.hd, pr = w.items_cap * md.nkv * w.rb_cap;
  struct Entry {
    const char* name;
    const void* p;
    int64_t bytes;
  };
  const Entry table[] = {
      {"h", w.h, R * md.d * 4}, {"u", w.u, R * md.d * 2}, {"q", w.q, R * nqhd * 2}, {"o", w.o, R * nqhd * 2},
      {"P", w.P, w.p_elems * 4}, {"pm", w.pm, pr * 4}, {"pl", w.pl, pr * 4}, {"po", w.po, pr * md.hd * 4},
      {"rows", w.rows, 4 * R * 4}, {"reqs", w.reqs, 4 * (int64_t)w.n_req_cap * 4},
      {"items", w.items, w.items_cap * 16}, {"order", w.order, w.items_cap * 4}, {"n_items", w.n_items, 16},
      {"tree", w.tree, 2 * R * 4}};
  for (const Entry& e : table)
    if (n == e.name) {
      *ptr = const_cast<void*>(e.p);
      *bytes = e.bytes;
      return WAR_OK;
    }
  return fail(WAR_ERR_INVALID_ARG, "unknown workspace buffer");
}

}  // extern "C"
