// Row-wise kernels of the decoder step: RoPE table, embedding + RMSNorm,
// split-K reduction fused with residual + RMSNorm, with RoPE + KV-page write,
// and with SwiGLU; and the argmax + greedy acceptance of the verify step.
//
// Rounding points (bf16 compute, fp32 accumulate): every value that feeds a
// matrix multiply (norm outputs, SwiGLU product) and the rotated q, k and the v
// stored in the KV pages are rounded to bf16 (nearest even).  The residual
// stream, norm statistics, rotation and SwiGLU arithmetic stay fp32.
#include "kernels.h"

namespace {

// cos/sin of pos * inv_freq[j], evaluated in double and stored as float.
__global__ void k_rope_table(int rows, const int32_t* pos, const double* inv_freq, int half,
                             float* cos_t, float* sin_t) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * half) return;
  const int r = i / half, j = i % half;
  const double ang = (double)pos[r] * inv_freq[j];
  cos_t[i] = (float)cos(ang);
  sin_t[i] = (float)sin(ang);
}

// u = bf16(h * rsqrt(mean(h^2) + eps) * g), h already in global memory.
__device__ void norm_row(const float* h, int d, const bf16_t* g, float eps, bf16_t* u, float ss,
                         float* red) {
  const float tot = block_sum(ss, red);
  const float rs = rsqrtf(tot / (float)d + eps);
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const float4 x = *reinterpret_cast<const float4*>(h + c);
    const uint2 gg = *reinterpret_cast<const uint2*>(g + c);
    const float g0 = bf2f(gg.x & 0xffff), g1 = bf2f(gg.x >> 16);
    const float g2 = bf2f(gg.y & 0xffff), g3 = bf2f(gg.y >> 16);
    uint2 o;
    o.x = pack2(x.x * rs * g0, x.y * rs * g1);
    o.y = pack2(x.z * rs * g2, x.w * rs * g3);
    *reinterpret_cast<uint2*>(u + c) = o;
  }
}

__global__ void __launch_bounds__(256) k_embed_norm(const int32_t* tok, const bf16_t* E,
                                                    const bf16_t* g, int d, float eps, float* h,
                                                    bf16_t* u) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  const bf16_t* e = E + (int64_t)tok[r] * d;
  float* hr = h + (int64_t)r * d;
  float ss = 0.f;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const uint2 v = *reinterpret_cast<const uint2*>(e + c);
    float4 x;
    x.x = bf2f(v.x & 0xffff);
    x.y = bf2f(v.x >> 16);
    x.z = bf2f(v.y & 0xffff);
    x.w = bf2f(v.y >> 16);
    ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
    *reinterpret_cast<float4*>(hr + c) = x;
  }
  norm_row(hr, d, g, eps, u + (int64_t)r * d, ss, red);
}

// Sum of the split-K partials of one float4 run, in split order: the loads of
// up to eight splits are issued before the first add, so the split counts the
// projections use cost one memory round trip.
__device__ __forceinline__ float4 sum_splits(const float* P, int64_t sstride, int splits, float4 x) {
  for (int s0 = 0; s0 < splits; s0 += 8) {
    float4 t[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < splits) t[u] = *reinterpret_cast<const float4*>(P + (s0 + u) * sstride);
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (s0 + u < splits) {
        x.x += t[u].x; x.y += t[u].y; x.z += t[u].z; x.w += t[u].w;
      }
  }
  return x;
}

// h += sum_s P[s]; u = norm(h) * g   (one 1024-thread workgroup per row).
// NV > 0: each thread keeps its NV float4 of the row in registers (d <= 4096 NV)
// and has its gains loaded before the reduction, so the normalisation needs no
// second pass over memory; NV = 0: any width, h re-read after the reduction.
template <int NV>
__global__ void __launch_bounds__(1024) k_residual_norm(int rows, int splits, const float* P, int d,
                                                        const bf16_t* g, float eps, float* h,
                                                        bf16_t* u) {
  __shared__ float red[16];
  const int r = blockIdx.x;
  float* hr = h + (int64_t)r * d;
  const int64_t sstride = (int64_t)rows * d;
  float ss = 0.f;
  if constexpr (NV == 0) {
    for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
      float4 x = *reinterpret_cast<const float4*>(hr + c);
      x = sum_splits(P + (int64_t)r * d + c, sstride, splits, x);
      ss += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
      *reinterpret_cast<float4*>(hr + c) = x;
    }
    norm_row(hr, d, g, eps, u + (int64_t)r * d, ss, red);
  } else {
    float4 x[NV];
    uint2 gg[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = (threadIdx.x + i * 1024) * 4;
      if (c < d) {
        gg[i] = *reinterpret_cast<const uint2*>(g + c);
        x[i] = sum_splits(P + (int64_t)r * d + c, sstride, splits, *reinterpret_cast<const float4*>(hr + c));
        ss += x[i].x * x[i].x + x[i].y * x[i].y + x[i].z * x[i].z + x[i].w * x[i].w;
        *reinterpret_cast<float4*>(hr + c) = x[i];
      }
    }
    const float rs = rsqrtf(block_sum(ss, red) / (float)d + eps);
    bf16_t* ur = u + (int64_t)r * d;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c = (threadIdx.x + i * 1024) * 4;
      if (c < d) {
        uint2 o;
        o.x = pack2(x[i].x * rs * bf2f(gg[i].x & 0xffff), x[i].y * rs * bf2f(gg[i].x >> 16));
        o.y = pack2(x[i].z * rs * bf2f(gg[i].y & 0xffff), x[i].w * rs * bf2f(gg[i].y >> 16));
        *reinterpret_cast<uint2*>(ur + c) = o;
      }
    }
  }
}

// Sum the QKV partials of one row, rotate q and k (rotate-half pairs (j, j+D/2)),
// round to bf16; q goes to its buffer, k and v of active rows into the KV page slot
// of the row's position (a tree node's own slot, when the step has tree drafts).
// Each thread takes four consecutive pairs (16-byte loads of the partials).
__global__ void __launch_bounds__(64) k_qkv_rope(int rows, int splits, const float* P, ModelDims md,
                                                  const float* cos_t, const float* sin_t,
                                                  StepMeta meta, const int32_t* row_req,
                                                  const int32_t* table, int max_pages, KvGeom kv,
                                                  int layer, bf16_t* q) {
  const int r = blockIdx.x;
  const int half = md.hd / 2;
  const int nq_pairs = md.nq * half, nk_pairs = md.nkv * half;
  const int n_pairs = md.qkv / 2;
  const bool act = meta.active[r] != 0;
  const int p = (blockIdx.y * blockDim.x + threadIdx.x) * 4;  // first of four pairs
  if (p >= n_pairs) return;
  int page = 0, slot = 0;
  if (act) {
    const int pos = meta.kvpos ? meta.kvpos[r] : meta.pos[r];
    const int seq = meta.req_seq[row_req[r]];
    page = table[(int64_t)seq * max_pages + pos / kv.page_size];
    slot = pos % kv.page_size;
  }
  const float* pr = P + (int64_t)r * md.qkv;
  const int64_t pstride = (int64_t)rows * md.qkv;
  int region, head, j;
  if (p < nq_pairs) {
    region = 0;
    head = p / half;
    j = p % half;
  } else if (p < nq_pairs + nk_pairs) {
    region = 1;
    head = (p - nq_pairs) / half;
    j = (p - nq_pairs) % half;
  } else {
    region = 2;
    head = (p - nq_pairs - nk_pairs) / half;
    j = (p - nq_pairs - nk_pairs) % half;
  }
  const int col = (region == 0 ? 0 : region == 1 ? md.nq * md.hd : (md.nq + md.nkv) * md.hd) +
                  head * md.hd + j;
  float x1[4] = {0.f, 0.f, 0.f, 0.f}, x2[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
  for (int s = 0; s < splits; ++s) {
    const float4 a1 = *reinterpret_cast<const float4*>(pr + s * pstride + col);
    const float4 a2 = *reinterpret_cast<const float4*>(pr + s * pstride + col + half);
    x1[0] += a1.x; x1[1] += a1.y; x1[2] += a1.z; x1[3] += a1.w;
    x2[0] += a2.x; x2[1] += a2.y; x2[2] += a2.z; x2[3] += a2.w;
  }
  bf16_t b1[4], b2[4];
  if (region < 2) {
    const float4 c = *reinterpret_cast<const float4*>(cos_t + r * half + j);
    const float4 sn = *reinterpret_cast<const float4*>(sin_t + r * half + j);
    const float cc[4] = {c.x, c.y, c.z, c.w}, ss[4] = {sn.x, sn.y, sn.z, sn.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      b1[e] = f2bf(x1[e] * cc[e] - x2[e] * ss[e]);
      b2[e] = f2bf(x2[e] * cc[e] + x1[e] * ss[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      b1[e] = f2bf(x1[e]);
      b2[e] = f2bf(x2[e]);
    }
  }
  auto pack4 = [](const bf16_t* v) {
    return make_uint2((uint32_t)v[0] | ((uint32_t)v[1] << 16), (uint32_t)v[2] | ((uint32_t)v[3] << 16));
  };
  if (region == 0) {
    bf16_t* qr = q + (int64_t)r * md.nq * md.hd + head * md.hd;
    *reinterpret_cast<uint2*>(qr + j) = pack4(b1);
    *reinterpret_cast<uint2*>(qr + j + half) = pack4(b2);
  } else if (act) {
    bf16_t* base = kv.kv + kv.page_elems(layer, page, head, region - 1);
    if (region == 1) {  // K in fragment order: dims j..j+3 stay within one 32-dim k-step
      *reinterpret_cast<uint2*>(base + key_elem(slot, j, md.hd)) = pack4(b1);
      *reinterpret_cast<uint2*>(base + key_elem(slot, j + half, md.hd)) = pack4(b2);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        base[(j + e) * kv.page_size + slot] = b1[e];
        base[(j + e + half) * kv.page_size + slot] = b2[e];
      }
    }
  }
}

// Per request: greedy token of each active row (best over the LM head's column
// blocks, ties -> lowest id), then the acceptance.  Chain drafts: the longest
// draft prefix that matches.  Tree drafts: a node is accepted when its parent
// is and its token is the parent's greedy token; the deepest accepted node
// (lowest index among equals) ends the accepted path.
__global__ void __launch_bounds__(1024) k_argmax_accept(const int32_t* ntok, int row_stride,
                                                       int n_blocks, const float* amax_v,
                                                       const int32_t* amax_i,
                                                       const int32_t* drafts, const int32_t* parents,
                                                       int k_max, int32_t* accept_lens, int32_t* next_tokens,
                                                       int32_t* accept_path) {
  __shared__ int greedy[64];
  __shared__ int s_par[64], s_dep[64], s_ok[64];
  const int b = blockIdx.x;
  const int n = ntok ? min(ntok[b], 64) : 1;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  // one wave per row (rows w, w + nw, ...): the rows' reductions run side by side
  for (int i = w; i < n; i += nw) {
    const int64_t row = (int64_t)b * row_stride + i;
    float v = -INFINITY;
    int idx = 0x7fffffff;
    // lane-strided blocks in ascending order, 16 loads in flight per batch
    for (int c0 = 0; c0 < n_blocks; c0 += 64 * 16) {
      float bv[16];
      int bi[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int c = c0 + u * 64 + lane;
        bv[u] = c < n_blocks ? amax_v[row * n_blocks + c] : -INFINITY;
        bi[u] = c < n_blocks ? amax_i[row * n_blocks + c] : 0x7fffffff;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (bv[u] > v || (bv[u] == v && bi[u] < idx)) {
          v = bv[u];
          idx = bi[u];
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const float ov = __shfl_xor(v, o, 64);
      const int oi = __shfl_xor(idx, o, 64);
      if (ov > v || (ov == v && oi < idx)) {
        v = ov;
        idx = oi;
      }
    }
    if (lane == 0) greedy[i] = idx;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  int a = 0, last = 0;
  if (parents && n > 0) {
    s_ok[0] = 1;
    s_dep[0] = 0;
    for (int j = 1; j < n; ++j) {
      int pj = parents[(int64_t)b * k_max + j - 1];
      if (pj < 0 || pj >= j) pj = j - 1;  // flagged by the step setup
      s_par[j] = pj;
      s_dep[j] = s_dep[pj] + 1;
      s_ok[j] = s_ok[pj] && drafts[(int64_t)b * k_max + j - 1] == greedy[pj];
      if (s_ok[j] && s_dep[j] > s_dep[last]) last = j;
    }
    a = s_dep[last];
    for (int d = a; d < k_max; ++d) accept_path[(int64_t)b * k_max + d] = -1;
    for (int j = last; j > 0; j = s_par[j]) accept_path[(int64_t)b * k_max + s_dep[j] - 1] = j;
  } else if (n > 0) {
    while (a < n - 1 && drafts && drafts[(int64_t)b * k_max + a] == greedy[a]) ++a;
    last = a;
  } else if (parents) {
    for (int d = 0; d < k_max; ++d) accept_path[(int64_t)b * k_max + d] = -1;
  }
  // no rows: the step's setup failed (war_pool_state reports why); -1 makes the
  // commit a discard
  if (accept_lens) accept_lens[b] = n > 0 ? a : -1;
  next_tokens[b] = n > 0 ? greedy[last] : -1;
}

// Tree drafts: one workgroup per (layer, kv-head, request) gathers the K rows and
// V^T columns of the accepted nodes into LDS, then writes them to slots
// ctx + 1 .. ctx + a (node d of the path has index >= d, so a sequential copy
// in depth order would also be safe; staging makes the order irrelevant).
constexpr int kCompactMaxNodes = 31, kCompactMaxDim = 128;
__global__ void __launch_bounds__(256) k_kv_compact(KvGeom kv, StepMeta meta, const int32_t* table,
                                                    int max_pages, const int32_t* accept_lens,
                                                    const int32_t* accept_path, int k_max) {
  __shared__ bf16_t s_k[kCompactMaxNodes][kCompactMaxDim], s_v[kCompactMaxNodes][kCompactMaxDim];
  __shared__ int s_src[kCompactMaxNodes];
  const int layer = blockIdx.x, kvh = blockIdx.y, b = blockIdx.z;
  const int n = meta.req_ntok[b];
  const int a = min(min(accept_lens[b], n - 1), k_max);
  if (a <= 0) return;
  const int D = kv.head_dim, P = kv.page_size;
  const int ctx = meta.req_pos0[b];
  const int32_t* trow = table + (int64_t)meta.req_seq[b] * max_pages;
  if (threadIdx.x < a) {
    const int src = accept_path[(int64_t)b * k_max + threadIdx.x];
    s_src[threadIdx.x] = (src >= 1 && src < n) ? src : threadIdx.x + 1;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a * D; e += blockDim.x) {
    const int d = e / D, c = e % D;
    const int sp = ctx + s_src[d];
    const int pg = trow[sp / P], sl = sp % P;
    s_k[d][c] = kv.kv[kv.page_elems(layer, pg, kvh, 0) + key_elem(sl, c, D)];
    s_v[d][c] = kv.kv[kv.page_elems(layer, pg, kvh, 1) + (int64_t)c * P + sl];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < a * D; e += blockDim.x) {
    const int d = e / D, c = e % D;
    const int dp = ctx + d + 1;
    const int pg = trow[dp / P], sl = dp % P;
    kv.kv[kv.page_elems(layer, pg, kvh, 0) + key_elem(sl, c, D)] = s_k[d][c];
    kv.kv[kv.page_elems(layer, pg, kvh, 1) + (int64_t)c * P + sl] = s_v[d][c];
  }
}

}  // namespace

void launch_rope_table(int rows, const int32_t* pos, const double* inv_freq, int half, float* cos_t,
                       float* sin_t, hipStream_t st) {
  k_rope_table<<<cdiv_i(rows * half, 256), 256, 0, st>>>(rows, pos, inv_freq, half, cos_t, sin_t);
}
void launch_embed_norm(int rows, const int32_t* tok, const bf16_t* E, const bf16_t* g, int d,
                       float eps, float* h, bf16_t* u, hipStream_t st) {
  k_embed_norm<<<rows, 256, 0, st>>>(tok, E, g, d, eps, h, u);
}
void launch_residual_norm(int rows, int splits, const float* P, int d, const bf16_t* g, float eps,
                          float* h, bf16_t* u, hipStream_t st) {
  if (d <= 4096)
    k_residual_norm<1><<<rows, 1024, 0, st>>>(rows, splits, P, d, g, eps, h, u);
  else if (d <= 8192)
    k_residual_norm<2><<<rows, 1024, 0, st>>>(rows, splits, P, d, g, eps, h, u);
  else
    k_residual_norm<0><<<rows, 1024, 0, st>>>(rows, splits, P, d, g, eps, h, u);
}
void launch_qkv_rope(int rows, int splits, const float* P, const ModelDims& md,
                     const float* cos_t, const float* sin_t, const StepMeta& meta,
                     const int32_t* row_req, const int32_t* table, int max_pages, const KvGeom& kv,
                     int layer, bf16_t* q, hipStream_t st) {
  dim3 grid(rows, cdiv_i(md.qkv / 8, 64));  // four pairs per thread, one wave per workgroup
  k_qkv_rope<<<grid, 64, 0, st>>>(rows, splits, P, md, cos_t, sin_t, meta, row_req, table,
                                   max_pages, kv, layer, q);
}
void launch_argmax_accept(int n_req, const int32_t* ntok, int row_stride, int n_blocks,
                          const float* amax_v, const int32_t* amax_i, const int32_t* draft_tokens,
                          const int32_t* parents, int k_max, int32_t* accept_lens, int32_t* next_tokens,
                          int32_t* accept_path, hipStream_t st) {
  k_argmax_accept<<<n_req, 1024, 0, st>>>(ntok, row_stride, n_blocks, amax_v, amax_i, draft_tokens,
                                         parents, k_max, accept_lens, next_tokens, accept_path);
}
void launch_kv_compact(const KvGeom& kv, int n_layers, int B, const StepMeta& meta, const int32_t* table,
                       int max_pages, const int32_t* accept_lens, const int32_t* accept_path, int k_max,
                       hipStream_t st) {
  dim3 grid(n_layers, kv.n_kv_heads, B);
  k_kv_compact<<<grid, 256, 0, st>>>(kv, meta, table, max_pages, accept_lens, accept_path, k_max);
}
