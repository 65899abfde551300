// Grouped-query verification attention over the paged KV cache (gfx950).
//
// Row r of a (request, kv-head) block is token t0 + r / G of that request for
// query head kvh*G + r % G; it sees keys 0 .. pos(row).  A verify step has
// G*(draft_len+1) such rows per request and kv-head (4..48); the keys number
// tens of thousands, so the kernel is bound by reading K and V from HBM once.
//
// Work item = (request, row block, key chunk) x kv-head, listed on the device
// by the step setup; a persistent grid strides over the items.  Inside an item
// the 4 waves split the chunk's keys; each wave walks 32-key blocks (two pages):
//   S^T = K Q^T  -- v_mfma_f32_16x16x32_bf16 with the keys as the M side: lane
//                   (m, g) loads 64 contiguous bytes of one key row, and key
//                   m of tile t is chosen as (m/4)*8 + 4t + m%4 so that every
//                   lane ends up holding 8 consecutive keys of one query row;
//   online softmax in fp32 (exp2, running max/sum per query row), P rounded
//                   to bf16 for the second product;
//   O^T += V^T P^T -- V is stored transposed inside a page ([dim][slot]), so
//                   each lane reads 16 contiguous bytes (8 keys of one dim).
// The waves' (max, sum, O) are merged through LDS in a fixed order and one
// partial per item goes to global memory; the combine kernel merges a
// request's chunks in item order (deterministic).
#include "kernels.h"

namespace {

// Keep the first n (0..8) bf16 elements of a fragment, zero the rest.  Slots at
// or beyond a sequence's end are never written and may hold any bit pattern;
// their softmax weight is 0, but 0 * NaN would still poison the product.
__device__ __forceinline__ uint4 keep_first(uint4 v, int n) {
  auto m = [n](int i) { return 2 * i + 1 < n ? 0xffffffffu : 2 * i < n ? 0x0000ffffu : 0u; };
  return make_uint4(v.x & m(0), v.y & m(1), v.z & m(2), v.w & m(3));
}

template <int NR, int HD>
__global__ void __launch_bounds__(256) k_attn(AttnArgs a) {
  constexpr int DPL = HD / 4;    // dims per lane group in the S^T operands
  constexpr int KSUB = HD / 32;  // MFMA k-steps over the head dim
  constexpr int NDT = HD / 16;   // 16-dim output tiles
  constexpr int RB = NR * 16;
  constexpr int OST = HD + 1;    // LDS row stride of the merge buffer
  __shared__ float s_m[4][RB], s_l[4][RB];
  __shared__ float s_o[RB * OST];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, ln = lane & 15, lg = lane >> 4;
  const int total = a.meta.n_items[0] * a.n_kv_heads;
  const int P = a.kv.page_size;

  for (int it = blockIdx.x; it < total; it += gridDim.x) {
    const int item = it / a.n_kv_heads, kvh = it % a.n_kv_heads;
    const int4 itm = a.meta.items[item];
    const int b = itm.x, t0 = itm.y * a.TB, chunk = itm.z;
    const int seq = a.meta.req_seq[b], pos0 = a.meta.req_pos0[b];
    const int row0 = a.meta.req_row0[b];
    const int nt = min(a.TB, a.meta.req_ntok[b] - t0);
    const int nrows = nt * a.G;
    const int last_pos = pos0 + t0 + nt - 1;
    const int S = last_pos + 1;
    const int kbeg = chunk * a.chunk, kend = min(S, kbeg + a.chunk);

    // queries (B operand of S^T): lane (n = ln, g = lg) of row tile rt
    int rpos[NR];
    bf16x8 qf[NR][KSUB];
#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      const int r = rt * 16 + ln;
      if (r < nrows) {
        const int ti = t0 + r / a.G, h = kvh * a.G + r % a.G;
        rpos[rt] = pos0 + ti;
        const bf16_t* qp = a.q + (int64_t)(row0 + ti) * a.q_stride + h * HD + lg * DPL;
#pragma unroll
        for (int j = 0; j < KSUB; ++j) qf[rt][j] = as_bf16x8(*reinterpret_cast<const uint4*>(qp + j * 8));
      } else {
        rpos[rt] = last_pos;
#pragma unroll
        for (int j = 0; j < KSUB; ++j) qf[rt][j] = as_bf16x8(make_uint4(0, 0, 0, 0));
      }
    }

    float m_run[NR], l_run[NR];
    f32x4 o_acc[NDT][NR];
#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      m_run[rt] = -INFINITY;
      l_run[rt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) o_acc[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    const int CW = a.chunk / 4;
    const int wk0 = kbeg + w * CW, wk1 = min(kend, wk0 + CW);
    const int32_t* trow = a.table + (int64_t)seq * a.max_pages;
    const bf16_t* kvl = a.kv.kv;
    // key row of this lane in S^T tile t (within a 32-key block)
    const int kk0 = (ln >> 2) * 8 + (ln & 3);  // tile 0; tile 1 adds 4

    for (int kb = wk0; kb < wk1; kb += 32) {
      const int pg0 = trow[kb / P];
      const int pg1 = (kb + 16 < S) ? trow[kb / P + 1] : pg0;
      // K fragments: A operand, lane (m = ln, g = lg)
      bf16x8 kf[2][KSUB];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int kk = kk0 + 4 * t;
        const int pg = kk < 16 ? pg0 : pg1;
        const bf16_t* kp = kvl + a.kv.page_elems(a.layer, pg, kvh, 0) + (kk & 15) * HD + lg * DPL;
#pragma unroll
        for (int j = 0; j < KSUB; ++j) kf[t][j] = as_bf16x8(*reinterpret_cast<const uint4*>(kp + j * 8));
      }
      // V^T fragments: A operand of the second product, lane (m = dim, g = lg) -> keys lg*8..+7
      bf16x8 vf[NDT];
      {
        const int pg = lg < 2 ? pg0 : pg1;
        const bf16_t* vp = kvl + a.kv.page_elems(a.layer, pg, kvh, 1) + (lg & 1) * 8;
        if (kb + 32 <= S) {
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
            vf[dt] = as_bf16x8(*reinterpret_cast<const uint4*>(vp + (dt * 16 + ln) * P));
        } else {  // the sequence ends inside this block
          const int nvalid = min(max(S - (kb + lg * 8), 0), 8);
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
            vf[dt] = as_bf16x8(keep_first(*reinterpret_cast<const uint4*>(vp + (dt * 16 + ln) * P), nvalid));
        }
      }
#pragma unroll
      for (int rt = 0; rt < NR; ++rt) {
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < KSUB; ++j) {
          s0 = mfma16(kf[0][j], qf[rt][j], s0);
          s1 = mfma16(kf[1][j], qf[rt][j], s1);
        }
        // lane holds S^T[key kb + lg*8 + 4t + i][row rt*16 + ln]
        float sv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k0 = kb + lg * 8 + i;
          sv[i] = k0 <= rpos[rt] ? s0[i] * a.scale_log2 : -INFINITY;
          sv[4 + i] = k0 + 4 <= rpos[rt] ? s1[i] * a.scale_log2 : -INFINITY;
        }
        float mx = sv[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float m_new = fmaxf(m_run[rt], mx);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m_run[rt] - m_use);
        float pe[8], sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          pe[e] = round_bf(exp2f(sv[e] - m_use));
          sum += pe[e];
        }
        l_run[rt] = l_run[rt] * alpha + sum;
        m_run[rt] = m_new;
        uint4 pp;
        pp.x = pack2(pe[0], pe[1]);
        pp.y = pack2(pe[2], pe[3]);
        pp.z = pack2(pe[4], pe[5]);
        pp.w = pack2(pe[6], pe[7]);
        const bf16x8 pf = as_bf16x8(pp);
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          o_acc[dt][rt] *= alpha;
          o_acc[dt][rt] = mfma16(vf[dt], pf, o_acc[dt][rt]);
        }
      }
    }

    // ---- merge the 4 waves (fixed order) and write the item's partial
#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      float l = l_run[rt];
      l += __shfl_xor(l, 16, 64);
      l += __shfl_xor(l, 32, 64);
      if (lg == 0) {
        s_m[w][rt * 16 + ln] = m_run[rt];
        s_l[w][rt * 16 + ln] = l;
      }
    }
    __syncthreads();
    float f_own[NR];
#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      const int r = rt * 16 + ln;
      const float mm = fmaxf(fmaxf(s_m[0][r], s_m[1][r]), fmaxf(s_m[2][r], s_m[3][r]));
      const float mu = mm == -INFINITY ? 0.f : mm;
      f_own[rt] = exp2f(m_run[rt] - mu);
    }
    for (int ww = 0; ww < 4; ++ww) {
      if (w == ww) {
#pragma unroll
        for (int rt = 0; rt < NR; ++rt)
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int idx = (rt * 16 + ln) * OST + dt * 16 + lg * 4 + i;
              const float v = o_acc[dt][rt][i] * f_own[rt];
              s_o[idx] = ww == 0 ? v : s_o[idx] + v;
            }
      }
      __syncthreads();
    }
    const int64_t pbase = ((int64_t)item * a.n_kv_heads + kvh) * RB;
    for (int e = tid; e < RB * HD; e += 256) {
      const int r = e / HD, d = e % HD;
      a.po[(pbase + r) * HD + d] = s_o[r * OST + d];
    }
    if (tid < RB) {
      const int r = tid;
      const float mm = fmaxf(fmaxf(s_m[0][r], s_m[1][r]), fmaxf(s_m[2][r], s_m[3][r]));
      const float mu = mm == -INFINITY ? 0.f : mm;
      float l = 0.f;
      for (int ww = 0; ww < 4; ++ww) l += s_l[ww][r] * exp2f(s_m[ww][r] - mu);
      a.pm[pbase + r] = mm;
      a.pl[pbase + r] = l;
    }
    __syncthreads();
  }
}

// Merge a (request, row block)'s chunk partials in item order; o = sum / l -> bf16.
template <int RB, int HD>
__global__ void __launch_bounds__(256) k_attn_combine(AttnArgs a) {
  const int seg = blockIdx.x, kvh = blockIdx.y;
  const int b = a.meta.seg_req[seg];
  const int t0 = a.meta.seg_rb[seg] * a.TB;
  const int nt = min(a.TB, a.meta.req_ntok[b] - t0);
  if (nt <= 0) return;
  const int nrows = nt * a.G;
  const int ib = a.meta.seg_begin[seg], ni = a.meta.seg_count[seg];
  const int row0 = a.meta.req_row0[b];
  for (int e = threadIdx.x; e < nrows * HD; e += blockDim.x) {
    const int r = e / HD, d = e % HD;
    float mm = -INFINITY;
    for (int i = 0; i < ni; ++i)
      mm = fmaxf(mm, a.pm[((int64_t)(ib + i) * a.n_kv_heads + kvh) * RB + r]);
    float l = 0.f, o = 0.f;
    for (int i = 0; i < ni; ++i) {
      const int64_t pb = ((int64_t)(ib + i) * a.n_kv_heads + kvh) * RB + r;
      const float f = exp2f(a.pm[pb] - mm);
      l += a.pl[pb] * f;
      o += a.po[pb * HD + d] * f;
    }
    const int ti = t0 + r / a.G, h = kvh * a.G + r % a.G;
    a.o[(int64_t)(row0 + ti) * a.q_stride + h * HD + d] = f2bf(o / l);
  }
}

template <int NR>
void launch_attn_nr(const AttnArgs& a, int head_dim, int grid, hipStream_t st) {
  if (head_dim == 128)
    k_attn<NR, 128><<<grid, 256, 0, st>>>(a);
  else
    k_attn<NR, 64><<<grid, 256, 0, st>>>(a);
}

template <int RB>
void launch_comb(const AttnArgs& a, int head_dim, int n_segs, hipStream_t st) {
  dim3 grid(n_segs, a.n_kv_heads);
  if (head_dim == 128)
    k_attn_combine<RB, 128><<<grid, 256, 0, st>>>(a);
  else
    k_attn_combine<RB, 64><<<grid, 256, 0, st>>>(a);
}

}  // namespace

int attn_rows_per_block(int G, int k_rows) {
  const int rows = G * k_rows;
  return rows <= 16 ? 16 : rows <= 32 ? 32 : 48;
}

void launch_attn(const AttnArgs& a, int RB, int head_dim, int grid, hipStream_t st) {
  if (RB == 16)
    launch_attn_nr<1>(a, head_dim, grid, st);
  else if (RB == 32)
    launch_attn_nr<2>(a, head_dim, grid, st);
  else
    launch_attn_nr<3>(a, head_dim, grid, st);
}

void launch_attn_combine(const AttnArgs& a, int RB, int head_dim, int n_segs, hipStream_t st) {
  if (RB == 16)
    launch_comb<16>(a, head_dim, n_segs, st);
  else if (RB == 32)
    launch_comb<32>(a, head_dim, n_segs, st);
  else
    launch_comb<48>(a, head_dim, n_segs, st);
}
