// Grouped-query verification attention over the paged KV cache (gfx950).
//
// Row r of a (request, kv-head) block is token t0 + r / G of that request for
// query head kvh*G + r % G; it sees keys 0 .. pos(row) (tree drafts: the context
// and the step slots of its node's root path).  A verify step has
// G*(draft_len+1) such rows per request and kv-head (4..48); the keys number
// tens of thousands, so the kernel is bound by reading K and V from HBM once.
//
// Work item = (request, row block, key chunk) x kv-head, listed on the device
// by the step setup; a persistent grid strides over the items.  Inside an item
// the 4 waves split the chunk's keys; each wave walks 32-key blocks (two pages):
//   S^T = K Q^T  -- v_mfma_f32_16x16x32_bf16 with the keys as the M side:
//                   k-step j covers dims 32j..32j+31, and the keys are
//                   stored in fragment order (key_elem), so one load of a
//                   wave reads 512 contiguous bytes from each of two pages;
//                   key m of tile t is chosen as (m/4)*8 + 4t + m%4 so that
//                   every lane ends up holding 8 consecutive keys of one row;
//   online softmax in fp32 (exp2, running max/sum per query row), P split
//                   into bf16 hi + lo for the second product;
//   O^T += V^T P^T -- V is stored transposed inside a page ([dim][slot]), so
//                   each lane reads 16 contiguous bytes (8 keys of one dim).
// Block bookkeeping (positions, page ids, page bases) is wave-uniform and kept
// in scalar registers; only the last blocks of a request take the causal /
// tree / end-of-sequence masks, in a loop of their own.
// The waves' (max, sum, O) are merged through LDS in a fixed order and one
// partial per item goes to global memory; the combine kernel merges a
// request's chunks in item order (deterministic).
#include <type_traits>

#include "kernels.h"

namespace {

// Keep the first n (0..8) bf16 elements of a fragment, zero the rest.  Slots at
// or beyond a sequence's end are never written and may hold any bit pattern;
// their softmax weight is 0, but 0 * NaN would still poison the product.
__device__ __forceinline__ uint4 keep_first(uint4 v, int n) {
  auto m = [n](int i) { return 2 * i + 1 < n ? 0xffffffffu : 2 * i < n ? 0x0000ffffu : 0u; };
  return make_uint4(v.x & m(0), v.y & m(1), v.z & m(2), v.w & m(3));
}

// K and V^T fragments of one 32-key block (see the file comment for the layout).
template <int HD>
struct KVFrag {
  uint4 k[2][HD / 32];
  uint4 v[HD / 16];
};

// DEPTH = blocks in flight per wave beyond the one being computed (0 or 1);
// QLDS = queries read from LDS instead of registers; WPE = waves per SIMD the
// register budget allows.  Two waves per SIMD let one wave's MFMA/softmax work
// overlap the other's memory waits.
// TREE = the step has tree drafts (rows carry node masks).
template <int NR, int HD, int DEPTH, bool QLDS, int WPE, bool TREE>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPE, WPE)))
k_attn(AttnArgs a) {
  constexpr int KSUB = HD / 32;  // MFMA k-steps over the head dim
  constexpr int NDT = HD / 16;   // 16-dim output tiles
  constexpr int RB = NR * 16;
  constexpr int OST = HD + 1;    // LDS row stride of the merge buffer
  constexpr int QST = HD + 8;    // LDS row stride (bf16) of the staged queries
  __shared__ float s_m[4][RB], s_l[4][RB];
  __shared__ float s_o[RB * OST];
  __shared__ __attribute__((aligned(16))) bf16_t s_q[QLDS ? RB * QST : 8];
  __shared__ uint32_t s_tm[TREE ? RB : 1];  // tree drafts: step slots each row sees
  const int tid = threadIdx.x, lane = tid & 63, ln = lane & 15, lg = lane >> 4;
  // the wave index is wave-uniform: block positions, page ids and page bases
  // derived from it live in scalar registers
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int total = a.meta.n_items[1] * a.n_kv_heads;  // units: work-order slots x kv-heads
  const int CH = a.meta.n_items[3];                     // keys per item (a multiple of 128)
  const int P = a.kv.page_size;
  // key row of this lane in S^T tile t (within a 32-key block); tile 1 adds 4
  const int kk0 = (ln >> 2) * 8 + (ln & 3);
  // Per-lane element offsets inside a page (kind 0 = K in fragment order, see
  // key_elem; kind 1 = V^T [dim][slot]): lanes ln < 8 read K rows of the
  // block's first page, the others its second; lane groups lg < 2 read V^T of
  // the first page.  K of tile t, k-step j is one 512-byte run per page.
  const int koff0 = key_elem(kk0 & 15, lg * 8, HD), koff1 = key_elem((kk0 + 4) & 15, lg * 8, HD);
  const int voff = P * HD + (lg & 1) * 8 + ln * P;
  const bool k_second = ln >= 8, v_second = lg >= 2;

  // Units are handed out by per-class counters (class = workgroup id mod NC):
  // a workgroup takes the next unit of its class when it finishes one, so
  // units of unequal length balance over the workgroups.  Workgroups are dealt
  // to the 8 XCDs round-robin, so with 8 kv-heads every unit of one kv-head
  // runs on the same XCD, and items that are neighbours in the work order (the
  // same prefix chunk of sibling requests) share its L2.  The combine kernel
  // that follows every launch resets the counters.
  //
  // The next unit is taken from the counter when the key loop of the current
  // one ends, so the counter's latency overlaps the merge; a unit starts with
  // one (scalar) load of its work-order slot's descriptor instead of a chain
  // of dependent loads (order, item, request fields).
  const int NC = min(8, (int)gridDim.x);
  const int cls = blockIdx.x % NC;
  __shared__ int s_it;
  if (tid == 0) s_it = atomicAdd(&a.unit_ctr[cls], 1) * NC + cls;
  __syncthreads();
  for (;;) {
    const int it = s_it;
    if (it >= total) break;
    const int kvh = it % a.n_kv_heads;
    const int4 u0 = a.meta.udesc[2 * (it / a.n_kv_heads)], u1 = a.meta.udesc[2 * (it / a.n_kv_heads) + 1];
    const int item = u0.x, b = u0.y, chunk = u0.z;
    const int t0 = u0.w & 0xffff, nt = u0.w >> 16;
    // a shared-prefix unit (.w = n > 0) covers the live rows of requests
    // b .. b+n-1, one after the other, and sees every key of its chunk (the
    // shared keys precede every member's rows): no causal mask
    const bool shared = u1.x > 0;
    const int nmem = shared ? u1.x : 1;
    const int seq = u1.y, pos0 = u1.z, row0 = u1.w;
    int nrows = nt * a.G;
    if (shared)
      for (int jm = 1; jm < nmem; ++jm) nrows += min(a.TB, a.meta.req_ntok[b + jm]) * a.G;
    const int last_pos = shared ? (chunk + 1) * CH - 1 : pos0 + t0 + nt - 1;
    const int qpos0 = shared ? last_pos + 1 : pos0 + t0;  // smallest row position
    // tree drafts: every key at or past the context needs its row's node mask
    // (a shared-prefix unit's keys all precede the context)
    const int mask_from = TREE ? pos0 - 1 : qpos0;
    if constexpr (TREE) {
      // the node mask relative to the row's own slot: bit d = slot rpos - d is
      // visible (bits past the node index: context keys, always visible)
      if (tid < RB) {
        uint32_t rm = 0xffffffffu;
        if (!shared && tid < nrows) {
          const int i = t0 + tid / a.G;
          rm = __brev(a.meta.tmask[row0 + i]) >> (31 - i);
          if (i < 31) rm |= 0xffffffffu << (i + 1);
        }
        s_tm[tid] = rm;
      }
      __syncthreads();
    }
    const int S = last_pos + 1;
    const int kbeg = chunk * CH, kend = min(S, kbeg + CH);
    const int CW = CH / 4;
    const int wk0 = kbeg + w * CW, wk1 = min(kend, wk0 + CW);
    const int nb = wk1 > wk0 ? (wk1 - wk0 + 31) / 32 : 0;
    // blocks before nfull lie at or below every row's position (and inside the
    // sequence): no causal, tree or end-of-sequence mask
    const int nfull = mask_from - 31 - wk0 < 0 ? 0 : min(nb, (mask_from - 31 - wk0) / 32 + 1);
    const int32_t* trow = a.table + (int64_t)seq * a.max_pages;
    // elements per page across kv-heads and kinds; this kv-head's part of page 0
    const int64_t pstride = (int64_t)a.kv.n_kv_heads * 2 * P * HD;
    const bf16_t* kvb = a.kv.kv + a.kv.page_elems(a.layer, 0, kvh, 0);

    // Keys and values are read once per step (a unit's 4 waves take disjoint
    // blocks, the 8 kv-head units of a chunk disjoint pieces of each page), so
    // they are loaded as non-temporal: they do not displace the lines that are
    // reused (queries, partials, block tables).  High load: attention 17.5 ->
    // 16.5 ms per step (6.0 -> 6.4 TB/s); low load and forked siblings
    // unchanged.
    typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
    auto ntload = [](const bf16_t* p) {
      return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p)));
    };
    auto load_block = [&](KVFrag<HD>& f, int kb) {
      const int pg0 = trow[kb / P];
      const int pg1 = (kb + 16 < S) ? trow[kb / P + 1] : pg0;
      const bf16_t* kp = kvb + (int64_t)(k_second ? pg1 : pg0) * pstride;
#pragma unroll
      for (int j = 0; j < KSUB; ++j) {
        f.k[0][j] = ntload(kp + koff0 + j * 256);
        f.k[1][j] = ntload(kp + koff1 + j * 256);
      }
      const bf16_t* vp = kvb + (int64_t)(v_second ? pg1 : pg0) * pstride + voff;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) f.v[dt] = ntload(vp + dt * 16 * P);
    };

    // The first block is requested before the queries are staged, and each
    // next block as soon as the current one is computed -- except with three
    // row tiles, which lack the registers for a block held across those points
    // and load each block right before computing it.
    constexpr bool kEarlyLoad = NR < 3;
    KVFrag<HD> f0;
    if (kEarlyLoad && nb > 0) load_block(f0, wk0);

    // row r -> (query row, query head) and its partial row; false if r is not live
    auto row_src = [&](int r, int& qrow, int& h, int64_t& prow) -> bool {
      if (r >= nrows) return false;
      int jm = 0, lr = r;
      if (shared) {
        int nr = min(a.TB, a.meta.req_ntok[b]) * a.G;
        while (lr >= nr) {
          lr -= nr;
          ++jm;
          nr = min(a.TB, a.meta.req_ntok[b + jm]) * a.G;
        }
      }
      qrow = a.meta.req_row0[b + jm] + t0 + lr / a.G;
      h = kvh * a.G + lr % a.G;
      const int pitem = shared ? a.meta.seg_begin[b + jm] + chunk : item;
      prow = ((int64_t)pitem * a.n_kv_heads + kvh) * a.prb + lr;
      return true;
    };

    // queries (B operand of S^T): lane (n = ln, g = lg) of row tile rt
    int rpos[NR];
    bf16x8 qf[QLDS ? 1 : NR][KSUB];
#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      const int r = rt * 16 + ln;
      rpos[rt] = (!shared && r < nrows) ? pos0 + t0 + r / a.G : last_pos;
    }
    if constexpr (QLDS) {
      for (int e = tid; e < RB * (HD / 8); e += 256) {
        const int r = e / (HD / 8), c = (e % (HD / 8)) * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        int qrow, h;
        int64_t prow;
        if (row_src(r, qrow, h, prow))
          v = *reinterpret_cast<const uint4*>(a.q + (int64_t)qrow * a.q_stride + h * HD + c);
        *reinterpret_cast<uint4*>(&s_q[r * QST + c]) = v;
      }
      __syncthreads();
    } else {
#pragma unroll
      for (int rt = 0; rt < (QLDS ? 1 : NR); ++rt) {
        const int r = rt * 16 + ln;
        int qrow, h;
        int64_t prow;
        if (row_src(r, qrow, h, prow)) {
          const bf16_t* qp = a.q + (int64_t)qrow * a.q_stride + h * HD + lg * 8;
#pragma unroll
          for (int j = 0; j < KSUB; ++j) qf[rt][j] = as_bf16x8(*reinterpret_cast<const uint4*>(qp + j * 32));
        } else {
#pragma unroll
          for (int j = 0; j < KSUB; ++j) qf[rt][j] = as_bf16x8(make_uint4(0, 0, 0, 0));
        }
      }
    }
    auto qfrag = [&](int rt, int j) -> bf16x8 {
      if constexpr (QLDS)
        return as_bf16x8(*reinterpret_cast<const uint4*>(&s_q[(rt * 16 + ln) * QST + j * 32 + lg * 8]));
      else
        return qf[rt][j];
    };

    float m_run[NR], l_run[NR];
    f32x4 o_acc[NDT][NR];
#pragma unroll
    for (int rt = 0; rt < NR; ++rt) {
      m_run[rt] = -INFINITY;
      l_run[rt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) o_acc[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // MASK: the block holds keys above some row's position or past the
    // sequence end (only the last blocks of a request)
    auto compute_block = [&](const KVFrag<HD>& fin, int kb, auto mask_tag) {
      constexpr bool MASK = decltype(mask_tag)::value;
      if constexpr (QLDS) asm volatile("" ::: "memory");  // re-read Q from LDS each block
      // phase 1: scores of every row tile (the K fragments die after this)
      float sc[NR][8];
#pragma unroll
      for (int rt = 0; rt < NR; ++rt) {
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < KSUB; ++j) {
          const bf16x8 q = qfrag(rt, j);
          s0 = mfma16(as_bf16x8(fin.k[0][j]), q, s0);
          s1 = mfma16(as_bf16x8(fin.k[1][j]), q, s1);
        }
        // lane holds S^T[key kb + lg*8 + 4t + i][row rt*16 + ln]
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sc[rt][i] = s0[i];
          sc[rt][4 + i] = s1[i];
        }
      }
      uint4 vf[NDT];
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) vf[dt] = fin.v[dt];
      if constexpr (MASK) {
        if (kb + 32 > S) {  // the sequence ends inside this block
          const int nvalid = min(max(S - (kb + lg * 8), 0), 8);
#pragma unroll
          for (int dt = 0; dt < NDT; ++dt) vf[dt] = keep_first(vf[dt], nvalid);
        }
      }
      // phase 2: online softmax and O^T += V^T P^T per row tile
#pragma unroll
      for (int rt = 0; rt < NR; ++rt) {
        float* sv = sc[rt];
        if constexpr (MASK) {
          if constexpr (TREE) {
            // a tree row sees the step slot pos0 + i only when node i is on its path
            const uint32_t tm = s_tm[rt * 16 + ln];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const int dd = rpos[rt] - (kb + lg * 8 + e);
              if (dd < 0 || !((tm >> min(dd, 31)) & 1u)) sv[e] = -INFINITY;
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (kb + lg * 8 + e > rpos[rt]) sv[e] = -INFINITY;
          }
        }
        float lm = sv[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) lm = fmaxf(lm, sv[e]);
        lm *= a.scale_log2;
        // Lazy rescaling: a row's running max only moves when one of its scores
        // exceeds it by more than 2^8 (weights stay below 256, exact in fp32).
        // Each row decides from its own maximum (the 4 lanes of a row agree), so
        // a row's result never depends on the other rows of its tile; the wave
        // skips the row maxima when no lane needs them.
        if (__any(lm > m_run[rt] + 8.f)) {
          float mx = fmaxf(lm, __shfl_xor(lm, 16, 64));
          mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
          if (mx > m_run[rt] + 8.f) {
            const float alpha = exp2f(m_run[rt] - mx);
            l_run[rt] *= alpha;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) o_acc[dt][rt] *= alpha;
            m_run[rt] = mx;
          }
        }
        const float m_use = m_run[rt] == -INFINITY ? 0.f : m_run[rt];
        // P = hi + lo, both bf16: the product keeps ~16 bits of each weight.
        // v_exp_f32 directly: weights below 2^-126 of the running max flush to 0.
        float sum = 0.f;
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[e], a.scale_log2, -m_use));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[e + 1], a.scale_log2, -m_use));
          sum += p0 + p1;
          hi[e / 2] = pack2(p0, p1);
          lo[e / 2] = pack2(p0 - lo_f(hi[e / 2]), p1 - hi_f(hi[e / 2]));
        }
        l_run[rt] += sum;
        const bf16x8 ph = as_bf16x8(make_uint4(hi[0], hi[1], hi[2], hi[3]));
        const bf16x8 pl = as_bf16x8(make_uint4(lo[0], lo[1], lo[2], lo[3]));
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          o_acc[dt][rt] = mfma16(as_bf16x8(vf[dt]), ph, o_acc[dt][rt]);
          o_acc[dt][rt] = mfma16(as_bf16x8(vf[dt]), pl, o_acc[dt][rt]);
        }
      }
    };
    using NoMask = std::integral_constant<bool, false>;
    using Mask = std::integral_constant<bool, true>;

    // Block i of this wave is at key wk0 + 32 i.  The unmasked blocks and the
    // masked tail (at most the last two blocks of a request) run in separate
    // loops, so that each loop body holds one instantiation of the block code.
    int i = 0;
    if constexpr (kEarlyLoad) {
      // at the top of every iteration f0 holds block i
      if constexpr (DEPTH == 1) {
        // one more block in flight while a block is computed
        KVFrag<HD> f1;
        for (; i + 1 < nfull; i += 2) {
          load_block(f1, wk0 + 32 * (i + 1));
          compute_block(f0, wk0 + 32 * i, NoMask{});
          if (i + 2 < nb) load_block(f0, wk0 + 32 * (i + 2));
          compute_block(f1, wk0 + 32 * (i + 1), NoMask{});
        }
      }
      for (; i < nfull; ++i) {
        compute_block(f0, wk0 + 32 * i, NoMask{});
        if (i + 1 < nb) load_block(f0, wk0 + 32 * (i + 1));
      }
      for (; i < nb; ++i) {
        compute_block(f0, wk0 + 32 * i, Mask{});
        if (i + 1 < nb) load_block(f0, wk0 + 32 * (i + 1));
      }
    } else {
      static_assert(DEPTH == 0, "a block in flight needs the early first load");
      for (; i < nfull; ++i) {
        load_block(f0, wk0 + 32 * i);
        compute_block(f0, wk0 + 32 * i, NoMask{});
      }
      for (; i < nb; ++i) {
        load_block(f0, wk0 + 32 * i);
        compute_block(f0, wk0 + 32 * i, Mask{});
      }
    }

    // the next unit: the counter's reply arrives during the merge
    int next_it = 0;
    if (tid == 0) next_it = atomicAdd(&a.unit_ctr[cls], 1) * NC + cls;

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
    // partial of the live rows only: [item][kvh][row][dim] with row stride HD
    // (a shared-prefix unit writes each member's rows into that member's item)
    for (int e = tid; e < nrows * (HD / 4); e += 256) {
      const int r = e / (HD / 4), d4 = (e % (HD / 4)) * 4;
      int qrow, h;
      int64_t prow;
      if (!row_src(r, qrow, h, prow)) continue;
      const float* src = &s_o[r * OST + d4];
      *reinterpret_cast<float4*>(&a.po[prow * HD + d4]) = make_float4(src[0], src[1], src[2], src[3]);
    }
    if (tid < nrows) {
      const int r = tid;
      int qrow, h;
      int64_t prow;
      if (row_src(r, qrow, h, prow)) {
        const float mm = fmaxf(fmaxf(s_m[0][r], s_m[1][r]), fmaxf(s_m[2][r], s_m[3][r]));
        const float mu = mm == -INFINITY ? 0.f : mm;
        float l = 0.f;
        for (int ww = 0; ww < 4; ++ww) l += s_l[ww][r] * exp2f(s_m[ww][r] - mu);
        a.pm[prow] = mm;
        a.pl[prow] = l;
      }
    }
    // every thread has read s_it at the top of this unit (the merge passed barriers)
    if (tid == 0) s_it = next_it;
    __syncthreads();
  }
}

// One unit's rows and keys, decoded from its work-order descriptor (the fields
// k_attn reads inline; prefill units are never shared-prefix units).
struct UnitRows {
  int item, b, chunk, t0, nt, seq, pos0, row0, nrows, last_pos;
  __device__ void decode(const AttnArgs& a, int it) {
    const int4 u0 = a.meta.udesc[2 * (it / a.n_kv_heads)], u1 = a.meta.udesc[2 * (it / a.n_kv_heads) + 1];
    item = u0.x;
    b = u0.y;
    chunk = u0.z;
    t0 = u0.w & 0xffff;
    nt = u0.w >> 16;
    seq = u1.y;
    pos0 = u1.z;
    row0 = u1.w;
    nrows = nt * a.G;
    last_pos = pos0 + t0 + nt - 1;
  }
  // row r -> (query row, query head) and its partial row; false if r is not live
  __device__ bool src(const AttnArgs& a, int kvh, int r, int& qrow, int& h, int64_t& prow) const {
    if (r >= nrows) return false;
    qrow = a.meta.req_row0[b] + t0 + r / a.G;
    h = kvh * a.G + r % a.G;
    prow = ((int64_t)item * a.n_kv_heads + kvh) * a.prb + r;
    return true;
  }
};

// Prefill attention over row blocks of NW * 32 rows (a causal run of a
// sequence's new tokens; G query heads per token).  Wave w owns rows
// [32w, 32w + 32): two 16-row tiles, queries in registers.  The NW waves share
// every 32-key block, which all threads stage through LDS (two buffers; the
// next three blocks in flight in three register sets, each block requested
// three blocks before it is computed; K rows and V^T rows padded against bank
// conflicts; V^T columns past the sequence end zeroed), so a key
// block is read from memory once per NW * 32 rows instead of once per 48 rows
// as in k_attn.  Per block and wave: S^T = K Q^T
// for both row tiles (each K fragment read once from LDS), the online softmax
// of k_attn, and O^T += V^T P^T with P as bf16 hi + lo (each V^T fragment read
// once for both tiles).  Work units, partials and the merge are k_attn's.
template <int NW, int HD>
__global__ void __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2)))
k_attn_rows(AttnArgs a) {
  constexpr int KSUB = HD / 32;  // MFMA k-steps over the head dim
  constexpr int NDT = HD / 16;   // 16-dim output tiles
  constexpr int NRW = 2;         // 16-row tiles per wave
  constexpr int NT = NW * 64;    // threads
  constexpr int KST = HD + 8;    // LDS row stride (bf16) of K [32 keys][HD]
  constexpr int VST = 32 + 8;    // LDS row stride (bf16) of V^T [HD][32 keys]
  __shared__ __attribute__((aligned(16))) bf16_t s_k[2][32 * KST];
  __shared__ __attribute__((aligned(16))) bf16_t s_v[2][HD * VST];
  const int tid = threadIdx.x, lane = tid & 63, ln = lane & 15, lg = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int total = a.meta.n_items[1] * a.n_kv_heads;
  const int CH = a.meta.n_items[3];
  const int P = a.kv.page_size;
  // key row of this lane in S^T tile t of a block: (ln/4)*8 + ln%4 + 4t
  const int kk0 = (ln >> 2) * 8 + (ln & 3);

  const int NC = min(8, (int)gridDim.x);
  const int cls = blockIdx.x % NC;
  __shared__ int s_it;
  if (tid == 0) s_it = atomicAdd(&a.unit_ctr[cls], 1) * NC + cls;
  __syncthreads();
  for (;;) {
    const int it = s_it;
    if (it >= total) break;
    const int kvh = it % a.n_kv_heads;
    UnitRows u;
    u.decode(a, it);
    const int S = u.last_pos + 1;
    const int qpos0 = u.pos0 + u.t0;  // the first row's position
    const int kbeg = u.chunk * CH, kend = min(S, kbeg + CH);
    const int nb = kend > kbeg ? (kend - kbeg + 31) / 32 : 0;
    // blocks before nfull lie at or below every row's position
    const int nfull = qpos0 - 31 - kbeg < 0 ? 0 : min(nb, (qpos0 - 31 - kbeg) / 32 + 1);
    const int32_t* trow = a.table + (int64_t)u.seq * a.max_pages;
    const int64_t pstride = (int64_t)a.kv.n_kv_heads * 2 * P * HD;
    const bf16_t* kvb = a.kv.kv + a.kv.page_elems(a.layer, 0, kvh, 0);

    // A 32-key block is four regions of 2 HD 16-byte pieces in memory: K and
    // V^T of its two pages.  Piece q of a region sits at q * 8 elements from
    // the region's start; in LDS, piece q of K page g goes to the key and dims
    // that key_elem places there (rows g*16 + slot), and piece q of V^T page g
    // is dim q/2, keys g*16 + (q%2)*8.  Thread t moves pieces t, t + NT, ... of
    // the 8 HD.
    constexpr int NPC = 8 * HD / NT;  // pieces per thread
    static_assert(8 * HD % NT == 0 && NT % (2 * HD) == 0 || (2 * HD) % NT == 0, "piece mapping");
    auto gload = [&](uint4 (&stg)[NPC], int kb) __attribute__((always_inline)) {
      const int pg0 = trow[kb / P];
      const int pg1 = (kb + 16 < S) ? trow[kb / P + 1] : pg0;
#pragma unroll
      for (int i = 0; i < NPC; ++i) {
        const int pc = tid + i * NT, reg = pc / (2 * HD), q = pc % (2 * HD);
        const bf16_t* base = kvb + (int64_t)((reg & 1) ? pg1 : pg0) * pstride + (reg >= 2 ? P * HD : 0);
        stg[i] = *reinterpret_cast<const uint4*>(base + q * 8);
      }
    };
    // V^T slots past the sequence end are zeroed on the way into LDS
    auto lstore = [&](int buf, uint4 (&stg)[NPC], int kb) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < NPC; ++i) {
        const int pc = tid + i * NT, reg = pc / (2 * HD), q = pc % (2 * HD);
        if (reg < 2) {
          // piece q of the page's K in fragment order (key_elem): dims j*32 +
          // (q%4)*8, slot (s8/4)*8 + t*4 + s8%4 with s8 = (q/4)%8, t*KSUB + j = q/32
          const int s8 = (q >> 2) & 7, tj = q >> 5, t = tj / KSUB, j = tj % KSUB;
          const int slot = ((s8 >> 2) << 3) | (t << 2) | (s8 & 3);
          *reinterpret_cast<uint4*>(&s_k[buf][((reg & 1) * 16 + slot) * KST + j * 32 + (q & 3) * 8]) = stg[i];
        } else {
          uint4 v = stg[i];
          if (kb + 32 > S) v = keep_first(v, min(max(S - (kb + (reg & 1) * 16 + (q & 1) * 8), 0), 8));
          *reinterpret_cast<uint4*>(&s_v[buf][(q >> 1) * VST + (reg & 1) * 16 + (q & 1) * 8]) = v;
        }
      }
    };
    // three register sets: while block i is computed from LDS, blocks i + 1 to
    // i + 3 are in flight, so a block's loads have two block computations to
    // arrive before it is stored to LDS
    uint4 stA[NPC], stB[NPC], stC[NPC];
    if (nb > 0) gload(stA, kbeg);
    if (nb > 1) gload(stB, kbeg + 32);
    if (nb > 2) gload(stC, kbeg + 64);

    // queries (B operand of S^T) and row positions of this wave's two tiles
    bf16x8 qf[NRW][KSUB];
    int rpos[NRW];
#pragma unroll
    for (int rt = 0; rt < NRW; ++rt) {
      const int r = (NRW * w + rt) * 16 + ln;
      int qrow, h;
      int64_t prow;
      rpos[rt] = r < u.nrows ? qpos0 + r / a.G : u.last_pos;
      if (u.src(a, kvh, r, qrow, h, prow)) {
        const bf16_t* qp = a.q + (int64_t)qrow * a.q_stride + h * HD + lg * 8;
#pragma unroll
        for (int j = 0; j < KSUB; ++j) qf[rt][j] = as_bf16x8(*reinterpret_cast<const uint4*>(qp + j * 32));
      } else {
#pragma unroll
        for (int j = 0; j < KSUB; ++j) qf[rt][j] = as_bf16x8(make_uint4(0, 0, 0, 0));
      }
    }
    if (nb > 0) lstore(0, stA, kbeg);
    __syncthreads();

    float m_run[NRW], l_run[NRW];
    f32x4 o_acc[NDT][NRW];
#pragma unroll
    for (int rt = 0; rt < NRW; ++rt) {
      m_run[rt] = -INFINITY;
      l_run[rt] = 0.f;
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) o_acc[dt][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // masked: the block holds keys above some row's position (wave-uniform)
    auto compute_block = [&](int buf, int kb, bool masked) __attribute__((always_inline)) {
      f32x4 sacc[NRW][2];
#pragma unroll
      for (int rt = 0; rt < NRW; ++rt) sacc[rt][0] = sacc[rt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < KSUB; ++j) {
        const bf16x8 k0 = as_bf16x8(*reinterpret_cast<const uint4*>(&s_k[buf][kk0 * KST + j * 32 + lg * 8]));
        const bf16x8 k1 = as_bf16x8(*reinterpret_cast<const uint4*>(&s_k[buf][(kk0 + 4) * KST + j * 32 + lg * 8]));
#pragma unroll
        for (int rt = 0; rt < NRW; ++rt) {
          sacc[rt][0] = mfma16(k0, qf[rt][j], sacc[rt][0]);
          sacc[rt][1] = mfma16(k1, qf[rt][j], sacc[rt][1]);
        }
      }
      // keep the V^T fragment reads below the softmax (registers)
      asm volatile("" ::: "memory");
      bf16x8 ph[NRW], pl[NRW];
#pragma unroll
      for (int rt = 0; rt < NRW; ++rt) {
        // lane holds S^T[key kb + lg*8 + e][row]
        float sv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sv[i] = sacc[rt][0][i];
          sv[4 + i] = sacc[rt][1][i];
        }
        if (masked) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (kb + lg * 8 + e > rpos[rt]) sv[e] = -INFINITY;
        }
        float lm = sv[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) lm = fmaxf(lm, sv[e]);
        lm *= a.scale_log2;
        // lazy rescaling, decided per row as in k_attn
        if (__any(lm > m_run[rt] + 8.f)) {
          float mx = fmaxf(lm, __shfl_xor(lm, 16, 64));
          mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
          if (mx > m_run[rt] + 8.f) {
            const float alpha = exp2f(m_run[rt] - mx);
            l_run[rt] *= alpha;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) o_acc[dt][rt] *= alpha;
            m_run[rt] = mx;
          }
        }
        const float m_use = m_run[rt] == -INFINITY ? 0.f : m_run[rt];
        float sum = 0.f;
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(sv[e], a.scale_log2, -m_use));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(sv[e + 1], a.scale_log2, -m_use));
          sum += p0 + p1;
          hi[e / 2] = pack2(p0, p1);
          lo[e / 2] = pack2(p0 - lo_f(hi[e / 2]), p1 - hi_f(hi[e / 2]));
        }
        l_run[rt] += sum;
        ph[rt] = as_bf16x8(make_uint4(hi[0], hi[1], hi[2], hi[3]));
        pl[rt] = as_bf16x8(make_uint4(lo[0], lo[1], lo[2], lo[3]));
      }
#pragma unroll
      for (int dt = 0; dt < NDT; ++dt) {
        const bf16x8 v = as_bf16x8(*reinterpret_cast<const uint4*>(&s_v[buf][(dt * 16 + ln) * VST + lg * 8]));
#pragma unroll
        for (int rt = 0; rt < NRW; ++rt) {
          o_acc[dt][rt] = mfma16(v, ph[rt], o_acc[dt][rt]);
          o_acc[dt][rt] = mfma16(v, pl[rt], o_acc[dt][rt]);
        }
        // at most two V^T fragments in registers at a time
        if (dt % 2 == 1) asm volatile("" ::: "memory");
      }
    };
    // Block i (keys kbeg + 32 i) is in LDS buffer i % 2 when step i starts;
    // blocks i + 1 and i + 2 are in register sets (i + 1) % 3 and (i + 2) % 3.
    // Step i requests block i + 3 into set i % 3 (block i left it for LDS at
    // the end of step i - 1), computes block i, and stores block i + 1 into the
    // other LDS buffer (whose block i - 1 every wave finished before the last
    // barrier).
#define ROWS_STEP(I, LD, ST, BUF)                                   \
    {                                                               \
      const int ii = i + (I);                                       \
      if (ii >= nb) break;                                          \
      const int kb = kbeg + 32 * ii;                                \
      if (ii + 3 < nb) gload(LD, kb + 96);                          \
      compute_block(BUF, kb, ii >= nfull);                          \
      if (ii + 1 < nb) lstore(1 - (BUF), ST, kb + 32);              \
      __syncthreads();                                              \
    }
    for (int i = 0; i < nb; i += 6) {
      ROWS_STEP(0, stA, stB, 0)
      ROWS_STEP(1, stB, stC, 1)
      ROWS_STEP(2, stC, stA, 0)
      ROWS_STEP(3, stA, stB, 1)
      ROWS_STEP(4, stB, stC, 0)
      ROWS_STEP(5, stC, stA, 1)
    }
#undef ROWS_STEP

    int next_it = 0;
    if (tid == 0) next_it = atomicAdd(&a.unit_ctr[cls], 1) * NC + cls;
    // this wave's rows: partial O, running max and sum
#pragma unroll
    for (int rt = 0; rt < NRW; ++rt) {
      const int r = (NRW * w + rt) * 16 + ln;
      float l = l_run[rt];
      l += __shfl_xor(l, 16, 64);
      l += __shfl_xor(l, 32, 64);
      int qrow, h;
      int64_t prow;
      if (u.src(a, kvh, r, qrow, h, prow)) {
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt) {
          const f32x4 v = o_acc[dt][rt];
          *reinterpret_cast<float4*>(&a.po[prow * HD + dt * 16 + lg * 4]) = make_float4(v[0], v[1], v[2], v[3]);
        }
        if (lg == 0) {
          a.pm[prow] = m_run[rt];
          a.pl[prow] = l;
        }
      }
    }
    if (tid == 0) s_it = next_it;
    __syncthreads();
  }
}

// Merge a (request, row block)'s chunk partials in item order; o = sum / l -> bf16.
// Workgroup = (segment, kv-head, slice of 1024/HD rows: 8 at head_dim 128), so
// a step's merge spreads over hundreds of workgroups.  One wave per row puts
// the per-item weights exp2(m_i - m) in LDS (lanes over items), then one thread
// per output float4 accumulates the items in order with independent loads.
constexpr int kCombMaxItems = 512;
template <int RB, int HD>
__global__ void __launch_bounds__(256) k_attn_combine(AttnArgs a) {
  constexpr int TPR = HD / 4;                 // threads per row
  constexpr int RPW = 256 / TPR;              // rows per workgroup
  constexpr int PF = 16;                      // partial-O loads issued before the weights are known
  constexpr int IPL = kCombMaxItems / 64;     // items per lane in the weight pass
  __shared__ float s_w[RPW][kCombMaxItems];
  __shared__ float s_il[RPW];
  const int seg = blockIdx.x, kvh = blockIdx.y, r0 = blockIdx.z * RPW;
  // the attention launch before this one is complete: its work counters restart
  if (seg == 0 && kvh == 0 && blockIdx.z == 0 && threadIdx.x < 8) a.unit_ctr[threadIdx.x] = 0;
  const int b = a.meta.seg_req[seg];
  const int t0 = a.meta.seg_rb[seg] * a.TB;
  const int nrows = min(a.TB, a.meta.req_ntok[b] - t0) * a.G;
  if (r0 >= nrows) return;
  const int rows = min(RPW, nrows - r0);
  const int ib = a.meta.seg_begin[seg], ni = min(a.meta.seg_count[seg], kCombMaxItems);
  const int64_t is = (int64_t)a.n_kv_heads * RB;  // pm / pl elements per item
  const float* pm = a.pm + ((int64_t)ib * a.n_kv_heads + kvh) * RB + r0;
  const float* pl = a.pl + ((int64_t)ib * a.n_kv_heads + kvh) * RB + r0;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  // this thread's output float4: the first PF items' partial O are requested
  // now, so their loads overlap the weight pass
  const int r = threadIdx.x / TPR, d4 = (threadIdx.x % TPR) * 4;
  const bool live = r < rows;
  const float* po = a.po + (((int64_t)ib * a.n_kv_heads + kvh) * RB + r0 + r) * HD + d4;
  float4 pre[PF];
#pragma unroll
  for (int i = 0; i < PF; ++i)
    if (live && i < ni) pre[i] = *reinterpret_cast<const float4*>(po + i * is * HD);
  // weight pass, one wave per row (rows w, w + 4, ...): each lane's items
  // (i = lane + 64 j) of all of the wave's rows are loaded first, once; max and
  // sum in ascending item order per lane
  constexpr int RPV = RPW / 4;                // rows per wave
  float vm[RPV][IPL], vl[RPV][IPL];
#pragma unroll
  for (int q = 0; q < RPV; ++q) {
    const int rr = w + 4 * q;
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const int i = lane + 64 * j;
      const bool ok = rr < rows && i < ni;
      vm[q][j] = ok ? pm[i * is + rr] : -INFINITY;
      vl[q][j] = ok ? pl[i * is + rr] : 0.f;
    }
  }
#pragma unroll
  for (int q = 0; q < RPV; ++q) {
    const int rr = w + 4 * q;
    if (rr >= rows) break;
    float mm = -INFINITY;
#pragma unroll
    for (int j = 0; j < IPL; ++j) mm = fmaxf(mm, vm[q][j]);
    mm = wave_max(mm);
    float l = 0.f;
#pragma unroll
    for (int j = 0; j < IPL; ++j) {
      const int i = lane + 64 * j;
      if (i < ni) {
        const float f = exp2f(vm[q][j] - mm);
        s_w[rr][i] = f;
        l += vl[q][j] * f;
      }
    }
    l = wave_sum(l);
    if (lane == 0) s_il[rr] = 1.f / l;
  }
  __syncthreads();
  if (!live) return;
  float4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < PF; ++i)
    if (i < ni) {
      const float f = s_w[r][i];
      acc.x += pre[i].x * f;
      acc.y += pre[i].y * f;
      acc.z += pre[i].z * f;
      acc.w += pre[i].w * f;
    }
#pragma unroll 8
  for (int i = PF; i < ni; ++i) {
    const float4 v = *reinterpret_cast<const float4*>(po + i * is * HD);
    const float f = s_w[r][i];
    acc.x += v.x * f;
    acc.y += v.y * f;
    acc.z += v.z * f;
    acc.w += v.w * f;
  }
  const float inv = s_il[r];
  const int rr = r0 + r;
  const int ti = t0 + rr / a.G, h = kvh * a.G + rr % a.G;
  bf16_t* dst = a.o + (int64_t)(a.meta.req_row0[b] + ti) * a.q_stride + h * HD + d4;
  uint2 o;
  o.x = pack2(acc.x * inv, acc.y * inv);
  o.y = pack2(acc.z * inv, acc.w * inv);
  *reinterpret_cast<uint2*>(dst) = o;
}

// Tuned per row-tile count: one tile prefetches one block and keeps Q in
// registers; two or three tiles keep Q in LDS and no prefetch buffer so that
// two waves fit each SIMD.
template <int NR>
void launch_attn_nr(const AttnArgs& a, int head_dim, int grid, hipStream_t st) {
  constexpr int DEPTH = NR == 1 ? 1 : 0;
  constexpr bool QLDS = NR > 1;
  const bool tree = a.meta.tmask != nullptr;
  if (head_dim == 128) {
    if (tree)
      k_attn<NR, 128, DEPTH, QLDS, 2, true><<<grid, 256, 0, st>>>(a);
    else
      k_attn<NR, 128, DEPTH, QLDS, 2, false><<<grid, 256, 0, st>>>(a);
  } else {
    if (tree)
      k_attn<NR, 64, DEPTH, QLDS, 2, true><<<grid, 256, 0, st>>>(a);
    else
      k_attn<NR, 64, DEPTH, QLDS, 2, false><<<grid, 256, 0, st>>>(a);
  }
}

template <int RB>
void launch_comb(const AttnArgs& a, int head_dim, int n_segs, hipStream_t st) {
  // slices only over the rows a segment can have (TB tokens x G heads)
  dim3 grid(n_segs, a.n_kv_heads, cdiv_i(std::min(RB, a.TB * a.G), 1024 / head_dim));
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
  if (RB == 128) {  // prefill row blocks
    if (head_dim == 128) k_attn_rows<4, 128><<<grid, 256, 0, st>>>(a);
    else k_attn_rows<4, 64><<<grid, 256, 0, st>>>(a);
    return;
  }
  if (RB == 16)
    launch_attn_nr<1>(a, head_dim, grid, st);
  else if (RB == 32)
    launch_attn_nr<2>(a, head_dim, grid, st);
  else
    launch_attn_nr<3>(a, head_dim, grid, st);
}

void launch_attn_combine(const AttnArgs& a, int RB, int head_dim, int n_segs, hipStream_t st) {
  if (RB == 128)
    launch_comb<128>(a, head_dim, n_segs, st);
  else if (RB == 16)
    launch_comb<16>(a, head_dim, n_segs, st);
  else if (RB == 32)
    launch_comb<32>(a, head_dim, n_segs, st);
  else
    launch_comb<48>(a, head_dim, n_segs, st);
}
