// Sampled verification: lossless speculative sampling with a deterministic
// drafter over top-k / temperature target distributions (gfx950).
//
// Target distribution of a row: keep the top_k largest logits (value
// descending, ties to the lowest token id), p = softmax(z_kept / T).  The
// draft d at row i is accepted iff u_i < p_i(d); at the first rejection the
// next token is drawn from p_i with d removed, and after the last draft from
// p_n; a draw with uniform v is the smallest token t (in id order) whose
// cumulative weight exceeds v times the total.  (The paper samples with
// temperature 1 and top-k 200 and requires lossless speculation; the rule is
// the standard one for a point-mass drafter.)
//
// k_sample_rows: one workgroup per row.  A 3-pass radix select on an
// order-preserving integer image of the logits finds the top_k-th largest
// value and how many of its ties are kept; ordered passes (each wave walks its
// own id segment in coalesced 64-id chunks, with wave scans) rank the ties
// and place both draws.  Each row's outcome (accepted?,
// token if rejected here, token if every draft up to here is accepted) is
// computed for every row; k_sample_accept then walks the rows of a request.
#include "kernels.h"

namespace {

constexpr int kST = 1024;   // threads per row workgroup
constexpr int kBins = 2048; // radix-select bins (11-bit digits)

__device__ __forceinline__ uint32_t fkey(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);  // larger float -> larger key
}

__device__ int block_excl_scan_i(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  __syncthreads();
  if (lane == 63) sh[w] = x;
  __syncthreads();
  int off = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) off += sh[i];
    tot += sh[i];
  }
  *total = tot;
  __syncthreads();
  return off + x - v;
}

// inclusive scan over the 64 lanes of a wave
template <class T>
__device__ __forceinline__ T wave_incl_scan(T x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const T y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

__global__ void __launch_bounds__(kST) k_sample_rows(SampleArgs s) {
  constexpr int NW = kST / 64;
  __shared__ int hist[2 * kBins];
  __shared__ int sh_i[NW];
  __shared__ float sh_f[NW], sh_g[NW];
  __shared__ uint32_t s_prefix;
  __shared__ int s_need;
  __shared__ float s_max, s_wd;
  __shared__ int s_tok[2], s_last[2];
  const int r = blockIdx.x;
  const int b = r / s.kp1, i = r % s.kp1;
  const int dl = s.ntok[b] - 1;  // drafts of the request (-1: inactive step)
  if (i > dl) return;
  const int d = i < dl ? s.drafts[(int64_t)b * s.k_max + i] : -1;
  const float* z = s.logits + (int64_t)r * s.V;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;

  // ---- radix select of the top_k-th largest key: digits of 11, 11 and 10
  // bits, high first (the first digit spans sign, exponent and two mantissa
  // bits, so that logits of similar size spread over many bins), into two
  // histogram copies (even and odd waves) to halve atomic contention
  if (t == 0) {
    s_prefix = 0;
    s_need = s.top_k;
    s_wd = 0.f;
    s_tok[0] = s_tok[1] = -1;
  }
  float mx = -INFINITY;
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 21 : pass == 1 ? 10 : 0;
    const int nbits = pass == 2 ? 10 : 11;
    const int nb = 1 << nbits;
    for (int k = t; k < 2 * kBins; k += kST) hist[k] = 0;
    __syncthreads();
    const uint32_t pre = s_prefix;
    const uint32_t hmask = pass == 0 ? 0u : (0xffffffffu << (shift + nbits));
    int* hh = hist + (w & 1) * kBins;
    for (int v = t; v < s.V; v += kST) {
      const float x = z[v];
      if (pass == 0) mx = fmaxf(mx, x);
      const uint32_t key = fkey(x);
      if ((key & hmask) == pre) atomicAdd(&hh[(key >> shift) & (nb - 1)], 1);
    }
    __syncthreads();
    // the bin holding the need-th largest: thread t looks at bins 2t and 2t+1
    const int c1 = 2 * t + 1 < nb ? hist[2 * t + 1] + hist[kBins + 2 * t + 1] : 0;
    const int c0 = 2 * t < nb ? hist[2 * t] + hist[kBins + 2 * t] : 0;
    int total;
    const int below = block_excl_scan_i(c0 + c1, sh_i, &total);
    const int above = total - below - c0 - c1;  // elements in bins above 2t+1
    const int need = s_need;
    __syncthreads();
    if (above < need && need <= above + c1) {
      s_prefix = pre | ((uint32_t)(2 * t + 1) << shift);
      s_need = need - above;
    } else if (above + c1 < need && need <= above + c1 + c0) {
      s_prefix = pre | ((uint32_t)(2 * t) << shift);
      s_need = need - above - c1;
    }
    __syncthreads();
  }
  const uint32_t kth = s_prefix;  // key of the top_k-th largest logit
  const int ties_kept = s_need;   // how many logits equal to it are kept (lowest ids first)
  // row maximum
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  if (lane == 0) sh_f[w] = mx;
  __syncthreads();
  if (t == 0) {
    float m = sh_f[0];
    for (int k = 1; k < NW; ++k) m = fmaxf(m, sh_f[k]);
    s_max = m;
  }
  __syncthreads();
  const float zmax = s_max;
  const float invT = 1.f / s.temperature;

  // ---- ordered passes: wave w owns ids [seg0, seg1), walked in 64-id chunks
  // (lane l reads id c + l: coalesced); prefixes inside a chunk come from
  // wave scans, across chunks from a running carry, across waves from a block
  // scan of the wave totals
  const int seg = (s.V + NW - 1) / NW;
  const int seg0 = min(s.V, w * seg), seg1 = min(s.V, seg0 + seg);
  // (1) ties per wave -> the rank of each wave's first tie
  int ties = 0;
  for (int c = seg0; c < seg1; c += 64) {
    const int v = c + lane;
    ties += (v < seg1 && fkey(z[v]) == kth) ? 1 : 0;
  }
  for (int o = 32; o >= 1; o >>= 1) ties += __shfl_xor(ties, o, 64);
  if (lane == 0) sh_i[w] = ties;
  __syncthreads();
  int tie0 = 0;
  for (int k = 0; k < w; ++k) tie0 += sh_i[k];
  __syncthreads();
  // weight of id v given the rank of the ties before it
  auto weight = [&](int v, int tie_rank_incl, bool is_tie, float x) -> float {
    const uint32_t key = fkey(x);
    const bool kept = key > kth || (is_tie && tie_rank_incl <= ties_kept);
    return kept ? expf((x - zmax) * invT) : 0.f;
  };
  // (2) weights per wave (all, and without the draft)
  float wsum = 0.f, wdr = 0.f;
  {
    int carry = tie0;
    for (int c = seg0; c < seg1; c += 64) {
      const int v = c + lane;
      const float x = v < seg1 ? z[v] : -INFINITY;
      const bool tie = v < seg1 && fkey(x) == kth;
      const int rank = carry + wave_incl_scan(tie ? 1 : 0);
      carry = __shfl(rank, 63, 64);
      const float wv = v < seg1 ? weight(v, rank, tie, x) : 0.f;
      wsum += wv;
      if (v == d) wdr = wv;
    }
  }
  for (int o = 32; o >= 1; o >>= 1) {
    wsum += __shfl_xor(wsum, o, 64);
    wdr += __shfl_xor(wdr, o, 64);
  }
  if (lane == 0) {
    sh_f[w] = wsum;
    sh_g[w] = wdr;
  }
  __syncthreads();
  float W = 0.f, wdraft = 0.f, off_all = 0.f, off_rej = 0.f;
  for (int k = 0; k < NW; ++k) {
    if (k < w) {
      off_all += sh_f[k];
      off_rej += sh_f[k] - sh_g[k];
    }
    W += sh_f[k];
    wdraft += sh_g[k];
  }
  const float Wr = W - wdraft;
  // the acceptance test, then the token for either outcome
  const float u = s.uniforms[(int64_t)r * 2], vv = s.uniforms[(int64_t)r * 2 + 1];
  const bool accept = d >= 0 && u * W < wdraft;
  // (3) cumulative weights in id order: the draws
  const float tgt_end = vv * W, tgt_rej = vv * Wr;
  int last_end = -1, last_rej = -1;  // highest kept ids (fallback below)
  {
    int carry = tie0;
    float ce = off_all, cr = off_rej;
    for (int c = seg0; c < seg1; c += 64) {
      const int v = c + lane;
      const float x = v < seg1 ? z[v] : -INFINITY;
      const bool tie = v < seg1 && fkey(x) == kth;
      const int rank = carry + wave_incl_scan(tie ? 1 : 0);
      carry = __shfl(rank, 63, 64);
      const float wv = v < seg1 ? weight(v, rank, tie, x) : 0.f;
      const float wr = v == d ? 0.f : wv;
      const float ie = wave_incl_scan(wv), ir = wave_incl_scan(wr);
      const float cum_e = ce + ie, cum_r = cr + ir;
      if (wv > 0.f) {
        last_end = v;
        if (v != d) last_rej = v;
        if (cum_e > tgt_end && cum_e - wv <= tgt_end) s_tok[1] = v;
        if (v != d && cum_r > tgt_rej && cum_r - wr <= tgt_rej) s_tok[0] = v;
      }
      ce += __shfl(ie, 63, 64);
      cr += __shfl(ir, 63, 64);
    }
  }
  // a target at the very top of the cumulative sum can miss every crossing
  // through rounding between partial sums: take the last kept token then
  for (int o = 32; o >= 1; o >>= 1) {
    last_end = max(last_end, __shfl_xor(last_end, o, 64));
    last_rej = max(last_rej, __shfl_xor(last_rej, o, 64));
  }
  if (lane == 0) {
    sh_i[w] = last_end;
    hist[w] = last_rej;
  }
  __syncthreads();
  if (t == 0) {
    int le = -1, lr = -1;
    for (int k = 0; k < NW; ++k) {
      le = max(le, sh_i[k]);
      lr = max(lr, hist[k]);
    }
    int* o = s.row_out + (int64_t)r * 3;
    o[0] = accept ? 1 : 0;
    o[1] = s_tok[0] >= 0 ? s_tok[0] : lr;
    o[2] = s_tok[1] >= 0 ? s_tok[1] : le;
  }
}

__global__ void k_sample_accept(SampleArgs s, int32_t* accept_lens, int32_t* next_tokens) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= s.B) return;
  const int dl = s.ntok[b] - 1;
  if (dl < 0) {  // no rows: the step's setup failed
    if (accept_lens) accept_lens[b] = -1;
    next_tokens[b] = -1;
    return;
  }
  int a = 0, nxt = -1;
  for (int i = 0; i <= dl; ++i) {
    const int* o = s.row_out + (int64_t)(b * s.kp1 + i) * 3;
    if (i < dl && o[0]) continue;
    a = i;
    nxt = i < dl ? o[1] : o[2];
    break;
  }
  if (accept_lens) accept_lens[b] = a;
  next_tokens[b] = nxt;
}

}  // namespace

void launch_sample(const SampleArgs& s, int32_t* accept_lens, int32_t* next_tokens, hipStream_t st) {
  k_sample_rows<<<s.B * s.kp1, kST, 0, st>>>(s);
  k_sample_accept<<<cdiv_i(s.B, 64), 64, 0, st>>>(s, accept_lens, next_tokens);
}
