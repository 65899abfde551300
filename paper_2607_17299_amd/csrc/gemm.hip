// Skinny-M bf16 GEMM on gfx950 MFMA for the decoder projections and the LM head.
//
// C[m][n] = sum_k A[m][k] * W[n][k]: A is the (few-row) activation matrix,
// W a weight matrix stored [out][in].  In the verify step M is 4..~600 rows
// against N x K weights of 16-310 MB, so the kernel is bound by streaming W
// from HBM: every weight byte is read exactly once per m-block.
//
// Weights are repacked once, when the model is created, into MFMA fragment
// order: for n-tile nt (16 output rows), k-step s (64 inputs) and half j, the
// 1 KB fragment holds, for lane l, the 8 values
//     W[nt*16 + l%16][s*64 + (l/16)*16 + j*8 + e],  e = 0..7.
// The 8 n-tiles of one workgroup form a group (16 KB per k-step), and the
// whole matrix is stored step-major: k-step s, then group g, then tile t
// (0..7), then half j.  A workgroup reads one contiguous 16 KB piece per
// k-step, and the workgroups of a split, which advance through k together,
// sweep one contiguous window of N/128 pieces: the access pattern of a plain
// copy.  (Row-major W would touch 16 rows 8-24 KB apart per load; one run per
// group, 16 KB per step, streamed 6-9% slower.)  For the stacked [gate; up]
// matrix, group g holds gate tiles 4g..4g+3 as t = 0..3 and the matching up
// tiles as t = 4..7.
//
// Workgroup = 4 waves = 128 output columns; each wave owns 32 columns (two
// 16-wide MFMA n-tiles: t = 2w, 2w+1, or gate t = w and up t = w + 4) and all
// MT 16-row m-tiles of the workgroup's m-block.
// K advances in steps of 64:
//   * W goes straight from HBM to registers (4 fragments per wave and step);
//   * the A tile (MT*16 rows x 64) is loaded into registers by all 256 threads
//     and staged through LDS (three buffers, rows padded to 144 bytes), shared
//     by the 4 waves;
//   * both are requested three steps ahead, A before W, so that the in-order
//     memory counter never makes a step wait for loads younger than its own;
//     the A tile of step s+1 goes to LDS at the end of step s (one barrier);
//   * v_mfma_f32_16x16x32_bf16 accumulates in fp32.  Inside a step the
//     k-index is permuted identically for A and W (lane group g holds k
//     g*16 .. g*16+15), which leaves the dot products unchanged.
// Split-K over blockIdx.y fills the 256 CUs when N is small; partial sums go to
// P[split][M][N] and a row kernel adds them in a fixed order (deterministic).
// The argmax epilogue (LM head, one split) writes optional fp32 logits and the
// best (value, lowest index) of each row within each 128-column block.  The
// SwiGLU epilogue (gate/up, one split) takes the paired [gate; up] groups,
// wave w of block nb owning gate n-tile 4nb + w and the matching up n-tile,
// and writes bf16 silu(gate) * up for its 16 columns.  At 97-192 rows the
// argmax epilogue runs in k_gemm_x2, and SwiGLU and the partial sums of
// splits of 8-64 k-steps in k_gemm_x2c (below); k_gemm_x2c also takes 33-64
// rows (SwiGLU and partial sums) and the 8- and 16-step splits at 65-80 rows.
#include "kernels.h"

namespace {

constexpr int KS = 64;
constexpr int ROWB = KS * 2 + 16;  // LDS bytes per A row (16-byte pad vs bank conflicts)

template <int MT>
struct Tile {
  static constexpr int CHUNKS = MT * 16 * (KS / 8);  // 16-byte chunks of the A tile
  static constexpr int PER_THREAD = (CHUNKS + 255) / 256;
  static constexpr int BYTES = MT * 16 * ROWB;
};

// NSTEPS > 0: every split covers exactly NSTEPS k-steps and the step loop is
// fully unrolled (straight-line code lets the compiler's memory-counter waits
// stay exact, so loads issued three steps ahead really stay in flight);
// NSTEPS == 0: a runtime loop over (K split) / 64 steps.
// MW = 2: two groups of 4 waves take the two m-blocks of one weight block in
// one workgroup (rows 97-192: one workgroup per CU instead of 1.5); both read
// the same W fragments, the second group mostly from L1/L2.
// WNT: the launch has one m-block, so each weight byte is used by a single
// workgroup and the weight loads are non-temporal (they do not displace the
// activations and partial sums that other workgroups reuse; 64-80-row steps
// 0.14-0.28 ms faster).  With several m-blocks (the append's row chunks) the
// m-blocks of a weight block find it in L2, so the loads stay temporal.
template <int MT, int NSTEPS, int EPI, int MW, bool WNT = false>
__global__ void __launch_bounds__(256 * MW) __attribute__((amdgpu_waves_per_eu(1, 2))) k_gemm(GemmArgs g) {
  static_assert(MW == 1 || EPI != EPI_ARGMAX, "the argmax epilogue has one m-block per workgroup");
  __shared__ __attribute__((aligned(16))) unsigned char sAll[MW][3][Tile<MT>::BYTES];
  const int tid = threadIdx.x & 255, lane = tid & 63, w = tid >> 6, ln = lane & 15, lg = lane >> 4;
  const int mg = MW > 1 ? __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 8) : 0;
  unsigned char (*sA)[Tile<MT>::BYTES] = sAll[mg];
  // Workgroups are dealt to the 8 XCDs round-robin by linear id.  The m-blocks
  // of one weight block get ids 8 apart (same XCD, dispatched together), so
  // all but the first find W in that XCD's L2; a ragged tail of fewer than 8
  // n-blocks falls back to consecutive ids.
  const int mblocks = (g.M + MT * 16 * MW - 1) / (MT * 16 * MW);  // workgroup m-blocks
  const int NB = g.N / 128;
  const int full = (NB / 8) * 8 * mblocks;
  int nb, mb;
  if ((int)blockIdx.x < full) {
    const int r = blockIdx.x % (8 * mblocks);
    nb = (blockIdx.x / (8 * mblocks)) * 8 + (r & 7);
    mb = r >> 3;
  } else {
    const int r = blockIdx.x - full;
    nb = (NB / 8) * 8 + r / mblocks;
    mb = r % mblocks;
  }
  const int split = blockIdx.y;
  const int m0 = (mb * MW + mg) * MT * 16;
  const int kb = split * g.kper;
  const int ke = min(g.K, kb + g.kper);
  const int nsteps = NSTEPS > 0 ? NSTEPS : (ke - kb) / KS;
  const int n0 = nb * 128;
  // SwiGLU: the block's first gate tile (output column tile of the epilogue)
  const int tb = nb * 4;
  const bf16_t* Wb = g.Wp + (int64_t)nb * (8 * KS * 16);
  const int NG = g.N / 128;  // groups; one k-step of all groups is contiguous

  // Loads are raw buffer loads (one descriptor for the W block, one for A): the
  // compiler does not re-issue them next to their use, so they stay in flight
  // for the steps in between.  A rows at or beyond M load row 0 instead (no
  // per-lane branch around the load): an output row depends only on its own A
  // row, and rows >= M are never written.
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(Wb), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ares =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(g.A), 0, 0x7fffffff, 0x00020000);
  // byte offsets of this lane's fragments of the split's first step (tiles
  // 2w and 2w+1, or gate tile w and up tile w + 4); a step is 16 KB further
  const int wv0 = (EPI == EPI_SWIGLU ? w : w * 2) * (KS * 32) + lane * 16;
  const int64_t sstride = (int64_t)NG * (KS * 256);  // bytes per k-step of the matrix
  const int s0 = kb / KS;
  const int wv1 = wv0 + (EPI == EPI_SWIGLU ? 4 : 1) * (KS * 32);
  int av[Tile<MT>::PER_THREAD];
  int aoff[Tile<MT>::PER_THREAD];
#pragma unroll
  for (int i = 0; i < Tile<MT>::PER_THREAD; ++i) {
    const int c = min(tid + 256 * i, Tile<MT>::CHUNKS - 1);
    const int r = c >> 3, q = c & 7;
    const int gm = m0 + r;
    aoff[i] = r * ROWB + q * 16;
    const int src = gm < g.M ? (g.a_rows ? g.a_rows[gm] : gm) : (g.a_rows ? g.a_rows[0] : 0);
    av[i] = (src * g.lda + kb + q * 8) * 2;
  }

  auto bload = [](__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
  };
  auto bload_w = [](__amdgpu_buffer_rsrc_t r, int voff, int soff) {  // cache policy 2: non-temporal
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, WNT ? 2 : 0));
  };
  auto load_w = [&](uint4* wr, int s) {
    const int so = (int)((s0 + s) * sstride);
    wr[0] = bload_w(wres, wv0, so);
    wr[1] = bload_w(wres, wv0 + 1024, so);
    wr[2] = bload_w(wres, wv1, so);
    wr[3] = bload_w(wres, wv1 + 1024, so);
  };
  auto load_a = [&](uint4* ar, int s) {
#pragma unroll
    for (int i = 0; i < Tile<MT>::PER_THREAD; ++i) ar[i] = bload(ares, av[i], s * KS * 2);
  };
  auto store_a = [&](const uint4* ar, int buf) {
#pragma unroll
    for (int i = 0; i < Tile<MT>::PER_THREAD; ++i)
      if (tid + 256 * i < Tile<MT>::CHUNKS)
        *reinterpret_cast<uint4*>(&sA[buf][aoff[i]]) = ar[i];
  };

  f32x4 acc[MT][2];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt][0] = acc[mt][1] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const uint4* wr, int buf) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bf16x8 b0 = as_bf16x8(wr[j]), b1 = as_bf16x8(wr[2 + j]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const bf16x8 a = as_bf16x8(
            *reinterpret_cast<const uint4*>(&sA[buf][(mt * 16 + ln) * ROWB + lg * 32 + j * 16]));
        acc[mt][0] = mfma16(a, b0, acc[mt][0]);
        acc[mt][1] = mfma16(a, b1, acc[mt][1]);
      }
    }
  };

  // register sets rotate with period 3: step s uses wr[s%3]; ar[s%3] holds A(s)
  // until it is stored, then receives A(s+3)
  uint4 wA[4], wB[4], wC[4];
  uint4 aA[Tile<MT>::PER_THREAD], aB[Tile<MT>::PER_THREAD], aC[Tile<MT>::PER_THREAD];
  if (nsteps > 0) { load_a(aA, 0); load_w(wA, 0); }
  if (nsteps > 1) { load_a(aB, 1); load_w(wB, 1); }
  if (nsteps > 2) { load_a(aC, 2); load_w(wC, 2); }
  __builtin_amdgcn_sched_barrier(0);
  if (nsteps > 0) store_a(aA, 0);
  __syncthreads();

// sched_barrier pins the loads where they are issued: otherwise the scheduler
// sinks each load next to its use and the step waits for it right away.
#define GEMM_STEP(S, AL, AS, WR, B)                    \
  if ((S) < nsteps) {                                  \
    if ((S) + 3 < nsteps) load_a(AL, (S) + 3);         \
    __builtin_amdgcn_sched_barrier(0);                 \
    compute(WR, B);                                    \
    if ((S) + 3 < nsteps) load_w(WR, (S) + 3);         \
    __builtin_amdgcn_sched_barrier(0);                 \
    if ((S) + 1 < nsteps) store_a(AS, ((B) + 1) % 3);  \
    __syncthreads();                                   \
  }
  if constexpr (NSTEPS > 0) {
#pragma unroll
    for (int s = 0; s < NSTEPS; s += 3) {
      GEMM_STEP(s, aA, aB, wA, 0)
      GEMM_STEP(s + 1, aB, aC, wB, 1)
      GEMM_STEP(s + 2, aC, aA, wC, 2)
    }
  } else {
    for (int s = 0; s < nsteps; s += 3) {
      GEMM_STEP(s, aA, aB, wA, 0)
      GEMM_STEP(s + 1, aB, aC, wB, 1)
      GEMM_STEP(s + 2, aC, aA, wC, 2)
    }
  }
#undef GEMM_STEP

  // lane holds C[mt*16 + lg*4 + i][n0 + w*32 + t*16 + ln]
  if constexpr (EPI == EPI_SWIGLU) {
    // t = 0: gate column (tb + w)*16 + ln, t = 1: the matching up column
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + mt * 16 + lg * 4 + i;
        const float a = acc[mt][0][i];
        if (m < g.M) g.out[(int64_t)m * g.ld_out + (tb + w) * 16 + ln] = f2bf(a / (1.f + expf(-a)) * acc[mt][1][i]);
      }
  } else if constexpr (EPI == EPI_PARTIAL) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = m0 + mt * 16 + lg * 4 + i;
          if (m < g.M)
            g.P[((int64_t)split * g.M + m) * g.N + n0 + w * 32 + t * 16 + ln] = acc[mt][t][i];
        }
  } else {
    float* sv = reinterpret_cast<float*>(&sA[0][0]);           // [4][MT*16]
    int* si = reinterpret_cast<int*>(&sA[1][0]);                // [4][MT*16]
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = mt * 16 + lg * 4 + i;
        const int m = m0 + r;
        const int c0 = n0 + w * 32 + ln, c1 = c0 + 16;
        float v = acc[mt][0][i];
        int idx = c0;
        const float v1 = acc[mt][1][i];
        if (v1 > v) {
          v = v1;
          idx = c1;
        }
        if (g.logits && m < g.M) {
          g.logits[(int64_t)m * g.ld_logits + c0] = acc[mt][0][i];
          g.logits[(int64_t)m * g.ld_logits + c1] = acc[mt][1][i];
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const float ov = __shfl_xor(v, o, 64);
          const int oi = __shfl_xor(idx, o, 64);
          if (ov > v || (ov == v && oi < idx)) {
            v = ov;
            idx = oi;
          }
        }
        if (ln == 0) {
          sv[w * MT * 16 + r] = v;
          si[w * MT * 16 + r] = idx;
        }
      }
    __syncthreads();
    for (int r = tid; r < MT * 16; r += 256) {
      const int m = m0 + r;
      if (m >= g.M) continue;
      float v = sv[r];
      int idx = si[r];
      for (int ww = 1; ww < 4; ++ww) {
        const float ov = sv[ww * MT * 16 + r];
        const int oi = si[ww * MT * 16 + r];
        if (ov > v || (ov == v && oi < idx)) {
          v = ov;
          idx = oi;
        }
      }
      g.amax_v[(int64_t)m * (g.N / 128) + nb] = v;
      g.amax_i[(int64_t)m * (g.N / 128) + nb] = idx;
    }
  }
}

// The SwiGLU and argmax epilogues at 97-192 rows (two m-blocks of MT = 4..6
// m-tiles, an m-half each): one 8-wave workgroup takes both m-blocks of its
// weight block.  Wave (m, h, c) owns m-half m, k-half h of every 64-wide
// k-step and the 64 columns of half c (four n-tiles: t = 4c .. 4c+3, or gate
// tiles 2c, 2c+1 with the matching up tiles), so each A fragment it reads
// from LDS feeds four MFMAs.  The two k-half waves of each (m-half, column
// half) add their sums through LDS at the end; wave (m, h, c) then writes
// m-tiles [h ? ceil(MT/2) : 0, h ? MT : ceil(MT/2)) of its m-half.  Same
// pipeline as k_gemm.  (Measured against k_gemm's two-group mode: gate/up 5%
// and the LM head 10% faster at 192 rows; the split-K projections slower, so
// they kept k_gemm.  Gate/up over 64 k-steps and the split-K projections now
// run in k_gemm_x2c; this kernel keeps the LM head and gate/up over other K.)
template <int MT, int NSTEPS, int EPI>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(1, 2))) k_gemm_x2(GemmArgs g) {
  constexpr int RT = 2 * MT;                             // m-tiles of the workgroup
  constexpr int A_CHUNKS = RT * 16 * (KS / 8);           // 16-byte chunks of the A tile
  constexpr int A_PER = (A_CHUNKS + 511) / 512;
  constexpr int A_BYTES = RT * 16 * ROWB;
  constexpr int MLO = (MT + 1) / 2;                      // m-tiles the k-half 0 waves write
  constexpr int X_BYTES = 2 * 2 * MT * 4 * 64 * 16;      // the k-half exchange
  constexpr int S_BYTES = 3 * A_BYTES > X_BYTES ? 3 * A_BYTES : X_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[S_BYTES];
  __shared__ float s_bv[2][RT * 16];                     // argmax: best per column half
  __shared__ int s_bi[2][RT * 16];
  auto sA = [&](int buf) { return smem + buf * A_BYTES; };
  const int tid = threadIdx.x, lane = tid & 63, ln = lane & 15, lg = lane >> 4;
  const int wi = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int mh = wi >> 2, kh = (wi >> 1) & 1, cw = wi & 1;  // m-half, k-half, column half
  // Workgroups are dealt to the 8 XCDs round-robin by linear id.  The m-blocks
  // of one weight block get ids 8 apart (same XCD, dispatched together), so
  // all but the first find W in that XCD's L2; a ragged tail of fewer than 8
  // n-blocks falls back to consecutive ids.
  const int mblocks = (g.M + RT * 16 - 1) / (RT * 16);
  const int NB = g.N / 128;
  const int full = (NB / 8) * 8 * mblocks;
  int nb, mb;
  if ((int)blockIdx.x < full) {
    const int r = blockIdx.x % (8 * mblocks);
    nb = (blockIdx.x / (8 * mblocks)) * 8 + (r & 7);
    mb = r >> 3;
  } else {
    const int r = blockIdx.x - full;
    nb = (NB / 8) * 8 + r / mblocks;
    mb = r % mblocks;
  }
  const int split = blockIdx.y;
  const int m0 = mb * RT * 16;            // the workgroup's first row
  const int mr = m0 + mh * MT * 16;       // this wave's m-half
  const int kb = split * g.kper;
  const int ke = min(g.K, kb + g.kper);
  const int nsteps = NSTEPS > 0 ? NSTEPS : (ke - kb) / KS;
  const int n0 = nb * 128;
  // SwiGLU: the block's first gate tile (output column tile of the epilogue)
  const int tb = nb * 4;
  const bf16_t* Wb = g.Wp + (int64_t)nb * (8 * KS * 16);
  const int NG = g.N / 128;  // groups; one k-step of all groups is contiguous

  // Loads are raw buffer loads (one descriptor for the W block, one for A): the
  // compiler does not re-issue them next to their use, so they stay in flight
  // for the steps in between.  A rows at or beyond M load row 0 instead (no
  // per-lane branch around the load): an output row depends only on its own A
  // row, and rows >= M are never written.
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(Wb), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ares =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(g.A), 0, 0x7fffffff, 0x00020000);
  // tile t of the group holds half j at byte (t*2 + j)*1024 of a step's piece;
  // this wave's four tiles (two gate and the two matching up tiles for SwiGLU)
  int tt[4];
#pragma unroll
  for (int n = 0; n < 4; ++n) tt[n] = EPI == EPI_SWIGLU ? (n < 2 ? 2 * cw + n : 4 + 2 * cw + n - 2) : 4 * cw + n;
  const int64_t sstride = (int64_t)NG * (KS * 256);  // bytes per k-step of the matrix
  const int s0 = kb / KS;
  int av[A_PER];
  int aoff[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    const int c = min(tid + 512 * i, A_CHUNKS - 1);
    const int r = c >> 3, q = c & 7;
    const int gm = m0 + r;
    aoff[i] = r * ROWB + q * 16;
    const int src = gm < g.M ? (g.a_rows ? g.a_rows[gm] : gm) : (g.a_rows ? g.a_rows[0] : 0);
    av[i] = (src * g.lda + kb + q * 8) * 2;
  }

  auto bload = [](__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
  };
  auto load_w = [&](uint4* wr, int s) {
    const int so = (int)((s0 + s) * sstride);
#pragma unroll
    for (int n = 0; n < 4; ++n) wr[n] = bload(wres, (tt[n] * 2 + kh) * 1024 + lane * 16, so);
  };
  auto load_a = [&](uint4* ar, int s) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i) ar[i] = bload(ares, av[i], s * KS * 2);
  };
  auto store_a = [&](const uint4* ar, int buf) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
      if (A_CHUNKS % 512 == 0 || tid + 512 * i < A_CHUNKS)
        *reinterpret_cast<uint4*>(sA(buf) + aoff[i]) = ar[i];
  };

  f32x4 acc[MT][4];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int n = 0; n < 4; ++n) acc[mt][n] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const uint4* wr, int buf) {
    bf16x8 b[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) b[n] = as_bf16x8(wr[n]);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const bf16x8 a =
          as_bf16x8(*reinterpret_cast<const uint4*>(sA(buf) + ((mh * MT + mt) * 16 + ln) * ROWB + lg * 32 + kh * 16));
#pragma unroll
      for (int n = 0; n < 4; ++n) acc[mt][n] = mfma16(a, b[n], acc[mt][n]);
    }
  };

  // register sets rotate with period 3: step s uses wr[s%3]; ar[s%3] holds A(s)
  // until it is stored, then receives A(s+3)
  uint4 wA[4], wB[4], wC[4];
  uint4 aA[A_PER], aB[A_PER], aC[A_PER];
  if (nsteps > 0) { load_a(aA, 0); load_w(wA, 0); }
  if (nsteps > 1) { load_a(aB, 1); load_w(wB, 1); }
  if (nsteps > 2) { load_a(aC, 2); load_w(wC, 2); }
  __builtin_amdgcn_sched_barrier(0);
  if (nsteps > 0) store_a(aA, 0);
  __syncthreads();

// sched_barrier pins the loads where they are issued: otherwise the scheduler
// sinks each load next to its use and the step waits for it right away.
#define GEMM_STEP(S, AL, AS, WR_, B)                   \
  if ((S) < nsteps) {                                  \
    if ((S) + 3 < nsteps) load_a(AL, (S) + 3);         \
    __builtin_amdgcn_sched_barrier(0);                 \
    compute(WR_, B);                                   \
    if ((S) + 3 < nsteps) load_w(WR_, (S) + 3);        \
    __builtin_amdgcn_sched_barrier(0);                 \
    if ((S) + 1 < nsteps) store_a(AS, ((B) + 1) % 3);  \
    __syncthreads();                                   \
  }
  if constexpr (NSTEPS > 0) {
#pragma unroll
    for (int s = 0; s < NSTEPS; s += 3) {
      GEMM_STEP(s, aA, aB, wA, 0)
      GEMM_STEP(s + 1, aB, aC, wB, 1)
      GEMM_STEP(s + 2, aC, aA, wC, 2)
    }
  } else {
    for (int s = 0; s < nsteps; s += 3) {
      GEMM_STEP(s, aA, aB, wA, 0)
      GEMM_STEP(s + 1, aB, aC, wB, 1)
      GEMM_STEP(s + 2, aC, aA, wC, 2)
    }
  }
#undef GEMM_STEP

  // k-half sums: each wave hands the m-tiles the other k-half wave of its
  // column half writes to LDS, then adds the ones handed to it (the last step's
  // barrier has ended every read of the A buffers)
  f32x4* xs = reinterpret_cast<f32x4*>(smem);
  auto mine = [&](int mt) { return (mt < MLO ? 0 : 1) == kh; };
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    if (!mine(mt))
#pragma unroll
      for (int n = 0; n < 4; ++n) xs[(((mh * 2 + cw) * MT + mt) * 4 + n) * 64 + lane] = acc[mt][n];
  __syncthreads();
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
    if (mine(mt))
#pragma unroll
      for (int n = 0; n < 4; ++n) acc[mt][n] += xs[(((mh * 2 + cw) * MT + mt) * 4 + n) * 64 + lane];

  // lane holds C[mt*16 + lg*4 + i][column of tile tt[n]: n0 + tt[n]*16 + ln]
  if constexpr (EPI == EPI_SWIGLU) {
    // n = 0, 1: gate tiles 2cw + n; n = 2, 3: the matching up tiles
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (!mine(mt)) continue;
#pragma unroll
      for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = mr + mt * 16 + lg * 4 + i;
          const float a = acc[mt][n][i];
          if (m < g.M)
            g.out[(int64_t)m * g.ld_out + (tb + 2 * cw + n) * 16 + ln] = f2bf(a / (1.f + expf(-a)) * acc[mt][n + 2][i]);
        }
    }
  } else if constexpr (EPI == EPI_PARTIAL) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (!mine(mt)) continue;
#pragma unroll
      for (int n = 0; n < 4; ++n)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = mr + mt * 16 + lg * 4 + i;
          if (m < g.M) g.P[((int64_t)split * g.M + m) * g.N + n0 + tt[n] * 16 + ln] = acc[mt][n][i];
        }
    }
  } else {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      if (!mine(mt)) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = (mh * MT + mt) * 16 + lg * 4 + i;
        const int m = m0 + r;
        // columns ascend with n: a strictly larger value replaces, ties keep the lower id
        float v = acc[mt][0][i];
        int idx = n0 + tt[0] * 16 + ln;
#pragma unroll
        for (int n = 1; n < 4; ++n)
          if (acc[mt][n][i] > v) {
            v = acc[mt][n][i];
            idx = n0 + tt[n] * 16 + ln;
          }
        if (g.logits && m < g.M)
#pragma unroll
          for (int n = 0; n < 4; ++n) g.logits[(int64_t)m * g.ld_logits + n0 + tt[n] * 16 + ln] = acc[mt][n][i];
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) {
          const float ov = __shfl_xor(v, o, 64);
          const int oi = __shfl_xor(idx, o, 64);
          if (ov > v || (ov == v && oi < idx)) {
            v = ov;
            idx = oi;
          }
        }
        if (ln == 0) {
          s_bv[cw][r] = v;
          s_bi[cw][r] = idx;
        }
      }
    }
    __syncthreads();
    for (int r = tid; r < RT * 16; r += 512) {
      const int m = m0 + r;
      if (m >= g.M) continue;
      float v = s_bv[0][r];
      int idx = s_bi[0][r];
      if (s_bv[1][r] > v || (s_bv[1][r] == v && s_bi[1][r] < idx)) {
        v = s_bv[1][r];
        idx = s_bi[1][r];
      }
      g.amax_v[(int64_t)m * (g.N / 128) + nb] = v;
      g.amax_i[(int64_t)m * (g.N / 128) + nb] = idx;
    }
  }
}

// SwiGLU (one split of 64 k-steps) and split-K partial sums at 33-192 rows,
// column-quarter waves: wave (kh, cq) owns k-half kh of every step and two
// n-tiles (gate tile cq with its up tile 4 + cq, or tiles 2cq, 2cq + 1) for
// all RT m-tiles (one A fragment read from LDS feeds two MFMAs), so no
// two waves load the same weight fragment and every weight byte is used by one
// workgroup (WNT: non-temporal weight loads).  The two k-halves' sums meet in
// LDS at the end, the kh = 0 waves writing the first ceil(RT/2) m-tiles and
// the kh = 1 waves the rest.  Gate/up at 100, 128
// and 192 rows: 45, 50 and 59 us against 56, 56 and 61 us for k_gemm_x2; at
// 192 rows qkv 21.8 -> 20.7 us, o 16.4 -> 15.2, down 35.8 -> 32.1 against
// k_gemm's two-group mode (weights rotated past the memory-side cache).
template <int RT, int NSTEPS, int EPI, bool WNT>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(1, 2))) k_gemm_x2c(GemmArgs g) {
  static_assert(EPI == EPI_SWIGLU || EPI == EPI_PARTIAL, "SwiGLU or partial sums");
  constexpr int A_CHUNKS = RT * 16 * (KS / 8);
  constexpr int A_PER = (A_CHUNKS + 511) / 512;
  constexpr int A_BYTES = RT * 16 * ROWB;
  constexpr int LO = (RT + 1) / 2, HI = RT - LO;     // m-tiles the k-half 0 / 1 waves keep
  constexpr int X_BYTES = 4 * 2 * LO * 2 * 64 * 16;
  constexpr int S_BYTES = 3 * A_BYTES > X_BYTES ? 3 * A_BYTES : X_BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char smem[S_BYTES];
  auto sA = [&](int buf) { return smem + buf * A_BYTES; };
  const int tid = threadIdx.x, lane = tid & 63, ln = lane & 15, lg = lane >> 4;
  const int wi = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kh = wi >> 2, cq = wi & 3;
  const int mblocks = (g.M + RT * 16 - 1) / (RT * 16);
  const int NB = g.N / 128;
  const int full = (NB / 8) * 8 * mblocks;
  int nb, mb;
  if ((int)blockIdx.x < full) {
    const int r = blockIdx.x % (8 * mblocks);
    nb = (blockIdx.x / (8 * mblocks)) * 8 + (r & 7);
    mb = r >> 3;
  } else {
    const int r = blockIdx.x - full;
    nb = (NB / 8) * 8 + r / mblocks;
    mb = r % mblocks;
  }
  const int m0 = mb * RT * 16;
  const int split = blockIdx.y;
  const int kb = split * g.kper;
  const int s0 = kb / KS;
  const int nsteps = NSTEPS;
  const int tb = nb * 4;
  const bf16_t* Wb = g.Wp + (int64_t)nb * (8 * KS * 16);
  const int NG = g.N / 128;
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(Wb), 0, 0x7fffffff, 0x00020000);
  const __amdgpu_buffer_rsrc_t ares =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(g.A), 0, 0x7fffffff, 0x00020000);
  const int64_t sstride = (int64_t)NG * (KS * 256);
  // the wave's two tiles: SwiGLU gate tile cq and up tile 4 + cq, else tiles 2cq, 2cq + 1
  const int t0 = EPI == EPI_SWIGLU ? cq : 2 * cq, t1 = EPI == EPI_SWIGLU ? 4 + cq : 2 * cq + 1;
  const int wg0 = (t0 * 2 + kh) * 1024 + lane * 16, wu0 = (t1 * 2 + kh) * 1024 + lane * 16;
  int av[A_PER];
  int aoff[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) {
    const int c = min(tid + 512 * i, A_CHUNKS - 1);
    const int r = c >> 3, q = c & 7;
    const int gm = m0 + r;
    aoff[i] = r * ROWB + q * 16;
    const int src = gm < g.M ? (g.a_rows ? g.a_rows[gm] : gm) : (g.a_rows ? g.a_rows[0] : 0);
    av[i] = (src * g.lda + kb + q * 8) * 2;
  }
  auto bload = [](__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
  };
  auto bload_w = [](__amdgpu_buffer_rsrc_t r, int voff, int soff) {  // cache policy 2: non-temporal
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, WNT ? 2 : 0));
  };
  auto load_w = [&](uint4* wr, int s) {
    const int so = (int)((s0 + s) * sstride);
    wr[0] = bload_w(wres, wg0, so);
    wr[1] = bload_w(wres, wu0, so);
  };
  auto load_a = [&](uint4* ar, int s) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i) ar[i] = bload(ares, av[i], s * KS * 2);
  };
  auto store_a = [&](const uint4* ar, int buf) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
      if (A_CHUNKS % 512 == 0 || tid + 512 * i < A_CHUNKS)
        *reinterpret_cast<uint4*>(sA(buf) + aoff[i]) = ar[i];
  };
  f32x4 acc[RT][2];
#pragma unroll
  for (int mt = 0; mt < RT; ++mt) acc[mt][0] = acc[mt][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const uint4* wr, int buf) {
    const bf16x8 b0 = as_bf16x8(wr[0]), b1 = as_bf16x8(wr[1]);
#pragma unroll
    for (int mt = 0; mt < RT; ++mt) {
      const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4*>(sA(buf) + (mt * 16 + ln) * ROWB + lg * 32 + kh * 16));
      acc[mt][0] = mfma16(a, b0, acc[mt][0]);
      acc[mt][1] = mfma16(a, b1, acc[mt][1]);
    }
  };
  uint4 wA[2], wB[2], wC[2];
  uint4 aA[A_PER], aB[A_PER], aC[A_PER];
  if (nsteps > 0) { load_a(aA, 0); load_w(wA, 0); }
  if (nsteps > 1) { load_a(aB, 1); load_w(wB, 1); }
  if (nsteps > 2) { load_a(aC, 2); load_w(wC, 2); }
  __builtin_amdgcn_sched_barrier(0);
  if (nsteps > 0) store_a(aA, 0);
  __syncthreads();
#define GEMM_STEP(S, AL, AS, WR_, B)                   \
  if ((S) < nsteps) {                                  \
    if ((S) + 3 < nsteps) load_a(AL, (S) + 3);         \
    __builtin_amdgcn_sched_barrier(0);                 \
    compute(WR_, B);                                   \
    if ((S) + 3 < nsteps) load_w(WR_, (S) + 3);        \
    __builtin_amdgcn_sched_barrier(0);                 \
    if ((S) + 1 < nsteps) store_a(AS, ((B) + 1) % 3);  \
    __syncthreads();                                   \
  }
#pragma unroll
  for (int s = 0; s < NSTEPS; s += 3) {
    GEMM_STEP(s, aA, aB, wA, 0)
    GEMM_STEP(s + 1, aB, aC, wB, 1)
    GEMM_STEP(s + 2, aC, aA, wC, 2)
  }
#undef GEMM_STEP
  // k-half sums: the kh = 0 wave keeps m-tiles [0, LO), the kh = 1 wave the rest
  // (compile-time tile indices in both branches: acc stays in registers)
  f32x4* xs = reinterpret_cast<f32x4*>(smem);
  auto xidx = [&](int k, int q, int n) { return (((cq * 2 + k) * LO + q) * 2 + n) * 64 + lane; };
  if (kh == 0) {
#pragma unroll
    for (int q = 0; q < HI; ++q)
#pragma unroll
      for (int n = 0; n < 2; ++n) xs[xidx(0, q, n)] = acc[LO + q][n];
  } else {
#pragma unroll
    for (int q = 0; q < LO; ++q)
#pragma unroll
      for (int n = 0; n < 2; ++n) xs[xidx(1, q, n)] = acc[q][n];
  }
  __syncthreads();
  auto out_tile = [&](int t, f32x4 gsum, f32x4 usum) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + t * 16 + lg * 4 + i;
      if (m >= g.M) continue;
      if constexpr (EPI == EPI_SWIGLU) {
        const float a = gsum[i];
        g.out[(int64_t)m * g.ld_out + (tb + cq) * 16 + ln] = f2bf(a / (1.f + expf(-a)) * usum[i]);
      } else {
        float* pr = g.P + ((int64_t)split * g.M + m) * g.N + nb * 128 + ln;
        pr[t0 * 16] = gsum[i];
        pr[t1 * 16] = usum[i];
      }
    }
  };
  if (kh == 0) {
#pragma unroll
    for (int q = 0; q < LO; ++q) out_tile(q, acc[q][0] + xs[xidx(1, q, 0)], acc[q][1] + xs[xidx(1, q, 1)]);
  } else {
#pragma unroll
    for (int q = 0; q < HI; ++q)
      out_tile(LO + q, acc[LO + q][0] + xs[xidx(0, q, 0)], acc[LO + q][1] + xs[xidx(0, q, 1)]);
  }
}

template <int MT, int MW, bool WNT>
void launch_mw(const GemmArgs& g, int epi, int splits, hipStream_t st) {
  dim3 grid((g.N / 128) * cdiv_i(g.M, MT * 16 * MW), splits, 1);
  const dim3 block(256 * MW);
  const int steps = g.kper / KS;
  const bool exact = (int64_t)g.kper * splits == g.K;
  if (epi == EPI_SWIGLU) {
    if (steps == 64) k_gemm<MT, 64, EPI_SWIGLU, MW, WNT><<<grid, block, 0, st>>>(g);
    else k_gemm<MT, 0, EPI_SWIGLU, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 4) {
    k_gemm<MT, 4, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 8) {
    k_gemm<MT, 8, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 12) {
    k_gemm<MT, 12, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 16) {
    k_gemm<MT, 16, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 32) {
    k_gemm<MT, 32, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 48) {
    k_gemm<MT, 48, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else if (exact && steps == 64) {
    k_gemm<MT, 64, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  } else {
    k_gemm<MT, 0, EPI_PARTIAL, MW, WNT><<<grid, block, 0, st>>>(g);
  }
}

template <int MT>
void launch_mt(const GemmArgs& g, int epi, int splits, hipStream_t st) {
  if constexpr (MT >= 4) {
    // two m-blocks (97-192 rows) come with 4-6 tiles each
    if (gemm_mw(g.M) == 2 && epi != EPI_PARTIAL) {
      dim3 grid((g.N / 128) * cdiv_i(g.M, MT * 32), splits, 1);
      if (epi == EPI_ARGMAX && g.kper == 64 * KS) k_gemm_x2<MT, 64, EPI_ARGMAX><<<grid, 512, 0, st>>>(g);
      else if (epi == EPI_ARGMAX) k_gemm_x2<MT, 0, EPI_ARGMAX><<<grid, 512, 0, st>>>(g);
      else if (g.kper == 64 * KS) k_gemm_x2c<2 * MT, 64, EPI_SWIGLU, true><<<grid, 512, 0, st>>>(g);
      else k_gemm_x2<MT, 0, EPI_SWIGLU><<<grid, 512, 0, st>>>(g);
      return;
    }
  }
  // one m-block (at most 6 tiles: every m-tile count below 4 is one)
  const bool single = MT < 4 || g.M <= MT * 16;
  if (epi == EPI_ARGMAX) {
    dim3 grid((g.N / 128) * cdiv_i(g.M, MT * 16), splits, 1);
    if (single && g.kper == 64 * KS) k_gemm<MT, 64, EPI_ARGMAX, 1, true><<<grid, 256, 0, st>>>(g);
    else if (single) k_gemm<MT, 0, EPI_ARGMAX, 1, true><<<grid, 256, 0, st>>>(g);
    else if (g.kper == 64 * KS) k_gemm<MT, 64, EPI_ARGMAX, 1><<<grid, 256, 0, st>>>(g);
    else k_gemm<MT, 0, EPI_ARGMAX, 1><<<grid, 256, 0, st>>>(g);
  } else if (gemm_mw(g.M) == 2) {
    if constexpr (MT >= 4) {
      const int steps = g.kper / KS;
      const bool exact = (int64_t)g.kper * splits == g.K;
      dim3 grid((g.N / 128) * cdiv_i(g.M, MT * 32), splits, 1);
      if (exact && steps == 8) { k_gemm_x2c<2 * MT, 8, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g); return; }
      if (exact && steps == 16) { k_gemm_x2c<2 * MT, 16, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g); return; }
      if (exact && steps == 32) { k_gemm_x2c<2 * MT, 32, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g); return; }
      if (exact && steps == 48) { k_gemm_x2c<2 * MT, 48, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g); return; }
      if (exact && steps == 64) { k_gemm_x2c<2 * MT, 64, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g); return; }
    }
    launch_mw<MT, 2, false>(g, epi, splits, st);
  } else if (single) {
    launch_mw<MT, 1, true>(g, epi, splits, st);
  } else {
    launch_mw<MT, 1, false>(g, epi, splits, st);
  }
}

// One 16-byte fragment chunk per thread: chunk c = (((s * NG + g) * 8 + t) * 2 + j) * 64 + l
// for tile t of group g (NG = N / 128 groups); W2 non-null: t < 4 is tile 4g + t of W, t >= 4 tile
// 4g + t - 4 of W2 (the gate/up pairing), else tile 8g + t of W.
__global__ void k_pack_weights(const bf16_t* __restrict__ W, const bf16_t* __restrict__ W2, int K,
                               int64_t chunks, uint4* __restrict__ dst, int NG) {
  for (int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; c < chunks;
       c += (int64_t)gridDim.x * blockDim.x) {
    const int l = (int)(c & 63);
    const int j = (int)((c >> 6) & 1);
    const int t = (int)((c >> 7) & 7);
    const int64_t sg = c >> 10;  // s * NG + g
    const int s = (int)(sg / NG);
    const int64_t grp = sg - (int64_t)s * NG;
    const bf16_t* src = W2 && t >= 4 ? W2 : W;
    const int64_t tile = W2 ? grp * 4 + (t & 3) : grp * 8 + t;
    const int64_t row = tile * 16 + (l & 15);
    const int col = s * KS + (l >> 4) * 16 + j * 8;
    dst[c] = *reinterpret_cast<const uint4*>(src + row * K + col);
  }
}

}  // namespace

void launch_pack_weights(const bf16_t* W, const bf16_t* W2, int N, int K, bf16_t* dst, hipStream_t st) {
  const int64_t chunks = (int64_t)N * K / 8;
  const int blocks = (int)std::min<int64_t>((chunks + 255) / 256, 16384);
  k_pack_weights<<<blocks, 256, 0, st>>>(W, W2, K, chunks, reinterpret_cast<uint4*>(dst), N / 128);
}

// 16-row tiles per m-block: up to 6 (96 rows); more rows take more m-blocks
int gemm_mt(int M) {
  const int t = std::max(1, cdiv_i(M, 16));
  if (t <= 6) return t;
  return cdiv_i(t, cdiv_i(t, 6));  // balanced m-blocks of at most 6 tiles
}

// m-blocks per workgroup: 2 when the rows make exactly two m-blocks
int gemm_mw(int M) { return cdiv_i(M, 16 * gemm_mt(M)) == 2 ? 2 : 1; }

// workgroups per 128-column block and split
int gemm_mblock_groups(int M) { return cdiv_i(M, 16 * gemm_mt(M) * gemm_mw(M)); }

// 33-64 rows: the column-quarter kernel with four m-tiles (its 64-row tile
// then holds the rows exactly), for SwiGLU and exact splits of 8-64 k-steps.
// At 64 rows qkv 13.1 -> 12.1 us, o 10.3 -> 9.5, gate/up 38.4 -> 37.8, down
// 22.8 -> 22.1 (weights rotated).
bool launch_x2c_64(const GemmArgs& g, int epi, int splits, hipStream_t st) {
  const int steps = g.kper / KS;
  if ((int64_t)g.kper * splits != g.K) return false;
  dim3 grid((g.N / 128) * cdiv_i(g.M, 64), splits, 1);
  if (epi == EPI_SWIGLU) {
    if (steps != 64) return false;
    k_gemm_x2c<4, 64, EPI_SWIGLU, true><<<grid, 512, 0, st>>>(g);
  } else if (steps == 8) {
    k_gemm_x2c<4, 8, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else if (steps == 16) {
    k_gemm_x2c<4, 16, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else if (steps == 32) {
    k_gemm_x2c<4, 32, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else if (steps == 48) {
    k_gemm_x2c<4, 48, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else if (steps == 64) {
    k_gemm_x2c<4, 64, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else {
    return false;
  }
  return true;
}

// 65-80 rows: the short split-K projections (splits of 8 and 16 k-steps: qkv
// and o) take the column-quarter kernel with five m-tiles; at 72 rows qkv and
// o run 3-4% faster than in k_gemm, while gate/up and the 32-step down
// projection run 1-4% slower and stay there (weights rotated).
bool launch_x2c_80(const GemmArgs& g, int epi, int splits, hipStream_t st) {
  const int steps = g.kper / KS;
  if (epi != EPI_PARTIAL || (int64_t)g.kper * splits != g.K) return false;
  dim3 grid((g.N / 128) * cdiv_i(g.M, 80), splits, 1);
  if (steps == 8) {
    k_gemm_x2c<5, 8, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else if (steps == 16) {
    k_gemm_x2c<5, 16, EPI_PARTIAL, true><<<grid, 512, 0, st>>>(g);
  } else {
    return false;
  }
  return true;
}

void launch_gemm(const GemmArgs& g, int epi, int splits, hipStream_t st) {
  if (g.M > 32 && g.M <= 64 && epi != EPI_ARGMAX && launch_x2c_64(g, epi, splits, st)) return;
  if (g.M > 64 && g.M <= 80 && launch_x2c_80(g, epi, splits, st)) return;
  switch (gemm_mt(g.M)) {
    case 1: launch_mt<1>(g, epi, splits, st); break;
    case 2: launch_mt<2>(g, epi, splits, st); break;
    case 3: launch_mt<3>(g, epi, splits, st); break;
    case 4: launch_mt<4>(g, epi, splits, st); break;
    case 5: launch_mt<5>(g, epi, splits, st); break;
    default: launch_mt<6>(g, epi, splits, st); break;  // gemm_mt never exceeds 6
  }
}
