// Shared device helpers and internal launch interfaces for the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // raw bfloat16 bits in memory

#define WAR_DEV __device__ __forceinline__

// ------------------------------------------------------------------ bf16 bits
WAR_DEV float bf2f(bf16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// float -> bfloat16 bits, round to nearest even (gfx950 v_cvt_pk_bf16_f32).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
WAR_DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// round a float to the nearest bfloat16 value, kept as float
WAR_DEV float round_bf(float f) { return bf2f(f2bf(f)); }

WAR_DEV uint32_t pack2(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// the two floats held by a packed bf16 pair
WAR_DEV float lo_f(uint32_t v) { return __uint_as_float(v << 16); }
WAR_DEV float hi_f(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

WAR_DEV bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

WAR_DEV f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------ wave reductions
WAR_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
WAR_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide sum over blockDim.x (multiple of 64, <= 1024) threads.
WAR_DEV float block_sum(float v, float* red /* [16] shared */) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63, nw = blockDim.x >> 6;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

__host__ __device__ inline int cdiv_i(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------- internal layouts
// Pool device state (one allocation, see PoolDev below).
struct PoolDev {
  int32_t* stack;      // [num_pages] free stack, top at stack[free_count-1]
  int32_t* refcount;   // [num_pages]
  int32_t* held;       // [max_seqs] pages held per sequence
  int32_t* base;       // [max_seqs] pages held before the last reservation
  int32_t* scalars;    // [0] free_count, [1] error flags, [2] 1 while a failed
                       // verify step waits for its commit
  int32_t* table;      // [max_seqs][max_pages] (caller memory)
  // host-mapped word the commit kernel writes when it ends: (commit sequence
  // number << 32) | free count, read by the host without waiting
  unsigned long long* report;
  int32_t num_pages, max_seqs, max_pages, page_size;
};

// Per-forward row metadata built on the device (verify) or host (prefill).
//   rows:     tok[r], pos[r], active[r] for r < n_rows
//   requests: seq[b], pos0[b] (position of the request's first row),
//             ntok[b] (active rows), row0[b] (row of token 0)
//   attention work list: items[i] = (b, row_block, key_chunk, 0), n_items,
//             segment (b, row_block) -> first item and item count
struct StepMeta {
  int32_t* tok;
  int32_t* pos;
  int32_t* active;
  int32_t* row_req;     // request index of each row
  int32_t* req_seq;
  int32_t* req_pos0;
  int32_t* req_ntok;
  int32_t* req_row0;
  int4* items;
  // nullable: the attention work order, n_items[1] item slots.  An item with
  // .w > 0 is a shared-prefix unit covering the rows of requests x .. x+w-1.
  int32_t* order;
  int32_t* n_items;     // [0] item slots, [1] units in the work order, [3] keys per item
  // the work order resolved: per slot of the order, two int4
  //   (item, request, key chunk, first token | rows' token count << 16),
  //   (.w of the item, sequence id, request position 0, request's first row)
  int4* udesc;
  int32_t* seg_begin;   // [n_segs]
  int32_t* seg_count;   // [n_segs]
  int32_t* seg_req;     // [n_segs]
  int32_t* seg_rb;      // [n_segs]
  // Tree drafts (both null otherwise): the KV slot of each row (its node index
  // past the context, while pos is the context plus the node's depth) and the
  // step slots the row sees, bit i = node i (its root-to-node path).
  int32_t* kvpos;
  uint32_t* tmask;
};

enum { ERR_BAD_TOKEN = 1, ERR_NO_PAGES = 2, ERR_BAD_PARENT = 4, ERR_DUP_SEQ = 8 };
